// Instantiations of the attention kernel (attn_kernel.hpp) for head
// dimension 64.
#include "attn_kernel.hpp"

int pulsar_attn::launch_d64(const KernelArgs& ka, bool causal, bool lse, int mode,
                            hipStream_t stream) {
  return launch_for_d<64, kQT, kCausalWaves, kPartialWaves>(ka, causal, lse, mode, stream);
}
