// Attention launches: the launch shape (workgroups, rows per workgroup)
// and the choice of kernel instantiation by head dimension, mask, LSE output
// and row-map mode.  The kernel itself is in attn_kernel.hpp.
#include "attn_kernel.hpp"

using pulsar_attn::KernelArgs;

int attn_rows_per_wg(int group, bool causal) {
  const int heads_per_wg = group >= 4 ? 4 : group;
  const int waves = causal ? kCausalWaves : kPartialWaves;
  return 32 * kQT * (waves / heads_per_wg);
}

int launch_attention(const AttnLaunch& a, hipStream_t stream) {
  // load offsets are formed with 24-bit multiplies: a K/V row of at most
  // 2^24 bytes (and, with buffers below 2 GiB, positions below 2^24)
  if ((int64_t)a.Hkv * a.d * 2 >= (1 << 24)) return PULSAR_EUNSUPPORTED;
  KernelArgs ka;
  ka.a = a;
  ka.group = a.Hq / a.Hkv;
  ka.heads_per_wg = ka.group >= 4 ? 4 : ka.group;
  ka.hsub = ka.group / ka.heads_per_wg;
  ka.rows_per_wg = attn_rows_per_wg(ka.group, a.causal != 0);
  ka.n_row_tiles = (a.n_q + ka.rows_per_wg - 1) / ka.rows_per_wg;
  ka.nz = a.nz_kv * a.nsplit;
  const bool lse = a.lse != nullptr;
  if (a.d == 128) return pulsar_attn::launch_d128(ka, a.causal != 0, lse, a.map.mode, stream);
  return pulsar_attn::launch_d64(ka, a.causal != 0, lse, a.map.mode, stream);
}
