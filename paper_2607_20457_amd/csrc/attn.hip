// Attention launches: the launch shape (workgroups, rows per workgroup)
// and the choice of kernel instantiation by head dimension, mask, LSE output
// and row-map mode.  The kernel itself is in attn_kernel.hpp.
#include <mutex>

#include "attn_kernel.hpp"

using pulsar_attn::KernelArgs;

namespace {

// Work counters of the persistent causal launches: a slot per (device,
// stream), since launches on one stream never overlap, while launches on
// different streams may.  A slot holds a counter per KV head and the count
// of finished workgroups; it is zero before and after every launch.  A
// stream beyond the slots, or one being captured into a graph (whose
// replays could run beside other launches from the same stream), gets the
// plain one-workgroup-per-item launch.
constexpr int kSchedSlots = 64;
constexpr int kSchedWords = 32;  // up to 31 KV heads
__device__ __align__(256) unsigned g_sched[kSchedSlots][kSchedWords];

struct SchedDevice {
  bool ready = false;
  unsigned* base = nullptr;  // device address of g_sched on this device
  int n_cu = 0;
  int used = 0;
  hipStream_t stream[kSchedSlots];
};
std::mutex g_sched_mu;
SchedDevice g_sched_dev[64];

// The counter slot of the current device and this stream (and the device's
// compute-unit count), or null.
unsigned* sched_slot(hipStream_t stream, int* n_cu) {
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(stream, &cap) != hipSuccess || cap != hipStreamCaptureStatusNone)
    return nullptr;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  std::lock_guard<std::mutex> lock(g_sched_mu);
  SchedDevice& sd = g_sched_dev[dev];
  if (!sd.ready) {
    void* p = nullptr;
    int cu = 0;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(g_sched)) != hipSuccess ||
        hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cu < 1)
      return nullptr;
    sd.base = static_cast<unsigned*>(p);
    sd.n_cu = cu;
    sd.ready = true;
  }
  int slot = -1;
  for (int i = 0; i < sd.used; ++i)
    if (sd.stream[i] == stream) slot = i;
  if (slot < 0) {
    if (sd.used == kSchedSlots) return nullptr;
    slot = sd.used++;
    sd.stream[slot] = stream;
  }
  *n_cu = sd.n_cu;
  return sd.base + (size_t)slot * kSchedWords;
}

}  // namespace

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
  ka.sched = nullptr;
  ka.grid = 0;
  if (a.causal && a.Hkv < kSchedWords) {
    int n_cu = 0;
    ka.sched = sched_slot(stream, &n_cu);
    ka.grid = n_cu;
  }
  const bool lse = a.lse != nullptr;
  if (a.d == 128) return pulsar_attn::launch_d128(ka, a.causal != 0, lse, a.map.mode, stream);
  return pulsar_attn::launch_d64(ka, a.causal != 0, lse, a.map.mode, stream);
}
