// Allocation-free variant of the attention backward (tps_op_attention_bwd):
// its row-dot workspace (D_i = dO_i . O_i, one f32 per (sequence, head,
// query)) lives in a fixed device array of this library instead of a
// caller-provided or library-allocated buffer.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>
#include <vector>

#include "errors.h"
#include "kernels.h"

using namespace tps;

namespace {

// Largest b * s * heads the fixed workspace serves (4 MiB of f32).
constexpr int64_t kScratchRows = int64_t(1) << 20;

// One copy per GPU the library runs on, alive until the process ends.  In
// host code this name is only a stand-in: the device address comes from
// hipGetSymbolAddress, per device.
__device__ __align__(256) float scratch[kScratchRows];

std::mutex g_mu;
std::vector<float*> g_ptr;   // per device id; nullptr until resolved

// The calling thread's current device's copy of `scratch`, resolved once per
// device (with that device current).
int scratch_for_current_device(float** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return check_hip(e, "attention_bwd_noalloc: hipGetDevice");
  std::lock_guard<std::mutex> lock(g_mu);
  if ((int)g_ptr.size() <= dev) g_ptr.resize(dev + 1, nullptr);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return check_hip(e, "attention_bwd_noalloc: hipGetSymbolAddress(scratch)");
    if (!p) return set_error(TPS_EHIP, "attention_bwd_noalloc: no device address for the workspace");
    g_ptr[dev] = static_cast<float*>(p);
  }
  *out = g_ptr[dev];
  return TPS_OK;
}

}  // namespace

extern "C" int64_t tps_op_attention_bwd_noalloc_max_rows(void) { return kScratchRows; }

extern "C" int tps_op_attention_bwd_noalloc(int dtype, int b, int s, int n_heads, int head_dim, const void* qkv,
                                            const void* o, const float* lse, const void* d_o, void* dqkv,
                                            void* stream) {
  clear_error();
  if (dtype != TPS_F32 && dtype != TPS_BF16) return set_error(TPS_EINVAL, "attention_bwd_noalloc: dtype");
  if (head_dim != 64 && head_dim != 128)
    return set_error(TPS_EINVAL, "attention_bwd_noalloc: head_dim must be 64 or 128");
  if (b < 0 || s < 0 || n_heads <= 0) return set_error(TPS_EINVAL, "attention_bwd_noalloc: shape");
  if (b == 0 || s == 0) return TPS_OK;
  const int64_t rows = (int64_t)b * s * n_heads;
  if (rows > kScratchRows)
    return set_error(TPS_EINVAL, "attention_bwd_noalloc: b * s * n_heads = " + std::to_string(rows) +
                                     " exceeds the fixed workspace of " + std::to_string(kScratchRows) +
                                     " rows; use tps_op_attention_bwd with a workspace");
  if (!qkv || !o || !lse || !d_o || !dqkv) return set_error(TPS_EINVAL, "attention_bwd_noalloc: null pointer");
  auto al16 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; };
  if (!al16(qkv) || !al16(o) || !al16(d_o)) return set_error(TPS_EINVAL, "attention_bwd_noalloc: alignment");
  float* ws = nullptr;
  const int rc = scratch_for_current_device(&ws);
  if (rc != TPS_OK) return rc;
  return check_hip(attention_bwd_launch(dtype, b, s, n_heads, n_heads, head_dim, qkv, o, lse, d_o, dqkv, ws,
                                        nullptr, static_cast<hipStream_t>(stream)),
                   "attention_bwd_noalloc launch");
}
