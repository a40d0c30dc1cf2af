// Host side of T-Offload's model-state path (paper, Section 5, "Hardware-
// agnostic T-Offload Solution by Co-design with T-Pipe"): after a layer's
// gradients have reached host DRAM its optimizer update runs on the CPU, and
// the updated weights go back to the device in a quantized form.  The paper
// fixes neither the optimizer nor the format; here the update is AdamW (bias-
// corrected moments, decoupled weight decay) in f32 on f32 master weights,
// and the reloaded block is the storage dtype (round to nearest even) or FP8
// E4M3 codes with one f32 scale per matrix row (scale = max|row| / 448,
// nearest code with ties to an even mantissa, saturating at 448).
#include <algorithm>
#include <cmath>
#include <cstring>
#include <thread>
#include <vector>

#include "errors.h"
#include "planner.h"

namespace {

uint16_t f32_to_bf16(float x) {
  uint32_t b;
  memcpy(&b, &x, 4);
  if ((b & 0x7F800000u) == 0x7F800000u && (b & 0x7FFFFFu)) return (uint16_t)((b >> 16) | 0x40);   // NaN stays NaN
  b += 0x7FFFu + ((b >> 16) & 1u);
  return (uint16_t)(b >> 16);
}

// Nearest E4M3 code of x (ties to an even mantissa), saturating at 448, no
// negative zero; branch-free so that the row loops vectorise.  Normal range:
// the f32 bit pattern rounded to 3 mantissa bits by an integer add (a carry
// moves into the exponent), then rebiased from 127 to 7.  Below 2^-6 the code
// is the value in steps of 2^-9, rounded by adding and subtracting 1.5 * 2^23.
inline uint8_t e4m3_encode(float x) {
  uint32_t b;
  memcpy(&b, &x, 4);
  const uint32_t sign = (b >> 24) & 0x80u;
  const uint32_t ab = b & 0x7FFFFFFFu;
  float a;
  memcpy(&a, &ab, 4);
  const int32_t normal = (int32_t)((ab + 0x7FFFFu + ((ab >> 20) & 1u)) >> 20) - (120 << 3);
  const float q = (a * 512.f + 12582912.f) - 12582912.f;
  int32_t c = a < 0.015625f ? (int32_t)q : normal;
  c = a < 448.f ? c : 0x7E;   // also infinities and NaN
  c = c > 0x7E ? 0x7E : c;
  return (uint8_t)(c == 0 ? 0u : (sign | (uint32_t)c));
}

struct Adam {
  float b1, b2, eps, lr_c, wd_c;   // lr_c = lr / (1 - b1^t) , wd_c = lr * wd
  float inv_bc2_sqrt;              // 1 / sqrt(1 - b2^t)
  bool update;
  // the element update; the device update (optim.hip) performs the same f32
  // operations in the same order
  void apply(float* __restrict__ w, float* __restrict__ m, float* __restrict__ v, const float* __restrict__ g,
             int64_t n) const {
    if (!update) return;
    for (int64_t i = 0; i < n; ++i) {
      const float gi = g[i];
      const float mi = b1 * m[i] + (1.f - b1) * gi;
      const float vi = b2 * v[i] + (1.f - b2) * gi * gi;
      m[i] = mi;
      v[i] = vi;
      const float denom = std::sqrt(vi) * inv_bc2_sqrt + eps;
      w[i] = w[i] - lr_c * mi / denom - wd_c * w[i];
    }
  }
};

template <typename F>
void parallel_for(int64_t n, int threads, F&& f) {
  if (threads <= 1 || n < 2) {
    f(0, n);
    return;
  }
  std::vector<std::thread> pool;
  const int64_t chunk = (n + threads - 1) / threads;
  for (int t = 0; t < threads; ++t) {
    const int64_t a = t * chunk, b = std::min(n, a + chunk);
    if (a >= b) break;
    pool.emplace_back([&f, a, b] { f(a, b); });
  }
  for (auto& th : pool) th.join();
}

}  // namespace

namespace tps {

AdamwCoef adamw_coef(const tps_adamw& opt, int32_t step) {
  AdamwCoef c{};
  c.b1 = opt.beta1;
  c.b2 = opt.beta2;
  c.eps = opt.eps;
  const double bc1 = 1.0 - std::pow((double)opt.beta1, step), bc2 = 1.0 - std::pow((double)opt.beta2, step);
  c.lr_c = (float)(opt.lr / bc1);
  c.inv_bc2_sqrt = (float)(1.0 / std::sqrt(bc2));
  c.wd_c = opt.lr * opt.weight_decay;
  return c;
}

int host_adamw(const Plan& p, const tps_adamw* opt, int32_t step, float* master, float* m, float* v,
               const float* grad, void* params_out, int32_t quant, int32_t n_threads) {
  if (!master || !params_out) return tps::set_error(TPS_EINVAL, "tps_host_adamw_layer: null argument");
  if (step < 0) return tps::set_error(TPS_EINVAL, "tps_host_adamw_layer: step must be >= 0");
  if (step > 0 && (!opt || !m || !v || !grad)) return tps::set_error(TPS_EINVAL, "tps_host_adamw_layer: optimizer state");
  if (quant != TPS_Q_NONE && quant != TPS_Q_FP8_ROW) return tps::set_error(TPS_EINVAL, "tps_host_adamw_layer: quant");
  if (quant == TPS_Q_FP8_ROW && p.dtype != TPS_BF16)
    return tps::set_error(TPS_EINVAL, "tps_host_adamw_layer: quantized blocks need bf16 storage");
  if (step > 0 && !(opt->lr >= 0.f && opt->beta1 >= 0.f && opt->beta1 < 1.f && opt->beta2 >= 0.f && opt->beta2 < 1.f &&
                    opt->eps >= 0.f && opt->weight_decay >= 0.f))
    return tps::set_error(TPS_EINVAL, "tps_host_adamw_layer: optimizer hyper-parameters out of range");
  Adam A{};
  A.update = step > 0;
  if (A.update) {
    const AdamwCoef c = adamw_coef(*opt, step);
    A.b1 = c.b1;
    A.b2 = c.b2;
    A.eps = c.eps;
    A.lr_c = c.lr_c;
    A.inv_bc2_sqrt = c.inv_bc2_sqrt;
    A.wd_c = c.wd_c;
  }
  const int threads = n_threads > 0 ? n_threads : std::max(1u, std::thread::hardware_concurrency());
  const int mat_slot[TPS_P_COUNT] = {0, -1, 1, -1, 2, -1, 3, -1, -1, -1, -1, -1};
  char* out = static_cast<char*>(params_out);
  for (int i = 0; i < TPS_P_COUNT; ++i) {
    if (p.prow[i] == 0) continue;   // a parameter the layer kind does not have
    float* W = master + p.goff[i] / 4;
    float* M = m ? m + p.goff[i] / 4 : nullptr;
    float* V = v ? v + p.goff[i] / 4 : nullptr;
    const float* G = grad ? grad + p.goff[i] / 4 : nullptr;
    const int64_t R = p.prow[i], Cn = p.pcol[i];
    const bool q8 = quant == TPS_Q_FP8_ROW && mat_slot[i] >= 0;
    // rows are the unit of work (a matrix row is quantized with its own scale)
    const int64_t units = R, per = Cn;
    parallel_for(units, R > 1 ? threads : 1, [&](int64_t a, int64_t b) {
      for (int64_t r = a; r < b; ++r) {
        const int64_t o = r * per;
        A.apply(W + o, M ? M + o : nullptr, V ? V + o : nullptr, G ? G + o : nullptr, per);
        if (q8) {
          // row maximum in 8 lanes (a max is exact, so the lane order does not matter)
          float lane[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
          const float* wr = W + o;
          int64_t c = 0;
          for (; c + 8 <= per; c += 8)
            for (int k = 0; k < 8; ++k) lane[k] = std::max(lane[k], std::fabs(wr[c + k]));
          for (; c < per; ++c) lane[0] = std::max(lane[0], std::fabs(wr[c]));
          float amax = 0.f;
          for (int k = 0; k < 8; ++k) amax = std::max(amax, lane[k]);
          const float scale = amax > 0.f ? amax / 448.f : 1.f;
          uint8_t* __restrict__ qd = reinterpret_cast<uint8_t*>(out + p.qoff[i]) + o;
          for (int64_t k = 0; k < per; ++k) qd[k] = e4m3_encode(wr[k] / scale);
          reinterpret_cast<float*>(out + p.qsoff[mat_slot[i]])[r] = scale;
        } else {
          const uint64_t base = quant == TPS_Q_FP8_ROW ? p.qoff[i] : p.poff[i];
          if (p.dtype == TPS_BF16) {
            uint16_t* d = reinterpret_cast<uint16_t*>(out + base) + o;
            for (int64_t c = 0; c < per; ++c) d[c] = f32_to_bf16(W[o + c]);
          } else {
            memcpy(reinterpret_cast<float*>(out + base) + o, W + o, (size_t)per * 4);
          }
        }
      }
    });
  }
  return TPS_OK;
}

}  // namespace tps

extern "C" int tps_host_adamw_layer(const tps_config* cfg, const tps_adamw* opt, int32_t step, float* master,
                                    float* m, float* v, const float* grad, void* params_out, int32_t quant,
                                    int32_t n_threads) {
  tps::clear_error();
  if (!cfg) return tps::set_error(TPS_EINVAL, "tps_host_adamw_layer: null argument");
  tps::Plan p;
  const int rc = tps::make_plan(cfg, &p);
  if (rc) return rc;
  return tps::host_adamw(p, opt, step, master, m, v, grad, params_out, quant, n_threads);
}
