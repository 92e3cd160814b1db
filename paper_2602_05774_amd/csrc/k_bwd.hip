// Gradient of the weighted-likelihood loss with respect to the draft logits
// (vsd_weighted_loss_bwd): the derivative of Eq. advance with the E-step
// quantities fixed,
//   g[v] = loss_scale / T_q * ((a + b) q(v) - a [v = z~] - b [v = z']),
// q(v) = exp(X[v] / T_q - lse_q).  One wavefront per row streams the draft
// row once (128-bit loads) and writes the gradient row once (128-bit stores);
// rows with a = b = 0 are written as zeros without reading X.  With the
// top-K renormalised KL term (Eq. klv) the row's K sparse coefficients are
// added to their elements before the store: each lane tests the K indices
// against its 8-element chunk (a hit is rare) and adds them in place.
#include "vsd_device.hpp"
#include "vsd_kernels.hpp"
#include "vsd_topk.hpp"

namespace vsd {

namespace {

constexpr int kRowsPerBlock = 4;

// The row's KL entries (index, coefficient); indices outside [0, Vd) (masked
// rows carry -1) never match a chunk.
template <bool KL>
struct KlRow {
  int idx[KL ? kMaxTopK : 1];
  float grad[KL ? kMaxTopK : 1];
  int K = 0;

  __device__ __forceinline__ void load(const BwdArgs& a, int64_t r) {
    if (!KL) return;
    K = a.kl_k;
#pragma unroll
    for (int k = 0; k < kMaxTopK; ++k) {
      idx[k] = k < K ? a.kl_idx[r * K + k] : -1;
      grad[k] = k < K ? a.kl_grad[r * K + k] : 0.0f;
    }
  }

  // Add the entries that fall in [base, base + 8) to g.
  __device__ __forceinline__ void add(int base, float (&g)[8]) const {
    if (!KL) return;
    uint32_t hit = 0;
#pragma unroll
    for (int k = 0; k < kMaxTopK; ++k) hit |= ((uint32_t)(idx[k] - base) < 8u ? 1u : 0u) << k;
    if (hit == 0u) return;
#pragma unroll
    for (int k = 0; k < kMaxTopK; ++k) {
      if ((hit >> k) & 1u) {
        const int j = idx[k] - base;
#pragma unroll
        for (int e = 0; e < 8; ++e) g[e] += (e == j) ? grad[k] : 0.0f;
      }
    }
  }
};

template <typename T, bool KL>
__global__ __launch_bounds__(256) void k_bwd(BwdArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t r = (int64_t)blockIdx.x * kRowsPerBlock + wave_id();
  if (r >= a.R) return;
  T* G = static_cast<T*>(a.G) + r * a.ld;
  const float ca = a.coef_a != nullptr ? a.coef_a[r] : 0.0f;
  const float cb = a.coef_b != nullptr ? a.coef_b[r] : 0.0f;
  KlRow<KL> kl;
  kl.load(a, r);
  constexpr int step = 8 * kWave;
  auto store_tail = [&](int base, const float (&g)[8]) {
    for (int v = base; v < a.Vd && v < base + 8; ++v) store1(G + v, g[v - base]);
  };
  if (ca == 0.0f && cb == 0.0f) {
    int base = lane * 8;
    for (; base + 8 <= a.Vd; base += step) {
      float g[8] = {0, 0, 0, 0, 0, 0, 0, 0};
      kl.add(base, g);
      store8(G + base, g);
    }
    if (base < a.Vd) {
      float g[8] = {0, 0, 0, 0, 0, 0, 0, 0};
      kl.add(base, g);
      store_tail(base, g);
    }
    return;
  }
  const T* X = static_cast<const T*>(a.X) + r * a.ld;
  const float c = a.inv_tq * kLog2e;
  const float lse2 = a.lse_q[r] * kLog2e;
  const float k = a.scale * a.inv_tq;
  const float kab = k * (ca + cb), ka = k * ca, kb = k * cb;
  const int zd = a.tok_d[r], zt = a.tok_t[r];
  int base = lane * 8;
  constexpr int U = 2;
  for (; base + (U - 1) * step + 8 <= a.Vd; base += U * step) {
    float x[U][8];
#pragma unroll
    for (int u = 0; u < U; ++u) load8(X + base + u * step, x[u]);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float g[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int v = base + u * step + j;
        float t = kab * __builtin_amdgcn_exp2f(fmaf(x[u][j], c, -lse2));
        t -= (v == zd) ? ka : 0.0f;
        t -= (v == zt) ? kb : 0.0f;
        g[j] = t;
      }
      kl.add(base + u * step, g);
      store8(G + base + u * step, g);
    }
  }
  for (; base + 8 <= a.Vd; base += step) {
    float x[8], g[8];
    load8(X + base, x);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int v = base + j;
      float t = kab * __builtin_amdgcn_exp2f(fmaf(x[j], c, -lse2));
      t -= (v == zd) ? ka : 0.0f;
      t -= (v == zt) ? kb : 0.0f;
      g[j] = t;
    }
    kl.add(base, g);
    store8(G + base, g);
  }
  if (base < a.Vd) {
    float g[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int v = base + j;
      float t = 0.0f;
      if (v < a.Vd) {
        t = kab * __builtin_amdgcn_exp2f(fmaf(load1(X + v), c, -lse2));
        t -= (v == zd) ? ka : 0.0f;
        t -= (v == zt) ? kb : 0.0f;
      }
      g[j] = t;
    }
    kl.add(base, g);
    store_tail(base, g);
  }
}

template <typename T>
hipError_t launch_t(const BwdArgs& a, hipStream_t s) {
  const dim3 grid((unsigned)((a.R + kRowsPerBlock - 1) / kRowsPerBlock));
  if (a.kl_idx != nullptr)
    hipLaunchKernelGGL((k_bwd<T, true>), grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((k_bwd<T, false>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_bwd(const BwdArgs& a, bool bf16, hipStream_t s) {
  return bf16 ? launch_t<bf16_t>(a, s) : launch_t<float>(a, s);
}

}  // namespace vsd
