// Decode-time verification of the draft paths (vsd_verify_paths).
//
// Speculative decoding keeps the draft token z~_i with probability
// alpha_i = min(1, p(z~_i) / q(z~_i)) (Sec. "Preliminary", Eq. acc) and, at
// the first rejection, draws a replacement from the residual distribution
// norm(max(0, p - q)) over the target vocabulary, which ends the path.  The
// count of kept tokens is an unbiased draw of the accepted length whose mean
// given the path is sum_k S_k (Eq. accepted_len_cond).
//
// One wavefront per path.  Lane i < d_s draws slot i's acceptance uniform
// (Philox counter (0, row, 2, offset), word 0) and tests
// Lambda(u) < log alpha (the normative log; log alpha from scoring); a ballot
// gives the first rejection.  The wavefront then streams the rejected row's
// target logits once (8 consecutive target indices per lane, 128-bit loads),
// forms p(t) and q(t) (draft logit through the inverse map, 0 for target
// tokens the draft cannot propose) from the row's log-sum-exps, and draws the
// residual token by Gumbel-max over log(max(0, p - q)) with the sampler's
// exact candidate filter (family 3, counters over the target index).
#include "vsd_device.hpp"
#include "vsd_draw.hpp"
#include "vsd_kernels.hpp"

namespace vsd {

namespace {

constexpr int kPathsPerBlock = 4;

template <typename T, bool MAPPED>
__global__ __launch_bounds__(256) void k_verify(VerifyArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t path = (int64_t)blockIdx.x * kPathsPerBlock + wave_id();
  if (path >= a.paths) return;
  int d = a.L;
  if (a.depth != nullptr) {
    d = a.depth[path];
    if (d < 1 || d > a.L) {
      if (lane == 0) report_error(a.err, VSD_DEVERR_DEPTH_RANGE);
      d = 0;
    }
  }
  bool reject = false;
  if (lane < d) {  // L <= 64: one slot per lane
    const int64_t r = path * a.L + lane;
    const uint4 w = philox4x32_10(0u, (uint32_t)r, 2u, a.offset, a.k0, a.k1);
    reject = !(spec_log(uniform_from_word(w.x)) < a.la[r * 3]);
  }
  const uint64_t rej = __ballot(reject);
  const int j = rej != 0ull ? __builtin_ctzll(rej) : d;
  if (lane == 0) a.accept_len[path] = j;
  if (j >= d) {
    if (lane == 0) a.resample[path] = -1;
    return;
  }
  // residual draw at the rejected slot
  const int64_t r = path * a.L + j;
  const T* X = static_cast<const T*>(a.X) + r * a.ld_d;
  const T* Y = static_cast<const T*>(a.Y) + r * a.ld_t;
  const float cq2 = a.inv_tq * kLog2e, cp2 = a.inv_tp * kLog2e;
  const float lq2 = a.lse_q[r] * kLog2e, lp2 = a.lse_p[r] * kLog2e;
  FamilyDraw f{(uint32_t)r, 3u, a.offset, a.k0, a.k1, 1.0f, kLog2e};
  // log(max(0, p - q)) of target indices base .. base+7, -inf where p <= q
  auto residual = [&](const float (&y)[8], const float (&x)[8], const bool (&mapped)[8], float (&v)[8]) {
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const float p = __builtin_amdgcn_exp2f(fmaf(y[k], cp2, -lp2));
      const float q = mapped[k] ? __builtin_amdgcn_exp2f(fmaf(x[k], cq2, -lq2)) : 0.0f;
      const float res = p - q;
      v[k] = res > 0.0f ? __builtin_amdgcn_logf(res) * kLn2 : -INFINITY;
    }
  };
  // whole 512-element chunks with every lane active (the draw's wavefront
  // reductions, including the seed of the first chunk, need all lanes), then
  // one partial chunk in which every lane takes part with its valid count
  const int nfull = a.Vt / (8 * kWave);
  for (int it = 0; it < nfull; ++it) {
    const int base = it * 8 * kWave + lane * 8;
    float y[8], x[8], v[8];
    bool mapped[8];
    load8(Y + base, y);
    if (MAPPED) {
      int32_t iv[8];
      load8(a.inv + base, iv);
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        mapped[k] = (uint32_t)iv[k] < (uint32_t)a.Vd;
        x[k] = mapped[k] ? load1(X + iv[k]) : 0.0f;
      }
    } else {
      load8(X + base, x);
#pragma unroll
      for (int k = 0; k < 8; ++k) mapped[k] = true;
    }
    residual(y, x, mapped, v);
    f.draw8(base, v, max8(v), it == 0);
  }
  if (nfull * 8 * kWave < a.Vt) {  // the partial last chunk
    const int base = nfull * 8 * kWave + lane * 8;
    const int nvalid = min(8, max(0, a.Vt - base));
    float y[8], x[8], v[8];
    bool mapped[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const bool in = k < nvalid;
      y[k] = in ? load1(Y + base + k) : 0.0f;
      int32_t iv = MAPPED ? (in ? a.inv[base + k] : -1) : (in ? base + k : -1);
      mapped[k] = (uint32_t)iv < (uint32_t)a.Vd;
      x[k] = mapped[k] ? load1(X + iv) : 0.0f;
    }
    residual(y, x, mapped, v);
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = k < nvalid ? v[k] : -INFINITY;
    f.draw(base, v, nvalid);
  }
  wave_argmax(f.best.key, f.best.idx);
  // no candidate at all: the residual mass vanished in float32 (alpha rounds
  // to 1 but the uniform exceeded it); reported as no replacement
  if (lane == 0) a.resample[path] = f.best.key == -INFINITY ? -1 : f.best.idx;
}

template <typename T>
hipError_t launch_t(const VerifyArgs& a, hipStream_t s) {
  const dim3 grid((unsigned)((a.paths + kPathsPerBlock - 1) / kPathsPerBlock));
  if (a.inv != nullptr)
    hipLaunchKernelGGL((k_verify<T, true>), grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((k_verify<T, false>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_verify(const VerifyArgs& a, bool bf16, hipStream_t s) {
  return bf16 ? launch_t<bf16_t>(a, s) : launch_t<float>(a, s);
}

}  // namespace vsd
