// Decode-time verification of the draft paths (vsd_verify_paths).
//
// Speculative decoding keeps the draft token z~_i with probability
// alpha_i = min(1, p(z~_i) / q(z~_i)) (Sec. "Preliminary", Eq. acc) and, at
// the first rejection, draws a replacement from the residual distribution
// norm(max(0, p - q)) over the target vocabulary, which ends the path.  The
// count of kept tokens is an unbiased draw of the accepted length whose mean
// given the path is sum_k S_k (Eq. accepted_len_cond).
//
// One workgroup of two wavefronts per path.  Lane i < d_s draws slot i's
// acceptance uniform (Philox counter (0, row, 2, offset), word 0) and tests
// Lambda(u) < log alpha (the normative log; log alpha from scoring); a ballot
// gives the first rejection (every wavefront of the workgroup takes the same
// decisions).  The two wavefronts then stream contiguous halves of the
// rejected row's target logits (8 consecutive target indices per lane,
// 128-bit loads), form p(t) and q(t) (draft logit through the inverse map, 0
// for target tokens the draft cannot propose) from the row's log-sum-exps,
// and draw the residual token by Gumbel-max over log(max(0, p - q)) with the
// sampler's exact candidate filter (family 3, counters over the target
// index); the halves' (key, index) maxima merge in index order.  The
// draft logits are gathered through the inverse map by every lane (an
// unmapped column reads element 0 and discards it), so a slice's eight
// gathers are in flight together.

#include "vsd_device.hpp"
#include "vsd_draw.hpp"
#include "vsd_kernels.hpp"

namespace vsd {

namespace {

constexpr int kWavesPerPath = 2;
constexpr int kChunkV = 8 * kWave;  // target indices per chunk: 8 per lane

// One 8-element slice of the residual draw with its values formed only where
// the filter needs them.  vmax is the log of the slice's largest residual:
// the logarithm is increasing, so it is the slice's largest value, and it
// takes the slice test; the eight logarithms are taken only when some lane's
// slice passes that test or the slice seeds the threshold.  Otherwise the
// steps and their order are those of FamilyDraw::draw8.
template <class Vals>
__device__ __forceinline__ void draw8_lazy(FamilyDraw& f, int base, float vmax, bool seed, Vals&& vals) {
  float v[8];
  if (seed) {
    vals(v);
    f.draw8(base, v, vmax, true);
    return;
  }
  if (!f.reachable(vmax)) return;
  const uint32_t c0 = (uint32_t)base >> 2;
  const uint4 p0 = f.philox(c0), p1 = f.philox(c0 + 1);
  const uint32_t wmax = max(max(max(p0.x, p0.y), max(p0.z, p0.w)), max(max(p1.x, p1.y), max(p1.z, p1.w)));
  const bool maybe = fmaf(vmax, f.c2, f.off) >= __builtin_amdgcn_logf((float)((~wmax) >> 8));
  if (__ballot(maybe) == 0ull) return;
  vals(v);
  f.exact(base, v, c0,
          maybe ? FamilyDraw::cand4(p0, v, f.c2, f.off) | (FamilyDraw::cand4(p1, v + 4, f.c2, f.off) << 4) : 0u);
}

template <typename T, bool MAPPED>
__global__ __launch_bounds__(kWavesPerPath * kWave) void k_verify(VerifyArgs a) {
  __shared__ Best part[kWavesPerPath];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = wave_id();
  const int64_t path = blockIdx.x;
  if (path >= a.paths) return;
  int d = a.L;
  if (a.depth != nullptr) {
    d = a.depth[path];
    if (d < 1 || d > a.L) {
      if (threadIdx.x == 0) report_error(a.err, VSD_DEVERR_DEPTH_RANGE);
      d = 0;
    }
  }
  // every wavefront of the block takes the same acceptance decisions
  bool reject = false;
  if (lane < d) {  // L <= 64: one slot per lane
    const int64_t r = path * a.L + lane;
    const uint4 w = philox4x32_10(0u, (uint32_t)r, 2u, a.offset, a.k0, a.k1);
    reject = !(spec_log(uniform_from_word(w.x)) < a.la[r * 3]);
  }
  const uint64_t rej = __ballot(reject);
  const int j = rej != 0ull ? __builtin_ctzll(rej) : d;
  if (j >= d) {
    if (threadIdx.x == 0) {
      a.accept_len[path] = j;
      a.resample[path] = -1;
    }
    return;
  }
  // residual draw at the rejected slot
  const int64_t r = path * a.L + j;
  const T* X = static_cast<const T*>(a.X) + r * a.ld_d;
  const T* Y = static_cast<const T*>(a.Y) + r * a.ld_t;
  const float cq2 = a.inv_tq * kLog2e, cp2 = a.inv_tp * kLog2e;
  const float lq2 = a.lse_q[r] * kLog2e, lp2 = a.lse_p[r] * kLog2e;
  FamilyDraw f{(uint32_t)r, 3u, a.offset, a.k0, a.k1, 1.0f, kLog2e};
  const __amdgpu_buffer_rsrc_t xrow = row_rsrc(X, row_bytes(X, a.Vd));
  // max(0, p - q) of target indices base .. base+7 (p from the target
  // logit, q from the draft logit through the inverse map, 0 if unmapped)
  auto load_res = [&](int base, float (&res)[8]) {
    float y[8], x[8];
    bool mapped[8];
    load8(Y + base, y);
    if (MAPPED) {
      int32_t iv[8];
      load8(a.inv + base, iv);
      // every lane loads, so the eight gathers issue together instead of one
      // per branch; they go through the draft row's buffer resource, which
      // answers an unmapped column's index (-1) with 0 without an access
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        mapped[k] = (uint32_t)iv[k] < (uint32_t)a.Vd;
        T raw;
        buf_gather(xrow, (uint32_t)iv[k], raw);
        x[k] = load1(&raw);
      }
    } else {
      load8(X + base, x);
#pragma unroll
      for (int k = 0; k < 8; ++k) mapped[k] = true;
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const float p = __builtin_amdgcn_exp2f(fmaf(y[k], cp2, -lp2));
      const float q = mapped[k] ? __builtin_amdgcn_exp2f(fmaf(x[k], cq2, -lq2)) : 0.0f;
      res[k] = fmaxf(p - q, 0.0f);
    }
  };
  // log(max(0, p - q)), -inf where p <= q
  auto log_res = [](float r) { return r > 0.0f ? __builtin_amdgcn_logf(r) * kLn2 : -INFINITY; };
  // the whole chunks are split into kWavesPerPath contiguous ranges, one per
  // wavefront, with every lane active (the draw's wavefront reductions,
  // including each range's seed, need all lanes); the last wavefront then
  // takes the partial chunk, in which every lane takes part with its valid
  // count
  const int nfull = a.Vt / kChunkV;
  const int c_begin = (int)((int64_t)nfull * wave / kWavesPerPath);
  const int c_end = (int)((int64_t)nfull * (wave + 1) / kWavesPerPath);
  for (int it = c_begin; it < c_end; ++it) {
    const int base = it * kChunkV + lane * 8;
    float res[8];
    load_res(base, res);
    draw8_lazy(f, base, log_res(max8(res)), it == c_begin, [&](float (&v)[8]) {
#pragma unroll
      for (int k = 0; k < 8; ++k) v[k] = log_res(res[k]);
    });
  }
  if (wave == kWavesPerPath - 1 && nfull * kChunkV < a.Vt) {
    const int base = nfull * kChunkV + lane * 8;
    const int nvalid = min(8, max(0, a.Vt - base));
    float v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const bool in = k < nvalid;
      const float y = in ? load1(Y + base + k) : 0.0f;
      const int32_t iv = MAPPED ? (in ? a.inv[base + k] : -1) : (in ? base + k : -1);
      const bool mapped = (uint32_t)iv < (uint32_t)a.Vd;
      const float x = mapped ? load1(X + iv) : 0.0f;
      const float p = __builtin_amdgcn_exp2f(fmaf(y, cp2, -lp2));
      const float q = mapped ? __builtin_amdgcn_exp2f(fmaf(x, cq2, -lq2)) : 0.0f;
      v[k] = in ? log_res(fmaxf(p - q, 0.0f)) : -INFINITY;
    }
    f.draw(base, v, nvalid);
  }
  wave_argmax(f.best.key, f.best.idx);
  if (lane == 0) part[wave] = f.best;
  __syncthreads();
  if (threadIdx.x == 0) {
    // the wavefronts' ranges are in index order, so the strict comparison
    // keeps the smallest index among equal keys
    Best b = part[0];
#pragma unroll
    for (int w = 1; w < kWavesPerPath; ++w)
      if (part[w].key > b.key) b = part[w];
    a.accept_len[path] = j;
    // no candidate at all: the residual mass vanished in float32 (alpha
    // rounds to 1 but the uniform exceeded it); reported as no replacement
    a.resample[path] = b.key == -INFINITY ? -1 : b.idx;
  }
}

template <typename T>
hipError_t launch_t(const VerifyArgs& a, hipStream_t s) {
  const dim3 grid((unsigned)a.paths);  // one workgroup of kWavesPerPath wavefronts per path
  if (a.inv != nullptr)
    hipLaunchKernelGGL((k_verify<T, true>), grid, dim3(kWavesPerPath * kWave), 0, s, a);
  else
    hipLaunchKernelGGL((k_verify<T, false>), grid, dim3(kWavesPerPath * kWave), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_verify(const VerifyArgs& a, bool bf16, hipStream_t s) {
  return bf16 ? launch_t<bf16_t>(a, s) : launch_t<float>(a, s);
}

}  // namespace vsd
