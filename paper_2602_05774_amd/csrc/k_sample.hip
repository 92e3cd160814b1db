// E-step sampling (Alg. 1 proposal z~ ~ q and correction z' ~ p; Alg. 2
// greedy reference z-bar), one wavefront per row.
//
// Each lane walks its 8-element chunks of the row (128-bit loads) and draws
// the Philox word of every element of both families.  The normative key
// float(x/T) + G costs two logarithms with a correctly rounded division each,
// so it is evaluated only for elements that can still win: with d = 1 - u
// (exact on the 2^-24 grid), G = -ln(-ln(1 - d)) <= -ln(d) because
// -ln(1 - d) >= d, and -ln(d) = (24 - log2(2^24 d)) ln 2 needs one hardware
// log2 of an exact integer.  An element whose bound x/T + (-ln d) + margin is
// below the running maximum (the lane's own, or the wavefront's, refreshed
// whenever a lane improves on it) cannot be the argmax; every other element
// gets its exact key.  The margin covers the hardware log2 error, the error of
// the normative log against the true one and the final rounding, so the
// tokens are exactly those of the definition.  Lanes visit indices in
// increasing order and keep the first of equal keys; a butterfly reduction
// with the same tie rule yields the row's tokens, independent of geometry.
#include "vsd_device.hpp"
#include "vsd_kernels.hpp"

namespace vsd {

namespace {

constexpr int kRowsPerBlock = 4;  // 256 threads = 4 wavefronts = 4 rows

struct Best {
  float key;
  int idx;
};

template <typename T>
__device__ __forceinline__ T neg_inf();
template <>
__device__ __forceinline__ float neg_inf<float>() { return -INFINITY; }
template <>
__device__ __forceinline__ bf16_t neg_inf<bf16_t>() { return (bf16_t)0xFF80u; }

__device__ __forceinline__ uint32_t word_of(const uint4& p, int k) {
  return k == 0 ? p.x : k == 1 ? p.y : k == 2 ? p.z : p.w;
}

// One 512-element chunk of a row: gather, draw, bound, and the exact keys of
// the candidates.  FULL chunks have every element in range and run without
// per-element guards; the row's last partial chunk runs with them.
template <typename T, bool MAPPED>
struct Chunk {
  const T* X;
  const T* Y;
  const int32_t* d2t;
  T* tile;
  int Vd, Vt;
  float inv_tq, inv_tp;
  uint32_t row, offset, k0, k1;
  int lane;
  float cq2, cp2;  // log2(e) / T of each family

  template <bool FULL>
  __device__ __forceinline__ void run(int chunk, Best& bd, Best& bt, Best& bg, float& wave_d, float& wave_t,
                                      bool& map_bad) const {
    const int base = chunk + lane * 8;
    float x[8], y[8];
    uint32_t wd[8], wt[8];
    if (MAPPED) {
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int v = chunk + k * kWave + lane;
        const bool in = FULL || v < Vd;
        const uint32_t t = (uint32_t)d2t[in ? v : 0];
        const bool ok = t < (uint32_t)Vt;
        map_bad |= in && !ok;
        const T val = Y[ok ? t : 0u];
        tile[k * kWave + lane] = (in && ok) ? val : neg_inf<T>();
      }
    }
    int nvalid = 8;
    if (FULL) {
      load8(X + base, x);
      if (MAPPED)
        load8(tile + lane * 8, y);
      else
        load8(Y + base, y);
    } else {
      nvalid = min(8, max(0, Vd - base));
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const bool in = k < nvalid;
        x[k] = in ? load1(X + base + k) : -INFINITY;
        y[k] = in ? (MAPPED ? load1(tile + lane * 8 + k) : load1(Y + base + k)) : -INFINITY;
      }
    }
    // Philox words: counter (v >> 2, row, family, offset), word v & 3.  A
    // chunk-aligned base is a multiple of 8, so the lane's 8 elements use the
    // four words of counters base/4 and base/4 + 1.
    const uint32_t c0 = (uint32_t)base >> 2;
    const uint4 d0 = philox4x32_10(c0, row, 0u, offset, k0, k1);
    const uint4 d1 = philox4x32_10(c0 + 1, row, 0u, offset, k0, k1);
    const uint4 t0 = philox4x32_10(c0, row, 1u, offset, k0, k1);
    const uint4 t1 = philox4x32_10(c0 + 1, row, 1u, offset, k0, k1);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      wd[k] = word_of(d0, k);
      wd[k + 4] = word_of(d1, k);
      wt[k] = word_of(t0, k);
      wt[k + 4] = word_of(t1, k);
    }
    // greedy reference: raw target maximum, first index wins
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const bool better = (FULL || k < nvalid) && y[k] > bg.key;
      bg.key = better ? y[k] : bg.key;
      bg.idx = better ? base + k : bg.idx;
    }
    // Candidates: elements whose key bound reaches the running maximum thr.
    // In log2 units the bound test reads  x * (log2e / T) + 24 - log2(j') >=
    // (thr - margin) log2e  with j' = (~w) >> 8 <= 2^24 (1 - u) (j' = 0 gives
    // an infinite bound).  The margin 2e-3 + 2e-6 |thr| exceeds every rounding
    // involved for elements with |x/T| <= |thr| + 100, and an element with
    // x/T < thr - 100 cannot reach thr because G < 16.7.
    const float thr_d = fmaxf(bd.key, wave_d), thr_t = fmaxf(bt.key, wave_t);
    const float od = 24.0f - (thr_d - (2e-3f + 2e-6f * fabsf(thr_d))) * kLog2e;
    const float ot = 24.0f - (thr_t - (2e-3f + 2e-6f * fabsf(thr_t))) * kLog2e;
    bool cd[8], ct[8];
    bool any = false;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const bool in = FULL || k < nvalid;
      cd[k] = in && fmaf(x[k], cq2, od) >= __builtin_amdgcn_logf((float)((~wd[k]) >> 8));
      ct[k] = in && fmaf(y[k], cp2, ot) >= __builtin_amdgcn_logf((float)((~wt[k]) >> 8));
      any |= cd[k] | ct[k];
    }
    if (__ballot(any) == 0ull) return;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      if (cd[k]) {
        const float kd = gumbel_key(x[k], inv_tq, wd[k]);
        if (kd > bd.key) {
          bd.key = kd;
          bd.idx = base + k;
        }
      }
      if (ct[k]) {
        const float kt = gumbel_key(y[k], inv_tp, wt[k]);
        if (kt > bt.key) {
          bt.key = kt;
          bt.idx = base + k;
        }
      }
    }
    if (__ballot(bd.key > wave_d || bt.key > wave_t) != 0ull) {
      wave_d = wave_max(bd.key);
      wave_t = wave_max(bt.key);
    }
  }
};

template <typename T, bool MAPPED>
__global__ __launch_bounds__(256) void k_sample(SampleArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t r = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  if (r >= a.R) return;
  const int i = (int)(r % a.L);
  const int64_t path = r / a.L;  // (b*T + t)*N + s
  int d = a.L;
  if (a.depth != nullptr) {
    d = a.depth[path];
    if (d < 1 || d > a.L) {
      if (lane == 0) report_error(a.err, VSD_DEVERR_DEPTH_RANGE);
      d = 0;
    }
  }
  if (i >= d) {
    if (lane == 0) {
      a.tok_d[r] = -1;
      a.tok_t[r] = -1;
      a.tok_g[r] = -1;
    }
    return;
  }
  const T* X = static_cast<const T*>(a.X) + r * a.ld_d;
  const T* Y = static_cast<const T*>(a.Y) + r * a.ld_t;
  const uint32_t row = (uint32_t)r;

  Best bd{-INFINITY, 0x7FFFFFFF}, bt{-INFINITY, 0x7FFFFFFF}, bg{-INFINITY, 0x7FFFFFFF};
  float wave_d = -INFINITY, wave_t = -INFINITY;  // wavefront maxima known so far
  bool map_bad = false;

  // Per-wavefront LDS tile: the mapped target logits of one 512-element chunk.
  // Gathers run in lane-strided order (instruction k loads draft indices
  // chunk + 64k + lane, which hit a few consecutive cache lines) and the tile
  // is read back in lane-contiguous order (lane j owns chunk + 8j .. +7, the
  // layout the Philox counters want).  LDS operations of one wavefront execute
  // in order, so no barrier is needed between its writes and reads.
  __shared__ __align__(16) T ytile[kRowsPerBlock][8 * kWave];
  T* tile = ytile[threadIdx.x >> 6];

  Chunk<T, MAPPED> c{X,     Y,        a.d2t, tile, a.Vd, a.Vt, a.inv_tq, a.inv_tp, row, a.offset, a.k0, a.k1,
                     lane,  a.inv_tq * kLog2e, a.inv_tp * kLog2e};
  int chunk = 0;
  for (; chunk + 8 * kWave <= a.Vd; chunk += 8 * kWave) c.template run<true>(chunk, bd, bt, bg, wave_d, wave_t, map_bad);
  if (chunk < a.Vd) c.template run<false>(chunk, bd, bt, bg, wave_d, wave_t, map_bad);
  if (map_bad) report_error(a.err, VSD_DEVERR_MAP_RANGE);
  wave_argmax(bd.key, bd.idx);
  wave_argmax(bt.key, bt.idx);
  wave_argmax(bg.key, bg.idx);
  if (lane == 0) {
    a.tok_d[r] = bd.idx;
    a.tok_t[r] = bt.idx;
    a.tok_g[r] = bg.idx;
  }
}

template <typename T>
hipError_t launch_t(const SampleArgs& a, hipStream_t s) {
  const dim3 grid((unsigned)((a.R + kRowsPerBlock - 1) / kRowsPerBlock));
  if (a.d2t != nullptr)
    hipLaunchKernelGGL((k_sample<T, true>), grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((k_sample<T, false>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_sample(const SampleArgs& a, bool bf16, hipStream_t s) {
  return bf16 ? launch_t<bf16_t>(a, s) : launch_t<float>(a, s);
}

}  // namespace vsd
