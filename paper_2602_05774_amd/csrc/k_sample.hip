// E-step sampling (Alg. 1 proposal z~ ~ q and correction z' ~ p; Alg. 2
// greedy reference z-bar), one wavefront per row.
//
// Each lane owns 8 consecutive vocabulary indices of every 512-element chunk
// (128-bit loads; the Philox counters of S2 cover 4 consecutive indices) and
// draws the Philox word of every element of both families.  The normative key
// float(x/T) + G costs two logarithms with a correctly rounded division each,
// so it is evaluated only for elements that can still win: with d = 1 - u
// (exact on the 2^-24 grid), G = -ln(-ln(1 - d)) <= -ln(d) because
// -ln(1 - d) >= d, and -ln(d) <= (24 - log2 j') ln 2 for the integer
// j' = (~w) >> 8 <= 2^24 d.  An element whose bound x/T - ln(d) + margin is
// below the running maximum (the lane's own, or the wavefront's, refreshed
// whenever a lane improves on it) cannot be the argmax; every other element
// gets its exact key.  The margin exceeds every rounding involved, so the
// tokens are exactly those of the definition.  Lanes visit indices in
// increasing order and keep the first of equal keys; a butterfly reduction
// with the same tie rule yields the row's tokens, independent of geometry.
//
// Mapped target logits are gathered in lane-strided order (gather k of a
// chunk loads indices chunk + 64k + lane: a few consecutive cache lines per
// instruction) and transposed to the lane-contiguous layout through a
// per-wavefront LDS tile.  Full chunks are software pipelined: the next
// chunk's map entries and draft row are loaded while the current chunk is
// drawn, and its target gathers are issued at the end of the current chunk
// and consumed after the next chunk's draft-family work.
#include "vsd_device.hpp"
#include "vsd_kernels.hpp"

namespace vsd {

namespace {

constexpr int kRowsPerBlock = 4;  // 256 threads = 4 wavefronts = 4 rows
constexpr int kChunk = 8 * kWave;  // elements per wavefront step

template <typename T>
__device__ __forceinline__ T neg_inf();
template <>
__device__ __forceinline__ float neg_inf<float>() { return -INFINITY; }
template <>
__device__ __forceinline__ bf16_t neg_inf<bf16_t>() { return (bf16_t)0xFF80u; }

__device__ __forceinline__ uint32_t word_of(const uint4& p, int k) {
  return k == 0 ? p.x : k == 1 ? p.y : k == 2 ? p.z : p.w;
}

// Raw 8-element slice of a row as loaded (bf16: one 128-bit load).
template <typename T>
struct Raw8;
template <>
struct Raw8<bf16_t> {
  uint4 v;
  __device__ __forceinline__ void load(const bf16_t* p) { v = *reinterpret_cast<const uint4*>(p); }
  __device__ __forceinline__ void unpack(float (&o)[8]) const {
    o[0] = bf16_lo(v.x); o[1] = bf16_hi(v.x);
    o[2] = bf16_lo(v.y); o[3] = bf16_hi(v.y);
    o[4] = bf16_lo(v.z); o[5] = bf16_hi(v.z);
    o[6] = bf16_lo(v.w); o[7] = bf16_hi(v.w);
  }
};
template <>
struct Raw8<float> {
  float4 a, b;
  __device__ __forceinline__ void load(const float* p) {
    a = reinterpret_cast<const float4*>(p)[0];
    b = reinterpret_cast<const float4*>(p)[1];
  }
  __device__ __forceinline__ void unpack(float (&o)[8]) const {
    o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
    o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
  }
};

struct Best {
  float key;
  int idx;
};

// Per-lane online log-sum-exp of v/T in the exactly consistent form of the
// scorer: mraw = largest raw value, mc = float(mraw * c), s = sum of
// exp2(fma(v, c, -mc)), c = log2(e)/T.  Elements equal to -inf add nothing.
struct LaneLse {
  float mraw = kNegBig, mc = kNegBig, s = 0.0f;

  template <int K>
  __device__ __forceinline__ void add(const float* v, float c) {
    float cm = v[0];
#pragma unroll
    for (int k = 1; k < K; ++k) cm = fmaxf(cm, v[k]);
    if (cm > mraw) {
      const float nmc = cm * c;
      s *= __builtin_amdgcn_exp2f(mc - nmc);
      mc = nmc;
      mraw = cm;
    }
#pragma unroll
    for (int k = 0; k < K; ++k) s += __builtin_amdgcn_exp2f(fmaf(v[k], c, -mc));
  }

  // Wavefront reduction; returns (max raw value, ln sum exp((v - max)/T)).
  __device__ __forceinline__ void finish(float c, float& m_out, float& tail_out) {
    float m = mc, t = s;
    wave_lse2(m, t);
    const float mr = wave_max(mraw);
    m_out = mr;
    tail_out = (log2f(t) - fmaf(mr, c, -m)) * kLn2;
  }
};

template <typename T, bool MAPPED, bool FUSED>
struct RowSampler {
  const T* X;
  const T* Y;
  const int32_t* d2t;
  T* tile;  // this wavefront's LDS tile, kChunk elements
  int Vd, Vt;
  float inv_tq, inv_tp;
  float cq2, cp2;  // log2(e) / T of each family
  uint32_t row, offset, k0, k1;
  int lane;
  int tblock;      // FUSED && MAPPED: target elements streamed per chunk
  Best bd{-INFINITY, 0x7FFFFFFF}, bt{-INFINITY, 0x7FFFFFFF}, bg{-INFINITY, 0x7FFFFFFF};
  float wave_d = -INFINITY, wave_t = -INFINITY;  // wavefront maxima known so far
  bool map_bad = false;
  LaneLse lq, lp;  // FUSED: draft and target log-sum-exp accumulators

  // FUSED && MAPPED: log-sum-exp of the target elements [lo, hi) of the row
  // (the target row is streamed in lock-step with the draft chunks, so the
  // mapped gathers of the same chunk find its cache lines in L2).
  __device__ __forceinline__ void stream_target(int lo, int hi) {
    for (int g = lo + lane * 8; g - lane * 8 < hi; g += kChunk) {
      float v[8];
      if (g + 8 <= hi) {
        load8(Y + g, v);
      } else {
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = (g + k < hi) ? load1(Y + g + k) : -INFINITY;
      }
      lp.template add<8>(v, cp2);
    }
  }

  __device__ __forceinline__ uint4 philox(uint32_t c0, uint32_t fam) const {
    return philox4x32_10(c0, row, fam, offset, k0, k1);
  }

  // Bound test of the 4 elements that share one Philox counter: bit k set
  // where x * log2e/T + off >= log2(j'), off = 24 - (thr - margin) log2e.
  __device__ __forceinline__ static uint32_t cand4(const uint4& w, const float* v, float c2, float off) {
    uint32_t m = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const bool c = fmaf(v[k], c2, off) >= __builtin_amdgcn_logf((float)((~word_of(w, k)) >> 8));
      m |= c ? (1u << k) : 0u;
    }
    return m;
  }

  // (thr - margin) log2e folded into the bound's constant.  The margin
  // 2e-3 + 2e-6 |thr| exceeds every rounding involved for elements with
  // |x/T| <= |thr| + 100; an element with x/T < thr - 100 cannot reach thr
  // because G < 16.7.
  __device__ __forceinline__ static float bound_offset(float thr) {
    return 24.0f - (thr - (2e-3f + 2e-6f * fabsf(thr))) * kLog2e;
  }

  // Exact keys of the candidates (rare); their Philox words are recomputed.
  __device__ __forceinline__ void exact(int base, const float (&x)[8], const float (&y)[8], uint32_t cd,
                                        uint32_t ct) {
    if (__ballot((cd | ct) != 0u) == 0ull) return;
    const uint32_t c0 = (uint32_t)base >> 2;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      if (cd & (1u << k)) {
        const float kd = gumbel_key(x[k], inv_tq, word_of(philox(c0 + (k >> 2), 0u), k & 3));
        if (kd > bd.key) {
          bd.key = kd;
          bd.idx = base + k;
        }
      }
      if (ct & (1u << k)) {
        const float kt = gumbel_key(y[k], inv_tp, word_of(philox(c0 + (k >> 2), 1u), k & 3));
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

  __device__ __forceinline__ void greedy(int base, const float (&y)[8], int nvalid) {
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const bool better = k < nvalid && y[k] > bg.key;
      bg.key = better ? y[k] : bg.key;
      bg.idx = better ? base + k : bg.idx;
    }
  }

  // Map entries of a full chunk in lane-strided order.
  __device__ __forceinline__ void load_map(int chunk, uint32_t (&t)[8]) const {
#pragma unroll
    for (int k = 0; k < 8; ++k) t[k] = (uint32_t)d2t[chunk + k * kWave + lane];
  }

  // Gathers of the mapped target logits; an out-of-range map entry reads
  // element 0 instead and is flagged in `bad`.
  __device__ __forceinline__ void gather(const uint32_t (&t)[8], T (&g)[8], uint32_t& bad) const {
    bad = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const bool ok = t[k] < (uint32_t)Vt;
      bad |= ok ? 0u : (1u << k);
      g[k] = Y[ok ? t[k] : 0u];
    }
  }

  // Transpose gathered values through the LDS tile into this lane's 8
  // lane-contiguous target logits (flagged entries become -inf).  LDS
  // operations of one wavefront execute in order: no barrier is needed.
  __device__ __forceinline__ void transpose(const T (&g)[8], uint32_t bad, float (&y)[8]) {
    map_bad |= bad != 0u;
#pragma unroll
    for (int k = 0; k < 8; ++k) tile[k * kWave + lane] = (bad & (1u << k)) ? neg_inf<T>() : g[k];
    load8(tile + lane * 8, y);
  }

  // Every chunk of the row whose 512 elements are all in range.
  __device__ void full_chunks(int nfull) {
    if (nfull == 0) return;
    uint32_t t[8];
    T g[8];
    uint32_t bad = 0;
    Raw8<T> xr, yr;
    if (MAPPED) {
      load_map(0, t);
      gather(t, g, bad);
    } else {
      yr.load(Y + lane * 8);
    }
    xr.load(X + lane * 8);
    for (int it = 0; it < nfull; ++it) {
      const int chunk = it * kChunk;
      const int base = chunk + lane * 8;
      const bool next = it + 1 < nfull;
      uint32_t tn[8];
      Raw8<T> xn, yn;
      if (next) {  // prefetch the next chunk's map entries and rows
        if (MAPPED)
          load_map(chunk + kChunk, tn);
        else
          yn.load(Y + base + kChunk);
        xn.load(X + base + kChunk);
      }
      const uint32_t c0 = (uint32_t)base >> 2;
      // draft family first: it does not wait for this chunk's gathers
      float x[8];
      xr.unpack(x);
      if (FUSED) lq.template add<8>(x, cq2);
      const float od = bound_offset(fmaxf(bd.key, wave_d));
      const uint32_t cd = cand4(philox(c0, 0u), x, cq2, od) | (cand4(philox(c0 + 1, 0u), x + 4, cq2, od) << 4);
      float y[8];
      if (MAPPED)
        transpose(g, bad, y);
      else
        yr.unpack(y);
      if (FUSED && !MAPPED) lp.template add<8>(y, cp2);
      if (FUSED && MAPPED) stream_target(it * tblock, min(Vt, (it + 1) * tblock));
      greedy(base, y, 8);
      const float ot = bound_offset(fmaxf(bt.key, wave_t));
      const uint32_t ct = cand4(philox(c0, 1u), y, cp2, ot) | (cand4(philox(c0 + 1, 1u), y + 4, cp2, ot) << 4);
      exact(base, x, y, cd, ct);
      if (next) {
        if (MAPPED)
          gather(tn, g, bad);
        else
          yr = yn;
        xr = xn;
      }
    }
  }

  // The row's last, partial chunk (guarded element by element).
  __device__ void tail_chunk(int chunk) {
    if (FUSED && MAPPED) stream_target((chunk / kChunk) * tblock, min(Vt, (chunk / kChunk + 1) * tblock));
    const int base = chunk + lane * 8;
    const int nvalid = min(8, max(0, Vd - base));
    if (MAPPED) {
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int v = chunk + k * kWave + lane;
        const bool in = v < Vd;
        const uint32_t t = (uint32_t)d2t[in ? v : 0];
        const bool ok = t < (uint32_t)Vt;
        map_bad |= in && !ok;
        const T val = Y[ok ? t : 0u];
        tile[k * kWave + lane] = (in && ok) ? val : neg_inf<T>();
      }
    }
    float x[8], y[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const bool in = k < nvalid;
      x[k] = in ? load1(X + base + k) : -INFINITY;
      y[k] = in ? (MAPPED ? load1(tile + lane * 8 + k) : load1(Y + base + k)) : -INFINITY;
    }
    if (FUSED) {
      lq.template add<8>(x, cq2);
      if (!MAPPED) lp.template add<8>(y, cp2);
    }
    greedy(base, y, nvalid);
    const uint32_t c0 = (uint32_t)base >> 2;
    const uint32_t valid = (1u << nvalid) - 1u;
    const float od = bound_offset(fmaxf(bd.key, wave_d));
    const float ot = bound_offset(fmaxf(bt.key, wave_t));
    const uint32_t cd = (cand4(philox(c0, 0u), x, cq2, od) | (cand4(philox(c0 + 1, 0u), x + 4, cq2, od) << 4)) & valid;
    const uint32_t ct = (cand4(philox(c0, 1u), y, cp2, ot) | (cand4(philox(c0 + 1, 1u), y + 4, cp2, ot) << 4)) & valid;
    exact(base, x, y, cd, ct);
  }
};

template <typename T, bool MAPPED, bool FUSED>
__global__ __launch_bounds__(256) void k_sample(SampleArgs a) {
  __shared__ __align__(16) T ytile[kRowsPerBlock][kChunk];
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
  if (i >= d) {  // masked slot: tokens -1, score outputs 0, nothing read
    if (lane == 0) {
      a.tok_d[r] = -1;
      a.tok_t[r] = -1;
      a.tok_g[r] = -1;
    }
    if (FUSED) {
      if (lane < 3) {
        a.la[r * 3 + lane] = 0.0f;
        a.lq[r * 3 + lane] = 0.0f;
      }
      if (lane == 0) {
        a.lse_q[r] = 0.0f;
        if (a.lse_p != nullptr) a.lse_p[r] = 0.0f;
      }
    }
    return;
  }
  const T* X = static_cast<const T*>(a.X) + r * a.ld_d;
  const T* Y = static_cast<const T*>(a.Y) + r * a.ld_t;
  RowSampler<T, MAPPED, FUSED> s{X,
                                 Y,
                                 a.d2t,
                                 ytile[threadIdx.x >> 6],
                                 a.Vd,
                                 a.Vt,
                                 a.inv_tq,
                                 a.inv_tp,
                                 a.inv_tq * kLog2e,
                                 a.inv_tp * kLog2e,
                                 (uint32_t)r,
                                 a.offset,
                                 a.k0,
                                 a.k1,
                                 lane,
                                 a.tblock};
  const int nfull = a.Vd / kChunk;
  s.full_chunks(nfull);
  if (nfull * kChunk < a.Vd) s.tail_chunk(nfull * kChunk);
  if (FUSED && MAPPED) {  // target elements past the last chunk's block (none when tblock covers the row)
    const int nchunks = (a.Vd + kChunk - 1) / kChunk;
    s.stream_target(min(a.Vt, nchunks * a.tblock), a.Vt);
  }
  if (s.map_bad) report_error(a.err, VSD_DEVERR_MAP_RANGE);
  wave_argmax(s.bd.key, s.bd.idx);
  wave_argmax(s.bt.key, s.bt.idx);
  wave_argmax(s.bg.key, s.bg.idx);
  if (FUSED) {
    // Row statistics of the scorer, in its exactly consistent shifted form,
    // and log q / log alpha of the three drawn tokens.
    float mq, tq, mp, tp;
    s.lq.finish(s.cq2, mq, tq);
    s.lp.finish(s.cp2, mp, tp);
    if (lane < 3) {
      const int z = lane == 0 ? s.bd.idx : lane == 1 ? s.bt.idx : s.bg.idx;
      float lqv = 0.0f, lav = 0.0f;
      if ((uint32_t)z < (uint32_t)a.Vd) {
        const int32_t zt = MAPPED ? a.d2t[z] : z;
        if ((uint32_t)zt < (uint32_t)a.Vt) {
          lqv = (load1(X + z) - mq) * a.inv_tq - tq;
          const float lp = (load1(Y + zt) - mp) * a.inv_tp - tp;
          lav = fminf(0.0f, lp - lqv);
        }
      }
      a.la[r * 3 + lane] = lav;
      a.lq[r * 3 + lane] = lqv;
    }
    if (lane == 0) {
      a.lse_q[r] = mq * a.inv_tq + tq;
      if (a.lse_p != nullptr) a.lse_p[r] = mp * a.inv_tp + tp;
    }
  }
  if (lane == 0) {
    a.tok_d[r] = s.bd.idx;
    a.tok_t[r] = s.bt.idx;
    a.tok_g[r] = s.bg.idx;
  }
}

template <typename T, bool FUSED>
hipError_t launch_t(const SampleArgs& a, hipStream_t s) {
  const dim3 grid((unsigned)((a.R + kRowsPerBlock - 1) / kRowsPerBlock));
  if (a.d2t != nullptr)
    hipLaunchKernelGGL((k_sample<T, true, FUSED>), grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((k_sample<T, false, FUSED>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_sample(const SampleArgs& a, bool bf16, hipStream_t s) {
  const bool fused = a.lse_q != nullptr;
  if (bf16) return fused ? launch_t<bf16_t, true>(a, s) : launch_t<bf16_t, false>(a, s);
  return fused ? launch_t<float, true>(a, s) : launch_t<float, false>(a, s);
}

}  // namespace vsd
