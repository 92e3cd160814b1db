// E-step sampling (Alg. 1 proposal z~ ~ q and correction z' ~ p; Alg. 2
// greedy reference z-bar), optionally fused with the row statistics of path
// scoring (log-sum-exps and the drawn tokens' log q / log alpha).
//
// Two wavefronts per row: the draft wavefront draws z~ from X (and, fused,
// accumulates the draft log-sum-exp); the target wavefront draws z' and z-bar
// from the mapped target logits.  Fused with a map, the target row is streamed
// for its log-sum-exp in lock-step with the draft chunks (2048 target
// elements per 512-element chunk, half by each wavefront), so the mapped
// gathers of a chunk find its cache lines in L2 and every logit is read from
// memory once.  The two wavefronts meet at one barrier at the end of the row.
//
// Each lane owns 8 consecutive vocabulary indices of every 512-element chunk
// (128-bit loads; the Philox counters of the sampler definition cover 4
// consecutive indices) and draws the Philox word of every element.  The
// normative key float(x/T) + G costs two logarithms with a correctly rounded
// division each, so it is evaluated only for elements that can still win:
// with d = 1 - u (exact on the 2^-24 grid), G = -ln(-ln(1 - d)) <= -ln(d)
// because -ln(1 - d) >= d, and -ln(d) <= (24 - log2 j') ln 2 for the integer
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
// per-row LDS tile.  Chunks are software pipelined: the next chunk's map
// entries and rows are loaded while the current chunk is drawn, and the target
// gathers of the next chunk are issued at the end of the current one.
//
// k_sample_step draws one depth of a rollout with exact context: three
// wavefronts per path, each on its own row (z~ from the draft row along z~,
// z' from the target row along z', z-bar from the target row along z-bar),
// with the counters of the slot's global row, so equal rows give exactly the
// tokens k_sample draws.
//
// With the top-K renormalised KL term (one-pass mode), the target wavefront
// also offers each chunk's mapped target logits, already in draft-index
// order, to an exact wavefront top-K (vsd_topk.hpp) and, after the row, forms
// the term over the K (as k_score_rows does).
#include "vsd_device.hpp"
#include "vsd_kernels.hpp"
#include "vsd_draw.hpp"
#include "vsd_topk.hpp"

namespace vsd {

namespace {

constexpr int kRowsPerBlock = 2;   // 256 threads = 2 rows x 2 wavefronts
constexpr int kChunk = 8 * kWave;  // draft elements per wavefront step
constexpr int kStream = 2 * kChunk;  // target elements each wavefront streams per chunk (fused, mapped)

template <typename T>
__device__ __forceinline__ T neg_inf();
template <>
__device__ __forceinline__ float neg_inf<float>() { return -INFINITY; }
template <>
__device__ __forceinline__ bf16_t neg_inf<bf16_t>() { return (bf16_t)0xFF80u; }

// Per-lane online log-sum-exp of v/T in the scorer's exactly consistent form:
// mraw = a raw reference value, mc = float(mraw * c), s = sum of
// exp2(fma(v, c, -mc)), c = log2(e)/T.  Elements equal to -inf add nothing.
// Every identity used after the row (the reduction, the rounding correction
// of mc, log q) holds for any reference, so the reference need not be the
// maximum:
//   add8        moves it up to the running maximum (the careful form);
//   add8_lazy   moves it only when the slice's maximum (already known to the
//               caller) exceeds it by more than 64 / c, so terms stay below
//               2^64: one compare per slice;
//   add8_fixed  keeps the reference start8 took from the lane's first slice
//               and tracks nothing: one fma, exp2 and add per element.
// A lane whose sum leaves [0, 2^120] (an element about 120 / c above its
// reference, or a NaN) is recomputed with add8 (bad()); 64 lanes and two
// wavefronts of such sums still merge below the float range.
struct LaneLse {
  float mraw = kNegBig, mc = kNegBig, s = 0.0f;

  __device__ __forceinline__ void start8(const float (&v)[8], float c) {
    const float cm = max8(v);
    if (cm > mraw) {
      s *= __builtin_amdgcn_exp2f(mc - cm * c);
      mc = cm * c;
      mraw = cm;
    }
  }

  __device__ __forceinline__ void add8_fixed(const float (&v)[8], float c) {
#pragma unroll
    for (int k = 0; k < 8; ++k) s += __builtin_amdgcn_exp2f(fmaf(v[k], c, -mc));
  }

  // add8_lazy's threshold in raw units, mraw + 64 / c (-inf while empty); only
  // add8_lazy moves the reference of an accumulator it is used on
  float lim = -INFINITY;
  __device__ __forceinline__ void add8_lazy(const float (&v)[8], float vmax, float c) {
    // a wavefront-uniform test first keeps the common case a scalar branch
    if (__ballot(vmax > lim) != 0ull && vmax > lim) {  // then vmax > mraw: mc does not decrease
      const float nmc = vmax * c;
      s *= __builtin_amdgcn_exp2f(mc - nmc);
      mc = nmc;
      mraw = vmax;
      lim = vmax + 64.0f / c;
    }
    add8_fixed(v, c);
  }

  __device__ __forceinline__ bool bad() const { return !(s <= 0x1p120f); }

  __device__ __forceinline__ void add8(const float (&v)[8], float c) {
    const float cm = max8(v);
    if (cm > mraw) {
      const float nmc = cm * c;
      s *= __builtin_amdgcn_exp2f(mc - nmc);
      mc = nmc;
      mraw = cm;
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) s += __builtin_amdgcn_exp2f(fmaf(v[k], c, -mc));
  }

  // Wavefront reduction (every lane ends with the row's values).
  __device__ __forceinline__ void reduce() {
    wave_lse2(mc, s);
    mraw = wave_max(mraw);
  }
};

// What the two wavefronts of a row hand to the epilogue.
struct RowShared {
  Best d, t, g;
  float q_mraw, q_mc, q_s;   // draft log-sum-exp (reduced)
  float p_mraw[2], p_mc[2], p_s[2];  // target log-sum-exp partials of the two wavefronts
};

// The lane's slice of a row at g (elements past n read as -inf).
template <typename T>
__device__ __forceinline__ void load_slice(const T* Y, int g, int n, float (&v)[8]) {
  if (g + 8 <= n) {
    load8(Y + g, v);
  } else {
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = (g + k < n) ? load1(Y + g + k) : -INFINITY;
  }
}

// Log-sum-exp of target elements [lo, hi) of a row (guarded at both ends);
// FIXED: against the lane's fixed reference, a whole range without guards.
template <bool FIXED, typename T>
__device__ __forceinline__ void stream_lse(const T* Y, int lo, int hi, int lane, float c2, LaneLse& acc) {
  if (FIXED && hi - lo == kStream) {
    float v0[8], v1[8];
    load8(Y + lo + lane * 8, v0);
    load8(Y + lo + kChunk + lane * 8, v1);
    acc.add8_fixed(v0, c2);
    acc.add8_fixed(v1, c2);
    return;
  }
  for (int g = lo + lane * 8; g - lane * 8 < hi; g += kChunk) {
    float v[8];
    load_slice(Y, g, hi, v);
    if (FIXED)
      acc.add8_fixed(v, c2);
    else
      acc.add8(v, c2);
  }
}

// Wavefront w of a row streams the target ranges [lo, lo + kStream) with
// lo = w kStream + j 2 kStream: the reference of its accumulator comes from
// its lane's first slice, and the careful recomputation repeats every range.
template <typename T>
__device__ __forceinline__ void stream_start(const T* Y, int w, int Vt, int lane, float c2, LaneLse& acc) {
  float v[8];
  load_slice(Y, w * kStream + lane * 8, min(w * kStream + kStream, Vt), v);
  acc.start8(v, c2);
}
template <typename T>
__device__ void stream_redo(const T* Y, int w, int Vt, int lane, float c2, LaneLse& acc) {
  acc = LaneLse{};
  for (int lo = w * kStream; lo < Vt; lo += 2 * kStream) stream_lse<false>(Y, lo, min(lo + kStream, Vt), lane, c2, acc);
}

// Careful recomputation over the lane's slices g = lane 8 + j kChunk of a row
// of n elements (the chunk layout of both wavefronts).
template <typename T>
__device__ void row_redo(const T* X, int n, int lane, float c, LaneLse& acc) {
  acc = LaneLse{};
  for (int g = lane * 8; g < n; g += kChunk) {
    float v[8];
    load_slice(X, g, n, v);
    acc.add8(v, c);
  }
}

// The draft wavefront of a row: z~ and, fused, the draft log-sum-exp and one
// half of the target stream.
template <typename T, bool MAPPED, bool FUSED>
__device__ void draft_wave(const T* X, const T* Y, int Vd, int Vt, FamilyDraw& f, LaneLse& lq, LaneLse& lp,
                           float cp2, int lane) {
  const int nfull = Vd / kChunk;
  if (FUSED && MAPPED) stream_start(Y, 0, Vt, lane, cp2, lp);
  if (nfull > 0) {
    Raw8<T> xr;
    xr.load(X + lane * 8);
    for (int it = 0; it < nfull; ++it) {
      const int base = it * kChunk + lane * 8;
      Raw8<T> xn;
      if (it + 1 < nfull) xn.load(X + base + kChunk);
      float x[8];
      xr.unpack(x);
      if (FUSED && MAPPED) {  // before the draws: the target wavefront's gathers of this
        // block's mapped elements then find its lines in L2 more often
        const int lo = it * 2 * kStream;
        stream_lse<true>(Y, min(lo, Vt), min(lo + kStream, Vt), lane, cp2, lp);
      }
      const float xmax = max8(x);
      if (FUSED) lq.add8_lazy(x, xmax, f.c2);
      f.draw8(base, x, xmax, it == 0);
      xr = xn;
    }
  }
  if (nfull * kChunk < Vd) {  // the partial last chunk
    const int base = nfull * kChunk + lane * 8;
    const int nvalid = min(8, max(0, Vd - base));
    float x[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) x[k] = k < nvalid ? load1(X + base + k) : -INFINITY;
    if (FUSED) lq.add8(x, f.c2);
    f.draw(base, x, nvalid);
    if (FUSED && MAPPED) {
      const int lo = nfull * 2 * kStream;
      stream_lse<true>(Y, min(lo, Vt), min(lo + kStream, Vt), lane, cp2, lp);
    }
  }
  if (FUSED && MAPPED) {  // target elements past the last chunk's block: even half-blocks
    const int nchunks = (Vd + kChunk - 1) / kChunk;
    for (int lo = nchunks * 2 * kStream; lo < Vt; lo += 2 * kStream)
      stream_lse<true>(Y, lo, min(lo + kStream, Vt), lane, cp2, lp);
  }
}

// The target wavefront of a row: z' and z-bar and, fused, the target
// log-sum-exp (unmapped) or the other half of the target stream (mapped).
template <typename T, bool MAPPED, bool FUSED, bool KL, bool DRAW = true>
__device__ void target_wave(const T* Y, const int32_t* d2t, T* tile, int Vd, int Vt, FamilyDraw& f, Best& bg,
                            LaneLse& lp, bool& map_bad, WaveTopK& tk, int lane) {
  auto same = [](int col) { return col; };
  const int nfull = Vd / kChunk;
  // Greedy maximum: each lane keeps the first of its largest values, gw is the
  // wavefront's largest so far.  A chunk in which no lane's maximum ymax
  // (elements past nvalid hold -inf) exceeds gw changes nothing: an element
  // below gw cannot be the row's maximum, and one equal to gw comes after the
  // element that reached gw (every earlier chunk holds smaller indices), so it
  // loses the tie.  gw rises a few times per row (each a new record of the
  // row so far), whereas some lane of 64 improves on its own maximum in
  // almost every chunk.
  float gw = -INFINITY;
  auto greedy = [&](int base, const float (&y)[8], int nvalid, float ymax) {
    if (__ballot(ymax > gw) == 0ull) return;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const bool better = k < nvalid && y[k] > bg.key;
      bg.key = better ? y[k] : bg.key;
      bg.idx = better ? base + k : bg.idx;
    }
    gw = wave_max(bg.key);
  };
  if (FUSED && MAPPED) stream_start(Y, 1, Vt, lane, f.c2, lp);
  if (nfull > 0) {
    uint32_t t[8];
    T g[8];
    Raw8<T> yr;
    auto load_map = [&](int chunk, uint32_t (&tt)[8]) {
#pragma unroll
      for (int k = 0; k < 8; ++k) tt[k] = (uint32_t)d2t[chunk + k * kWave + lane];
    };
    // map entries are range-checked before the launch (k_map_check reports
    // an out-of-range entry); the buffer's range check keeps every access in
    // the row
    const __amdgpu_buffer_rsrc_t yrow = row_rsrc(Y, row_bytes(Y, Vt));
    auto gather = [&](const uint32_t (&tt)[8]) {
#pragma unroll
      for (int k = 0; k < 8; ++k) buf_gather(yrow, tt[k], g[k]);
    };
    if (MAPPED) {
      load_map(0, t);
      gather(t);
    } else {
      yr.load(Y + lane * 8);
    }
    for (int it = 0; it < nfull; ++it) {
      const int chunk = it * kChunk;
      const int base = chunk + lane * 8;
      const bool next = it + 1 < nfull;
      uint32_t tn[8];
      Raw8<T> yn;
      if (next) {
        if (MAPPED)
          load_map(chunk + kChunk, tn);
        else
          yn.load(Y + base + kChunk);
      }
      if (FUSED && MAPPED) {  // this chunk's target block, second half
        const int lo = it * 2 * kStream + kStream;
        stream_lse<true>(Y, min(lo, Vt), min(lo + kStream, Vt), lane, f.c2, lp);
      }
      float y[8];
      if (MAPPED) {
        // transpose the gathered values through the LDS tile; LDS operations
        // of one wavefront execute in order, so no barrier is needed
#pragma unroll
        for (int k = 0; k < 8; ++k) tile[k * kWave + lane] = g[k];
        load8(tile + lane * 8, y);
      } else {
        yr.unpack(y);
      }
      const float ymax = max8(y);
      if (FUSED && !MAPPED) lp.add8_lazy(y, ymax, f.c2);
      greedy(base, y, 8, ymax);
      if (DRAW) f.draw8(base, y, ymax, it == 0);
      if (KL) {  // a slice whose largest mapped value is below the top-K threshold offers nothing
        if (it == 0) tk.seed_lane_max(ymax, lane);
        if (it == 0 || __ballot(ymax >= tk.thv) != 0ull) tk.append8(y, base, 0xFFu, same, lane);
      }
      if (next) {
        if (MAPPED)
          gather(tn);
        else
          yr = yn;
      }
    }
  }
  if (nfull * kChunk < Vd) {  // the partial last chunk
    const int chunk = nfull * kChunk;
    const int base = chunk + lane * 8;
    const int nvalid = min(8, max(0, Vd - base));
    if (FUSED && MAPPED) {
      const int lo = nfull * 2 * kStream + kStream;
      stream_lse<true>(Y, min(lo, Vt), min(lo + kStream, Vt), lane, f.c2, lp);
    }
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
    float y[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const bool in = k < nvalid;
      y[k] = in ? (MAPPED ? load1(tile + lane * 8 + k) : load1(Y + base + k)) : -INFINITY;
    }
    if (FUSED && !MAPPED) lp.add8(y, f.c2);
    greedy(base, y, nvalid, max8(y));
    if (DRAW) f.draw(base, y, nvalid);
    if (KL) tk.offer8(y, base, nvalid > 0 ? (1u << nvalid) - 1u : 0u, same, lane);
  }
  if (FUSED && MAPPED) {  // target elements past the last chunk's block: odd half-blocks
    const int nchunks = (Vd + kChunk - 1) / kChunk;
    for (int lo = nchunks * 2 * kStream + kStream; lo < Vt; lo += 2 * kStream)
      stream_lse<true>(Y, lo, min(lo + kStream, Vt), lane, f.c2, lp);
  }
}

template <typename T, bool MAPPED, bool FUSED, bool KL>
__global__ __launch_bounds__(256) void k_sample(SampleArgs a) {
  __shared__ __align__(16) T ytile[kRowsPerBlock][kChunk];
  __shared__ RowShared sh[kRowsPerBlock];
  __shared__ float kl_bv[KL ? kRowsPerBlock * kTopKCap : 1];
  __shared__ int kl_bi[KL ? kRowsPerBlock * kTopKCap : 1];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = wave_id();
  const int slot = wave >> 1;       // row within the block
  const bool draft_role = (wave & 1) == 0;
  const int64_t r = (int64_t)blockIdx.x * kRowsPerBlock + slot;
  const bool active = r < a.R;
  bool live = false;
  if (active) {
    const int i = (int)(r % a.L);
    int d = a.L;
    if (a.depth != nullptr) {
      d = a.depth[r / a.L];
      if (d < 1 || d > a.L) {
        if (lane == 0 && draft_role) report_error(a.err, VSD_DEVERR_DEPTH_RANGE);
        d = 0;
      }
    }
    live = i < d;
  }
  const T* X = static_cast<const T*>(a.X) + (active ? r : 0) * a.ld_d;
  const T* Y = static_cast<const T*>(a.Y) + (active ? r : 0) * a.ld_t;
  const float cq2 = a.inv_tq * kLog2e, cp2 = a.inv_tp * kLog2e;
  LaneLse lq, lp;
  if (live) {
    if (draft_role) {
      FamilyDraw f{(uint32_t)r, 0u, a.offset, a.k0, a.k1, a.inv_tq, cq2};
      draft_wave<T, MAPPED, FUSED>(X, Y, a.Vd, a.Vt, f, lq, lp, cp2, lane);
      if (FUSED && lq.bad()) row_redo(X, a.Vd, lane, cq2, lq);
      if (FUSED && MAPPED && lp.bad()) stream_redo(Y, 0, a.Vt, lane, cp2, lp);
      wave_argmax(f.best.key, f.best.idx);
      if (FUSED) {
        lq.reduce();
        lp.reduce();
      }
      if (lane == 0) {
        sh[slot].d = f.best;
        sh[slot].q_mraw = lq.mraw;
        sh[slot].q_mc = lq.mc;
        sh[slot].q_s = lq.s;
        sh[slot].p_mraw[0] = lp.mraw;
        sh[slot].p_mc[0] = lp.mc;
        sh[slot].p_s[0] = lp.s;
      }
    } else {
      FamilyDraw f{(uint32_t)r, 1u, a.offset, a.k0, a.k1, a.inv_tp, cp2};
      Best bg{-INFINITY, 0x7FFFFFFF};
      bool map_bad = false;
      WaveTopK tk;
      if (KL) tk.init(kl_bv + slot * kTopKCap, kl_bi + slot * kTopKCap, a.kl_k);
      target_wave<T, MAPPED, FUSED, KL>(Y, a.d2t, ytile[slot], a.Vd, a.Vt, f, bg, lp, map_bad, tk, lane);
      if (FUSED && lp.bad()) {
        if (MAPPED)
          stream_redo(Y, 1, a.Vt, lane, cp2, lp);
        else
          row_redo(Y, a.Vt, lane, cp2, lp);
      }
      if (map_bad) report_error(a.err, VSD_DEVERR_MAP_RANGE);
      if (KL) {
        tk.finish(lane);
        kl_row_term(tk, X, a.Vd, a.inv_tq, a.inv_tp, a.kl_gscale, a.kl_idx + r * a.kl_k, a.kl_grad + r * a.kl_k,
                    a.kl_row + r, lane);
      }
      wave_argmax(f.best.key, f.best.idx);
      wave_argmax(bg.key, bg.idx);
      if (FUSED) lp.reduce();
      if (lane == 0) {
        sh[slot].t = f.best;
        sh[slot].g = bg;
        sh[slot].p_mraw[1] = lp.mraw;
        sh[slot].p_mc[1] = lp.mc;
        sh[slot].p_s[1] = lp.s;
      }
    }
  }
  __syncthreads();
  if (!active || draft_role) return;
  // epilogue, by the target wavefront's first three lanes
  if (!live) {  // masked slot: tokens -1, score outputs 0, nothing read
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
    if (KL) {
      if (lane < a.kl_k) {
        a.kl_idx[r * a.kl_k + lane] = -1;
        a.kl_grad[r * a.kl_k + lane] = 0.0f;
      }
      if (lane == 0) a.kl_row[r] = 0.0f;
    }
    return;
  }
  const RowShared& s = sh[slot];
  if (lane == 0) {
    a.tok_d[r] = s.d.idx;
    a.tok_t[r] = s.t.idx;
    a.tok_g[r] = s.g.idx;
  }
  if (FUSED && lane < 3) {
    // row statistics in the scorer's shifted form: log q(z) = (x_z - max)/T
    // - ln sum exp((x - max)/T), the scaled maximum's rounding corrected
    const float qt = (log2f(s.q_s) - fmaf(s.q_mraw, cq2, -s.q_mc)) * kLn2;
    const float pmc = fmaxf(s.p_mc[0], s.p_mc[1]);
    const float ps = s.p_s[0] * __builtin_amdgcn_exp2f(s.p_mc[0] - pmc) +
                     s.p_s[1] * __builtin_amdgcn_exp2f(s.p_mc[1] - pmc);
    const float pmraw = fmaxf(s.p_mraw[0], s.p_mraw[1]);
    const float pt = (log2f(ps) - fmaf(pmraw, cp2, -pmc)) * kLn2;
    const int z = lane == 0 ? s.d.idx : lane == 1 ? s.t.idx : s.g.idx;
    const float gap = lse_gap(pmraw, pt, a.inv_tp, s.q_mraw, qt, a.inv_tq);
    float lqv = 0.0f, lav = 0.0f;
    if ((uint32_t)z < (uint32_t)a.Vd) {
      const int32_t zt = MAPPED ? a.d2t[z] : z;
      if ((uint32_t)zt < (uint32_t)a.Vt) {
        const float xz = load1(X + z);
        lqv = (xz - s.q_mraw) * a.inv_tq - qt;
        lav = log_alpha_of(xz, load1(Y + zt), a.inv_tq, a.inv_tp, gap);
      }
    }
    a.la[r * 3 + lane] = lav;
    a.lq[r * 3 + lane] = lqv;
    if (lane == 0) {
      a.lse_q[r] = s.q_mraw * a.inv_tq + qt;
      if (a.lse_p != nullptr) a.lse_p[r] = pmraw * a.inv_tp + pt;
    }
  }
}

template <typename T, bool MAPPED>
__global__ __launch_bounds__(192) void k_sample_step(SampleStepArgs a) {
  __shared__ __align__(16) T ytile[2][kChunk];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = wave_id();  // 0: z~, 1: z', 2: z-bar
  const int64_t path = blockIdx.x;     // the grid has exactly one workgroup per path
  int d = a.L;
  if (a.depth != nullptr) {
    d = a.depth[path];
    if (d < 1 || d > a.L) {
      if (lane == 0 && wave == 0) report_error(a.err, VSD_DEVERR_DEPTH_RANGE);
      d = 0;
    }
  }
  const int64_t r = path * a.L + a.step;
  int32_t* out = wave == 0 ? a.tok_d : wave == 1 ? a.tok_t : a.tok_g;
  if (a.step >= d) {  // masked slot
    if (lane == 0) out[r] = -1;
    return;
  }
  LaneLse unused_q, unused_p;
  if (wave == 0) {
    const T* X = static_cast<const T*>(a.X) + path * a.ld_d;
    FamilyDraw f{(uint32_t)r, 0u, a.offset, a.k0, a.k1, a.inv_tq, a.inv_tq * kLog2e};
    draft_wave<T, MAPPED, false>(X, nullptr, a.Vd, a.Vt, f, unused_q, unused_p, 0.0f, lane);
    wave_argmax(f.best.key, f.best.idx);
    if (lane == 0) out[r] = f.best.idx;
    return;
  }
  const T* Y = static_cast<const T*>(wave == 1 ? a.Y : a.Yg) + path * a.ld_t;
  FamilyDraw f{(uint32_t)r, 1u, a.offset, a.k0, a.k1, a.inv_tp, a.inv_tp * kLog2e};
  Best bg{-INFINITY, 0x7FFFFFFF};
  bool map_bad = false;
  WaveTopK unused_tk;
  if (wave == 1) {
    target_wave<T, MAPPED, false, false, true>(Y, a.d2t, ytile[0], a.Vd, a.Vt, f, bg, unused_p, map_bad, unused_tk,
                                               lane);
    wave_argmax(f.best.key, f.best.idx);
  } else {
    target_wave<T, MAPPED, false, false, false>(Y, a.d2t, ytile[1], a.Vd, a.Vt, f, bg, unused_p, map_bad,
                                                unused_tk, lane);
    wave_argmax(bg.key, bg.idx);
  }
  if (map_bad) report_error(a.err, VSD_DEVERR_MAP_RANGE);
  if (lane == 0) out[r] = wave == 1 ? f.best.idx : bg.idx;
}

// Range check of the map (the sampling kernels clamp map entries instead of
// testing each one): the first entry outside [0, Vt) is reported.
__global__ __launch_bounds__(256) void k_map_check(const int32_t* d2t, int Vd, int Vt, int32_t* err) {
  const int v = blockIdx.x * 256 + threadIdx.x;
  if (v < Vd && (uint32_t)d2t[v] >= (uint32_t)Vt) report_error(err, VSD_DEVERR_MAP_RANGE);
}

template <typename T>
hipError_t launch_step_t(const SampleStepArgs& a, hipStream_t s) {
  if (a.d2t != nullptr) {
    const hipError_t e = launch_map_check(a.d2t, a.Vd, a.Vt, a.err, s);
    if (e != hipSuccess) return e;
  }
  const dim3 grid((unsigned)a.paths);
  if (a.d2t != nullptr)
    hipLaunchKernelGGL((k_sample_step<T, true>), grid, dim3(3 * kWave), 0, s, a);
  else
    hipLaunchKernelGGL((k_sample_step<T, false>), grid, dim3(3 * kWave), 0, s, a);
  return hipGetLastError();
}

template <typename T, bool FUSED, bool KL>
hipError_t launch_t(const SampleArgs& a, hipStream_t s) {
  if (a.d2t != nullptr) {
    const hipError_t e = launch_map_check(a.d2t, a.Vd, a.Vt, a.err, s);
    if (e != hipSuccess) return e;
  }
  const dim3 grid((unsigned)((a.R + kRowsPerBlock - 1) / kRowsPerBlock));
  if (a.d2t != nullptr)
    hipLaunchKernelGGL((k_sample<T, true, FUSED, KL>), grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((k_sample<T, false, FUSED, KL>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_map_check(const int32_t* d2t, int Vd, int Vt, int32_t* err, hipStream_t s) {
  hipLaunchKernelGGL(k_map_check, dim3((unsigned)((Vd + 255) / 256)), dim3(256), 0, s, d2t, Vd, Vt, err);
  return hipGetLastError();
}

hipError_t launch_sample(const SampleArgs& a, bool bf16, hipStream_t s) {
  const bool fused = a.lse_q != nullptr;
  const bool kl = fused && a.kl_k > 0;
  if (bf16) {
    if (kl) return launch_t<bf16_t, true, true>(a, s);
    return fused ? launch_t<bf16_t, true, false>(a, s) : launch_t<bf16_t, false, false>(a, s);
  }
  if (kl) return launch_t<float, true, true>(a, s);
  return fused ? launch_t<float, true, false>(a, s) : launch_t<float, false, false>(a, s);
}

hipError_t launch_sample_step(const SampleStepArgs& a, bool bf16, hipStream_t s) {
  return bf16 ? launch_step_t<bf16_t>(a, s) : launch_step_t<float>(a, s);
}

}  // namespace vsd
