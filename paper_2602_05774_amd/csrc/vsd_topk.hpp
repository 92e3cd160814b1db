// Exact top-K of (value, index) pairs offered by one wavefront, K <= kMaxTopK.
//
// Order: the larger value first, equal values by the smaller index.  An offer
// takes part only if it is not below the current K-th best (a
// wavefront-uniform threshold, -inf until K entries are known); such offers
// are appended to a per-wavefront LDS buffer at positions counted from one
// ballot per slice position.  Whenever more than 64 entries are buffered the
// wavefront selects the K best (K rounds of wavefront argmax), keeps them at
// the front in order and raises the threshold.  An element below the
// threshold is worse than K known elements, so it cannot be in the final top
// K: the result is exact.  After finish() the K best are at the front of the
// buffer, in order.  -inf marks empty slots: a -inf offer never becomes an
// entry.
// Every call must be made by all 64 lanes of the wavefront.
#pragma once

#include "vsd_device.hpp"

namespace vsd {

constexpr int kMaxTopK = 16;
constexpr int kTopKCap = 640;   // entries per wavefront buffer (a full round of 8 offers per lane fits)

struct WaveTopK {
  float* bv;   // LDS [kTopKCap]
  int* bi;     // LDS [kTopKCap]
  int n;       // buffered entries (wavefront-uniform)
  int K;
  float thv;   // threshold (K-th best so far)
  int thi;

  __device__ __forceinline__ static bool beats(float v, int i, float ov, int oi) {
    return v > ov || (v == ov && i < oi);
  }

  __device__ __forceinline__ void init(float* v, int* i, int k) {
    bv = v;
    bi = i;
    n = 0;
    K = k;
    thv = -INFINITY;
    thi = 0x7FFFFFFF;
  }

  // Before the first offer: raise the threshold to the K-th largest of the
  // lanes' slice maxima vmax.  K lanes hold an element at least that large,
  // so an element below it is worse than K elements that the first offer
  // appends: the selection stays exact, and the first chunk appends about K
  // entries instead of all of them.
  __device__ void seed_lane_max(float vmax, int lane) {
    if (K > kWave) return;
    float v = vmax, kth = -INFINITY;
    int r = 0;
    for (; r < K; ++r) {
      const float m = wave_max(v);
      if (m == -INFINITY) break;
      const uint64_t b = __ballot(v == m);
      if (lane == __builtin_ctzll(b)) v = -INFINITY;  // one occurrence
      kth = m;
    }
    if (r == K && kth > thv) {
      thv = kth;
      thi = 0x7FFFFFFF;
    }
  }

  // Offer a lane's 8 values x of columns base .. base+7 (bit k of `bits`:
  // column base+k takes part).  A value equal to the threshold is appended
  // too (its index decides at the next compaction).  Returns at once when no
  // lane has a candidate; idx_of(col) gives the index kept with an entry.
  template <class IdxOf>
  __device__ __forceinline__ void offer8(const float (&x)[8], int base, uint32_t bits, IdxOf idx_of, int lane) {
    float best = -INFINITY;
#pragma unroll
    for (int k = 0; k < 8; ++k) best = ((bits >> k) & 1u) ? fmaxf(best, x[k]) : best;
    if (__ballot(best >= thv) == 0ull) return;
    append8(x, base, bits, idx_of, lane);
  }

  // append8 without the early exit: for callers that already know some
  // lane's offered maximum reaches the threshold.
  template <class IdxOf>
  __device__ __forceinline__ void append8(const float (&x)[8], int base, uint32_t bits, IdxOf idx_of, int lane) {
    uint32_t q = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) q |= (((bits >> k) & 1u) && x[k] >= thv) ? (1u << k) : 0u;
    if (__ballot((q & (q - 1u)) != 0u) == 0ull) {
      // At most one candidate per lane, the common case once the threshold
      // has risen: one ballot places them, and the lane's entry is picked
      // from its slice by selects.  (n <= 64 before the call, so the at
      // most 64 new entries fit.)
      const uint64_t has = __ballot(q != 0u);
      const int total = __builtin_popcountll(has);
      if (q != 0u) {
        // the entry at slice position k = ctz(q), by a tree of selects on
        // k's bits (no indexed access to the register arrays)
        const uint32_t k = (uint32_t)__builtin_ctz(q);
        const bool b0 = (k & 1u) != 0u, b1 = (k & 2u) != 0u, b2 = (k & 4u) != 0u;
        const float v01 = b0 ? x[1] : x[0], v23 = b0 ? x[3] : x[2];
        const float v45 = b0 ? x[5] : x[4], v67 = b0 ? x[7] : x[6];
        const float v = b2 ? (b1 ? v67 : v45) : (b1 ? v23 : v01);
        const int i01 = b0 ? idx_of(base + 1) : idx_of(base), i23 = b0 ? idx_of(base + 3) : idx_of(base + 2);
        const int i45 = b0 ? idx_of(base + 5) : idx_of(base + 4), i67 = b0 ? idx_of(base + 7) : idx_of(base + 6);
        const int id = b2 ? (b1 ? i67 : i45) : (b1 ? i23 : i01);
        const int pos = n + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(has >> 32),
                                                           __builtin_amdgcn_mbcnt_lo((uint32_t)has, 0u));
        bv[pos] = v;
        bi[pos] = id;
      }
      n += total;
    } else {
      append8_dense(x, base, q, idx_of);
    }
    if (n > kWave) compact(lane);  // keeps the threshold close to the K-th best so far
  }

  // The general append: q holds each lane's candidate positions.
  template <class IdxOf>
  __device__ __forceinline__ void append8_dense(const float (&x)[8], int base, uint32_t q, IdxOf idx_of) {
    // positions by slice position k, then by lane: one ballot per k and the
    // count of lower lanes in it (the buffer's order is irrelevant to the
    // selection, which orders by value and index)
    uint64_t bal[8];
    int total = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      bal[k] = __ballot((q >> k) & 1u);
      total += __builtin_popcountll(bal[k]);
    }
    int pos0 = n;  // n <= 64 before the call and total <= 512: the buffer holds them
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      if ((q >> k) & 1u) {
        const int pos = pos0 + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(bal[k] >> 32),
                                                              __builtin_amdgcn_mbcnt_lo((uint32_t)bal[k], 0u));
        bv[pos] = x[k];
        bi[pos] = idx_of(base + k);
      }
      pos0 += __builtin_popcountll(bal[k]);
    }
    n += total;
  }

  // Keep the K best buffered entries, in order, at the front.  Selected
  // entries are marked in LDS (value -inf); the K winners are written after
  // the last scan.
  __device__ void compact(int lane) {
    if (n <= kWave) {
      compact_small(lane);
      return;
    }
    float kv = -INFINITY;
    int ki = 0x7FFFFFFF;
    int cnt = 0;
    for (int r = 0; r < K; ++r) {
      float lv = -INFINITY;
      int li = 0x7FFFFFFF, lj = -1;
      for (int j = lane; j < n; j += kWave) {
        const float v = bv[j];
        const int i = bi[j];
        if (beats(v, i, lv, li)) {
          lv = v;
          li = i;
          lj = j;
        }
      }
      float wv = lv;
      int wi = li;
      wave_argmax(wv, wi);
      if (wv == -INFINITY) break;
      if (lj >= 0 && li == wi && lv == wv) bv[lj] = -INFINITY;  // indices are unique: one owner
      if (lane == r) {
        kv = wv;
        ki = wi;
      }
      ++cnt;
    }
    if (lane < cnt) {
      bv[lane] = kv;
      bi[lane] = ki;
    }
    n = cnt;
    if (cnt == K) {
      thv = lane_f(kv, K - 1);
      thi = lane_i(ki, K - 1);
    }
  }

  // compact() for at most one entry per lane.
  __device__ void compact_small(int lane) {
    float ev = lane < n ? bv[lane] : -INFINITY;
    int ei = lane < n ? bi[lane] : 0x7FFFFFFF;
    float kv = -INFINITY;
    int ki = 0x7FFFFFFF;
    int cnt = 0;
    for (int r = 0; r < K; ++r) {
      float wv = ev;
      int wi = ei;
      wave_argmax(wv, wi);
      if (wv == -INFINITY) break;
      if (ei == wi && ev == wv) {
        ev = -INFINITY;
        ei = 0x7FFFFFFF;
      }
      if (lane == r) {
        kv = wv;
        ki = wi;
      }
      ++cnt;
    }
    if (lane < cnt) {
      bv[lane] = kv;
      bi[lane] = ki;
    }
    n = cnt;
    if (cnt == K) {
      thv = lane_f(kv, K - 1);
      thi = lane_i(ki, K - 1);
    }
  }

  __device__ __forceinline__ void finish(int lane) { compact(lane); }
};

// The KL term of one row (Eq. klv) from its members' values held by the
// lanes: lane k < K holds member k (mine), its draft index v (-1: none),
// target logit y and draft logit x.  p_hat and q_hat (from y / T_p and
// x / T_q) are renormalised over the members, the row term
// -sum p_hat log q_hat goes to *row_out (lane 0) and the gradient
// coefficients gscale (q_hat - p_hat) with the indices to idx_out / grad_out
// (index -1 and coefficient 0 past the members).
__device__ inline void kl_row_term_xy(bool mine, int v, float y, float x, int K, float inv_tq, float inv_tp,
                                      float gscale, int32_t* idx_out, float* grad_out, float* row_out, int lane) {
  const float pa = mine ? y * inv_tp : -INFINITY;
  const float qa = v >= 0 ? x * inv_tq : -INFINITY;
  const float pm = wave_max(pa), qm = wave_max(qa);
  const float pe = mine ? expf(pa - pm) : 0.0f;
  const float qe = mine ? expf(qa - qm) : 0.0f;
  const float ps = wave_sum(pe), qs = wave_sum(qe);
  const float p_hat = pe / ps, q_hat = qe / qs;
  const float log_q_hat = qa - qm - logf(qs);
  const float term = wave_sum(mine ? -p_hat * log_q_hat : 0.0f);
  if (lane < K) {
    idx_out[lane] = mine ? v : -1;
    grad_out[lane] = mine ? gscale * (q_hat - p_hat) : 0.0f;
  }
  if (lane == 0) *row_out = term;
}

// The same term from a materialised row's top K, after WaveTopK::finish():
// lane k < K takes the k-th entry (draft index v, target logit y) and reads
// x = X[v].  Only finite values become entries (a -inf offer is dropped at the next
// compaction), so a row with fewer than K finite mapped target logits has
// fewer than K entries: the distributions are renormalised over those, and
// the slots past them get index -1 and coefficient 0.  An index is read from
// X only if it lies in [0, Vd).
template <typename T>
__device__ void kl_row_term(const WaveTopK& tk, const T* X, int Vd, float inv_tq, float inv_tp, float gscale,
                            int32_t* idx_out, float* grad_out, float* row_out, int lane) {
  const bool mine = lane < tk.n && lane < tk.K;
  int v = mine ? tk.bi[lane] : -1;
  v = (uint32_t)v < (uint32_t)Vd ? v : -1;
  const float y = mine ? tk.bv[lane] : -INFINITY;
  const float x = v >= 0 ? load1(X + v) : -INFINITY;
  kl_row_term_xy(mine, v, y, x, tk.K, inv_tq, inv_tp, gscale, idx_out, grad_out, row_out, lane);
}

}  // namespace vsd
