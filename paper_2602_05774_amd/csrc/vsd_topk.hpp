// Exact top-K of (value, index) pairs offered by one wavefront, K <= kMaxTopK.
//
// Order: the larger value first, equal values by the smaller index.  An offer
// qualifies only if it beats the current K-th best (a wavefront-uniform
// threshold, -inf until K entries are known); qualifying offers are appended
// to a per-wavefront LDS buffer at positions given by a ballot prefix count.
// When the next round of offers could overflow the buffer the wavefront
// selects the K best buffered entries (K rounds of wavefront argmax), keeps
// them at the front in order and raises the threshold.  An element that fails
// the threshold is worse than K known elements, so it cannot be in the final
// top K: the result is exact.  After finish() the K best are at the front of
// the buffer, in order.  Values must not be -inf (sentinel of empty slots).
#pragma once

#include "vsd_device.hpp"

namespace vsd {

constexpr int kMaxTopK = 16;
constexpr int kTopKCap = 1024;  // entries per wavefront buffer

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

  // One offer per lane: value v of column col (valid lanes only); idx_of(col)
  // gives the index the order and the result use (evaluated for lanes that
  // reach the threshold only).  At most 64 entries are appended.
  template <class IdxOf>
  __device__ __forceinline__ void offer(float v, int col, bool valid, IdxOf idx_of, int lane) {
    bool q = valid && v >= thv;
    if (__ballot(q) == 0ull) return;
    int idx = 0x7FFFFFFF;
    if (q) {
      idx = idx_of(col);
      q = beats(v, idx, thv, thi);
    }
    const uint64_t m = __ballot(q);
    if (m == 0ull) return;
    if (q) {
      const int pos = n + (int)__builtin_popcountll(m & ((1ull << lane) - 1ull));
      bv[pos] = v;
      bi[pos] = idx;
    }
    n += (int)__builtin_popcountll(m);
  }

  // Room for `upcoming` more entries, compacting first if needed.
  __device__ __forceinline__ void reserve(int upcoming, int lane) {
    if (n + upcoming > kTopKCap) compact(lane);
  }

  // Keep the K best buffered entries, in order, at the front.
  __device__ void compact(int lane) {
    constexpr int kPer = kTopKCap / kWave;
    float ev[kPer];
    int ei[kPer];
    const int nt = (n + kWave - 1) / kWave;
#pragma unroll
    for (int t = 0; t < kPer; ++t) {
      const int j = lane + kWave * t;
      const bool in = t < nt && j < n;
      ev[t] = in ? bv[j] : -INFINITY;
      ei[t] = in ? bi[j] : 0x7FFFFFFF;
    }
    float kv = -INFINITY;
    int ki = 0x7FFFFFFF;
    int cnt = 0;
    for (int r = 0; r < K; ++r) {
      float lv = -INFINITY;
      int li = 0x7FFFFFFF;
#pragma unroll
      for (int t = 0; t < kPer; ++t) {
        if (t < nt && beats(ev[t], ei[t], lv, li)) {
          lv = ev[t];
          li = ei[t];
        }
      }
      float wv = lv;
      int wi = li;
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) {
        const float ov = __shfl_xor(wv, off, kWave);
        const int oi = __shfl_xor(wi, off, kWave);
        if (beats(ov, oi, wv, wi)) {
          wv = ov;
          wi = oi;
        }
      }
      if (wv == -INFINITY) break;  // fewer than K entries buffered
      // indices are unique, so exactly one entry matches the winner
#pragma unroll
      for (int t = 0; t < kPer; ++t) {
        if (t < nt && ei[t] == wi && ev[t] == wv) {
          ev[t] = -INFINITY;
          ei[t] = 0x7FFFFFFF;
        }
      }
      if (lane == r) {
        kv = wv;
        ki = wi;
      }
      ++cnt;
    }
    // this wavefront's LDS reads above precede these writes (in order)
    if (lane < cnt) {
      bv[lane] = kv;
      bi[lane] = ki;
    }
    n = cnt;
    if (cnt == K) {
      thv = __shfl(kv, K - 1, kWave);
      thi = __shfl(ki, K - 1, kWave);
    }
  }

  __device__ __forceinline__ void finish(int lane) { compact(lane); }
};

}  // namespace vsd
