// Draw machinery shared by the sampling kernels: raw 8-element row slices,
// the (key, index) state of a draw and one family's Philox draws with the
// exact candidate filter (k_sample.hip states why the filter is exact).
#pragma once

#include "vsd_device.hpp"

namespace vsd {

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

// State and steps common to both wavefronts of a row: the Philox draws and
// the exact filter of one family.  Every call must be made by all 64 lanes
// of the wavefront (lanes without elements pass values of -inf): the seed and
// the threshold's refresh are wavefront reductions.
struct FamilyDraw {
  uint32_t row, fam, offset, k0, k1;
  float inv_t, c2;  // 1/T and log2(e)/T
  Best best{-INFINITY, 0x7FFFFFFF};
  // A lower bound of the row's best key: the wavefront maximum of the keys
  // found so far, or the seeded bound of draw8 while that is larger.
  float wave_best = -INFINITY;
  // bound_offset(wave_best): after every draw no lane's best exceeds
  // wave_best, so the threshold is wave_best itself and the offset changes
  // only when wave_best changes
  float off = INFINITY;

  __device__ __forceinline__ uint4 philox(uint32_t c0) const { return philox4x32_10(c0, row, fam, offset, k0, k1); }

  // (thr - margin) log2e folded into the bound's constant.  The margin
  // 2e-3 + 2e-6 |thr| exceeds every rounding involved for elements with
  // |x/T| <= |thr| + 100; an element with x/T < thr - 100 cannot reach thr
  // because G < 16.7.
  __device__ __forceinline__ static float bound_offset(float thr) {
    return 24.0f - (thr - (2e-3f + 2e-6f * fabsf(thr))) * kLog2e;
  }

  // Whether any lane's slice with maximum vmax can reach the threshold at
  // all: every word gives G < 24 ln 2 (u <= 1 - 2^-24), which is the bound
  // (24 - log2 j') ln 2 at j' = 1, so a slice failing it for log2 j' = 0
  // fails for every word and needs no Philox draw.  Peaked rows skip most of
  // their slices this way once their top elements are known.
  __device__ __forceinline__ bool reachable(float vmax) const {
    return __ballot(fmaf(vmax, c2, off) >= 0.0f) != 0ull;
  }

  // Bound test of the 4 elements that share one Philox counter: bit k set
  // where v * log2e/T + off >= log2(j').
  __device__ __forceinline__ static uint32_t cand4(const uint4& w, const float* v, float c2, float off) {
    uint32_t m = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const bool c = fmaf(v[k], c2, off) >= __builtin_amdgcn_logf((float)((~word_of(w, k)) >> 8));
      m |= c ? (1u << k) : 0u;
    }
    return m;
  }

  // Draw the lane's 8 elements at `base` (values v, the first nvalid valid).
  // A full slice is first tested as a whole: the largest value vmax against
  // the largest Philox word (the smallest j').  If that pair fails the bound,
  // every element fails it: v_k c2 + off <= vmax c2 + off < log2(j'_min) <=
  // log2(j'_k) up to the same rounding of the one log that the margin already
  // covers.
  __device__ __forceinline__ void draw(int base, const float (&v)[8], int nvalid) {
    if (nvalid == 8) {
      draw8(base, v, max8(v));
      return;
    }
    if (!reachable(max8(v))) return;  // elements past nvalid hold -inf
    const uint32_t c0 = (uint32_t)base >> 2;
    const uint32_t cand = (cand4(philox(c0), v, c2, off) | (cand4(philox(c0 + 1), v + 4, c2, off) << 4)) &
                          ((1u << nvalid) - 1u);
    exact(base, v, c0, cand);
  }
  // seed = true (the row's first full slice): before the test, raise the
  // wavefront threshold to a lower bound of the row's best key taken from
  // these elements.  With d = 1 - u (exact on the 2^-24 grid), -ln u <= d / u,
  // so G = -ln(-ln u) >= ln u - ln d; x/T + ln u - ln d less a margin that
  // covers the hardware logarithms and the key's two roundings is below the
  // element's normative key, hence below the row's best.  The element that
  // attains the wavefront maximum of that bound still passes the filter, so
  // the best key found afterwards reaches the seeded threshold.  Without the
  // seed every element of a row's first chunk would take the exact key.
  __device__ __forceinline__ void draw8(int base, const float (&v)[8], float vmax, bool seed = false) {
    const uint32_t c0 = (uint32_t)base >> 2;
    if (seed) {
      const uint4 p0 = philox(c0), p1 = philox(c0 + 1);
      float lo[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float u = uniform_from_word(word_of(k < 4 ? p0 : p1, k & 3));
        const float g = (__builtin_amdgcn_logf(u) - __builtin_amdgcn_logf(1.0f - u)) * kLn2;
        lo[k] = v[k] * inv_t + g;
      }
      float thr = wave_max(max8(lo));
      thr -= 1e-3f + 1e-5f * fabsf(thr);
      if (thr > wave_best && thr < INFINITY) {
        wave_best = thr;
        off = bound_offset(thr);
      }
    }
    if (!reachable(vmax)) return;
    const uint4 p0 = philox(c0), p1 = philox(c0 + 1);
    const uint32_t wmax = max(max(max(p0.x, p0.y), max(p0.z, p0.w)), max(max(p1.x, p1.y), max(p1.z, p1.w)));
    const bool maybe = fmaf(vmax, c2, off) >= __builtin_amdgcn_logf((float)((~wmax) >> 8));
    if (__ballot(maybe) == 0ull) return;
    exact(base, v, c0, maybe ? cand4(p0, v, c2, off) | (cand4(p1, v + 4, c2, off) << 4) : 0u);
  }
  // Exact keys of the candidates (bit k of cand: element base + k).  Each
  // round takes every lane's lowest remaining candidate, so a round evaluates
  // one key per lane that has one and the rounds number the largest count in
  // a lane (a single key's code, not one per slice position).  A lane's
  // candidates come in increasing index order, after the smaller indices of
  // its earlier chunks, so the strict comparison keeps the first of equal
  // keys.
  __device__ __forceinline__ void exact(int base, const float (&v)[8], uint32_t c0, uint32_t cand) {
    if (__ballot(cand != 0u) == 0ull) return;
    // the candidate's Philox word is recomputed (the counter made opaque), so
    // no word of the slice stays alive through the exact keys
    asm volatile("" : "+v"(c0));
    while (cand != 0u) {
      const int k = __builtin_ctz(cand);
      cand &= cand - 1u;
      // v[k] by selects; the empty asm keeps the compiler from turning the
      // chain into an indexed stack array
      float x = v[0];
#pragma unroll
      for (int j = 1; j < 8; ++j) {
        x = k == j ? v[j] : x;
        asm volatile("" : "+v"(x));
      }
      const float key = gumbel_key(x, inv_t, word_of(philox(c0 + ((uint32_t)k >> 2)), k & 3));
      if (key > best.key) {
        best.key = key;
        best.idx = base + k;
      }
    }
    if (__ballot(best.key > wave_best) != 0ull) {
      wave_best = wave_max(best.key);
      off = bound_offset(wave_best);
    }
  }
};

}  // namespace vsd
