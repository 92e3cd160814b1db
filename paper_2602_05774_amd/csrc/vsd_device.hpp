// Device-side helpers shared by the VSD kernels (gfx950, wave64).
//
//  * Philox4x32-10 (Salmon et al., SC'11) and the library's normative float32
//    logarithm / Gumbel variate, exactly as the sampler definition in vsd.h
//    states them: one IEEE binary32 operation per step, no contraction.
//  * 128-bit loads of 8 logits (bf16 or fp32) and 128-bit bf16 stores.
//  * Wavefront reductions (butterfly over all 64 lanes, so every lane ends
//    with the same, order-independent result).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/vsd.h"

namespace vsd {

constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kNegBig = -3.402823466e+38f;  // -FLT_MAX: an "empty" max

using bf16_t = uint16_t;  // bf16 storage

// ---------------------------------------------------------------- Philox ---
__device__ __forceinline__ void mulhilo32(uint32_t a, uint32_t b, uint32_t& hi, uint32_t& lo) {
  const uint64_t p = (uint64_t)a * (uint64_t)b;  // v_mad_u64_u32
  hi = (uint32_t)(p >> 32);
  lo = (uint32_t)p;
}

// a ^ b ^ c in one gfx950 instruction (v_bitop3_b32, truth table 0x96).
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c) {
  return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);
}

// Ten Philox4x32 rounds on counter (c0,c1,c2,c3) with key (k0,k1): per round
// two 32x32->64 multiplies (v_mad_u64_u32) and two three-way XORs.
__device__ __forceinline__ uint4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                               uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int j = 0; j < 10; ++j) {
    uint32_t hi0, lo0, hi1, lo1;
    mulhilo32(0xD2511F53u, c0, hi0, lo0);
    mulhilo32(0xCD9E8D57u, c2, hi1, lo1);
    const uint32_t n0 = xor3(hi1, c1, k0);
    const uint32_t n2 = xor3(hi0, c3, k1);
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return make_uint4(c0, c1, c2, c3);
}

// ------------------------------------------------- normative log / Gumbel ---
// Natural log of a positive normal float: x = 2^e m, m in (sqrt(1/2), sqrt(2)],
// log m = 2 atanh(f / (2 + f)) by its odd series through s^9, e ln2 split
// hi/lo.  Every line is one correctly rounded binary32 operation.
__device__ __forceinline__ float spec_log(float x) {
#pragma clang fp contract(off)
  const uint32_t b = __float_as_uint(x);
  int e = (int)((b >> 23) & 0xFFu) - 127;
  float m = __uint_as_float((b & 0x7FFFFFu) | 0x3F800000u);
  if (m > __uint_as_float(0x3FB504F3u)) {
    m = m * 0.5f;
    e = e + 1;
  }
  const float f = m - 1.0f;
  const float s = f / (2.0f + f);
  const float z = s * s;
  float p = __uint_as_float(0x3DE38E39u);        // 1/9
  p = __uint_as_float(0x3E124925u) + z * p;      // 1/7
  p = __uint_as_float(0x3E4CCCCDu) + z * p;      // 1/5
  p = __uint_as_float(0x3EAAAAABu) + z * p;      // 1/3
  const float t2 = s + s;
  const float lm = t2 + t2 * (z * p);
  const float ef = (float)e;
  return ef * __uint_as_float(0x3F317200u) + (lm + ef * __uint_as_float(0x35BFBE8Eu));
}

// u = (2 (w >> 9) + 1) 2^-24: 2^23 equally spaced values in (0, 1), exact.
__device__ __forceinline__ float uniform_from_word(uint32_t w) {
  return (float)(2u * (w >> 9) + 1u) * 5.9604644775390625e-8f;
}

// G = -log(-log u), u = uniform_from_word(w).
__device__ __forceinline__ float gumbel_from_word(uint32_t w) {
#pragma clang fp contract(off)
  const float u = uniform_from_word(w);
  const float e = -spec_log(u);
  return -spec_log(e);
}

// key = float(logit * invT) + G   (two roundings, as the definition fixes).
__device__ __forceinline__ float gumbel_key(float logit, float inv_t, uint32_t w) {
#pragma clang fp contract(off)
  const float xs = logit * inv_t;
  return xs + gumbel_from_word(w);
}

// ----------------------------------------------------------- loads/stores ---
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

__device__ __forceinline__ void load8(const float* p, float (&v)[8]) {
  const float4 a = reinterpret_cast<const float4*>(p)[0];
  const float4 b = reinterpret_cast<const float4*>(p)[1];
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

__device__ __forceinline__ void load8(const bf16_t* p, float (&v)[8]) {
  const uint4 a = *reinterpret_cast<const uint4*>(p);
  v[0] = bf16_lo(a.x); v[1] = bf16_hi(a.x);
  v[2] = bf16_lo(a.y); v[3] = bf16_hi(a.y);
  v[4] = bf16_lo(a.z); v[5] = bf16_hi(a.z);
  v[6] = bf16_lo(a.w); v[7] = bf16_hi(a.w);
}

__device__ __forceinline__ void load8(const int32_t* p, int32_t (&v)[8]) {
  const int4 a = reinterpret_cast<const int4*>(p)[0];
  const int4 b = reinterpret_cast<const int4*>(p)[1];
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

__device__ __forceinline__ float load1(const float* p) { return *p; }
__device__ __forceinline__ float load1(const bf16_t* p) { return __uint_as_float((uint32_t)(*p) << 16); }

// Gathers from one row through a raw buffer resource (the row's base and
// size wave-uniform, so the descriptor lives in scalar registers): the byte
// offset is the only per-lane address arithmetic (no 64-bit address, no
// clamp), and the hardware returns 0 for an offset at or past the row's
// size, so no access leaves the row whatever the index.  Callers use it for
// indices from a map whose range is checked and reported elsewhere.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(const void* row, uint32_t bytes) {
  // word 3 of a gfx9 buffer descriptor: 32-bit data format, no swizzle
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(row), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ uint32_t row_bytes(const float*, int n) { return (uint32_t)n * 4u; }
__device__ __forceinline__ uint32_t row_bytes(const bf16_t*, int n) { return (uint32_t)n * 2u; }
// raw element idx of the row (the byte offset is formed modulo 2^32; any
// value of it is inside the row or answered with zero by the range check)
__device__ __forceinline__ void buf_gather(__amdgpu_buffer_rsrc_t r, uint32_t idx, float& out) {
  out = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)(idx * 4u), 0, 0));
}
__device__ __forceinline__ void buf_gather(__amdgpu_buffer_rsrc_t r, uint32_t idx, bf16_t& out) {
  out = __builtin_amdgcn_raw_buffer_load_b16(r, (int)(idx * 2u), 0, 0);
}

// fp32 -> bf16, round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const __bf16 a = (__bf16)lo;
  const __bf16 b = (__bf16)hi;
  return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

__device__ __forceinline__ void store8(float* p, const float (&v)[8]) {
  reinterpret_cast<float4*>(p)[0] = make_float4(v[0], v[1], v[2], v[3]);
  reinterpret_cast<float4*>(p)[1] = make_float4(v[4], v[5], v[6], v[7]);
}

__device__ __forceinline__ void store8(bf16_t* p, const float (&v)[8]) {
  *reinterpret_cast<uint4*>(p) = make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                                            pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7]));
}

__device__ __forceinline__ void store1(float* p, float v) { *p = v; }
__device__ __forceinline__ void store1(bf16_t* p, float v) {
  *p = __builtin_bit_cast(uint16_t, (__bf16)v);
}

// log alpha = min(0, log p(z) - log q(z)) (Eq. acc) of a token with draft
// logit x and target logit y, grouped as (y/T_p - x/T_q) - gap with the row
// constant gap = lse_p - lse_q.  At temperatures that are powers of two the
// first difference is exact for bf16 logits, so tokens of one row with equal
// y/T_p - x/T_q (common on bf16 grids) get bitwise equal values and the
// oracle gate sees their tie exactly (equality accepts).
__device__ __forceinline__ float log_alpha_of(float x, float y, float inv_tq, float inv_tp, float gap) {
#pragma clang fp contract(off)
  return fminf(0.0f, (y * inv_tp - x * inv_tq) - gap);
}

// gap = lse_p - lse_q from each log-sum-exp's raw maximum m and tail t (lse =
// m/T + t): the maxima are logit values, so their tempered difference is
// exact wherever y/T_p - x/T_q is, and only the small tails round.
__device__ __forceinline__ float lse_gap(float pm, float pt, float inv_tp, float qm, float qt, float inv_tq) {
#pragma clang fp contract(off)
  return (pm * inv_tp - qm * inv_tq) + (pt - qt);
}

// Index of the calling wavefront within its workgroup, as a wavefront-uniform
// (scalar) value: everything derived from it (row indices, row pointers,
// Philox counter words) then lives in scalar registers.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// ------------------------------------------------------------ lane math ---
// max(a, b, c) in one instruction (v_max3_f32).
__device__ __forceinline__ float max3f(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// Largest of 8 values in four instructions (all v_max3_f32: a plain fmaxf of
// the asm results would first quiet both operands).
__device__ __forceinline__ float max8(const float (&v)[8]) {
  return max3f(max3f(v[0], v[1], v[2]), max3f(v[3], v[4], v[5]), max3f(v[6], v[7], v[7]));
}

// ------------------------------------------------------ wave reductions ---
// Every lane must be active.  Within each row of 16 lanes the values meet
// through DPP lane permutations (quad_perm [1,0,3,2], quad_perm [2,3,0,1],
// row_half_mirror, row_mirror: after them every lane holds its row's
// result); the four row results are then read with readlane and combined in
// a fixed order, so every lane ends with the same, run-to-run identical
// value and no LDS permute is needed.
template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(dpp_i<CTRL>(__float_as_int(v)));
}
__device__ __forceinline__ float lane_f(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
__device__ __forceinline__ int lane_i(int v, int l) { return __builtin_amdgcn_readlane(v, l); }
constexpr int kDppQuad1 = 0xB1;       // quad_perm [1,0,3,2]
constexpr int kDppQuad2 = 0x4E;       // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141; // row_half_mirror
constexpr int kDppMirror = 0x140;     // row_mirror

// (key, index) maximum; equal keys resolve to the smaller index.
__device__ __forceinline__ void argmax_merge(float& key, int& idx, float ok, int oi) {
  if (ok > key || (ok == key && oi < idx)) {
    key = ok;
    idx = oi;
  }
}
template <int CTRL>
__device__ __forceinline__ void argmax_step(float& key, int& idx) {
  argmax_merge(key, idx, dpp_f<CTRL>(key), dpp_i<CTRL>(idx));
}
__device__ __forceinline__ void wave_argmax(float& key, int& idx) {
  argmax_step<kDppQuad1>(key, idx);
  argmax_step<kDppQuad2>(key, idx);
  argmax_step<kDppHalfMirror>(key, idx);
  argmax_step<kDppMirror>(key, idx);
  float k = lane_f(key, 0);
  int i = lane_i(idx, 0);
#pragma unroll
  for (int r = 1; r < 4; ++r) argmax_merge(k, i, lane_f(key, 16 * r), lane_i(idx, 16 * r));
  key = k;
  idx = i;
}

// Combine per-lane (max, sum of exp2(x - max)) pairs in the log2 domain.
__device__ __forceinline__ void lse2_merge(float& m, float& s, float om, float os) {
  const float nm = fmaxf(m, om);
  s = s * __builtin_amdgcn_exp2f(m - nm) + os * __builtin_amdgcn_exp2f(om - nm);
  m = nm;
}
template <int CTRL>
__device__ __forceinline__ void lse2_step(float& m, float& s) {
  lse2_merge(m, s, dpp_f<CTRL>(m), dpp_f<CTRL>(s));
}
__device__ __forceinline__ void wave_lse2(float& m, float& s) {
  lse2_step<kDppQuad1>(m, s);
  lse2_step<kDppQuad2>(m, s);
  lse2_step<kDppHalfMirror>(m, s);
  lse2_step<kDppMirror>(m, s);
  float rm = lane_f(m, 0), rs = lane_f(s, 0);
#pragma unroll
  for (int r = 1; r < 4; ++r) lse2_merge(rm, rs, lane_f(m, 16 * r), lane_f(s, 16 * r));
  m = rm;
  s = rs;
}

__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f<kDppQuad1>(v);
  v += dpp_f<kDppQuad2>(v);
  v += dpp_f<kDppHalfMirror>(v);
  v += dpp_f<kDppMirror>(v);
  return (lane_f(v, 0) + lane_f(v, 16)) + (lane_f(v, 32) + lane_f(v, 48));
}

__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_f<kDppQuad1>(v));
  v = fmaxf(v, dpp_f<kDppQuad2>(v));
  v = fmaxf(v, dpp_f<kDppHalfMirror>(v));
  v = fmaxf(v, dpp_f<kDppMirror>(v));
  return fmaxf(fmaxf(lane_f(v, 0), lane_f(v, 16)), fmaxf(lane_f(v, 32), lane_f(v, 48)));
}

__device__ __forceinline__ int wave_sum_int(int v) {
  v += dpp_i<kDppQuad1>(v);
  v += dpp_i<kDppQuad2>(v);
  v += dpp_i<kDppHalfMirror>(v);
  v += dpp_i<kDppMirror>(v);
  return (lane_i(v, 0) + lane_i(v, 16)) + (lane_i(v, 32) + lane_i(v, 48));
}

// First device-side data error wins; later ones are dropped.
__device__ __forceinline__ void report_error(int32_t* err, int32_t code) {
  atomicCAS(err, 0, code);
}

}  // namespace vsd
