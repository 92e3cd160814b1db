// Internal kernel arguments and launchers (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vsd {

constexpr int kMaxL = 64;

struct SampleArgs {
  const void* X;             // [R, ld_d]
  const void* Y;             // [R, ld_t]
  const int32_t* d2t;        // [Vd] or null (identity)
  const int32_t* depth;      // [P*N] or null
  int32_t* tok_d;
  int32_t* tok_t;
  int32_t* tok_g;
  int32_t* err;
  int64_t R, ld_d, ld_t;
  int32_t L, Vd, Vt;
  float inv_tq, inv_tp;      // float(1/T)
  uint32_t k0, k1, offset;   // Philox key words and counter word 3
  // Fused sample + row statistics (all null for plain sampling):
  float* lse_q;              // [R]
  float* lse_p;              // [R] optional
  float* la;                 // [R,3]
  float* lq;                 // [R,3]
  int32_t tblock;            // mapped: target elements streamed per 512-element chunk
};

struct ScoreRowArgs {
  const void* X;
  const void* Y;
  const int32_t* d2t;
  const int32_t* depth;
  const int32_t* tok[3];     // draft, target, greedy
  float* lse_q;              // [R] required
  float* lse_p;              // [R] optional
  float* la;                 // [R,3]
  float* lq;                 // [R,3]
  int32_t* err;
  int64_t R, ld_d, ld_t;
  int32_t L, Vd, Vt;
  float inv_tq, inv_tp;
};

struct CombineArgs {
  const float* la;           // [R,3]
  const float* lq;           // [R,3]
  const int32_t* depth;      // [P*N] or null
  float* survival;           // optional [R]
  float* ea;                 // optional [P*N]
  uint8_t* acc_flag;         // optional [R]
  uint8_t* val_flag;         // optional [R]
  float* o_prime;            // optional [R]
  float* beta;               // optional [R]
  float* zeta;               // optional [R]
  float* coef_a;             // [R]
  float* coef_b;             // [R]
  float* loss_pos;           // [P]
  int32_t* err;
  int32_t P, N, L;
  int32_t mode, car_input;
  float inv_tau;
  float w[kMaxL];            // w(l) = w_base^l, l = 1..L
};

struct BwdArgs {
  const void* X;
  void* G;
  const float* lse_q;
  const int32_t* tok_d;
  const int32_t* tok_t;
  const float* coef_a;
  const float* coef_b;
  int64_t R, ld;
  int32_t Vd;
  float inv_tq, scale;
};

hipError_t launch_sample(const SampleArgs& a, bool bf16, hipStream_t s);
hipError_t launch_score_rows(const ScoreRowArgs& a, bool bf16, hipStream_t s);
hipError_t launch_combine(const CombineArgs& a, hipStream_t s);
hipError_t launch_loss_total(const float* loss_pos, int32_t P, float scale, float* out, hipStream_t s);
hipError_t launch_bwd(const BwdArgs& a, bool bf16, hipStream_t s);

}  // namespace vsd
