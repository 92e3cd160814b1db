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
  // top-K renormalised KL term (fused only; kl_k > 0 turns it on)
  int32_t kl_k;
  int32_t* kl_idx;           // [R, kl_k]
  float* kl_grad;            // [R, kl_k]
  float* kl_row;             // [R]
  float kl_gscale;           // loss_scale * kl_weight / N / T_q
};

// One depth of a rollout with exact context (vsd_sample_step): path p's rows
// are X + p ld_d (along z~), Y + p ld_t (along z'), Yg + p ld_t (along
// z-bar); its tokens go to row p L + step of the token arrays.
struct SampleStepArgs {
  const void* X;
  const void* Y;
  const void* Yg;
  const int32_t* d2t;        // [Vd] or null
  const int32_t* depth;      // [paths] or null
  int32_t* tok_d;
  int32_t* tok_t;
  int32_t* tok_g;
  int32_t* err;
  int64_t paths, ld_d, ld_t;
  int32_t L, step, Vd, Vt;
  float inv_tq, inv_tp;
  uint32_t k0, k1, offset;
};

// Decode-time verification of the draft paths (vsd_verify_paths).
struct VerifyArgs {
  const void* X;             // [R, ld_d]
  const void* Y;             // [R, ld_t]
  const int32_t* inv;        // [Vt] draft index of target column t, -1 unmapped; null = identity
  const int32_t* depth;      // [paths] or null
  const float* la;           // [R, 3] log alpha of the three families (column 0: z~)
  const float* lse_q;        // [R]
  const float* lse_p;        // [R]
  int32_t* accept_len;       // [paths]
  int32_t* resample;         // [paths] target index, -1 when every token is kept
  int32_t* err;
  int64_t paths, ld_d, ld_t;
  int32_t L, Vd, Vt;
  float inv_tq, inv_tp;
  uint32_t k0, k1, offset;
};

struct ScoreRowArgs {
  const void* X;
  const void* Y;
  const int32_t* d2t;
  const int32_t* depth;
  const int32_t* tok[3];     // draft, target, greedy
  float* lse_q;              // [R] optional
  float* lse_p;              // [R] optional
  float* la;                 // [R,3]
  float* lq;                 // [R,3]
  int32_t* err;
  int64_t R, ld_d, ld_t;
  int32_t L, Vd, Vt;
  float inv_tq, inv_tp;
  int32_t fam_lo, fam_hi;    // families [fam_lo, fam_hi) gathered on these rows (columns of la / lq)
  // top-K renormalised KL term (kl_k > 0 turns it on)
  int32_t kl_k;
  int32_t* kl_idx;           // [R, kl_k]
  float* kl_grad;            // [R, kl_k]
  float* kl_row;             // [R]
  float kl_gscale;           // loss_scale * kl_weight / N / T_q
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
  const float* kl_row;       // [R] KL row terms, or null (term off)
  float* kl_pos;             // optional [P]
  float kl_weight;
  float w[kMaxL];            // w(l) = w_base^l, l = 1..L
};

struct BwdArgs {
  const void* X;
  void* G;
  const float* lse_q;
  const int32_t* tok_d;
  const int32_t* tok_t;
  const float* coef_a;       // [R], or null: a = 0
  const float* coef_b;       // [R], or null: b = 0
  int64_t R, ld;
  int32_t Vd;
  float inv_tq, scale;
  const int32_t* kl_idx;     // [R, kl_k] or null: sparse KL gradient terms added to the row
  const float* kl_grad;      // [R, kl_k]
  int32_t kl_k;
};

// ------------------------------------------------ fused LM-head variant ---
constexpr int kLmTile = 256;           // rows and vocabulary columns per logit tile
constexpr int kLmTilesPerSlice = 16;   // vocabulary tiles one forward workgroup walks

// Vocabulary slices of a V-column pass (a function of V only, so the float
// outputs of a row do not depend on the batch size).
inline int lm_nslice(int V) {
  const int tiles = (V + kLmTile - 1) / kLmTile;
  return (tiles + kLmTilesPerSlice - 1) / kLmTilesPerSlice;
}

// One slice's running state of one row (32 bytes).
struct LmPartial {
  float mraw, mc, s;   // log-sum-exp in shifted form
  float key;           // best Gumbel key
  int32_t idx;         // its draft index
  float gval;          // greedy maximum (target pass)
  int32_t gidx;
  int32_t pad;
};

// Top-K renormalised KL term on the fused head: every row segment of the
// target pass keeps its few best mapped target logits; a slice's record
// holds the best kLmKlM of its four segments' lists and an upper bound of
// every value they dropped (-inf: none dropped).
constexpr int kLmKlM = 8;
struct LmKlEntry {
  float val;                 // raw target logit
  int32_t idx;               // its draft index
};

// A row the slice lists cannot decide is recomputed exactly over slices of
// the draft vocabulary, whose records (kLmRedoM entries each) take the place
// of the row's target-slice lists once the combine has read them: as many
// slices as fit there (at least one; the row's region is padded when one
// does not fit).
constexpr int kLmRedoM = 16;
inline int lm_redo_nslice(int Vd, int Vt) {
  const int tiles = (Vd + kLmTile - 1) / kLmTile;
  const int fit = lm_nslice(Vt) * kLmKlM / kLmRedoM;
  return fit < 1 ? 1 : fit < tiles ? fit : tiles;
}
// LmKlEntry records per row of the KL lists' region.
inline int lm_kl_stride(int Vd, int Vt) {
  const int lists = lm_nslice(Vt) * kLmKlM, redo = lm_redo_nslice(Vd, Vt) * kLmRedoM;
  return lists > redo ? lists : redo;
}

struct LmFwdArgs {
  const void* Hd;            // [R, H] bf16
  const void* Ht;            // [R, H] bf16
  const void* Wd;            // [Vd, H] bf16
  const void* Wt;            // [Vt, H] bf16
  const int32_t* inv;        // [Vt] draft index of each target column (-1: none); null = identity
  LmPartial* part;           // [R, nslice_t + nslice_d], target slices first
  LmKlEntry* kl_part;        // KL term: [R, kl_stride] rows of nslice_t slice lists of kLmKlM, or
                             // null (term off)
  float* kl_bound;           // KL term: [R, nslice_t] bound of the dropped values
  int64_t R;
  int32_t kl_stride;         // KL term: LmKlEntry records per row of kl_part
  int32_t H, Vd, Vt;
  int32_t nslice_t, nslice_d;
  int32_t sample;            // 0: log-sum-exp only (scoring given tokens)
  float inv_tq, inv_tp;
  uint32_t k0, k1, offset;
};

struct LmCombineArgs {
  const LmPartial* part;
  const void* Hd;
  const void* Ht;
  const void* Wd;
  const void* Wt;
  const int32_t* d2t;
  const int32_t* depth;
  const int32_t* tok_in[3];  // scoring: given tokens; sampling: null
  int32_t* tok_out[3];       // sampling: drawn tokens
  float* lse_q;
  float* lse_p;              // optional
  float* la;                 // [R,3]
  float* lq;                 // [R,3]
  int32_t* err;
  int64_t R;
  int32_t L, H, Vd, Vt;
  int32_t nslice_t, nslice_d;
  float inv_tq, inv_tp;
  // top-K renormalised KL term (kl_k > 0 turns it on)
  int32_t kl_k;
  LmKlEntry* kl_part;        // [R, kl_stride]: the forward's slice lists; rows listed for the
                             // recompute then hold its kl_nslice records of kLmRedoM
  int32_t kl_stride;         // lm_kl_stride(Vd, Vt)
  const float* kl_bound;     // [R, nslice_t]
  int32_t* kl_count;         // [1] rows the slice lists could not decide (reset before the combine)
  int32_t* kl_list;          // [R] those rows, in the order they were found
  int32_t kl_nslice;         // lm_redo_nslice(Vd, Vt)
  int32_t* kl_idx;           // [R, kl_k]
  float* kl_grad;            // [R, kl_k]
  float* kl_row;             // [R]
  float kl_gscale;           // loss_scale * kl_weight / N / T_q
};

struct LmBwdArgs {
  const void* Hd;
  const void* Wd;
  void* G;                   // [R, ldg] bf16: gradient w.r.t. the draft logits
  void* dH;                  // [R, H] bf16
  float* dW;                 // [Vd, H] fp32 or null: gradient w.r.t. the draft head's weight
  const float* lse_q;
  const int32_t* tok_d;
  const int32_t* tok_t;
  const float* coef_a;
  const float* coef_b;
  const int32_t* kl_idx;     // [R, kl_k] or null: the KL term's sparse gradient, added to G
  const float* kl_grad;      // [R, kl_k]
  int32_t kl_k;
  int64_t R, ldg;
  int32_t H, Vd;
  float inv_tq, scale;
};

// C = A^T B with A [K, M] and B [K, N] row-major bf16, C [M, N] fp32.
struct LmGemmTNArgs {
  const void* A;
  const void* B;
  float* C;
  int64_t M, lda;
  int64_t ldb, ldc;
  int32_t N, K;
};

struct LmGemmNNArgs {
  const void* A;             // [M, K] bf16
  const void* B;             // [K, N] bf16
  void* C;                   // [M, N] bf16
  int64_t M, lda;
  int64_t ldb, ldc;
  int32_t N, K;
};

hipError_t launch_lm_inv(const int32_t* d2t, int Vd, int Vt, int32_t* inv, int32_t* err, hipStream_t s);
hipError_t launch_lm_fwd(const LmFwdArgs& a, hipStream_t s);
hipError_t launch_lm_combine(const LmCombineArgs& a, hipStream_t s);
hipError_t launch_lm_kl_reset(const LmCombineArgs& a, hipStream_t s);
hipError_t launch_lm_kl_redo(const LmCombineArgs& a, hipStream_t s);
hipError_t launch_lm_bwd(const LmBwdArgs& a, hipStream_t s);

// Range check of a draft-to-target map: the first entry outside [0, Vt) is
// reported as VSD_DEVERR_MAP_RANGE (kernels that gather through the map
// without testing each entry run it first).
hipError_t launch_map_check(const int32_t* d2t, int Vd, int Vt, int32_t* err, hipStream_t s);
hipError_t launch_sample(const SampleArgs& a, bool bf16, hipStream_t s);
hipError_t launch_sample_step(const SampleStepArgs& a, bool bf16, hipStream_t s);
hipError_t launch_verify(const VerifyArgs& a, bool bf16, hipStream_t s);
hipError_t launch_score_rows(const ScoreRowArgs& a, bool bf16, hipStream_t s);
hipError_t launch_combine(const CombineArgs& a, hipStream_t s);
hipError_t launch_loss_total(const float* loss_pos, int32_t P, float scale, float* out, hipStream_t s);
hipError_t launch_bwd(const BwdArgs& a, bool bf16, hipStream_t s);

}  // namespace vsd
