/*
 * vsd.h -- C ABI of the Variational Speculative Decoding (VSD) EM path-scoring
 * library for AMD Instinct MI355X (gfx950).
 *
 * The library computes, for a batch of training positions, the data-parallel
 * part of one VSD EM step (Appendix "Algorithm Detail": Alg. 1, the MC-based EM
 * framework, and Alg. 2, the oracle):
 *
 *   vsd_sample_paths      E-step proposals: N draft paths, N target correction
 *                         paths and N greedy target reference paths of depth L
 *                         per position (Alg. 1 proposal/correction draws,
 *                         Alg. 2 greedy baseline).
 *   vsd_score_paths       Row softmax statistics, acceptance ratios (Sec.
 *                         "Preliminary", Eq. acc), survival and expected
 *                         accepted length (Sec. "Theoretical Analysis",
 *                         Eqs. survival_def / accepted_len_cond), the oracle
 *                         gate (Alg. 2), target correction (Alg. 1), ARW beta
 *                         (Eq. beta_update), CAR zeta (Eq. zeta_update), the
 *                         weighted-likelihood loss (Eq. advance / Eq. basic)
 *                         and the per-row gradient coefficients.
 *   vsd_weighted_loss_bwd Gradient of that loss with respect to the draft
 *                         logits (derivative of Eq. advance).
 *
 * Every call takes the logits either materialised ([R, ld] arrays) or, in
 * the fused LM-head variant (dims->hidden_dim > 0), as hidden states and an
 * LM-head weight: logits = hidden @ weight^T, computed tile by tile on the
 * matrix cores and never stored (see "Fused LM head" below).
 *
 * Terminology and layout
 * ----------------------
 *   position x = (b, t), b < B, t < T;  P = B*T positions.
 *   path slot s < N (the paper's sample size S);  depth i = 1..L (the paper's
 *   sampling length L).
 *   row r = ((b*T + t)*N + s)*L + (i-1);  R = P*N*L rows.  One row is one
 *   "path-token": it owns one draft logit row X_r (v_draft entries) and one
 *   target logit row Y_r (v_target entries).  Rows are given per slot: all
 *   three path families at slot (s,i) are scored against the same two rows
 *   (the draft and target conditionals along the sampled draft path).
 *   Level l = 1..L of slot s denotes the length-l prefix of path s.
 *   Per-row quantities indexed by level (flags, o', beta, zeta) live at row
 *   ((b*T + t)*N + s)*L + (l-1).
 *   Families: 0 = draft proposal z~, 1 = target correction z', 2 = greedy z-bar.
 *   All tokens are in draft-index space [0, v_draft).  When v_draft !=
 *   v_target an injective map d2t: [0, v_draft) -> [0, v_target) is required;
 *   the target probability of draft token v is p(d2t[v]) with the target
 *   softmax taken over all v_target entries.  Without a map, d2t is the
 *   identity.
 *   valid_depth[b,t,s] = d_s in [1, L] (NULL means d_s = L for all paths):
 *   slot (s,i) exists iff i <= d_s.  Rows with i > d_s are "masked": their
 *   tokens are -1, their score outputs are 0 and their gradient rows are 0.
 *
 * Memory, ownership, streams
 * --------------------------
 *   Every array argument is a DEVICE pointer owned by the caller; struct
 *   arguments (vsd_dims, vsd_params, vsd_src, vsd_score_out, vsd_grad) are
 *   HOST pointers read during the call only.  The library never allocates or
 *   frees memory, never synchronises, never reads device memory on the host
 *   and keeps no mutable global state other than a thread-local error string
 *   and, for vsd_sample_score_paths_static, its static scratch array and that
 *   array's address per device.
 *   All work is enqueued on `hip_stream` (a hipStream_t; NULL = default
 *   stream) and is complete only when that stream is.
 *   Logit rows: row r starts at element r*ld of its array; the array holds R
 *   rows of ld elements (ld >= v).  Base pointers and ld*element_size must be
 *   multiples of 16 bytes (rows are read with 128-bit loads).
 *
 * Errors
 * ------
 *   Host-side validation runs before anything is launched; on failure the
 *   call returns a non-zero vsd_status, launches nothing and writes nothing.
 *   vsd_last_error() then holds a message naming the offending argument.
 *   Data errors only visible on the device (a token outside [-1, v_draft), a
 *   d2t entry outside [0, v_target), a depth outside [1, L]) never make a
 *   kernel access memory outside the arrays it was given (the offending
 *   access is skipped, clamped into the array, or answered with zero by the
 *   hardware range check of a row's buffer descriptor), and the first
 *   VSD_DEVERR_* code is stored atomically into *device_error (a slot the
 *   caller zeroes beforehand; the library only ever replaces 0 by a non-zero
 *   code).  The outputs of such a call are unspecified.  A failed HIP launch returns VSD_ERR_HIP.
 *
 * Determinism
 * -----------
 *   Every output is a pure function of the inputs: bitwise identical run to
 *   run and independent of launch geometry.  Tokens depend only on (seed,
 *   offset, row index, vocabulary index) and the logits, so a resumed trainer
 *   reproduces them exactly by passing the same offset.
 *
 * Normative sampler definition (draft proposal z~ and target correction z')
 * ------------------------------------------------------------------------
 *   The paper draws z~ ~ q and z' ~ p (Alg. 1) without naming a sampler; this
 *   library fixes one so that the sampled tokens are unique and reproducible
 *   bit for bit by any implementation of this definition.  Every operation
 *   below is one IEEE-754 binary32 operation rounded to nearest-even (no fused
 *   multiply-add, correctly rounded division); integers are unsigned 32-bit.
 *
 *   S1 Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers:
 *      as easy as 1, 2, 3", SC'11).  Key (k0,k1) = (low 32 bits of seed,
 *      high 32 bits of seed).  Ten rounds; round j uses the key
 *      (k0 + j*0x9E3779B9, k1 + j*0xBB67AE85) mod 2^32, j = 0..9.  A round
 *      maps (c0,c1,c2,c3) to
 *        (hi(0xCD9E8D57*c2) ^ c1 ^ k0', lo(0xCD9E8D57*c2),
 *         hi(0xD2511F53*c0) ^ c3 ^ k1', lo(0xD2511F53*c0))
 *      where hi/lo are the upper/lower 32 bits of the 64-bit product.
 *   S2 For vocabulary index v of row r and family f (0 = z~, 1 = z'), the
 *      counter is (v >> 2, r, f, offset) and the word used is output word
 *      (v & 3).  (For a mapped target row, v is the draft index.)
 *   S3 u = float(2*(w >> 9) + 1) * 2^-24, exactly representable, in (0,1).
 *   S4 Lambda(x), the normative log of a positive normal float x:
 *        e = ((bits(x) >> 23) & 0xFF) - 127;
 *        m = float with bits (bits(x) & 0x7FFFFF) | 0x3F800000;   (m in [1,2))
 *        if m > 1.41421354f (0x3FB504F3): m = m * 0.5f; e = e + 1;
 *        f = m - 1;   s = f / (2 + f);   z = s * s;
 *        p = 1/9;  p = 1/7 + z*p;  p = 1/5 + z*p;  p = 1/3 + z*p;
 *            (each constant c is float(c): 0x3DE38E39, 0x3E124925,
 *             0x3E4CCCCD, 0x3EAAAAAB; every * and + rounds separately)
 *        t2 = s + s;   lm = t2 + t2 * (z * p);
 *        ef = float(e);
 *        Lambda = ef * 0.693145751953125f (0x3F317200)
 *                 + (lm + ef * 1.42860677e-06f (0x35BFBE8E)).
 *      (The series is 2*atanh(s) = log(m); the constant split is exact for
 *      the ef*hi product.)
 *   S5 G = -Lambda(-Lambda(u))  (a Gumbel(0,1) variate).
 *   S6 key_v = float(logit_v * invT) + G, with invT = float(1/T) and
 *      logit_v = X[r][v] (z~, T = temp_draft) or Y[r][d2t[v]] (z',
 *      T = temp_target).  The token is the v in [0, v_draft) with the largest
 *      key; among equal keys the smallest v.
 *   S7 The greedy reference z-bar is the v in [0, v_draft) maximising the raw
 *      target logit Y[r][d2t[v]]; among equal logits the smallest v
 *      (Alg. 2, greedy target policy).
 *   Logits must be finite.
 *
 * Fused LM head (dims->hidden_dim = H > 0)
 * ----------------------------------------
 *   Both sources give `hidden` [R, H] and `weight` [V, H] (bf16, rows
 *   contiguous, 16-byte aligned; `logits` NULL; dims->dtype = VSD_BF16;
 *   H a multiple of 64).  X_r = hidden_d[r] . weight_d^T and Y_r likewise,
 *   accumulated in fp32; every definition above applies to these values.
 *   The fp32 sum's order is the library's (not fixed by this header), so
 *   tokens are reproducible run to run but a different implementation
 *   agrees with them only where the top two keys (or greedy values) of a row
 *   are further apart than the products' rounding.
 *   vsd_sample_paths does not accept fused sources (it has no workspace);
 *   vsd_sample_score_paths draws and scores, vsd_score_paths scores given
 *   tokens.  The map d2t, when given, must be injective (it is inverted on
 *   the device; a duplicate entry sets VSD_DEVERR_MAP_DUPLICATE).  The workspace (vsd_score_workspace_bytes with the same
 *   dims) then also holds per-slice partial row statistics.
 *   Backward: grad->grad_logits (bf16, row stride dims->ld_draft, a multiple
 *   of 8 >= v_draft) receives g as defined at vsd_weighted_loss_bwd, and
 *   grad->grad_hidden [R, H] (bf16) receives g . weight_d.
 *   grad->grad_weight [V_d, H] fp32, optional (NULL: not computed), receives
 *   the gradient with respect to the draft head's weight, g^T . hidden_d
 *   (fp32 accumulation of the bf16 g; written, not accumulated into).
 *   dims->ld_target is unused.
 *
 * VSD (KL): the top-K renormalised KL term (params->kl_weight > 0)
 * ---------------------------------------------------------------
 *   The paper's KL variant (Eq. klv) adds a token-level distillation term
 *   over the K target tokens of highest probability.  Per live row r, with
 *   y_v = Y[r][d2t[v]] over the draft vocabulary:
 *     Omega_r  = the K draft indices with the largest finite y_v (equal
 *                values: the smaller index first), in that order; a row
 *                with fewer than K finite y_v (entries of zero target
 *                probability, y_v = -inf) has that many members, its
 *                kl_idx / kl_grad slots past them hold -1 / 0 (none: the
 *                row's term is 0);
 *     p_hat(v) = exp(y_v/T_p) / sum_{u in Omega_r} exp(y_u/T_p),
 *     q_hat(v) = exp(X[r][v]/T_q) / sum_{u in Omega_r} exp(X[r][u]/T_q);
 *     kl_row[r] = - sum_{v in Omega_r} p_hat(v) log q_hat(v).
 *   Per position KL_x = (1/N) sum over live rows of kl_row (the path-level
 *   divergence is the expected sum of the per-step ones), and
 *   loss_pos[x] = L_x + kl_weight KL_x.  The gradient gains
 *   kl_grad[r][k] = loss_scale kl_weight / N (q_hat - p_hat)(Omega_r[k]) / T_q
 *   at draft index kl_idx[r][k] = Omega_r[k]; vsd_weighted_loss_bwd adds
 *   these when given kl_idx and kl_grad.  K <= v_draft.  Computed by
 *   vsd_score_paths and vsd_sample_score_paths (same outputs, same results),
 *   on materialised logits and with the fused LM head alike; fused, the
 *   backward adds the sparse gradient to g before g is contracted with the
 *   weight (so grad_hidden and grad_weight include the term).
 *
 * Exact context (vsd_sample_step, vsd_score_paths_ctx, vsd_weighted_loss_bwd_ctx)
 * ------------------------------------------------------------------------------
 *   By default the three families of a slot read the same rows: the
 *   conditionals along the draft path.  The paper's acceptance test
 *   (Sec. "Preliminary", Eq. acc) and survival (Eq. survival_def) are taken
 *   along each path with its own prefix, p(.|x, z_<i) and q(.|x, z_<i); a
 *   caller that runs the models along every path can pass those rows instead:
 *   family f (0: z~, 1: z', 2: z-bar) then has draft rows X_f and target rows
 *   Y_f ([R, ld] each, the layout of the shared rows), and
 *     log alpha^f, log q^f  come from X_f, Y_f at z^f,
 *     every later quantity  as before (flags, o', beta, zeta, a, b, loss),
 *     the gradient          a-part on X_0 (the rows along z~), b-part on X_1
 *                           (along z'); X_2 only gates.
 *   The KL term, when on, is taken on X_0, Y_0.  vsd_sample_step draws one
 *   depth of such a rollout: the models' rows at depth i depend on the
 *   tokens at depths < i, so the draws go depth by depth, each with the
 *   Philox counters of the slot's global row (equal rows at every depth give
 *   exactly the tokens of vsd_sample_paths).
 */
#ifndef VSD_H
#define VSD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define VSD_ABI_VERSION 4

typedef enum vsd_status {
  VSD_OK = 0,
  VSD_ERR_NULL_POINTER = 1,  /* a required pointer is NULL */
  VSD_ERR_INVALID_SHAPE = 2, /* B,T,N,L,v,ld or hidden_dim out of range */
  VSD_ERR_INVALID_VALUE = 3, /* temperature, w_base, tau, mode ... invalid */
  VSD_ERR_MISALIGNED = 4,    /* base pointer or row stride not 16-B aligned */
  VSD_ERR_MAP_REQUIRED = 5,  /* v_draft != v_target and d2t == NULL */
  VSD_ERR_UNSUPPORTED = 6,   /* combination this build does not implement */
  VSD_ERR_WORKSPACE = 7,     /* workspace NULL or smaller than required */
  VSD_ERR_HIP = 8            /* a HIP runtime call failed */
} vsd_status;

/* Codes written to *device_error by the kernels. */
enum {
  VSD_DEVERR_NONE = 0,
  VSD_DEVERR_TOKEN_RANGE = 1, /* token outside [-1, v_draft) or -1 on a live slot */
  VSD_DEVERR_MAP_RANGE = 2,   /* d2t entry outside [0, v_target) */
  VSD_DEVERR_DEPTH_RANGE = 3, /* valid_depth entry outside [1, L] */
  VSD_DEVERR_MAP_DUPLICATE = 4 /* two d2t entries name the same target token
                                  (detected where the map is inverted: the
                                  fused LM head's draws, verification) */
};

typedef enum vsd_dtype { VSD_F32 = 0, VSD_BF16 = 1 } vsd_dtype;

/* Which M-step estimator the coefficients implement (Alg. 1, M-step). */
typedef enum vsd_grad_mode {
  VSD_GRAD_BASIC = 0,  /* Eq. basic: c = 0 */
  VSD_GRAD_ARW = 1,    /* Eq. advance with zeta = 1: c = beta */
  VSD_GRAD_ARW_CAR = 2 /* Eq. advance: c = beta * zeta (default) */
} vsd_grad_mode;

/* What CAR's softmax is taken over (Eq. zeta_update). */
typedef enum vsd_car_input {
  VSD_CAR_PROB = 0,   /* exp(Q/tau), Q = draft path probability (as printed) */
  VSD_CAR_LOGPROB = 1 /* exp(log Q / tau), an alternative reading */
} vsd_car_input;

typedef struct vsd_dims {
  int32_t B, T, N, L;  /* 1 <= B,T; 1 <= N <= 1024; 1 <= L <= 64; R = B*T*N*L < 2^24 */
  int32_t v_draft;     /* draft vocabulary size, >= 1 */
  int32_t v_target;    /* target vocabulary size, >= v_draft */
  int32_t dtype;       /* vsd_dtype of the logit (or hidden/weight) arrays */
  int32_t hidden_dim;  /* fused LM-head variant: H (multiple of 64); 0 otherwise */
  int64_t ld_draft;    /* row stride of the draft logit array (fused: of the
                          bf16 logit-gradient buffer), elements */
  int64_t ld_target;   /* row stride of the target logit array, elements */
} vsd_dims;

typedef struct vsd_params {
  float temp_draft;    /* T_q > 0: q = softmax(X / T_q) */
  float temp_target;   /* T_p > 0: p = softmax(Y / T_p) */
  float w_base;        /* > 0; oracle length weight w(l) = w_base^l (1.05) */
  float car_tau;       /* > 0; CAR temperature tau (0.2) */
  int32_t mode;        /* vsd_grad_mode */
  int32_t car_input;   /* vsd_car_input */
  float loss_scale;    /* multiplies the summed loss and the gradient */
  float kl_weight;     /* >= 0; weight of the top-K renormalised KL term (0 = off) */
  int32_t kl_topk;     /* K of that term, 1..16 (used when kl_weight > 0) */
} vsd_params;

/* Source of one model's logits.  Materialised (dims->hidden_dim == 0):
 * `logits` != NULL, an [R, ld] array of dims->dtype.  Fused LM head
 * (dims->hidden_dim > 0): `logits` == NULL, logits are hidden[R, H] @
 * weight[V, H]^T computed on the fly (bf16 only). */
typedef struct vsd_src {
  const void* logits;
  const void* hidden;
  const void* weight;
} vsd_src;

typedef struct vsd_score_out {
  float* lse_draft;       /* [R]   required: log-sum-exp of X_r / T_q */
  float* lse_target;      /* [R]   optional: log-sum-exp of Y_r / T_p */
  float* log_alpha;       /* [R,3] optional: min(0, log p - log q) per family */
  float* log_q_tok;       /* [R,3] optional: log q(token) per family */
  float* survival;        /* [R]   optional: S_i of z~ (prefix product) */
  float* exp_accept_len;  /* [P*N] optional: sum_{k<=d_s} S_k of z~ */
  uint8_t* accept_flag;   /* [R]   optional: I~ = oracle accepts z~ at level */
  uint8_t* valid_flag;    /* [R]   optional: I' = oracle accepts the used path */
  float* o_prime;         /* [R]   optional: o' = w(l) * I' */
  float* beta;            /* [R]   optional: ARW coefficient */
  float* zeta;            /* [R]   optional: CAR weight */
  float* coef_a;          /* [R]   required: coefficient of -log q(z~) */
  float* coef_b;          /* [R]   required: coefficient of -log q(z') */
  float* loss_pos;        /* [P]   optional: L_x + kl_weight KL_x (unscaled) */
  float* loss_total;      /* [1]   optional: loss_scale * sum_x loss_pos */
  int32_t* device_error;  /* [1]   required */
  /* Top-K renormalised KL term (kl_weight > 0; see "VSD (KL)" above): */
  int32_t* kl_idx;        /* [R,K] required with the term: the row's top-K draft indices (-1 masked) */
  float* kl_grad;         /* [R,K] required with the term: the term's gradient at kl_idx */
  float* kl_row;          /* [R]   optional: the row's term (0 masked) */
  float* kl_pos;          /* [P]   optional: KL_x */
} vsd_score_out;

/* Exact context: the rows of each family's own conditionals (see above). */
typedef struct vsd_ctx_rows {
  const void* draft[3];   /* [R, ld_draft] each: draft logits along z~, z', z-bar */
  const void* target[3];  /* [R, ld_target] each: target logits along z~, z', z-bar */
} vsd_ctx_rows;

typedef struct vsd_grad {
  void* grad_logits;      /* [R, ld_draft]: dtype of X; fused: bf16 */
  void* grad_hidden;      /* fused: [R, H] bf16, required */
  float* grad_weight;     /* fused, optional: [V_d, H] fp32, g^T . hidden_d */
} vsd_grad;

/* E-step sampling (Alg. 1: z~ ~ q and z' ~ p; Alg. 2: z-bar greedy).
 * Writes tok_draft, tok_target, tok_greedy ([R] int32 each, draft-index
 * space, -1 on masked rows) following the normative sampler definition above.
 * Reads X (draft) over [0, v_draft) and Y (target) at d2t[v] for every v.
 * Materialised logits only (fused sources: VSD_ERR_UNSUPPORTED). */
vsd_status vsd_sample_paths(const vsd_dims* dims, const vsd_src* draft,
                            const vsd_src* target, const int32_t* d2t,
                            const int32_t* valid_depth, float temp_draft,
                            float temp_target, uint64_t seed, uint32_t offset,
                            int32_t* tok_draft, int32_t* tok_target,
                            int32_t* tok_greedy, int32_t* device_error,
                            void* hip_stream);

/* Path scoring and M-step weights for given tokens (any tokens the caller
 * supplies, not only those of vsd_sample_paths).  Per row: q and p log-sum-exp
 * over the full draft / target vocabularies, log alpha and log q of the three
 * families.  Per position: prefix sums over depth, oracle flags (equality
 * accepts), o', beta (leave-one-out over paths alive at the level; 0 when the
 * denominator is 0), zeta (softmax over paths alive at the level), W = sum o',
 * L_x (0 when W = 0), and
 *   a_{s,i} = (1/W) sum_{l=i..d_s} o'_{l,s} (I~_{l,s} - c_{l,s})
 *   b_{s,i} = (1/W) sum_{l=i..d_s} o'_{l,s} (1 - I~_{l,s}).
 * `workspace` must hold vsd_score_workspace_bytes() bytes (16-B aligned). */
vsd_status vsd_score_paths(const vsd_dims* dims, const vsd_params* params,
                           const vsd_src* draft, const vsd_src* target,
                           const int32_t* d2t, const int32_t* valid_depth,
                           const int32_t* tok_draft, const int32_t* tok_target,
                           const int32_t* tok_greedy, const vsd_score_out* out,
                           void* workspace, size_t workspace_bytes,
                           void* hip_stream);

/* vsd_sample_paths followed by vsd_score_paths on the drawn tokens, in one
 * pass over the logits: the sampling kernel also accumulates both
 * log-sum-exps and gathers the drawn tokens' logits, so X and Y are read from
 * memory once instead of twice.  Temperatures come from `params`.  Tokens are
 * identical to vsd_sample_paths'; the float outputs agree with
 * vsd_score_paths' up to float32 summation order.  Same workspace as
 * vsd_score_paths. */
vsd_status vsd_sample_score_paths(const vsd_dims* dims, const vsd_params* params,
                                  const vsd_src* draft, const vsd_src* target,
                                  const int32_t* d2t, const int32_t* valid_depth,
                                  uint64_t seed, uint32_t offset,
                                  int32_t* tok_draft, int32_t* tok_target,
                                  int32_t* tok_greedy, const vsd_score_out* out,
                                  void* workspace, size_t workspace_bytes,
                                  void* hip_stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * vsd_sample_score_paths with the library's own scratch in place of the
 * caller's workspace.  Same arguments, outputs and results otherwise (the
 * same kernels run).
 *   Scratch: a static device array of VSD_STATIC_SCRATCH_BYTES (256 MiB) that
 *   every device the library runs on holds from the library's first use there
 *   until the process ends; the call uses the one of the calling thread's
 *   current device (hip_stream must belong to that device).  Its address is
 *   looked up once per device (hipGetSymbolAddress); the call itself
 *   allocates nothing.
 *   Limit: dims whose vsd_score_workspace_bytes() exceeds
 *   VSD_STATIC_SCRATCH_BYTES return VSD_ERR_WORKSPACE before anything is
 *   launched (the five reference workloads need at most 164 MiB, the
 *   fused 128k-vocabulary head with its KL lists).
 *   Sharing: every call on a device uses that device's one array, which keeps
 *   the last call's contents; nothing in it needs to start at zero (each call
 *   writes every region before reading it).  Calls that overlap on one device
 *   (different streams, or threads without ordering between them) race on the
 *   scratch and their outputs are undefined: order them on one stream. */
#define VSD_STATIC_SCRATCH_BYTES ((size_t)256 << 20)
vsd_status vsd_sample_score_paths_static(const vsd_dims* dims, const vsd_params* params,
                                         const vsd_src* draft, const vsd_src* target,
                                         const int32_t* d2t, const int32_t* valid_depth,
                                         uint64_t seed, uint32_t offset,
                                         int32_t* tok_draft, int32_t* tok_target,
                                         int32_t* tok_greedy, const vsd_score_out* out,
                                         void* hip_stream);

/* Gradient of loss_scale * sum_x L_x with respect to the draft logits (the
 * derivative of Eq. advance, with o', beta, zeta and the tokens held fixed):
 *   g[r][v] = loss_scale / T_q * ((a+b) q_r(v) - a [v = z~] - b [v = z'])
 * with q_r(v) = exp(X[r][v] / T_q - lse_draft[r]).  Columns [0, v_draft) of
 * every row are written; rows with a = b = 0 (masked rows among them) are
 * written as zeros without reading X; padding columns [v_draft, ld) are not
 * touched.  grad_logits has the layout of X (stride ld_draft) and its dtype
 * (bf16 rounded to nearest-even).  Fused LM head: X is recomputed from the
 * draft hidden states, g is written to grad_logits in bf16, and grad_hidden
 * = g . weight_d (fp32 accumulation of the bf16 g, bf16 result).
 * kl_idx / kl_grad ([R, K] from vsd_score_paths) add the top-K KL term's
 * gradient: required when params->kl_weight > 0, ignored otherwise. */
vsd_status vsd_weighted_loss_bwd(const vsd_dims* dims, const vsd_params* params,
                                 const vsd_src* draft, const float* lse_draft,
                                 const int32_t* tok_draft,
                                 const int32_t* tok_target, const float* coef_a,
                                 const float* coef_b, const int32_t* kl_idx,
                                 const float* kl_grad, const vsd_grad* grad,
                                 int32_t* device_error, void* hip_stream);

/* One depth of a rollout with exact context (Alg. 1 draws and Alg. 2's
 * greedy reference, depth by depth).  step in [0, L).  draft_rows: the draft
 * logits at this depth along z~ of every path, path p at draft_rows + p *
 * ld_draft (P*N rows, P = B*T, paths in (b, t, s) order); target_rows and
 * greedy_rows: the target logits along z' and along z-bar, stride ld_target.
 * Writes row p*L + step of tok_draft, tok_target, tok_greedy ([R] each), -1
 * where step >= valid_depth[p]; other rows are not touched.  The draws are
 * those of vsd_sample_paths for that row (same counters), so a rollout whose
 * rows are equal for the three families reproduces vsd_sample_paths exactly.
 * Materialised logits only (dims->hidden_dim must be 0). */
vsd_status vsd_sample_step(const vsd_dims* dims, int32_t step,
                           const void* draft_rows, const void* target_rows,
                           const void* greedy_rows, const int32_t* d2t,
                           const int32_t* valid_depth, float temp_draft,
                           float temp_target, uint64_t seed, uint32_t offset,
                           int32_t* tok_draft, int32_t* tok_target,
                           int32_t* tok_greedy, int32_t* device_error,
                           void* hip_stream);

/* vsd_score_paths with exact context: family f's log alpha and log q from
 * rows->draft[f] and rows->target[f].  out->lse_draft (and lse_target) are
 * those of the rows along z~; lse_draft_corr [R] (required) receives the
 * draft log-sum-exp of the rows along z' (the backward needs it).  KL term
 * (kl_weight > 0) on the rows along z~.  Same workspace as vsd_score_paths.
 * Materialised logits only. */
vsd_status vsd_score_paths_ctx(const vsd_dims* dims, const vsd_params* params,
                               const vsd_ctx_rows* rows, const int32_t* d2t,
                               const int32_t* valid_depth,
                               const int32_t* tok_draft, const int32_t* tok_target,
                               const int32_t* tok_greedy, const vsd_score_out* out,
                               float* lse_draft_corr, void* workspace,
                               size_t workspace_bytes, void* hip_stream);

/* vsd_weighted_loss_bwd with exact context: grad_draft_path [R, ld_draft]
 * receives loss_scale / T_q (a q(v) - a [v = z~]) (+ the KL term's gradient)
 * on the rows along z~ (rows->draft[0], lse_draft), and grad_corr_path
 * receives loss_scale / T_q (b q(v) - b [v = z']) on the rows along z'
 * (rows->draft[1], lse_draft_corr).  The two buffers must be distinct (the
 * caller adds them where the rows are the same).  Layout and dtype as
 * vsd_weighted_loss_bwd's grad_logits. */
vsd_status vsd_weighted_loss_bwd_ctx(const vsd_dims* dims, const vsd_params* params,
                                     const vsd_ctx_rows* rows, const float* lse_draft,
                                     const float* lse_draft_corr,
                                     const int32_t* tok_draft, const int32_t* tok_target,
                                     const float* coef_a, const float* coef_b,
                                     const int32_t* kl_idx, const float* kl_grad,
                                     void* grad_draft_path, void* grad_corr_path,
                                     int32_t* device_error, void* hip_stream);

/* Decode-time verification of the draft paths (Sec. "Preliminary", Eq.
 * acc): slot by slot, z~_i is kept iff Lambda(u_i) < log alpha_i, with u_i
 * the uniform of Philox counter (0, row, 2, offset) word 0 (the sampler
 * definition's u and normative log) and log alpha from vsd_score_paths
 * (log_alpha [R,3], column 0); at the first rejection a replacement is drawn
 * from norm(max(0, p - q)) over the whole target vocabulary (q(t) = q(v) for
 * t = d2t[v], 0 for target tokens the draft cannot propose; p and q from the
 * row's logits and lse_target / lse_draft) by Gumbel-max of
 * log(max(0, p - q)) with the sampler's Gumbel variates over target indices
 * t (counter (t >> 2, row, 3, offset), word t & 3), and the path ends.
 * accept_len [P*N] receives the number of kept tokens (its mean given the
 * path is the expected accepted length sum_k S_k); resample_tok [P*N] the
 * replacement's target index, -1 when every live token was kept (no bonus
 * token is drawn: there is no row for it) or, with probability ~1e-7, when
 * the residual mass vanishes in float32.  With a map, `workspace` must hold
 * vsd_score_workspace_bytes() bytes (its inverse-map region is rebuilt);
 * without one it may be NULL.  Materialised logits only. */
vsd_status vsd_verify_paths(const vsd_dims* dims, const vsd_params* params,
                            const vsd_src* draft, const vsd_src* target,
                            const int32_t* d2t, const int32_t* valid_depth,
                            const float* log_alpha, const float* lse_draft,
                            const float* lse_target, uint64_t seed, uint32_t offset,
                            int32_t* accept_len, int32_t* resample_tok,
                            void* workspace, size_t workspace_bytes,
                            int32_t* device_error, void* hip_stream);

/* Bytes of workspace vsd_score_paths needs for `dims` (host only). */
vsd_status vsd_score_workspace_bytes(const vsd_dims* dims, size_t* bytes);

const char* vsd_status_string(vsd_status status); /* static string */
const char* vsd_last_error(void);                 /* thread-local detail */
int32_t vsd_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* VSD_H */
