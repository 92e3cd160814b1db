// Host side of the C ABI declared in include/vsd.h: argument validation
// (before any launch), workspace layout, launch geometry, error reporting.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>

#include "vsd_device.hpp"
#include "vsd_kernels.hpp"
#include "vsd_topk.hpp"

// Scratch of vsd_sample_score_paths_static: one copy of this array lives on
// every device the library's code object is loaded on, until the process
// ends.  Host code never passes the array's name to a kernel (on the host it
// is a stand-in, not a device address): static_scratch() looks up this
// device's address once and every launch takes that pointer.
static __device__ __align__(256) unsigned char scratch[VSD_STATIC_SCRATCH_BYTES];

namespace {

thread_local std::string g_last_error;

vsd_status fail(vsd_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

vsd_status ok() {
  g_last_error.clear();
  return VSD_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool finite_pos(float v) { return std::isfinite(v) && v > 0.0f; }

// A grid's size is a 32-bit count of work-items; the largest launch per row
// is one 192-thread workgroup per path (per-depth sampling, L = 1), so rows
// stay below 2^24, and the fused LM head's workgroups of 512 threads below
// 2^23.
constexpr int64_t kMaxRows = (int64_t)1 << 24;
constexpr int64_t kMaxLmWorkgroups = (int64_t)1 << 23;
constexpr int32_t kMaxHidden = 65536;

size_t align_up(size_t n) { return (n + 255) & ~(size_t)255; }

int64_t rows_of(const vsd_dims* d) { return (int64_t)d->B * d->T * d->N * d->L; }

// Shape checks shared by every entry point.
vsd_status check_dims(const vsd_dims* d) {
  if (d == nullptr) return fail(VSD_ERR_NULL_POINTER, "dims is NULL");
  if (d->B < 1 || d->T < 1) return fail(VSD_ERR_INVALID_SHAPE, "B=%d T=%d must be >= 1", d->B, d->T);
  if (d->N < 1 || d->N > 1024) return fail(VSD_ERR_INVALID_SHAPE, "N=%d outside [1,1024]", d->N);
  if (d->L < 1 || d->L > vsd::kMaxL) return fail(VSD_ERR_INVALID_SHAPE, "L=%d outside [1,64]", d->L);
  if (d->v_draft < 1) return fail(VSD_ERR_INVALID_SHAPE, "v_draft=%d must be >= 1", d->v_draft);
  if (d->v_target < d->v_draft)
    return fail(VSD_ERR_INVALID_SHAPE, "v_target=%d < v_draft=%d (the map must be injective)", d->v_target,
                d->v_draft);
  if (d->dtype != VSD_F32 && d->dtype != VSD_BF16) return fail(VSD_ERR_INVALID_VALUE, "dtype=%d", d->dtype);
  const int64_t R = rows_of(d);
  if (R >= kMaxRows) return fail(VSD_ERR_INVALID_SHAPE, "R=B*T*N*L=%lld must be < 2^24", (long long)R);
  if (d->hidden_dim < 0 || d->hidden_dim > kMaxHidden || d->hidden_dim % 64 != 0)
    return fail(VSD_ERR_INVALID_SHAPE, "hidden_dim=%d must be 0 or a multiple of 64 up to %d", d->hidden_dim,
                kMaxHidden);
  if (d->hidden_dim > 0) {
    if (d->dtype != VSD_BF16) return fail(VSD_ERR_UNSUPPORTED, "the fused LM head takes bf16 operands only");
    // the fused kernels launch row tiles x vocabulary tiles workgroups
    const int64_t nrt = (R + vsd::kLmTile - 1) / vsd::kLmTile;
    const int64_t vt = std::max<int64_t>(
        std::max<int64_t>((d->v_draft + vsd::kLmTile - 1) / vsd::kLmTile, (d->hidden_dim + vsd::kLmTile - 1) / vsd::kLmTile),
        vsd::lm_nslice(d->v_target) + vsd::lm_nslice(d->v_draft));
    if (nrt * vt >= kMaxLmWorkgroups)
      return fail(VSD_ERR_INVALID_SHAPE, "fused LM head: R=%lld rows x %lld vocabulary tiles too large",
                  (long long)R, (long long)vt);
  }
  return VSD_OK;
}

bool is_fused(const vsd_dims* d) { return d->hidden_dim > 0; }

// Fused LM-head checks for one source: hidden [R, H] and weight [V, H], bf16,
// rows contiguous.
vsd_status check_fused_src(const vsd_src* src, const char* name) {
  if (src == nullptr) return fail(VSD_ERR_NULL_POINTER, "%s source is NULL", name);
  if (src->logits != nullptr)
    return fail(VSD_ERR_UNSUPPORTED, "%s: hidden_dim > 0 selects the fused LM head, but logits were given", name);
  if (src->hidden == nullptr || src->weight == nullptr)
    return fail(VSD_ERR_NULL_POINTER, "%s: the fused LM head needs hidden and weight", name);
  if (!aligned16(src->hidden) || !aligned16(src->weight))
    return fail(VSD_ERR_MISALIGNED, "%s hidden / weight pointer not 16-byte aligned", name);
  return VSD_OK;
}

// Materialised-logit checks for one source.
vsd_status check_logits(const vsd_dims* d, const vsd_src* src, const char* name, int64_t ld, int32_t v) {
  if (src == nullptr) return fail(VSD_ERR_NULL_POINTER, "%s source is NULL", name);
  if (src->logits == nullptr) {
    if (src->hidden != nullptr || src->weight != nullptr)
      return fail(VSD_ERR_UNSUPPORTED, "%s: a fused LM-head source needs dims->hidden_dim > 0 (and is not "
                  "accepted by vsd_sample_paths)", name);
    return fail(VSD_ERR_NULL_POINTER, "%s logits are NULL", name);
  }
  const int64_t es = d->dtype == VSD_F32 ? 4 : 2;
  if (ld < v) return fail(VSD_ERR_INVALID_SHAPE, "%s ld=%lld < v=%d", name, (long long)ld, v);
  if ((ld * es) % 16 != 0)
    return fail(VSD_ERR_MISALIGNED, "%s row stride %lld bytes is not a multiple of 16", name, (long long)(ld * es));
  if (!aligned16(src->logits)) return fail(VSD_ERR_MISALIGNED, "%s logits pointer not 16-byte aligned", name);
  return VSD_OK;
}

// check_logits for a bare row pointer (the exact-context calls).
vsd_status check_rows(const vsd_dims* d, const void* rows, const char* name, int64_t ld, int32_t v) {
  const vsd_src src{rows, nullptr, nullptr};
  return check_logits(d, &src, name, ld, v);
}

// Every row set of an exact-context call: materialised logits, draft rows
// of the first `ndraft` families and target rows of the first `ntarget`.
vsd_status check_ctx_rows(const vsd_dims* d, const vsd_ctx_rows* rows, int ndraft, int ntarget) {
  if (is_fused(d)) return fail(VSD_ERR_UNSUPPORTED, "exact context: materialised logits only (hidden_dim must be 0)");
  if (rows == nullptr) return fail(VSD_ERR_NULL_POINTER, "rows is NULL");
  static const char* const dn[3] = {"draft rows along z~", "draft rows along z'", "draft rows along z-bar"};
  static const char* const tn[3] = {"target rows along z~", "target rows along z'", "target rows along z-bar"};
  vsd_status st;
  for (int f = 0; f < ndraft; ++f)
    if ((st = check_rows(d, rows->draft[f], dn[f], d->ld_draft, d->v_draft)) != VSD_OK) return st;
  for (int f = 0; f < ntarget; ++f)
    if ((st = check_rows(d, rows->target[f], tn[f], d->ld_target, d->v_target)) != VSD_OK) return st;
  return VSD_OK;
}

vsd_status check_map(const vsd_dims* d, const int32_t* d2t) {
  if (d->v_draft != d->v_target && d2t == nullptr)
    return fail(VSD_ERR_MAP_REQUIRED, "v_draft=%d != v_target=%d requires d2t", d->v_draft, d->v_target);
  if (d2t != nullptr && !aligned16(d2t)) return fail(VSD_ERR_MISALIGNED, "d2t pointer not 16-byte aligned");
  return VSD_OK;
}

// Both sources materialised (hidden_dim == 0) or both fused LM heads
// (hidden_dim > 0).
vsd_status check_sources(const vsd_dims* d, const vsd_src* draft, const vsd_src* target) {
  vsd_status st;
  if (d->hidden_dim > 0) {
    if ((st = check_fused_src(draft, "draft")) != VSD_OK) return st;
    return check_fused_src(target, "target");
  }
  if ((st = check_logits(d, draft, "draft", d->ld_draft, d->v_draft)) != VSD_OK) return st;
  return check_logits(d, target, "target", d->ld_target, d->v_target);
}

vsd_status check_params(const vsd_params* p) {
  if (p == nullptr) return fail(VSD_ERR_NULL_POINTER, "params is NULL");
  if (!finite_pos(p->temp_draft) || !finite_pos(p->temp_target))
    return fail(VSD_ERR_INVALID_VALUE, "temperatures must be finite and > 0");
  if (!finite_pos(p->w_base)) return fail(VSD_ERR_INVALID_VALUE, "w_base must be finite and > 0");
  if (!finite_pos(p->car_tau)) return fail(VSD_ERR_INVALID_VALUE, "car_tau must be finite and > 0");
  if (p->mode < VSD_GRAD_BASIC || p->mode > VSD_GRAD_ARW_CAR) return fail(VSD_ERR_INVALID_VALUE, "mode=%d", p->mode);
  if (p->car_input != VSD_CAR_PROB && p->car_input != VSD_CAR_LOGPROB)
    return fail(VSD_ERR_INVALID_VALUE, "car_input=%d", p->car_input);
  if (!std::isfinite(p->loss_scale)) return fail(VSD_ERR_INVALID_VALUE, "loss_scale must be finite");
  if (!std::isfinite(p->kl_weight) || p->kl_weight < 0.0f)
    return fail(VSD_ERR_INVALID_VALUE, "kl_weight must be finite and >= 0");
  if (p->kl_weight > 0.0f && (p->kl_topk < 1 || p->kl_topk > vsd::kMaxTopK))
    return fail(VSD_ERR_INVALID_VALUE, "kl_topk=%d outside [1,%d]", p->kl_topk, vsd::kMaxTopK);
  return VSD_OK;
}

bool kl_on(const vsd_params* p) { return p->kl_weight > 0.0f; }

vsd_status hip_fail(hipError_t e, const char* what) {
  return fail(VSD_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

struct WorkspaceLayout {
  size_t la, lq, loss, klrow, inv, part, klpart, klbound, klcount, kllist, total;
};

// la [R,3], lq [R,3], loss [P], KL row terms [R] fp32; the inverse map
// [v_target] int32 (fused LM head draws, verification); fused LM head also
// the slice partials [R, nslice_t + nslice_d] and, for the KL term, the
// target slices' lists [R, lm_kl_stride] (a recomputed row's records take
// their place), their bounds [R, nslice_t] and the count [1] and list [R]
// of the rows to recompute.
WorkspaceLayout workspace_layout(const vsd_dims* d) {
  const int64_t R = rows_of(d);
  const int64_t P = (int64_t)d->B * d->T;
  WorkspaceLayout w;
  w.la = 0;
  w.lq = w.la + align_up((size_t)R * 3 * sizeof(float));
  w.loss = w.lq + align_up((size_t)R * 3 * sizeof(float));
  w.klrow = w.loss + align_up((size_t)P * sizeof(float));
  w.inv = w.klrow + align_up((size_t)R * sizeof(float));
  w.part = w.inv + align_up((size_t)d->v_target * sizeof(int32_t));
  w.total = w.klpart = w.klbound = w.klcount = w.kllist = w.part;
  if (d->hidden_dim > 0) {
    const size_t nst = (size_t)vsd::lm_nslice(d->v_target);
    const size_t nsl = nst + (size_t)vsd::lm_nslice(d->v_draft);
    const size_t stride = (size_t)vsd::lm_kl_stride(d->v_draft, d->v_target);
    w.klpart = w.part + align_up((size_t)R * nsl * sizeof(vsd::LmPartial));
    w.klbound = w.klpart + align_up((size_t)R * stride * sizeof(vsd::LmKlEntry));
    w.klcount = w.klbound + align_up((size_t)R * nst * sizeof(float));
    w.kllist = w.klcount + align_up(sizeof(int32_t));
    w.total = w.kllist + align_up((size_t)R * sizeof(int32_t));
  }
  return w;
}

// Validation of the score outputs and workspace shared by the scoring calls.
vsd_status check_score_out_fields(const vsd_score_out* out) {
  if (out == nullptr) return fail(VSD_ERR_NULL_POINTER, "out is NULL");
  if (out->lse_draft == nullptr || out->coef_a == nullptr || out->coef_b == nullptr)
    return fail(VSD_ERR_NULL_POINTER, "out->lse_draft, coef_a and coef_b are required");
  if (out->device_error == nullptr) return fail(VSD_ERR_NULL_POINTER, "out->device_error is NULL");
  return VSD_OK;
}

vsd_status check_score_out(const vsd_dims* dims, const vsd_score_out* out, const void* workspace,
                           size_t workspace_bytes) {
  vsd_status st = check_score_out_fields(out);
  if (st != VSD_OK) return st;
  const WorkspaceLayout wl = workspace_layout(dims);
  if (workspace == nullptr || workspace_bytes < wl.total)
    return fail(VSD_ERR_WORKSPACE, "workspace of %zu bytes required, %zu given", wl.total,
                workspace == nullptr ? (size_t)0 : workspace_bytes);
  if (!aligned16(workspace)) return fail(VSD_ERR_MISALIGNED, "workspace not 16-byte aligned");
  return VSD_OK;
}

// Validation of the KL outputs (kl_weight > 0) shared by the scoring calls.
vsd_status check_kl_out(const vsd_dims* dims, const vsd_params* params, const vsd_score_out* out) {
  if (!kl_on(params)) return VSD_OK;
  if (params->kl_topk > dims->v_draft)
    return fail(VSD_ERR_INVALID_VALUE, "kl_topk=%d > v_draft=%d", params->kl_topk, dims->v_draft);
  if (out->kl_idx == nullptr || out->kl_grad == nullptr)
    return fail(VSD_ERR_NULL_POINTER, "out->kl_idx and out->kl_grad are required with kl_weight > 0");
  return VSD_OK;
}

// Row statistics of the materialised scoring calls.  Shared rows: one
// launch gathers the three families on X[0], Y[0].  Exact context: family f
// on X[f], Y[f] (one launch each); the draft log-sum-exp of the rows along z'
// goes to lse_corr.  The KL term, when on, rides on the launch that covers
// z~'s rows; *kl_row_out receives its [R] row terms (null when off).
vsd_status score_rows(const vsd_dims* dims, const vsd_params* params, const void* const X[3],
                      const void* const Y[3], bool ctx, const int32_t* d2t, const int32_t* valid_depth,
                      const int32_t* const tok[3], const vsd_score_out* out, float* lse_corr, char* ws,
                      const WorkspaceLayout& wl, float* la, float* lq, float** kl_row_out, hipStream_t s) {
  float* kl_row = nullptr;
  hipError_t e;
  if (kl_on(params))
    kl_row = out->kl_row != nullptr ? out->kl_row : reinterpret_cast<float*>(ws + wl.klrow);
  *kl_row_out = kl_row;
  for (int f = 0; f < (ctx ? 3 : 1); ++f) {
    vsd::ScoreRowArgs ra{};
    ra.X = X[f];
    ra.Y = Y[f];
    ra.d2t = d2t;
    ra.depth = valid_depth;
    for (int k = 0; k < 3; ++k) ra.tok[k] = tok[k];
    ra.fam_lo = ctx ? f : 0;
    ra.fam_hi = ctx ? f + 1 : 3;
    ra.lse_q = f == 0 ? out->lse_draft : f == 1 ? lse_corr : nullptr;
    ra.lse_p = f == 0 ? out->lse_target : nullptr;
    ra.la = la;
    ra.lq = lq;
    ra.err = out->device_error;
    ra.R = rows_of(dims);
    ra.ld_d = dims->ld_draft;
    ra.ld_t = dims->ld_target;
    ra.L = dims->L;
    ra.Vd = dims->v_draft;
    ra.Vt = dims->v_target;
    ra.inv_tq = 1.0f / params->temp_draft;
    ra.inv_tp = 1.0f / params->temp_target;
    if (kl_on(params) && f == 0) {
      ra.kl_k = params->kl_topk;
      ra.kl_idx = out->kl_idx;
      ra.kl_grad = out->kl_grad;
      ra.kl_row = kl_row;
      ra.kl_gscale = params->loss_scale * params->kl_weight / (float)dims->N / params->temp_draft;
    }
    e = vsd::launch_score_rows(ra, dims->dtype == VSD_BF16, s);
    if (e != hipSuccess) return hip_fail(e, "k_score_rows launch");
  }
  return VSD_OK;
}

// The per-position combine (and the loss total) over row statistics already
// in la / lq.
vsd_status launch_combine_and_total(const vsd_dims* dims, const vsd_params* params, const int32_t* valid_depth,
                                    const vsd_score_out* out, const float* la, const float* lq, float* loss_pos,
                                    const float* kl_row, hipStream_t s) {
  vsd::CombineArgs ca{};
  ca.la = la;
  ca.lq = lq;
  ca.depth = valid_depth;
  ca.survival = out->survival;
  ca.ea = out->exp_accept_len;
  ca.acc_flag = out->accept_flag;
  ca.val_flag = out->valid_flag;
  ca.o_prime = out->o_prime;
  ca.beta = out->beta;
  ca.zeta = out->zeta;
  ca.coef_a = out->coef_a;
  ca.coef_b = out->coef_b;
  ca.loss_pos = loss_pos;
  ca.err = out->device_error;
  ca.P = dims->B * dims->T;
  ca.N = dims->N;
  ca.L = dims->L;
  ca.mode = params->mode;
  ca.car_input = params->car_input;
  ca.inv_tau = 1.0f / params->car_tau;
  ca.kl_row = kl_row;
  ca.kl_pos = kl_row != nullptr ? out->kl_pos : nullptr;
  ca.kl_weight = params->kl_weight;
  for (int l = 0; l < dims->L; ++l) ca.w[l] = (float)std::pow((double)params->w_base, (double)(l + 1));
  hipError_t e = vsd::launch_combine(ca, s);
  if (e != hipSuccess) return hip_fail(e, "k_combine launch");
  if (out->loss_total != nullptr) {
    e = vsd::launch_loss_total(loss_pos, ca.P, params->loss_scale, out->loss_total, s);
    if (e != hipSuccess) return hip_fail(e, "k_loss_total launch");
  }
  return VSD_OK;
}

// The KL row terms' buffer of a fused call: the caller's kl_row or the
// workspace's (null with the term off).
float* fused_kl_row(const vsd_params* params, const vsd_score_out* out, char* ws, const WorkspaceLayout& wl) {
  if (!kl_on(params)) return nullptr;
  return out->kl_row != nullptr ? out->kl_row : reinterpret_cast<float*>(ws + wl.klrow);
}

// Fused LM head: the forward GEMM pass over both vocabularies (sampling
// or log-sum-exp only), then the slice combine into tokens and row
// statistics.  tok_in != null scores the given tokens; otherwise draws.
vsd_status lm_forward(const vsd_dims* dims, const vsd_params* params, const vsd_src* draft, const vsd_src* target,
                      const int32_t* d2t, const int32_t* valid_depth, uint64_t seed, uint32_t offset,
                      const int32_t* const tok_in[3], int32_t* const tok_out[3], const vsd_score_out* out,
                      char* ws, const WorkspaceLayout& wl, float* la, float* lq, float* kl_row, hipStream_t s) {
  const bool sampling = tok_in == nullptr;
  int32_t* inv = nullptr;
  hipError_t e;
  if ((sampling || kl_on(params)) && d2t != nullptr) {  // the target draws and the KL lists go through it
    inv = reinterpret_cast<int32_t*>(ws + wl.inv);
    e = vsd::launch_lm_inv(d2t, dims->v_draft, dims->v_target, inv, out->device_error, s);
    if (e != hipSuccess) return hip_fail(e, "k_lm_inv launch");
  }
  vsd::LmPartial* part = reinterpret_cast<vsd::LmPartial*>(ws + wl.part);
  vsd::LmFwdArgs f{};
  f.Hd = draft->hidden;
  f.Ht = target->hidden;
  f.Wd = draft->weight;
  f.Wt = target->weight;
  f.inv = inv;
  f.part = part;
  f.R = rows_of(dims);
  f.H = dims->hidden_dim;
  f.Vd = dims->v_draft;
  f.Vt = dims->v_target;
  f.nslice_t = vsd::lm_nslice(dims->v_target);
  f.nslice_d = vsd::lm_nslice(dims->v_draft);
  f.sample = sampling ? 1 : 0;
  f.inv_tq = 1.0f / params->temp_draft;
  f.inv_tp = 1.0f / params->temp_target;
  f.k0 = (uint32_t)(seed & 0xFFFFFFFFu);
  f.k1 = (uint32_t)(seed >> 32);
  f.offset = offset;
  if (kl_on(params)) {
    f.kl_part = reinterpret_cast<vsd::LmKlEntry*>(ws + wl.klpart);
    f.kl_stride = vsd::lm_kl_stride(dims->v_draft, dims->v_target);
    f.kl_bound = reinterpret_cast<float*>(ws + wl.klbound);
  }
  e = vsd::launch_lm_fwd(f, s);
  if (e != hipSuccess) return hip_fail(e, "k_lm_fwd launch");
  vsd::LmCombineArgs c{};
  c.part = part;
  c.Hd = draft->hidden;
  c.Ht = target->hidden;
  c.Wd = draft->weight;
  c.Wt = target->weight;
  c.d2t = d2t;
  c.depth = valid_depth;
  for (int k = 0; k < 3; ++k) {
    c.tok_in[k] = sampling ? nullptr : tok_in[k];
    c.tok_out[k] = sampling ? tok_out[k] : nullptr;
  }
  c.lse_q = out->lse_draft;
  c.lse_p = out->lse_target;
  c.la = la;
  c.lq = lq;
  c.err = out->device_error;
  c.R = f.R;
  c.L = dims->L;
  c.H = f.H;
  c.Vd = f.Vd;
  c.Vt = f.Vt;
  c.nslice_t = f.nslice_t;
  c.nslice_d = f.nslice_d;
  c.inv_tq = f.inv_tq;
  c.inv_tp = f.inv_tp;
  if (kl_on(params)) {
    c.kl_k = params->kl_topk;
    c.kl_part = f.kl_part;
    c.kl_bound = f.kl_bound;
    c.kl_count = reinterpret_cast<int32_t*>(ws + wl.klcount);
    c.kl_list = reinterpret_cast<int32_t*>(ws + wl.kllist);
    c.kl_stride = f.kl_stride;
    c.kl_nslice = vsd::lm_redo_nslice(dims->v_draft, dims->v_target);
    c.kl_idx = out->kl_idx;
    c.kl_grad = out->kl_grad;
    c.kl_row = kl_row;
    c.kl_gscale = params->loss_scale * params->kl_weight / (float)dims->N / params->temp_draft;
  }
  if (kl_on(params)) {
    e = vsd::launch_lm_kl_reset(c, s);
    if (e != hipSuccess) return hip_fail(e, "k_lm_kl_reset launch");
  }
  e = vsd::launch_lm_combine(c, s);
  if (e != hipSuccess) return hip_fail(e, "k_lm_combine launch");
  if (kl_on(params)) {
    e = vsd::launch_lm_kl_redo(c, s);
    if (e != hipSuccess) return hip_fail(e, "k_lm_kl_redo launch");
  }
  return VSD_OK;
}

// Device address of `scratch` on the calling thread's current device, looked
// up with that device current on the first call there and kept per device.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

vsd_status static_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(VSD_ERR_UNSUPPORTED, "device %d: at most %d devices", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (p == nullptr) return fail(VSD_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return VSD_OK;
}

}  // namespace

extern "C" {

int32_t vsd_abi_version(void) { return VSD_ABI_VERSION; }

const char* vsd_status_string(vsd_status s) {
  switch (s) {
    case VSD_OK: return "VSD_OK";
    case VSD_ERR_NULL_POINTER: return "VSD_ERR_NULL_POINTER";
    case VSD_ERR_INVALID_SHAPE: return "VSD_ERR_INVALID_SHAPE";
    case VSD_ERR_INVALID_VALUE: return "VSD_ERR_INVALID_VALUE";
    case VSD_ERR_MISALIGNED: return "VSD_ERR_MISALIGNED";
    case VSD_ERR_MAP_REQUIRED: return "VSD_ERR_MAP_REQUIRED";
    case VSD_ERR_UNSUPPORTED: return "VSD_ERR_UNSUPPORTED";
    case VSD_ERR_WORKSPACE: return "VSD_ERR_WORKSPACE";
    case VSD_ERR_HIP: return "VSD_ERR_HIP";
  }
  return "VSD_ERR_UNKNOWN";
}

const char* vsd_last_error(void) { return g_last_error.c_str(); }

vsd_status vsd_score_workspace_bytes(const vsd_dims* dims, size_t* bytes) {
  vsd_status st = check_dims(dims);
  if (st != VSD_OK) return st;
  if (bytes == nullptr) return fail(VSD_ERR_NULL_POINTER, "bytes is NULL");
  *bytes = workspace_layout(dims).total;
  return ok();
}

vsd_status vsd_sample_paths(const vsd_dims* dims, const vsd_src* draft, const vsd_src* target,
                            const int32_t* d2t, const int32_t* valid_depth, float temp_draft,
                            float temp_target, uint64_t seed, uint32_t offset, int32_t* tok_draft,
                            int32_t* tok_target, int32_t* tok_greedy, int32_t* device_error,
                            void* hip_stream) {
  vsd_status st = check_dims(dims);
  if (st != VSD_OK) return st;
  if (is_fused(dims))
    return fail(VSD_ERR_UNSUPPORTED, "the fused LM head needs a workspace: use vsd_sample_score_paths");
  if ((st = check_logits(dims, draft, "draft", dims->ld_draft, dims->v_draft)) != VSD_OK) return st;
  if ((st = check_logits(dims, target, "target", dims->ld_target, dims->v_target)) != VSD_OK) return st;
  if ((st = check_map(dims, d2t)) != VSD_OK) return st;
  if (!finite_pos(temp_draft) || !finite_pos(temp_target))
    return fail(VSD_ERR_INVALID_VALUE, "temperatures must be finite and > 0");
  if (tok_draft == nullptr || tok_target == nullptr || tok_greedy == nullptr)
    return fail(VSD_ERR_NULL_POINTER, "token outputs must not be NULL");
  if (device_error == nullptr) return fail(VSD_ERR_NULL_POINTER, "device_error is NULL");

  vsd::SampleArgs a{};
  a.X = draft->logits;
  a.Y = target->logits;
  a.d2t = d2t;
  a.depth = valid_depth;
  a.tok_d = tok_draft;
  a.tok_t = tok_target;
  a.tok_g = tok_greedy;
  a.err = device_error;
  a.R = rows_of(dims);
  a.ld_d = dims->ld_draft;
  a.ld_t = dims->ld_target;
  a.L = dims->L;
  a.Vd = dims->v_draft;
  a.Vt = dims->v_target;
  a.inv_tq = 1.0f / temp_draft;
  a.inv_tp = 1.0f / temp_target;
  a.k0 = (uint32_t)(seed & 0xFFFFFFFFu);
  a.k1 = (uint32_t)(seed >> 32);
  a.offset = offset;
  hipError_t e = vsd::launch_sample(a, dims->dtype == VSD_BF16, static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return hip_fail(e, "k_sample launch");
  return ok();
}

vsd_status vsd_score_paths(const vsd_dims* dims, const vsd_params* params, const vsd_src* draft,
                           const vsd_src* target, const int32_t* d2t, const int32_t* valid_depth,
                           const int32_t* tok_draft, const int32_t* tok_target, const int32_t* tok_greedy,
                           const vsd_score_out* out, void* workspace, size_t workspace_bytes,
                           void* hip_stream) {
  vsd_status st = check_dims(dims);
  if (st != VSD_OK) return st;
  if ((st = check_params(params)) != VSD_OK) return st;
  if ((st = check_sources(dims, draft, target)) != VSD_OK) return st;
  if ((st = check_map(dims, d2t)) != VSD_OK) return st;
  if (tok_draft == nullptr || tok_target == nullptr || tok_greedy == nullptr)
    return fail(VSD_ERR_NULL_POINTER, "token inputs must not be NULL");
  if ((st = check_score_out(dims, out, workspace, workspace_bytes)) != VSD_OK) return st;
  if ((st = check_kl_out(dims, params, out)) != VSD_OK) return st;
  const WorkspaceLayout wl = workspace_layout(dims);

  char* ws = static_cast<char*>(workspace);
  float* la = out->log_alpha != nullptr ? out->log_alpha : reinterpret_cast<float*>(ws + wl.la);
  float* lq = out->log_q_tok != nullptr ? out->log_q_tok : reinterpret_cast<float*>(ws + wl.lq);
  float* loss_pos = out->loss_pos != nullptr ? out->loss_pos : reinterpret_cast<float*>(ws + wl.loss);
  hipStream_t s = static_cast<hipStream_t>(hip_stream);

  if (is_fused(dims)) {
    const int32_t* const tin[3] = {tok_draft, tok_target, tok_greedy};
    float* kl_row = fused_kl_row(params, out, ws, wl);
    st = lm_forward(dims, params, draft, target, d2t, valid_depth, 0, 0, tin, nullptr, out, ws, wl, la, lq, kl_row,
                    s);
    if (st != VSD_OK) return st;
    if ((st = launch_combine_and_total(dims, params, valid_depth, out, la, lq, loss_pos, kl_row, s)) != VSD_OK)
      return st;
    return ok();
  }

  const void* const X[3] = {draft->logits, draft->logits, draft->logits};
  const void* const Y[3] = {target->logits, target->logits, target->logits};
  const int32_t* const tok[3] = {tok_draft, tok_target, tok_greedy};
  float* kl_row = nullptr;
  if ((st = score_rows(dims, params, X, Y, false, d2t, valid_depth, tok, out, nullptr, ws, wl, la, lq, &kl_row, s)) !=
      VSD_OK)
    return st;

  vsd_status st2 = launch_combine_and_total(dims, params, valid_depth, out, la, lq, loss_pos, kl_row, s);
  if (st2 != VSD_OK) return st2;
  return ok();
}

// The body of vsd_sample_score_paths, shared with its static-scratch variant.
static vsd_status sample_score_impl(const vsd_dims* dims, const vsd_params* params, const vsd_src* draft,
                                    const vsd_src* target, const int32_t* d2t, const int32_t* valid_depth,
                                    uint64_t seed, uint32_t offset, int32_t* tok_draft, int32_t* tok_target,
                                    int32_t* tok_greedy, const vsd_score_out* out, void* workspace,
                                    size_t workspace_bytes, void* hip_stream) {
  vsd_status st = check_dims(dims);
  if (st != VSD_OK) return st;
  if ((st = check_params(params)) != VSD_OK) return st;
  if ((st = check_sources(dims, draft, target)) != VSD_OK) return st;
  if ((st = check_map(dims, d2t)) != VSD_OK) return st;
  if (tok_draft == nullptr || tok_target == nullptr || tok_greedy == nullptr)
    return fail(VSD_ERR_NULL_POINTER, "token outputs must not be NULL");
  if ((st = check_score_out(dims, out, workspace, workspace_bytes)) != VSD_OK) return st;
  if ((st = check_kl_out(dims, params, out)) != VSD_OK) return st;

  const WorkspaceLayout wl = workspace_layout(dims);
  char* ws = static_cast<char*>(workspace);
  float* la = out->log_alpha != nullptr ? out->log_alpha : reinterpret_cast<float*>(ws + wl.la);
  float* lq = out->log_q_tok != nullptr ? out->log_q_tok : reinterpret_cast<float*>(ws + wl.lq);
  float* loss_pos = out->loss_pos != nullptr ? out->loss_pos : reinterpret_cast<float*>(ws + wl.loss);
  hipStream_t s = static_cast<hipStream_t>(hip_stream);

  if (is_fused(dims)) {
    int32_t* const tout[3] = {tok_draft, tok_target, tok_greedy};
    float* kl_row = fused_kl_row(params, out, ws, wl);
    st = lm_forward(dims, params, draft, target, d2t, valid_depth, seed, offset, nullptr, tout, out, ws, wl, la,
                    lq, kl_row, s);
    if (st != VSD_OK) return st;
    if ((st = launch_combine_and_total(dims, params, valid_depth, out, la, lq, loss_pos, kl_row, s)) != VSD_OK)
      return st;
    return ok();
  }

  vsd::SampleArgs a{};
  a.X = draft->logits;
  a.Y = target->logits;
  a.d2t = d2t;
  a.depth = valid_depth;
  a.tok_d = tok_draft;
  a.tok_t = tok_target;
  a.tok_g = tok_greedy;
  a.err = out->device_error;
  a.R = rows_of(dims);
  a.ld_d = dims->ld_draft;
  a.ld_t = dims->ld_target;
  a.L = dims->L;
  a.Vd = dims->v_draft;
  a.Vt = dims->v_target;
  a.inv_tq = 1.0f / params->temp_draft;
  a.inv_tp = 1.0f / params->temp_target;
  a.k0 = (uint32_t)(seed & 0xFFFFFFFFu);
  a.k1 = (uint32_t)(seed >> 32);
  a.offset = offset;
  a.lse_q = out->lse_draft;
  a.lse_p = out->lse_target;
  a.la = la;
  a.lq = lq;
  float* kl_row = nullptr;
  if (kl_on(params)) {
    kl_row = out->kl_row != nullptr ? out->kl_row : reinterpret_cast<float*>(ws + wl.klrow);
    a.kl_k = params->kl_topk;
    a.kl_idx = out->kl_idx;
    a.kl_grad = out->kl_grad;
    a.kl_row = kl_row;
    a.kl_gscale = params->loss_scale * params->kl_weight / (float)dims->N / params->temp_draft;
  }
  hipError_t e = vsd::launch_sample(a, dims->dtype == VSD_BF16, s);
  if (e != hipSuccess) return hip_fail(e, "k_sample (fused) launch");
  st = launch_combine_and_total(dims, params, valid_depth, out, la, lq, loss_pos, kl_row, s);
  if (st != VSD_OK) return st;
  return ok();
}

vsd_status vsd_sample_score_paths(const vsd_dims* dims, const vsd_params* params, const vsd_src* draft,
                                  const vsd_src* target, const int32_t* d2t, const int32_t* valid_depth,
                                  uint64_t seed, uint32_t offset, int32_t* tok_draft, int32_t* tok_target,
                                  int32_t* tok_greedy, const vsd_score_out* out, void* workspace,
                                  size_t workspace_bytes, void* hip_stream) {
  return sample_score_impl(dims, params, draft, target, d2t, valid_depth, seed, offset, tok_draft, tok_target,
                           tok_greedy, out, workspace, workspace_bytes, hip_stream);
}

vsd_status vsd_sample_score_paths_static(const vsd_dims* dims, const vsd_params* params, const vsd_src* draft,
                                         const vsd_src* target, const int32_t* d2t, const int32_t* valid_depth,
                                         uint64_t seed, uint32_t offset, int32_t* tok_draft, int32_t* tok_target,
                                         int32_t* tok_greedy, const vsd_score_out* out, void* hip_stream) {
  // everything the shared body checks except the workspace, before the
  // device is asked for the scratch's address
  vsd_status st = check_dims(dims);
  if (st != VSD_OK) return st;
  if ((st = check_params(params)) != VSD_OK) return st;
  if ((st = check_sources(dims, draft, target)) != VSD_OK) return st;
  if ((st = check_map(dims, d2t)) != VSD_OK) return st;
  if (tok_draft == nullptr || tok_target == nullptr || tok_greedy == nullptr)
    return fail(VSD_ERR_NULL_POINTER, "token outputs must not be NULL");
  if ((st = check_score_out_fields(out)) != VSD_OK) return st;
  if ((st = check_kl_out(dims, params, out)) != VSD_OK) return st;
  const size_t need = workspace_layout(dims).total;
  if (need > VSD_STATIC_SCRATCH_BYTES)
    return fail(VSD_ERR_WORKSPACE,
                "these dims need %zu bytes of workspace; the static scratch holds %zu (use vsd_sample_score_paths)",
                need, (size_t)VSD_STATIC_SCRATCH_BYTES);
  void* ws = nullptr;
  if ((st = static_scratch(&ws)) != VSD_OK) return st;
  return sample_score_impl(dims, params, draft, target, d2t, valid_depth, seed, offset, tok_draft, tok_target,
                           tok_greedy, out, ws, VSD_STATIC_SCRATCH_BYTES, hip_stream);
}

vsd_status vsd_weighted_loss_bwd(const vsd_dims* dims, const vsd_params* params, const vsd_src* draft,
                                 const float* lse_draft, const int32_t* tok_draft, const int32_t* tok_target,
                                 const float* coef_a, const float* coef_b, const int32_t* kl_idx,
                                 const float* kl_grad, const vsd_grad* grad, int32_t* device_error,
                                 void* hip_stream) {
  vsd_status st = check_dims(dims);
  if (st != VSD_OK) return st;
  if ((st = check_params(params)) != VSD_OK) return st;
  if (is_fused(dims)) {
    if ((st = check_fused_src(draft, "draft")) != VSD_OK) return st;
  } else if ((st = check_logits(dims, draft, "draft", dims->ld_draft, dims->v_draft)) != VSD_OK) {
    return st;
  }
  if (lse_draft == nullptr || tok_draft == nullptr || tok_target == nullptr || coef_a == nullptr ||
      coef_b == nullptr)
    return fail(VSD_ERR_NULL_POINTER, "lse_draft, tokens and coefficients are required");
  if (grad == nullptr || grad->grad_logits == nullptr) return fail(VSD_ERR_NULL_POINTER, "grad->grad_logits is NULL");
  if (!aligned16(grad->grad_logits)) return fail(VSD_ERR_MISALIGNED, "grad_logits not 16-byte aligned");
  if (device_error == nullptr) return fail(VSD_ERR_NULL_POINTER, "device_error is NULL");
  if (kl_on(params) && (kl_idx == nullptr || kl_grad == nullptr))
    return fail(VSD_ERR_NULL_POINTER, "kl_idx and kl_grad are required with kl_weight > 0");

  if (is_fused(dims)) {
    // grad_logits receives g (bf16, stride ld_draft), then dH = g W_d
    if (dims->ld_draft < dims->v_draft || (dims->ld_draft * 2) % 16 != 0)
      return fail(VSD_ERR_INVALID_SHAPE, "fused: ld_draft=%lld must be >= v_draft and a multiple of 8",
                  (long long)dims->ld_draft);
    if (grad->grad_hidden == nullptr) return fail(VSD_ERR_NULL_POINTER, "fused: grad->grad_hidden is NULL");
    if (!aligned16(grad->grad_hidden)) return fail(VSD_ERR_MISALIGNED, "grad_hidden not 16-byte aligned");
    if (grad->grad_weight != nullptr && !aligned16(grad->grad_weight))
      return fail(VSD_ERR_MISALIGNED, "grad_weight not 16-byte aligned");
    vsd::LmBwdArgs b{};
    b.Hd = draft->hidden;
    b.Wd = draft->weight;
    b.G = grad->grad_logits;
    b.dH = grad->grad_hidden;
    b.dW = grad->grad_weight;
    b.lse_q = lse_draft;
    b.tok_d = tok_draft;
    b.tok_t = tok_target;
    b.coef_a = coef_a;
    b.coef_b = coef_b;
    b.R = rows_of(dims);
    b.ldg = dims->ld_draft;
    b.H = dims->hidden_dim;
    b.Vd = dims->v_draft;
    b.inv_tq = 1.0f / params->temp_draft;
    b.scale = params->loss_scale;
    if (kl_on(params)) {
      b.kl_idx = kl_idx;
      b.kl_grad = kl_grad;
      b.kl_k = params->kl_topk;
    }
    hipError_t e = vsd::launch_lm_bwd(b, static_cast<hipStream_t>(hip_stream));
    if (e != hipSuccess) return hip_fail(e, "k_lm_bwd launch");
    return ok();
  }

  vsd::BwdArgs a{};
  a.X = draft->logits;
  a.G = grad->grad_logits;
  a.lse_q = lse_draft;
  a.tok_d = tok_draft;
  a.tok_t = tok_target;
  a.coef_a = coef_a;
  a.coef_b = coef_b;
  a.R = rows_of(dims);
  a.ld = dims->ld_draft;
  a.Vd = dims->v_draft;
  a.inv_tq = 1.0f / params->temp_draft;
  a.scale = params->loss_scale;
  if (kl_on(params)) {
    a.kl_idx = kl_idx;
    a.kl_grad = kl_grad;
    a.kl_k = params->kl_topk;
  }
  hipError_t e = vsd::launch_bwd(a, dims->dtype == VSD_BF16, static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return hip_fail(e, "k_bwd launch");
  return ok();
}

vsd_status vsd_sample_step(const vsd_dims* dims, int32_t step, const void* draft_rows, const void* target_rows,
                           const void* greedy_rows, const int32_t* d2t, const int32_t* valid_depth, float temp_draft,
                           float temp_target, uint64_t seed, uint32_t offset, int32_t* tok_draft,
                           int32_t* tok_target, int32_t* tok_greedy, int32_t* device_error, void* hip_stream) {
  vsd_status st = check_dims(dims);
  if (st != VSD_OK) return st;
  const vsd_ctx_rows rows{{draft_rows, nullptr, nullptr}, {target_rows, greedy_rows, nullptr}};
  if ((st = check_ctx_rows(dims, &rows, 1, 2)) != VSD_OK) return st;
  if (step < 0 || step >= dims->L) return fail(VSD_ERR_INVALID_VALUE, "step=%d outside [0, L=%d)", step, dims->L);
  if ((st = check_map(dims, d2t)) != VSD_OK) return st;
  if (!finite_pos(temp_draft) || !finite_pos(temp_target))
    return fail(VSD_ERR_INVALID_VALUE, "temperatures must be finite and > 0");
  if (tok_draft == nullptr || tok_target == nullptr || tok_greedy == nullptr)
    return fail(VSD_ERR_NULL_POINTER, "token outputs must not be NULL");
  if (device_error == nullptr) return fail(VSD_ERR_NULL_POINTER, "device_error is NULL");

  vsd::SampleStepArgs a{};
  a.X = draft_rows;
  a.Y = target_rows;
  a.Yg = greedy_rows;
  a.d2t = d2t;
  a.depth = valid_depth;
  a.tok_d = tok_draft;
  a.tok_t = tok_target;
  a.tok_g = tok_greedy;
  a.err = device_error;
  a.paths = (int64_t)dims->B * dims->T * dims->N;
  a.ld_d = dims->ld_draft;
  a.ld_t = dims->ld_target;
  a.L = dims->L;
  a.step = step;
  a.Vd = dims->v_draft;
  a.Vt = dims->v_target;
  a.inv_tq = 1.0f / temp_draft;
  a.inv_tp = 1.0f / temp_target;
  a.k0 = (uint32_t)(seed & 0xFFFFFFFFu);
  a.k1 = (uint32_t)(seed >> 32);
  a.offset = offset;
  hipError_t e = vsd::launch_sample_step(a, dims->dtype == VSD_BF16, static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return hip_fail(e, "k_sample_step launch");
  return ok();
}

vsd_status vsd_score_paths_ctx(const vsd_dims* dims, const vsd_params* params, const vsd_ctx_rows* rows,
                               const int32_t* d2t, const int32_t* valid_depth, const int32_t* tok_draft,
                               const int32_t* tok_target, const int32_t* tok_greedy, const vsd_score_out* out,
                               float* lse_draft_corr, void* workspace, size_t workspace_bytes, void* hip_stream) {
  vsd_status st = check_dims(dims);
  if (st != VSD_OK) return st;
  if ((st = check_params(params)) != VSD_OK) return st;
  if ((st = check_ctx_rows(dims, rows, 3, 3)) != VSD_OK) return st;
  if ((st = check_map(dims, d2t)) != VSD_OK) return st;
  if (tok_draft == nullptr || tok_target == nullptr || tok_greedy == nullptr)
    return fail(VSD_ERR_NULL_POINTER, "token inputs must not be NULL");
  if ((st = check_score_out(dims, out, workspace, workspace_bytes)) != VSD_OK) return st;
  if ((st = check_kl_out(dims, params, out)) != VSD_OK) return st;
  if (lse_draft_corr == nullptr) return fail(VSD_ERR_NULL_POINTER, "lse_draft_corr is NULL");

  const WorkspaceLayout wl = workspace_layout(dims);
  char* ws = static_cast<char*>(workspace);
  float* la = out->log_alpha != nullptr ? out->log_alpha : reinterpret_cast<float*>(ws + wl.la);
  float* lq = out->log_q_tok != nullptr ? out->log_q_tok : reinterpret_cast<float*>(ws + wl.lq);
  float* loss_pos = out->loss_pos != nullptr ? out->loss_pos : reinterpret_cast<float*>(ws + wl.loss);
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  const int32_t* const tok[3] = {tok_draft, tok_target, tok_greedy};
  float* kl_row = nullptr;
  if ((st = score_rows(dims, params, rows->draft, rows->target, true, d2t, valid_depth, tok, out, lse_draft_corr, ws,
                       wl, la, lq, &kl_row, s)) != VSD_OK)
    return st;
  if ((st = launch_combine_and_total(dims, params, valid_depth, out, la, lq, loss_pos, kl_row, s)) != VSD_OK)
    return st;
  return ok();
}

vsd_status vsd_weighted_loss_bwd_ctx(const vsd_dims* dims, const vsd_params* params, const vsd_ctx_rows* rows,
                                     const float* lse_draft, const float* lse_draft_corr, const int32_t* tok_draft,
                                     const int32_t* tok_target, const float* coef_a, const float* coef_b,
                                     const int32_t* kl_idx, const float* kl_grad, void* grad_draft_path,
                                     void* grad_corr_path, int32_t* device_error, void* hip_stream) {
  vsd_status st = check_dims(dims);
  if (st != VSD_OK) return st;
  if ((st = check_params(params)) != VSD_OK) return st;
  if ((st = check_ctx_rows(dims, rows, 2, 0)) != VSD_OK) return st;
  if (lse_draft == nullptr || lse_draft_corr == nullptr || tok_draft == nullptr || tok_target == nullptr ||
      coef_a == nullptr || coef_b == nullptr)
    return fail(VSD_ERR_NULL_POINTER, "log-sum-exps, tokens and coefficients are required");
  if (grad_draft_path == nullptr || grad_corr_path == nullptr)
    return fail(VSD_ERR_NULL_POINTER, "grad_draft_path and grad_corr_path are required");
  if (grad_draft_path == grad_corr_path)
    return fail(VSD_ERR_INVALID_VALUE, "grad_draft_path and grad_corr_path must be distinct buffers");
  if (!aligned16(grad_draft_path) || !aligned16(grad_corr_path))
    return fail(VSD_ERR_MISALIGNED, "gradient buffers not 16-byte aligned");
  if (device_error == nullptr) return fail(VSD_ERR_NULL_POINTER, "device_error is NULL");
  if (kl_on(params) && (kl_idx == nullptr || kl_grad == nullptr))
    return fail(VSD_ERR_NULL_POINTER, "kl_idx and kl_grad are required with kl_weight > 0");

  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  for (int f = 0; f < 2; ++f) {  // a-part on the rows along z~, b-part on the rows along z'
    vsd::BwdArgs a{};
    a.X = rows->draft[f];
    a.G = f == 0 ? grad_draft_path : grad_corr_path;
    a.lse_q = f == 0 ? lse_draft : lse_draft_corr;
    a.tok_d = tok_draft;
    a.tok_t = tok_target;
    a.coef_a = f == 0 ? coef_a : nullptr;
    a.coef_b = f == 0 ? nullptr : coef_b;
    a.R = rows_of(dims);
    a.ld = dims->ld_draft;
    a.Vd = dims->v_draft;
    a.inv_tq = 1.0f / params->temp_draft;
    a.scale = params->loss_scale;
    if (kl_on(params) && f == 0) {
      a.kl_idx = kl_idx;
      a.kl_grad = kl_grad;
      a.kl_k = params->kl_topk;
    }
    hipError_t e = vsd::launch_bwd(a, dims->dtype == VSD_BF16, s);
    if (e != hipSuccess) return hip_fail(e, "k_bwd launch");
  }
  return ok();
}

vsd_status vsd_verify_paths(const vsd_dims* dims, const vsd_params* params, const vsd_src* draft,
                            const vsd_src* target, const int32_t* d2t, const int32_t* valid_depth,
                            const float* log_alpha, const float* lse_draft, const float* lse_target, uint64_t seed,
                            uint32_t offset, int32_t* accept_len, int32_t* resample_tok, void* workspace,
                            size_t workspace_bytes, int32_t* device_error, void* hip_stream) {
  vsd_status st = check_dims(dims);
  if (st != VSD_OK) return st;
  if ((st = check_params(params)) != VSD_OK) return st;
  if (is_fused(dims)) return fail(VSD_ERR_UNSUPPORTED, "verification: materialised logits only (hidden_dim must be 0)");
  if ((st = check_sources(dims, draft, target)) != VSD_OK) return st;
  if ((st = check_map(dims, d2t)) != VSD_OK) return st;
  if (log_alpha == nullptr || lse_draft == nullptr || lse_target == nullptr)
    return fail(VSD_ERR_NULL_POINTER, "log_alpha, lse_draft and lse_target (from scoring) are required");
  if (accept_len == nullptr || resample_tok == nullptr)
    return fail(VSD_ERR_NULL_POINTER, "accept_len and resample_tok are required");
  if (device_error == nullptr) return fail(VSD_ERR_NULL_POINTER, "device_error is NULL");
  const WorkspaceLayout wl = workspace_layout(dims);
  if (d2t != nullptr) {
    if (workspace == nullptr || workspace_bytes < wl.total)
      return fail(VSD_ERR_WORKSPACE, "workspace of %zu bytes required, %zu given", wl.total,
                  workspace == nullptr ? (size_t)0 : workspace_bytes);
    if (!aligned16(workspace)) return fail(VSD_ERR_MISALIGNED, "workspace not 16-byte aligned");
  }

  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  int32_t* inv = nullptr;
  if (d2t != nullptr) {
    inv = reinterpret_cast<int32_t*>(static_cast<char*>(workspace) + wl.inv);
    hipError_t e = vsd::launch_lm_inv(d2t, dims->v_draft, dims->v_target, inv, device_error, s);
    if (e != hipSuccess) return hip_fail(e, "k_lm_inv launch");
  }
  vsd::VerifyArgs a{};
  a.X = draft->logits;
  a.Y = target->logits;
  a.inv = inv;
  a.depth = valid_depth;
  a.la = log_alpha;
  a.lse_q = lse_draft;
  a.lse_p = lse_target;
  a.accept_len = accept_len;
  a.resample = resample_tok;
  a.err = device_error;
  a.paths = (int64_t)dims->B * dims->T * dims->N;
  a.ld_d = dims->ld_draft;
  a.ld_t = dims->ld_target;
  a.L = dims->L;
  a.Vd = dims->v_draft;
  a.Vt = dims->v_target;
  a.inv_tq = 1.0f / params->temp_draft;
  a.inv_tp = 1.0f / params->temp_target;
  a.k0 = (uint32_t)(seed & 0xFFFFFFFFu);
  a.k1 = (uint32_t)(seed >> 32);
  a.offset = offset;
  hipError_t e = vsd::launch_verify(a, dims->dtype == VSD_BF16, s);
  if (e != hipSuccess) return hip_fail(e, "k_verify launch");
  return ok();
}

}  // extern "C"
