// Path scoring (vsd_score_paths).
//
// k_score_rows   one wavefront per row: online log-sum-exp of X/T_q over the
//                draft vocabulary and of Y/T_p over the whole target
//                vocabulary (128-bit loads, exp2 with folded scales, per-lane
//                chunk max), then the token gathers giving log q, log p and
//                log alpha = min(0, log p - log q) of the three families
//                (Sec. "Preliminary", Eq. acc).
// k_combine      one workgroup per position, one thread per path: prefix sums
//                over depth (Eqs. kappa, survival_def, accepted_len_cond), the
//                oracle gate and the correction (Alg. 2, Alg. 1), ARW beta
//                (Eq. beta_update), CAR zeta (Eq. zeta_update), the loss of
//                Eq. advance / Eq. basic and the per-row coefficients a, b.
// k_loss_total   one workgroup: loss_scale * sum over positions, fixed order.
//
// With the top-K renormalised KL term on (VSD (KL) variant, Eq. klv),
// k_score_rows also selects, while it streams the target row, the K mapped
// target tokens with the largest logits (exact wavefront top-K, vsd_topk.hpp;
// the mapped values are gathered through the map next to the block being
// streamed), then forms p_hat and q_hat renormalised over them, the row's term
// -sum p_hat log q_hat and its gradient coefficients; k_combine adds the
// per-position average over paths to the loss.
#include "vsd_device.hpp"
#include "vsd_kernels.hpp"
#include "vsd_topk.hpp"

namespace vsd {

namespace {

constexpr int kRowsPerBlock = 4;

// Online log-sum-exp of row[v] / T over v < V, reduced over the wavefront.
//
// With c = float(log2(e) / T), each lane keeps mraw (its largest raw logit),
// mc = float(mraw * c) and s = sum_v exp2(fma(x_v, c, -mc)); the fused
// multiply-add forms x_v * c exactly, so s is exactly consistent with mc.
// Because float(mraw * c) differs from mraw * c by delta = fma(mraw, c, -mc)
// (exactly representable), log2 sum_v 2^((x_v - mraw) c) = log2(s) - delta.
// Callers then form log q(z) = (x_z - mraw)/T - ln2 (log2 s - delta), which
// keeps full float32 precision even when |x/T| is in the hundreds (the
// shifted difference never rounds against a large log-sum-exp).
struct RowLse {
  float mraw;  // wavefront max of the raw logits
  float tail;  // ln sum_v exp((x_v - mraw)/T)  (>= 0)
};

template <typename T>
__device__ __forceinline__ RowLse row_lse(const T* row, int V, float c, int lane) {
  float mraw = kNegBig, mc = kNegBig, s = 0.0f;
  constexpr int U = 4;          // chunks in flight per lane
  constexpr int step = 8 * kWave;
  int base = lane * 8;
  for (; base + (U - 1) * step + 8 <= V; base += U * step) {
    float x[U][8];
#pragma unroll
    for (int u = 0; u < U; ++u) load8(row + base + u * step, x[u]);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float cm = max8(x[u]);
      if (cm > mraw) {
        const float nmc = cm * c;
        s *= __builtin_amdgcn_exp2f(mc - nmc);
        mc = nmc;
        mraw = cm;
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) s += __builtin_amdgcn_exp2f(fmaf(x[u][k], c, -mc));
    }
  }
  for (; base + 8 <= V; base += step) {
    float x[8];
    load8(row + base, x);
    const float cm = max8(x);
    if (cm > mraw) {
      const float nmc = cm * c;
      s *= __builtin_amdgcn_exp2f(mc - nmc);
      mc = nmc;
      mraw = cm;
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) s += __builtin_amdgcn_exp2f(fmaf(x[k], c, -mc));
  }
  if (base < V) {  // the one partial chunk of the row
    for (int v = base; v < V; ++v) {
      const float xv = load1(row + v);
      if (xv > mraw) {
        const float nmc = xv * c;
        s *= __builtin_amdgcn_exp2f(mc - nmc);
        mc = nmc;
        mraw = xv;
      }
      s += __builtin_amdgcn_exp2f(fmaf(xv, c, -mc));
    }
  }
  wave_lse2(mc, s);            // every lane's mc = float(its mraw * c): the max commutes
  mraw = wave_max(mraw);
  const float delta = fmaf(mraw, c, -mc);
  return RowLse{mraw, (log2f(s) - delta) * kLn2};
}

// row_lse of the target row, also selecting the K mapped target logits of
// largest value (wavefront top-K; value = raw target logit, index = its
// draft index).  Four chunks are in flight per lane as in row_lse, so one
// iteration streams a 2048-column block.  With a map, the same iteration
// offers draft chunk it = 512 indices: each lane gathers Y[d2t[v]] for
// v = 512 it + 64 k + lane, k < 8.  For an ascending map (about four target
// columns per draft index) those columns lie in the block just streamed, so
// the gathers find their lines in L2.  Draft chunks left when the stream ends
// (a map onto fewer columns than 4 per index) are offered after it.  Without
// a map the streamed values themselves are offered.  Only values at or above
// the top-K threshold are ever appended, so a slice whose largest value is
// below it in every lane offers nothing: one ballot decides.  Map entries
// outside [0, Vt) are reported by k_map_check, launched first.
template <typename T, bool MAPPED>
__device__ RowLse row_lse_topk(const T* row, int V, float c, int lane, WaveTopK& tk, const int32_t* d2t, int Vd) {
  float mraw = kNegBig, mc = kNegBig, s = 0.0f;
  constexpr int U = 4;
  constexpr int step = 8 * kWave;
  bool seeded = false;
  auto offer = [&](const float (&x)[8], int base, uint32_t bits, float vmax, auto idx_of) {
    if (!seeded) {  // the threshold from the lanes' largest offered values of the first slice
      seeded = true;
      tk.seed_lane_max(vmax, lane);
      tk.offer8(x, base, bits, idx_of, lane);
      return;
    }
    if (__ballot(vmax >= tk.thv) == 0ull) return;  // vmax: the lane's largest offered value
    tk.append8(x, base, bits, idx_of, lane);
  };
  auto lse8 = [&](const float (&x)[8], float cm) {
    if (cm > mraw) {
      const float nmc = cm * c;
      s *= __builtin_amdgcn_exp2f(mc - nmc);
      mc = nmc;
      mraw = cm;
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) s += __builtin_amdgcn_exp2f(fmaf(x[k], c, -mc));
  };
  // Draft chunk dc (512 indices; lane-strided: k-th value of a lane is draft
  // index 512 dc + 64 k + lane) is offered from gathered raw values.  Its map
  // entries are loaded one iteration ahead and its gathers are issued right
  // after the stream loads of the iteration that offers it, so the
  // log-sum-exp work of the block covers their latency.  The map's range is
  // checked before the launch (k_map_check); the gathers go through the
  // row's buffer resource, which keeps every access in the row.  Only the
  // last chunk can hold indices past V_d (their slots offer nothing).
  const int ndc = MAPPED ? (Vd + step - 1) / step : 0;
  const int nfull_dc = MAPPED ? Vd / step : 0;
  int dc = 0;
  uint32_t tmap[8];
  T graw[8];
  const __amdgpu_buffer_rsrc_t yrow = row_rsrc(row, row_bytes(row, V));
  auto load_map = [&](int d) {
    if (d < nfull_dc) {
#pragma unroll
      for (int k = 0; k < 8; ++k) tmap[k] = (uint32_t)d2t[d * step + k * kWave + lane];
    } else {
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int v = d * step + k * kWave + lane;
        tmap[k] = v < Vd ? (uint32_t)d2t[v] : 0u;
      }
    }
  };
  auto gather = [&]() {
#pragma unroll
    for (int k = 0; k < 8; ++k) buf_gather(yrow, tmap[k], graw[k]);
  };
  auto offer_gathered = [&](int d) {
    float y[8];
    uint32_t bits = 0xFFu;
#pragma unroll
    for (int k = 0; k < 8; ++k) y[k] = load1(&graw[k]);
    if (d >= nfull_dc) {
      bits = 0u;
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const bool in = d * step + k * kWave + lane < Vd;
        y[k] = in ? y[k] : -INFINITY;
        bits |= in ? (1u << k) : 0u;
      }
    }
    const int base = d * step + lane;
    offer(y, 0, bits, max8(y), [&](int k) { return base + k * kWave; });
  };
  if (MAPPED && ndc > 0) load_map(0);
  int chunk = 0;
  for (; chunk + U * step <= V; chunk += U * step) {
    float x[U][8];
#pragma unroll
    for (int u = 0; u < U; ++u) load8(row + chunk + u * step + lane * 8, x[u]);
    const bool g = MAPPED && dc < ndc;
    if (g) gather();
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float cm = max8(x[u]);
      lse8(x[u], cm);
      if (!MAPPED) offer(x[u], chunk + u * step + lane * 8, 0xFFu, cm, [](int col) { return col; });
    }
    if (g) {
      offer_gathered(dc);
      if (++dc < ndc) load_map(dc);
    }
  }
  for (; chunk < V; chunk += step) {
    const int base = chunk + lane * 8;
    const int nvalid = min(8, V - base);
    float x[8];
    if (nvalid >= 8) {
      load8(row + base, x);
    } else {
#pragma unroll
      for (int k = 0; k < 8; ++k) x[k] = k < nvalid ? load1(row + base + k) : -INFINITY;
    }
    const float cm = max8(x);
    lse8(x, cm);
    if (!MAPPED) {
      const uint32_t bits = nvalid <= 0 ? 0u : nvalid >= 8 ? 0xFFu : (1u << nvalid) - 1u;
      offer(x, base, bits, cm, [](int col) { return col; });
    }
  }
  for (; MAPPED && dc < ndc;) {  // draft chunks past the streamed blocks
    gather();
    offer_gathered(dc);
    if (++dc < ndc) load_map(dc);
  }
  wave_lse2(mc, s);
  mraw = wave_max(mraw);
  const float delta = fmaf(mraw, c, -mc);
  return RowLse{mraw, (log2f(s) - delta) * kLn2};
}

template <typename T, bool MAPPED, bool KL>
__global__ __launch_bounds__(256) void k_score_rows(ScoreRowArgs a) {
  __shared__ float kl_bv[KL ? kRowsPerBlock * kTopKCap : 1];
  __shared__ int kl_bi[KL ? kRowsPerBlock * kTopKCap : 1];
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t r = (int64_t)blockIdx.x * kRowsPerBlock + wave_id();
  if (r >= a.R) return;
  const int i = (int)(r % a.L);
  const int64_t path = r / a.L;
  int d = a.L;
  if (a.depth != nullptr) {
    d = a.depth[path];
    if (d < 1 || d > a.L) {
      if (lane == 0) report_error(a.err, VSD_DEVERR_DEPTH_RANGE);
      d = 0;
    }
  }
  if (i >= d) {  // masked slot: nothing is read, every output is zero
    if (lane < 3) {
      a.la[r * 3 + lane] = 0.0f;
      a.lq[r * 3 + lane] = 0.0f;
    }
    if (lane == 0) {
      if (a.lse_q != nullptr) a.lse_q[r] = 0.0f;
      if (a.lse_p != nullptr) a.lse_p[r] = 0.0f;
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
  const T* X = static_cast<const T*>(a.X) + r * a.ld_d;
  const T* Y = static_cast<const T*>(a.Y) + r * a.ld_t;
  const RowLse q = row_lse(X, a.Vd, a.inv_tq * kLog2e, lane);
  WaveTopK tk;
  RowLse p;
  if (KL) {
    const int slot = wave_id();
    tk.init(kl_bv + slot * kTopKCap, kl_bi + slot * kTopKCap, a.kl_k);
    p = row_lse_topk<T, MAPPED>(Y, a.Vt, a.inv_tp * kLog2e, lane, tk, a.d2t, a.Vd);
  } else {
    p = row_lse(Y, a.Vt, a.inv_tp * kLog2e, lane);
  }
  const float lse_q = q.mraw * a.inv_tq + q.tail;
  const float lse_p = p.mraw * a.inv_tp + p.tail;
  const float gap = lse_gap(p.mraw, p.tail, a.inv_tp, q.mraw, q.tail, a.inv_tq);
  if (lane >= a.fam_lo && lane < a.fam_hi) {  // lane f gathers family f
    const int32_t z = a.tok[lane][r];
    float lq = 0.0f, la = 0.0f;
    if ((uint32_t)z >= (uint32_t)a.Vd) {
      report_error(a.err, VSD_DEVERR_TOKEN_RANGE);
    } else {
      const int32_t zt = MAPPED ? a.d2t[z] : z;
      if ((uint32_t)zt >= (uint32_t)a.Vt) {
        report_error(a.err, VSD_DEVERR_MAP_RANGE);
      } else {
        const float xz = load1(X + z);
        lq = (xz - q.mraw) * a.inv_tq - q.tail;
        la = log_alpha_of(xz, load1(Y + zt), a.inv_tq, a.inv_tp, gap);
      }
    }
    a.la[r * 3 + lane] = la;
    a.lq[r * 3 + lane] = lq;
  }
  if (lane == 0) {
    if (a.lse_q != nullptr) a.lse_q[r] = lse_q;
    if (a.lse_p != nullptr) a.lse_p[r] = lse_p;
  }
  if (KL) {
    tk.finish(lane);
    kl_row_term(tk, X, a.Vd, a.inv_tq, a.inv_tp, a.kl_gscale, a.kl_idx + r * a.kl_k, a.kl_grad + r * a.kl_k,
                a.kl_row + r, lane);
  }
}

// Deterministic block reductions: butterfly within each wavefront, then the
// per-wavefront partials combined in wavefront order by every thread.
__device__ __forceinline__ float block_sum(float v, float* smem) {
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = wave_sum(v);
  __syncthreads();
  if (lane == 0) smem[w] = v;
  __syncthreads();
  float t = 0.0f;
  for (int k = 0; k < nw; ++k) t += smem[k];
  return t;
}

__device__ __forceinline__ float block_max(float v, float* smem) {
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = wave_max(v);
  __syncthreads();
  if (lane == 0) smem[w] = v;
  __syncthreads();
  float t = kNegBig;
  for (int k = 0; k < nw; ++k) t = fmaxf(t, smem[k]);
  return t;
}

__device__ __forceinline__ int block_sum_int(int v, int* smem) {
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = wave_sum_int(v);
  __syncthreads();
  if (lane == 0) smem[w] = v;
  __syncthreads();
  int t = 0;
  for (int k = 0; k < nw; ++k) t += smem[k];
  return t;
}

__global__ __launch_bounds__(1024) void k_combine(CombineArgs a) {
  __shared__ float redf[16];
  __shared__ int redi[16];
  const int pos = blockIdx.x;
  const int s = threadIdx.x;
  const bool real = s < a.N;
  int d = 0;
  if (real) {
    d = a.depth != nullptr ? a.depth[(int64_t)pos * a.N + s] : a.L;
    if (d < 1 || d > a.L) {
      report_error(a.err, VSD_DEVERR_DEPTH_RANGE);
      d = 0;
    }
  }
  const int64_t row0 = ((int64_t)pos * a.N + s) * a.L;
  float LSd = 0.0f, LSt = 0.0f, LSg = 0.0f, LQd = 0.0f, LQt = 0.0f;
  float ea = 0.0f, wsum = 0.0f, lsum = 0.0f, klsum = 0.0f;
  for (int l = 0; l < a.L; ++l) {
    const bool live = real && l < d;
    const int64_t row = row0 + l;
    if (live && a.kl_row != nullptr) klsum += a.kl_row[row];
    if (live) {  // prefix sums of log alpha (log survival) and of log q
      LSd += a.la[row * 3 + 0];
      LSt += a.la[row * 3 + 1];
      LSg += a.la[row * 3 + 2];
      LQd += a.lq[row * 3 + 0];
      LQt += a.lq[row * 3 + 1];
    }
    // Alg. 2 gate on z~; Alg. 1 substitutes z' when it fails.
    const bool acc = live && (LSd >= LSg);
    const bool val = live && (acc || LSt >= LSg);
    // ARW: leave-one-out acceptance rate among live paths with o' > 0; all
    // o' at one level share w(l), which cancels (acc implies val).
    const int n_acc = block_sum_int(acc ? 1 : 0, redi);
    const int n_val = block_sum_int(val ? 1 : 0, redi);
    const int num = n_acc - (acc ? 1 : 0);
    const int den = n_val - (val ? 1 : 0);
    const float beta = (live && den > 0) ? (float)num / (float)den : 0.0f;
    // CAR: softmax over live paths of confidence / tau.
    const float conf = a.car_input == VSD_CAR_PROB ? expf(LQd) : LQd;
    const float cmax = block_max(live ? conf : kNegBig, redf);
    const float e = live ? expf((conf - cmax) * a.inv_tau) : 0.0f;
    const float esum = block_sum(e, redf);
    const float zeta = live ? e / esum : 0.0f;
    const float c = a.mode == VSD_GRAD_ARW_CAR ? beta * zeta : a.mode == VSD_GRAD_ARW ? beta : 0.0f;
    const float o = val ? a.w[l] : 0.0f;
    const float surv = live ? expf(LSd) : 0.0f;
    ea += surv;
    wsum += o;
    if (live) lsum += o * ((acc ? LQd : LQt) - c * LQd);
    if (real) {
      if (a.survival) a.survival[row] = surv;
      if (a.acc_flag) a.acc_flag[row] = acc ? 1 : 0;
      if (a.val_flag) a.val_flag[row] = val ? 1 : 0;
      if (a.o_prime) a.o_prime[row] = o;
      if (a.beta) a.beta[row] = beta;
      if (a.zeta) a.zeta[row] = zeta;
      // level-l terms of the coefficient suffix sums, finished below
      a.coef_a[row] = o * ((acc ? 1.0f : 0.0f) - c);
      a.coef_b[row] = o * (acc ? 0.0f : 1.0f);
    }
  }
  const float W = block_sum(wsum, redf);
  const float total = block_sum(lsum, redf);
  if (real) {
    // a_{s,i} = (1/W) sum_{l>=i} o'(I~ - c),  b_{s,i} = (1/W) sum_{l>=i} o'(1 - I~)
    float acc_a = 0.0f, acc_b = 0.0f;
    for (int l = a.L - 1; l >= 0; --l) {
      const int64_t row = row0 + l;
      if (l < d && W > 0.0f) {
        acc_a += a.coef_a[row];
        acc_b += a.coef_b[row];
        a.coef_a[row] = acc_a / W;
        a.coef_b[row] = acc_b / W;
      } else {
        a.coef_a[row] = 0.0f;
        a.coef_b[row] = 0.0f;
      }
    }
    if (a.ea) a.ea[(int64_t)pos * a.N + s] = ea;
  }
  if (a.kl_row != nullptr) {
    // KL_x = (1/N) sum over live slots of the row terms, weighted into the loss
    const float kl = block_sum(klsum, redf) / (float)a.N;
    if (threadIdx.x == 0) {
      a.loss_pos[pos] = (W > 0.0f ? -total / W : 0.0f) + a.kl_weight * kl;
      if (a.kl_pos != nullptr) a.kl_pos[pos] = kl;
    }
  } else if (threadIdx.x == 0) {
    a.loss_pos[pos] = W > 0.0f ? -total / W : 0.0f;
  }
}

__global__ __launch_bounds__(256) void k_loss_total(const float* loss_pos, int32_t P, float scale, float* out) {
  __shared__ float red[16];
  float t = 0.0f;
  for (int p = threadIdx.x; p < P; p += blockDim.x) t += loss_pos[p];
  t = block_sum(t, red);
  if (threadIdx.x == 0) *out = scale * t;
}

template <typename T>
hipError_t launch_rows_t(const ScoreRowArgs& a, hipStream_t s) {
  const dim3 grid((unsigned)((a.R + kRowsPerBlock - 1) / kRowsPerBlock));
  if (a.kl_k > 0 && a.d2t != nullptr) {  // the top-K gathers through the map unchecked
    const hipError_t e = launch_map_check(a.d2t, a.Vd, a.Vt, a.err, s);
    if (e != hipSuccess) return e;
  }
  if (a.kl_k > 0) {
    if (a.d2t != nullptr)
      hipLaunchKernelGGL((k_score_rows<T, true, true>), grid, dim3(256), 0, s, a);
    else
      hipLaunchKernelGGL((k_score_rows<T, false, true>), grid, dim3(256), 0, s, a);
  } else if (a.d2t != nullptr) {
    hipLaunchKernelGGL((k_score_rows<T, true, false>), grid, dim3(256), 0, s, a);
  } else {
    hipLaunchKernelGGL((k_score_rows<T, false, false>), grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_score_rows(const ScoreRowArgs& a, bool bf16, hipStream_t s) {
  return bf16 ? launch_rows_t<bf16_t>(a, s) : launch_rows_t<float>(a, s);
}

hipError_t launch_combine(const CombineArgs& a, hipStream_t s) {
  const int threads = ((a.N + kWave - 1) / kWave) * kWave;
  hipLaunchKernelGGL(k_combine, dim3((unsigned)a.P), dim3(threads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_loss_total(const float* loss_pos, int32_t P, float scale, float* out, hipStream_t s) {
  hipLaunchKernelGGL(k_loss_total, dim3(1), dim3(256), 0, s, loss_pos, P, scale, out);
  return hipGetLastError();
}

}  // namespace vsd
