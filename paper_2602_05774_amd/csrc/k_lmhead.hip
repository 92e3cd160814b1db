// Fused LM-head variant: the draft and target logits X = H_d W_d^T and
// Y = H_t W_t^T (bf16 operands, fp32 accumulation on MFMA) are never written
// to memory.
//
// Forward.  One launch covers both models.  A workgroup (four wavefronts)
// owns 128 rows and one slice of a vocabulary; for every 128-column tile of
// the slice it computes the 128x128 logit tile on v_mfma_f32_32x32x16_bf16
// (each wavefront a 64x64 quadrant of 2x2 MFMA tiles, operands staged
// through double-buffered LDS) and consumes it in place: the online
// log-sum-exp (row softmax normalisers, Sec. "Preliminary"), the Gumbel-max
// draws with the exact candidate filter (Alg. 1 draws z~ ~ q and z' ~ p under
// the library's normative sampler) and the greedy maximum (Alg. 2).  Per-row
// running state stays in LDS across the tiles of the slice; the slice's
// result goes to a partial record.  A combine kernel merges the slices, forms
// the drawn tokens' logits by dot products (H_r . W_z) and writes tokens and
// the per-row statistics (log q, log alpha of Eq. acc) that the per-position
// combine then turns into weights and the loss.
//
// Backward (derivative of Eq. advance through the LM head).  The draft
// logits are recomputed tile by tile; g = loss_scale/T_q ((a+b) q - a e_z~ -
// b e_z') is written in bf16 (the gradient with respect to the logits); then
// dH_d = g W_d on MFMA, the W_d tiles read column-wise out of LDS.
#include "vsd_device.hpp"
#include "vsd_kernels.hpp"

namespace vsd {

namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int LDK = BK + 8;     // padded K-contiguous LDS row (bf16): 144 B, conflict-free 16-B reads
constexpr int LDN = BN + 8;     // padded N-contiguous LDS row (bf16) of the NN GEMM's B tile
constexpr int LDT = BN + 4;     // padded fp32 epilogue tile row
constexpr int kStageElems = (BM + BN) * LDK;        // A and B tiles of one stage (bf16)
constexpr int kLdsBytes = 2 * kStageElems * 2;      // double buffer; also holds the fp32 tile
constexpr int kXcds = 8;                            // MI355X: 8 XCDs, workgroups dealt round-robin
constexpr int kGroupRows = 8;                       // row tiles per L2 reuse group
static_assert(BM * LDT * 4 <= kLdsBytes, "epilogue tile must fit the operand buffers");
static_assert(BM * LDK + BK * LDN <= kStageElems, "NN stage must fit");
static_assert(kLmTile == BN, "vocabulary tile width");

__device__ __forceinline__ f32x16 mfma(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Workgroup -> (row tile, column index) so that the workgroups resident on
// one XCD at a time share few operand tiles: the dispatcher deals workgroup
// ids round-robin over the XCDs, so ids are first regrouped per XCD
// (a bijection), then walked in groups of kGroupRows row tiles, column index
// fastest within a group.
__device__ __forceinline__ void tile_of(int pid, int nrt, int ncol, int& rt, int& col) {
  const int total = nrt * ncol;
  const int xcd = pid % kXcds, local = pid / kXcds;
  const int per = total / kXcds, extra = total % kXcds;
  const int lpid = xcd * per + min(xcd, extra) + local;
  const int gsize = kGroupRows * ncol;
  const int g = lpid / gsize, in = lpid % gsize;
  const int first = g * kGroupRows;
  const int rows = min(nrt - first, kGroupRows);
  rt = first + in % rows;
  col = in / rows;
}

// ---------------------------------------------------------------- NT GEMM ---
// acc = A[row0 .. +BM, 0 .. K) * B[col0 .. +BN, 0 .. K)^T; A and B are bf16,
// row-major along K with row strides lda / ldb; rows >= nrow and columns
// >= ncol read as zero; K % BK == 0.  Wavefront w owns the 64x64 quadrant
// (w >> 1, w & 1): acc[ti*2 + tj] is its 32x32 tile (ti, tj).
struct NtTile {
  const bf16_t* A;
  const bf16_t* B;
  int64_t lda, ldb;
  int64_t row0, nrow;
  int col0, ncol, K;

  __device__ __forceinline__ void load_stage(int k0, uint4 (&ra)[4], uint4 (&rb)[4]) const {
    const int t = threadIdx.x;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = t + 256 * j;  // 16-byte chunk of the 128 x 64 tile
      const int r = c >> 3, kc = (c & 7) * 8;
      ra[j] = (row0 + r < nrow) ? *reinterpret_cast<const uint4*>(A + (row0 + r) * lda + k0 + kc)
                                : make_uint4(0, 0, 0, 0);
      rb[j] = (col0 + r < ncol) ? *reinterpret_cast<const uint4*>(B + (int64_t)(col0 + r) * ldb + k0 + kc)
                                : make_uint4(0, 0, 0, 0);
    }
  }

  __device__ __forceinline__ static void store_stage(bf16_t* lds, const uint4 (&ra)[4], const uint4 (&rb)[4]) {
    const int t = threadIdx.x;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = t + 256 * j;
      const int r = c >> 3, kc = (c & 7) * 8;
      *reinterpret_cast<uint4*>(lds + r * LDK + kc) = ra[j];
      *reinterpret_cast<uint4*>(lds + BM * LDK + r * LDK + kc) = rb[j];
    }
  }

  // Ends with a barrier: on return the LDS operand buffers are free.
  __device__ void run(bf16_t* lds, f32x16 (&acc)[4]) const {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int wr = w >> 1, wc = w & 1;
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[q] = f32x16{};
    uint4 ra[4], rb[4];
    const int nst = K / BK;
    load_stage(0, ra, rb);
    store_stage(lds, ra, rb);
    __syncthreads();
    for (int st = 0; st < nst; ++st) {
      const bf16_t* cur = lds + (st & 1) * kStageElems;
      if (st + 1 < nst) load_stage((st + 1) * BK, ra, rb);
#pragma unroll
      for (int ks = 0; ks < BK / 16; ++ks) {
        bf16x8 a[2], b[2];
#pragma unroll
        for (int ti = 0; ti < 2; ++ti) {
          const int ar = wr * 64 + ti * 32 + (lane & 31);
          a[ti] = *reinterpret_cast<const bf16x8*>(cur + ar * LDK + ks * 16 + (lane >> 5) * 8);
          const int br = wc * 64 + ti * 32 + (lane & 31);
          b[ti] = *reinterpret_cast<const bf16x8*>(cur + BM * LDK + br * LDK + ks * 16 + (lane >> 5) * 8);
        }
#pragma unroll
        for (int ti = 0; ti < 2; ++ti)
#pragma unroll
          for (int tj = 0; tj < 2; ++tj) acc[ti * 2 + tj] = mfma(a[ti], b[tj], acc[ti * 2 + tj]);
      }
      if (st + 1 < nst) store_stage(lds + ((st + 1) & 1) * kStageElems, ra, rb);
      __syncthreads();
    }
  }
};

// The four quadrants' accumulators into the fp32 tile T[BM][LDT].
__device__ __forceinline__ void spill(const f32x16 (&acc)[4], float* T) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wr = w >> 1, wc = w & 1;
#pragma unroll
  for (int ti = 0; ti < 2; ++ti)
#pragma unroll
    for (int tj = 0; tj < 2; ++tj)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int row = wr * 64 + ti * 32 + 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
        const int col = wc * 64 + tj * 32 + (lane & 31);
        T[row * LDT + col] = acc[ti * 2 + tj][i];
      }
}

// --------------------------------------------------------- epilogue helpers ---
__device__ __forceinline__ uint32_t word_of(const uint4& p, int k) {
  return k == 0 ? p.x : k == 1 ? p.y : k == 2 ? p.z : p.w;
}

// Candidate filter of the Gumbel-max draw.  With u from word w (S3) and
// j' = (~w) >> 8 <= 2^24 (1 - u), the variate obeys
// G = -ln(-ln u) <= -ln(1 - u) <= (24 - log2 j') ln 2, so an element whose
// bound x/T + (24 - log2 j') ln 2 stays below the best key so far, thr, less
// a rounding margin, cannot win.  (thr - margin) log2(e) is folded into the
// bound's constant; the margin 2e-3 + 2e-6 |thr| exceeds every rounding
// involved for |x/T| <= |thr| + 100, and an element with x/T < thr - 100
// cannot reach thr because G < 16.7.
__device__ __forceinline__ float bound_offset(float thr) {
  return 24.0f - (thr - (2e-3f + 2e-6f * fabsf(thr))) * kLog2e;
}

__device__ __forceinline__ bool bound_ok(float v, uint32_t w, float c2, float off) {
  return fmaf(v, c2, off) >= __builtin_amdgcn_logf((float)((~w) >> 8));
}

// Reductions over the 16 lanes that share a row (lanes 16g .. 16g+15).
__device__ __forceinline__ void lse_merge(float& mraw, float& mc, float& s, float omraw, float omc, float os) {
  const float nm = fmaxf(mc, omc);
  s = s * __builtin_amdgcn_exp2f(mc - nm) + os * __builtin_amdgcn_exp2f(omc - nm);
  mc = nm;
  mraw = fmaxf(mraw, omraw);
}

__device__ __forceinline__ void best_merge(float& key, int& idx, float okey, int oidx) {
  if (okey > key || (okey == key && oidx < idx)) {
    key = okey;
    idx = oidx;
  }
}

__device__ __forceinline__ void group_lse(float& mraw, float& mc, float& s) {
#pragma unroll
  for (int off = 8; off >= 1; off >>= 1)
    lse_merge(mraw, mc, s, __shfl_xor(mraw, off, kWave), __shfl_xor(mc, off, kWave), __shfl_xor(s, off, kWave));
}

__device__ __forceinline__ void group_best(float& key, int& idx) {
#pragma unroll
  for (int off = 8; off >= 1; off >>= 1) best_merge(key, idx, __shfl_xor(key, off, kWave), __shfl_xor(idx, off, kWave));
}

struct RowState {
  float mraw, mc, s;  // log-sum-exp: raw maximum, its scaled value, sum of exp2(x c2 - mc)
  float key;          // best Gumbel key so far
  int idx;            // its draft index
  float gval;         // target: greedy maximum (raw logit) ...
  int gidx;           // ... and its draft index
  int pad;
};
static_assert(sizeof(RowState) == sizeof(LmPartial), "partial record layout");

// One pass over the column tiles of one slice of one model for rows
// row0 .. row0+127.  TARGET = false: draft logits, keys of family 0 over
// every column.  TARGET = true: target logits, log-sum-exp over every column,
// keys of family 1 and the greedy maximum over the mapped columns, each
// identified by its draft index.
template <bool TARGET>
__device__ void lm_pass(const LmFwdArgs& a, int64_t row0, int slice, bf16_t* lds, float* T, RowState* rs) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int V = TARGET ? a.Vt : a.Vd;
  const int nslice = TARGET ? a.nslice_t : a.nslice_d;
  const int ntiles = (V + BN - 1) / BN;
  const int t_begin = (int)((int64_t)ntiles * slice / nslice);
  const int t_end = (int)((int64_t)ntiles * (slice + 1) / nslice);
  const float inv_t = TARGET ? a.inv_tp : a.inv_tq;
  const float c2 = inv_t * kLog2e;
  const uint32_t fam = TARGET ? 1u : 0u;
  if (threadIdx.x < BM)
    rs[threadIdx.x] = RowState{kNegBig, kNegBig, 0.0f, -INFINITY, 0x7FFFFFFF, -INFINITY, 0x7FFFFFFF, 0};
  const bf16_t* Hs = static_cast<const bf16_t*>(TARGET ? a.Ht : a.Hd);
  const bf16_t* Ws = static_cast<const bf16_t*>(TARGET ? a.Wt : a.Wd);
  NtTile g{Hs, Ws, a.H, a.H, row0, a.R, 0, V, a.H};
  for (int tile = t_begin; tile < t_end; ++tile) {
    g.col0 = tile * BN;
    f32x16 acc[4];
    g.run(lds, acc);
    spill(acc, T);
    __syncthreads();
    // wavefront w: rows w*32 .. +31, four at a time; 16 lanes per row, 8 columns per lane
#pragma unroll 1
    for (int it = 0; it < 8; ++it) {
      const int rl = w * 32 + it * 4 + (lane >> 4);
      const int64_t r = row0 + rl;
      const int c = g.col0 + (lane & 15) * 8;
      float x[8];
      load8(T + rl * LDT + (lane & 15) * 8, x);
      const int nvalid = r < a.R ? min(8, max(0, V - c)) : 0;
#pragma unroll
      for (int k = 0; k < 8; ++k)
        if (k >= nvalid) x[k] = -INFINITY;
      float mraw = kNegBig, mc = kNegBig, s = 0.0f;
      {
        float cm = x[0];
#pragma unroll
        for (int k = 1; k < 8; ++k) cm = fmaxf(cm, x[k]);
        if (cm > mraw) {
          mraw = cm;
          mc = cm * c2;
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) s += __builtin_amdgcn_exp2f(fmaf(x[k], c2, -mc));
      }
      float bkey = -INFINITY, gval = -INFINITY;
      int bidx = 0x7FFFFFFF, gidx = 0x7FFFFFFF;
      if (a.sample) {
        const float off = bound_offset(rs[rl].key);
        if (!TARGET) {
          const uint32_t c0 = (uint32_t)c >> 2;
          const uint4 p0 = philox4x32_10(c0, (uint32_t)r, fam, a.offset, a.k0, a.k1);
          const uint4 p1 = philox4x32_10(c0 + 1, (uint32_t)r, fam, a.offset, a.k0, a.k1);
          uint32_t cand = 0;
#pragma unroll
          for (int k = 0; k < 8; ++k) {
            const bool ok = k < nvalid && bound_ok(x[k], word_of(k < 4 ? p0 : p1, k & 3), c2, off);
            cand |= ok ? (1u << k) : 0u;
          }
          if (__ballot(cand != 0u) != 0ull) {
#pragma unroll
            for (int k = 0; k < 8; ++k) {
              if (cand & (1u << k)) {  // columns increase with k: strict > keeps the smallest index
                const float key = gumbel_key(x[k], inv_t, word_of(k < 4 ? p0 : p1, k & 3));
                if (key > bkey) {
                  bkey = key;
                  bidx = c + k;
                }
              }
            }
          }
        } else {
          // Draft indices of the lane's columns (-1: unmapped).  For an
          // ascending map they are consecutive, v_a .. v_a + m - 1 with
          // m <= 8, and lie in the Philox counters v_a>>2 .. (v_a>>2) + 2;
          // any other index (a map that is not ascending) gets its own call.
          int v[8];
          int va = 0x7FFFFFFF;
#pragma unroll
          for (int k = 0; k < 8; ++k) {
            v[k] = k < nvalid ? (a.inv != nullptr ? a.inv[c + k] : c + k) : -1;
            va = (v[k] >= 0 && v[k] < va) ? v[k] : va;
          }
          const uint32_t gb = va == 0x7FFFFFFF ? 0u : (uint32_t)va >> 2;
          const uint4 p0 = philox4x32_10(gb, (uint32_t)r, fam, a.offset, a.k0, a.k1);
          const uint4 p1 = philox4x32_10(gb + 1, (uint32_t)r, fam, a.offset, a.k0, a.k1);
          const uint4 p2 = philox4x32_10(gb + 2, (uint32_t)r, fam, a.offset, a.k0, a.k1);
          uint32_t wv[8];
          uint32_t cand = 0;
#pragma unroll
          for (int k = 0; k < 8; ++k) {
            wv[k] = 0;
            if (v[k] >= 0) {
              const uint32_t gi = ((uint32_t)v[k] >> 2) - gb;
              const int e = v[k] & 3;
              wv[k] = gi == 0 ? word_of(p0, e)
                    : gi == 1 ? word_of(p1, e)
                    : gi == 2 ? word_of(p2, e)
                              : word_of(philox4x32_10((uint32_t)v[k] >> 2, (uint32_t)r, fam, a.offset, a.k0, a.k1), e);
              best_merge(gval, gidx, x[k], v[k]);
              cand |= bound_ok(x[k], wv[k], c2, off) ? (1u << k) : 0u;
            }
          }
          if (__ballot(cand != 0u) != 0ull) {
#pragma unroll
            for (int k = 0; k < 8; ++k)
              if (cand & (1u << k)) best_merge(bkey, bidx, gumbel_key(x[k], inv_t, wv[k]), v[k]);
          }
        }
      }
      group_lse(mraw, mc, s);
      if (a.sample) {
        group_best(bkey, bidx);
        if (TARGET) group_best(gval, gidx);
      }
      if ((lane & 15) == 0 && r < a.R) {
        RowState st = rs[rl];
        lse_merge(st.mraw, st.mc, st.s, mraw, mc, s);
        if (a.sample) {
          best_merge(st.key, st.idx, bkey, bidx);
          if (TARGET) best_merge(st.gval, st.gidx, gval, gidx);
        }
        rs[rl] = st;
      }
    }
    __syncthreads();  // the tile buffer is the next GEMM's operand buffer
  }
  if (threadIdx.x < BM && row0 + threadIdx.x < a.R) {
    const RowState st = rs[threadIdx.x];
    const int col = TARGET ? slice : a.nslice_t + slice;
    a.part[(row0 + threadIdx.x) * (a.nslice_t + a.nslice_d) + col] =
        LmPartial{st.mraw, st.mc, st.s, st.key, st.idx, st.gval, st.gidx, 0};
  }
}

__global__ __launch_bounds__(256, 2) void k_lm_fwd(LmFwdArgs a) {
  __shared__ __align__(16) unsigned char smem[kLdsBytes];
  __shared__ RowState rs[BM];
  bf16_t* lds = reinterpret_cast<bf16_t*>(smem);
  float* T = reinterpret_cast<float*>(smem);
  const int nrt = (int)((a.R + BM - 1) / BM);
  int rt, col;
  tile_of(blockIdx.x, nrt, a.nslice_t + a.nslice_d, rt, col);
  if (col < a.nslice_t)
    lm_pass<true>(a, (int64_t)rt * BM, col, lds, T, rs);
  else
    lm_pass<false>(a, (int64_t)rt * BM, col - a.nslice_t, lds, T, rs);
}

// Inverse of the draft->target map: inv[t] = v where d2t[v] = t, else -1.
__global__ void k_lm_inv_fill(int32_t* inv, int Vt) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t < Vt) inv[t] = -1;
}

__global__ void k_lm_inv_scatter(const int32_t* d2t, int Vd, int Vt, int32_t* inv, int32_t* err) {
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= Vd) return;
  const int t = d2t[v];
  if ((uint32_t)t >= (uint32_t)Vt) {
    report_error(err, VSD_DEVERR_MAP_RANGE);
    return;
  }
  inv[t] = v;
}

// Dot product of two bf16 rows of length H (H % 8 == 0), one wavefront; the
// result is the same in every lane.
__device__ __forceinline__ float wave_dot(const bf16_t* x, const bf16_t* y, int H, int lane) {
  float acc = 0.0f;
  for (int k = lane * 8; k < H; k += kWave * 8) {
    float xv[8], yv[8];
    load8(x + k, xv);
    load8(y + k, yv);
#pragma unroll
    for (int j = 0; j < 8; ++j) acc = fmaf(xv[j], yv[j], acc);
  }
  return wave_sum(acc);
}

// Merge the slices of both models, write tokens (sampling) and the row
// statistics.  One wavefront per row.
__global__ __launch_bounds__(256) void k_lm_combine(LmCombineArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= a.R) return;
  const int i = (int)(r % a.L);
  int d = a.L;
  if (a.depth != nullptr) {
    d = a.depth[r / a.L];
    if (d < 1 || d > a.L) {
      if (lane == 0) report_error(a.err, VSD_DEVERR_DEPTH_RANGE);
      d = 0;
    }
  }
  const bool sampling = a.tok_in[0] == nullptr;
  if (i >= d) {  // masked slot: tokens -1 (sampling), every statistic 0
    if (lane < 3) {
      a.la[r * 3 + lane] = 0.0f;
      a.lq[r * 3 + lane] = 0.0f;
      if (sampling) a.tok_out[lane][r] = -1;
    }
    if (lane == 0) {
      a.lse_q[r] = 0.0f;
      if (a.lse_p != nullptr) a.lse_p[r] = 0.0f;
    }
    return;
  }
  const int nsl = a.nslice_t + a.nslice_d;
  const LmPartial* pr = a.part + r * nsl;
  // slices in index order, so equal keys resolve to the smaller index as in one pass
  float pmraw = kNegBig, pmc = kNegBig, ps = 0.0f, tkey = -INFINITY, gval = -INFINITY;
  int tidx = 0x7FFFFFFF, gidx = 0x7FFFFFFF;
  for (int sl = 0; sl < a.nslice_t; ++sl) {
    const LmPartial p = pr[sl];
    lse_merge(pmraw, pmc, ps, p.mraw, p.mc, p.s);
    best_merge(tkey, tidx, p.key, p.idx);
    best_merge(gval, gidx, p.gval, p.gidx);
  }
  float qmraw = kNegBig, qmc = kNegBig, qs = 0.0f, dkey = -INFINITY;
  int didx = 0x7FFFFFFF;
  for (int sl = 0; sl < a.nslice_d; ++sl) {
    const LmPartial p = pr[a.nslice_t + sl];
    lse_merge(qmraw, qmc, qs, p.mraw, p.mc, p.s);
    best_merge(dkey, didx, p.key, p.idx);
  }
  const float cq2 = a.inv_tq * kLog2e, cp2 = a.inv_tp * kLog2e;
  const float qt = (log2f(qs) - fmaf(qmraw, cq2, -qmc)) * kLn2;
  const float pt = (log2f(ps) - fmaf(pmraw, cp2, -pmc)) * kLn2;
  int tok[3];
  if (sampling) {
    tok[0] = didx;
    tok[1] = tidx;
    tok[2] = gidx;
  } else {
#pragma unroll
    for (int f = 0; f < 3; ++f) tok[f] = a.tok_in[f][r];
  }
  const bf16_t* hd = static_cast<const bf16_t*>(a.Hd) + r * a.H;
  const bf16_t* ht = static_cast<const bf16_t*>(a.Ht) + r * a.H;
  const bf16_t* Wd = static_cast<const bf16_t*>(a.Wd);
  const bf16_t* Wt = static_cast<const bf16_t*>(a.Wt);
  float lqv[3], lav[3];
#pragma unroll
  for (int f = 0; f < 3; ++f) {
    const int z = tok[f];
    lqv[f] = 0.0f;
    lav[f] = 0.0f;
    if ((uint32_t)z >= (uint32_t)a.Vd) {
      if (lane == 0) report_error(a.err, VSD_DEVERR_TOKEN_RANGE);
      continue;
    }
    const int zt = a.d2t != nullptr ? a.d2t[z] : z;
    if ((uint32_t)zt >= (uint32_t)a.Vt) {
      if (lane == 0) report_error(a.err, VSD_DEVERR_MAP_RANGE);
      continue;
    }
    const float xz = wave_dot(hd, Wd + (int64_t)z * a.H, a.H, lane);
    const float yz = wave_dot(ht, Wt + (int64_t)zt * a.H, a.H, lane);
    lqv[f] = (xz - qmraw) * a.inv_tq - qt;
    lav[f] = fminf(0.0f, (yz - pmraw) * a.inv_tp - pt - lqv[f]);
  }
  if (lane < 3) {
    a.la[r * 3 + lane] = lane == 0 ? lav[0] : lane == 1 ? lav[1] : lav[2];
    a.lq[r * 3 + lane] = lane == 0 ? lqv[0] : lane == 1 ? lqv[1] : lqv[2];
    if (sampling) a.tok_out[lane][r] = lane == 0 ? tok[0] : lane == 1 ? tok[1] : tok[2];
  }
  if (lane == 0) {
    a.lse_q[r] = qmraw * a.inv_tq + qt;
    if (a.lse_p != nullptr) a.lse_p[r] = pmraw * a.inv_tp + pt;
  }
}

// ----------------------------------------------------------- backward pass ---
// g for one 128x128 tile of the recomputed draft logits, written in bf16 to
// G [R, ldg] (columns [0, Vd) only).
__global__ __launch_bounds__(256, 2) void k_lm_bwd_g(LmBwdArgs a) {
  __shared__ __align__(16) unsigned char smem[kLdsBytes];
  bf16_t* lds = reinterpret_cast<bf16_t*>(smem);
  float* T = reinterpret_cast<float*>(smem);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nrt = (int)((a.R + BM - 1) / BM);
  int rt, ct;
  tile_of(blockIdx.x, nrt, (a.Vd + BN - 1) / BN, rt, ct);
  const int64_t row0 = (int64_t)rt * BM;
  const int col0 = ct * BN;
  NtTile g{static_cast<const bf16_t*>(a.Hd), static_cast<const bf16_t*>(a.Wd), a.H, a.H, row0, a.R, col0, a.Vd,
           a.H};
  f32x16 acc[4];
  g.run(lds, acc);
  spill(acc, T);
  __syncthreads();
  const float c2 = a.inv_tq * kLog2e;
  const float k = a.scale * a.inv_tq;
  bf16_t* G = static_cast<bf16_t*>(a.G);
#pragma unroll 1
  for (int it = 0; it < 8; ++it) {
    const int rl = w * 32 + it * 4 + (lane >> 4);
    const int64_t r = row0 + rl;
    const int c = col0 + (lane & 15) * 8;
    const int nvalid = min(8, a.Vd - c);
    if (r >= a.R || nvalid <= 0) continue;
    const float ca = a.coef_a[r], cb = a.coef_b[r];
    float gv[8];
    if (ca == 0.0f && cb == 0.0f) {
#pragma unroll
      for (int j = 0; j < 8; ++j) gv[j] = 0.0f;
    } else {
      float x[8];
      load8(T + rl * LDT + (lane & 15) * 8, x);
      const float lse2 = a.lse_q[r] * kLog2e;
      const float kab = k * (ca + cb), ka = k * ca, kb = k * cb;
      const int zd = a.tok_d[r], zt = a.tok_t[r];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        float t = kab * __builtin_amdgcn_exp2f(fmaf(x[j], c2, -lse2));
        t -= (c + j == zd) ? ka : 0.0f;
        t -= (c + j == zt) ? kb : 0.0f;
        gv[j] = t;
      }
    }
    bf16_t* out = G + r * a.ldg + c;
    if (nvalid == 8) {
      store8(out, gv);
    } else {
      for (int j = 0; j < nvalid; ++j) store1(out + j, gv[j]);
    }
  }
}

// C[M, N] = A[M, K] B[K, N], bf16 operands (row-major, strides lda / ldb),
// fp32 accumulation, bf16 result (stride ldc).  A's tile is staged
// K-contiguous; B's tile is staged as it lies in memory (N-contiguous) and
// each lane gathers its eight K values of one column with 16-bit LDS reads.
// N % 8 == 0; K is arbitrary (the tail reads as zero).
__global__ __launch_bounds__(256, 2) void k_lm_gemm_nn(LmGemmNNArgs a) {
  __shared__ __align__(16) bf16_t lds[2 * kStageElems];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wr = w >> 1, wc = w & 1;
  const int nrt = (int)((a.M + BM - 1) / BM);
  int rt, ct;
  tile_of(blockIdx.x, nrt, (a.N + BN - 1) / BN, rt, ct);
  const int64_t row0 = (int64_t)rt * BM;
  const int n0 = ct * BN;
  const int t = threadIdx.x;
  const bf16_t* A = static_cast<const bf16_t*>(a.A);
  const bf16_t* B = static_cast<const bf16_t*>(a.B);
  f32x16 acc[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) acc[q] = f32x16{};
  const int nst = (a.K + BK - 1) / BK;
  uint4 ra[4], rb[4];
  auto load = [&](int k0) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = t + 256 * j;
      {  // A: row r, K offset kc .. kc+7
        const int r = c >> 3, kc = (c & 7) * 8;
        const int64_t gr = row0 + r;
        const int gk = k0 + kc;
        if (gr < a.M && gk + 8 <= a.K) {
          ra[j] = *reinterpret_cast<const uint4*>(A + gr * a.lda + gk);
        } else {
          uint32_t wv[4] = {0, 0, 0, 0};
          if (gr < a.M)
            for (int e = 0; e < 8; ++e)
              if (gk + e < a.K) wv[e >> 1] |= (uint32_t)A[gr * a.lda + gk + e] << (16 * (e & 1));
          ra[j] = make_uint4(wv[0], wv[1], wv[2], wv[3]);
        }
      }
      {  // B: K row kr, N offset nc .. nc+7
        const int kr = c >> 4, nc = (c & 15) * 8;
        const int gk = k0 + kr, gn = n0 + nc;
        rb[j] = (gk < a.K && gn < a.N) ? *reinterpret_cast<const uint4*>(B + (int64_t)gk * a.ldb + gn)
                                      : make_uint4(0, 0, 0, 0);
      }
    }
  };
  auto store = [&](bf16_t* buf) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = t + 256 * j;
      const int r = c >> 3, kc = (c & 7) * 8;
      *reinterpret_cast<uint4*>(buf + r * LDK + kc) = ra[j];
      const int kr = c >> 4, nc = (c & 15) * 8;
      *reinterpret_cast<uint4*>(buf + BM * LDK + kr * LDN + nc) = rb[j];
    }
  };
  load(0);
  store(lds);
  __syncthreads();
  for (int st = 0; st < nst; ++st) {
    const bf16_t* cur = lds + (st & 1) * kStageElems;
    const bf16_t* curb = cur + BM * LDK;
    if (st + 1 < nst) load((st + 1) * BK);
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8 av[2], bv[2];
#pragma unroll
      for (int ti = 0; ti < 2; ++ti) {
        const int ar = wr * 64 + ti * 32 + (lane & 31);
        av[ti] = *reinterpret_cast<const bf16x8*>(cur + ar * LDK + ks * 16 + (lane >> 5) * 8);
        const int bn = wc * 64 + ti * 32 + (lane & 31);
        const int kb = ks * 16 + (lane >> 5) * 8;
#pragma unroll
        for (int e = 0; e < 8; ++e) bv[ti][e] = __builtin_bit_cast(__bf16, curb[(kb + e) * LDN + bn]);
      }
#pragma unroll
      for (int ti = 0; ti < 2; ++ti)
#pragma unroll
        for (int tj = 0; tj < 2; ++tj) acc[ti * 2 + tj] = mfma(av[ti], bv[tj], acc[ti * 2 + tj]);
    }
    if (st + 1 < nst) store(lds + ((st + 1) & 1) * kStageElems);
    __syncthreads();
  }
  bf16_t* C = static_cast<bf16_t*>(a.C);
#pragma unroll
  for (int ti = 0; ti < 2; ++ti)
#pragma unroll
    for (int tj = 0; tj < 2; ++tj)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int64_t row = row0 + wr * 64 + ti * 32 + 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
        const int col = n0 + wc * 64 + tj * 32 + (lane & 31);
        if (row < a.M && col < a.N) store1(C + row * a.ldc + col, acc[ti * 2 + tj][i]);
      }
}

}  // namespace

hipError_t launch_lm_inv(const int32_t* d2t, int Vd, int Vt, int32_t* inv, int32_t* err, hipStream_t s) {
  hipLaunchKernelGGL(k_lm_inv_fill, dim3((unsigned)((Vt + 255) / 256)), dim3(256), 0, s, inv, Vt);
  hipLaunchKernelGGL(k_lm_inv_scatter, dim3((unsigned)((Vd + 255) / 256)), dim3(256), 0, s, d2t, Vd, Vt, inv, err);
  return hipGetLastError();
}

hipError_t launch_lm_fwd(const LmFwdArgs& a, hipStream_t s) {
  const int64_t nrt = (a.R + BM - 1) / BM;
  hipLaunchKernelGGL(k_lm_fwd, dim3((unsigned)(nrt * (a.nslice_t + a.nslice_d))), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_lm_combine(const LmCombineArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_lm_combine, dim3((unsigned)((a.R + 3) / 4)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_lm_bwd(const LmBwdArgs& a, hipStream_t s) {
  const int64_t nrt = (a.R + BM - 1) / BM;
  hipLaunchKernelGGL(k_lm_bwd_g, dim3((unsigned)(nrt * ((a.Vd + BN - 1) / BN))), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  LmGemmNNArgs gm{a.G, a.Wd, a.dH, a.R, a.ldg, a.H, a.H, a.H, a.Vd};
  hipLaunchKernelGGL(k_lm_gemm_nn, dim3((unsigned)(nrt * ((a.H + BN - 1) / BN))), dim3(256), 0, s, gm);
  return hipGetLastError();
}

}  // namespace vsd
