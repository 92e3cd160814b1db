// Fused LM-head variant: the draft and target logits X = H_d W_d^T and
// Y = H_t W_t^T (bf16 operands, fp32 accumulation on MFMA) are never written
// to memory.
//
// Matrix core tiling.  A workgroup of eight wavefronts (two per SIMD) owns a
// 256x256 output tile; wavefront (wr, wc) computes rows wr*128 .. +127 and
// columns wc*64 .. +63 as 4x2 tiles of v_mfma_f32_32x32x16_bf16.  Operands
// stream through a double-buffered LDS stage of 64 K values per row.  Rows
// that are K-contiguous in memory (hidden states, weights in the forward) are
// staged as they are and read as one 16-byte fragment per lane; a K-major
// operand (the weight in dH = g W_d) is staged N-contiguous and read with the
// gfx950 transpose load (ds_read_b64_tr_b16), two per fragment.
//
// Forward.  One launch covers both models.  A workgroup owns 256 rows and one
// slice of a vocabulary; for every 256-column tile of the slice it computes
// the logit tile and consumes it in place: the online log-sum-exp (row
// softmax normalisers, Sec. "Preliminary"), the Gumbel-max draws with the
// exact candidate filter (Alg. 1 draws z~ ~ q and z' ~ p under the library's
// normative sampler) and the greedy maximum (Alg. 2).  Per-row running state
// stays in LDS across the tiles of the slice; the slice's result goes to a
// partial record.  A combine kernel merges the slices, forms the drawn
// tokens' logits by dot products (H_r . W_z) and writes tokens and the
// per-row statistics (log q, log alpha of Eq. acc).
//
// Backward (derivative of Eq. advance through the LM head).  The draft
// logits are recomputed tile by tile; g = loss_scale/T_q ((a+b) q - a e_z~ -
// b e_z') is written in bf16 (the gradient with respect to the logits); then
// dH_d = g W_d and, when asked for, dW_d = g^T H_d (fp32).
#include "vsd_device.hpp"
#include "vsd_kernels.hpp"
#include "vsd_topk.hpp"

namespace vsd {

namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) short s16x4;
typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
typedef __attribute__((ext_vector_type(16))) float f32x16;

constexpr int TM = 256, TN = 256, TK = 64;   // workgroup tile and K per stage
constexpr int kThreads = 512;                // eight wavefronts
constexpr int LDK = TK + 8;                  // K-contiguous LDS row (bf16): 144 B, conflict-free 16-B reads
constexpr int LDN = TN + 32;                 // N-contiguous LDS row (bf16) of a K-major operand: 576 B
constexpr int LDT = TN + 4;                  // fp32 epilogue row
constexpr int kStageElems = 2 * TM * LDK;    // A and B of one stage (bf16), padded rows
constexpr int kStageNT = 2 * TM * TK;        // A and B of one stage, direct-loaded NT operands
constexpr int kLdsBytes = 2 * kStageElems * 2;
constexpr int kXcds = 8;                     // MI355X: 8 XCDs, workgroups dealt round-robin
constexpr int kGroupRows = 4;                // row tiles per L2 reuse group
static_assert(TM * LDK == TK * LDN, "both operand layouts fill the same stage slot");
static_assert(2 * 64 * LDT * 4 <= kLdsBytes, "two 64-row epilogue buffers fit the operand buffers");
static_assert(kLmTile == TN && kLmTile == TM, "tile width shared with the host");
static_assert(2 * kStageNT * 2 <= kLdsBytes, "two direct-loaded NT stages fit");
constexpr int kLmSegM = 6;                   // KL term: list length of one row segment
static_assert(kLmRedoM >= kMaxTopK, "a recompute record holds every member a slice can have");
static_assert(TM * 4 * kLmRedoM * 8 <= kLdsBytes, "the recompute's segment lists fit");
static_assert(TM * 4 * (32 + kLmSegM * 8 + 4) <= kLdsBytes, "the slice merge's row states and KL lists fit");

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

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) const void global_void;

// ------------------------------------------------------------- GEMM core ---
// acc = A[row0 .. +TM, 0 .. K) * B, accumulated over K in order.  A is bf16
// [*, K] row-major (stride lda), or with TA = true [K, *] row-major (the
// tile takes its columns row0 .. +TM).  NN = false: B is [N, K] row-major
// (stride ldb) and the tile takes rows col0 .. +TN of it; NN = true: B is
// [K, N] row-major and the tile takes columns col0 .. +TN.  K-major operands
// are staged N-contiguous and read with transpose loads.  Rows >= nrow, columns
// >= ncol and K >= K read as zero; NN needs ncol % 8 == 0, NT needs K % 8 ==
// 0 (A's K tail is read element-wise when K % TK != 0).
// Wavefront w = (wr, wc) = (w >> 2, w & 3) accumulates acc[ti*2 + tj] =
// rows wr*128 + ti*32 .. +31, columns wc*64 + tj*32 .. +31.
template <bool NN, bool TA = false>
struct Core {
  const bf16_t* A;
  const bf16_t* B;
  int64_t lda, ldb;
  int64_t row0, nrow;
  int col0, ncol, K;
  // NT only: tile row i reads row arow[i] of A and tile column j row
  // brow[j] of B (null: i and j themselves); a B row index outside
  // [0, brow_n) reads row 0 (its results are the caller's to discard)
  const int32_t* arow = nullptr;
  const int32_t* brow = nullptr;
  int brow_n = 0;

  __device__ __forceinline__ uint4 load_a(int64_t r, int k) const {
    if (r >= nrow) return make_uint4(0, 0, 0, 0);
    const bf16_t* p = A + r * lda + k;
    if (k + 8 <= K) return *reinterpret_cast<const uint4*>(p);
    uint32_t w[4] = {0, 0, 0, 0};
    for (int e = 0; e < 8; ++e)
      if (k + e < K) w[e >> 1] |= (uint32_t)p[e] << (16 * (e & 1));
    return make_uint4(w[0], w[1], w[2], w[3]);
  }

  // 8 consecutive columns m .. m+7 of K row k of a K-major A (zeros past
  // the matrix).
  __device__ __forceinline__ uint4 load_ta(int k, int64_t m) const {
    if (k >= K || m >= nrow) return make_uint4(0, 0, 0, 0);
    const bf16_t* p = A + (int64_t)k * lda + m;
    if (m + 8 <= nrow) return *reinterpret_cast<const uint4*>(p);
    uint32_t w[4] = {0, 0, 0, 0};
    for (int e = 0; e < 8; ++e)
      if (m + e < nrow) w[e >> 1] |= (uint32_t)p[e] << (16 * (e & 1));
    return make_uint4(w[0], w[1], w[2], w[3]);
  }

  __device__ __forceinline__ void load(int k0, uint4 (&ra)[4], uint4 (&rb)[4]) const {
    const int t = threadIdx.x;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = t + kThreads * j;  // 16-byte chunk of the 256 x 64 tile
      const int r = c >> 3, kc = (c & 7) * 8;
      if (TA) {
        const int kr = c >> 5, mc = (c & 31) * 8;  // 64 K rows x 256 columns
        ra[j] = load_ta(k0 + kr, row0 + mc);
      } else {
        ra[j] = load_a(row0 + r, k0 + kc);
      }
      if (!NN) {
        rb[j] = (col0 + r < ncol && k0 + kc < K)
                    ? *reinterpret_cast<const uint4*>(B + (int64_t)(col0 + r) * ldb + k0 + kc)
                    : make_uint4(0, 0, 0, 0);
      } else {
        const int kr = c >> 5, nc = (c & 31) * 8;  // 64 K rows x 256 columns
        rb[j] = (k0 + kr < K && col0 + nc < ncol)
                    ? *reinterpret_cast<const uint4*>(B + (int64_t)(k0 + kr) * ldb + col0 + nc)
                    : make_uint4(0, 0, 0, 0);
      }
    }
  }

  __device__ __forceinline__ static void store(bf16_t* L, const uint4 (&ra)[4], const uint4 (&rb)[4]) {
    const int t = threadIdx.x;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = t + kThreads * j;
      const int r = c >> 3, kc = (c & 7) * 8;
      if (TA)
        *reinterpret_cast<uint4*>(L + (c >> 5) * LDN + (c & 31) * 8) = ra[j];
      else
        *reinterpret_cast<uint4*>(L + r * LDK + kc) = ra[j];
      if (!NN) {
        *reinterpret_cast<uint4*>(L + TM * LDK + r * LDK + kc) = rb[j];
      } else {
        const int kr = c >> 5, nc = (c & 31) * 8;
        *reinterpret_cast<uint4*>(L + TM * LDK + kr * LDN + nc) = rb[j];
      }
    }
  }

  // NT: both operands K-contiguous.  A stage goes from global memory to LDS
  // directly (global_load_lds_dwordx4: lane i's 16 bytes land at the
  // instruction's LDS base + 16 i), 8 rows of 64 K values per instruction;
  // rows are unpadded (128 B) and lane i of a row loads global 16-byte chunk
  // (i ^ row) & 7, so chunk c of row r sits at position c ^ (r & 7).  The
  // LDS serves a 16-byte read to 16 lanes at a time from 64 four-byte banks,
  // so a fragment read of 16 consecutive rows meets each bank twice (rows r
  // and r + 8 coincide).  A swizzle by (r >> 1) & 7 removes that two-way
  // conflict and halves the LDS busy cycles, but left the forward's time
  // unchanged and raised what it fetches from beyond L2 by about 1.7x (the
  // workgroups sharing operand tiles drift further apart), so this one
  // stays.  Rows past
  // nrow / ncol read the last valid row (their results are never used); K is
  // a multiple of TK.  The lane's source addresses at K offset 0 are formed
  // once per tile (row clamp and row stride); a stage only adds k0.
  struct NtSrc {
    const bf16_t* a[4];
    const bf16_t* b[4];
  };
  __device__ __forceinline__ NtSrc nt_src() const {
    const int lane = threadIdx.x & 63, w = wave_id();
    const int lr = lane >> 3, lc = lane & 7;
    NtSrc s;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = w * 32 + j * 8 + lr;
      const int cg = (lc ^ r) & 7;
      int64_t ra = min(row0 + r, nrow - 1);
      int rb = min(col0 + r, ncol - 1);
      if (arow != nullptr) ra = arow[ra];
      if (brow != nullptr) {
        rb = brow[rb];
        rb = (uint32_t)rb < (uint32_t)brow_n ? rb : 0;
      }
      s.a[j] = A + ra * lda + cg * 8;
      s.b[j] = B + (int64_t)rb * ldb + cg * 8;
    }
    return s;
  }
  __device__ __forceinline__ static void issue(const NtSrc& s, int k0, bf16_t* L) {
    const int w = wave_id();
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      __builtin_amdgcn_global_load_lds((const global_void*)(s.a[j] + k0), (lds_void*)(L + (w * 32 + j * 8) * TK),
                                       16, 0, 0);
      __builtin_amdgcn_global_load_lds((const global_void*)(s.b[j] + k0),
                                       (lds_void*)(L + TM * TK + (w * 32 + j * 8) * TK), 16, 0, 0);
    }
  }

  // Fragment of rows r0 .. r0+31 (one per lane & 31) at K offset ks*16 of a
  // direct-loaded NT operand block.
  __device__ __forceinline__ static bf16x8 frag_nt(const bf16_t* L, int r0, int ks, int lane) {
    const int r = r0 + (lane & 31), c = ks * 2 + (lane >> 5);
    return *reinterpret_cast<const bf16x8*>(L + r * TK + (((c ^ r) & 7) << 3));
  }

  // The B fragment of tile column n0 (32 wide) at K offset ks*16.
  __device__ __forceinline__ static bf16x8 frag_b(const bf16_t* L, int n0, int ks, int lane) {
    if (!NN) return frag_nt(L + TM * TK, n0, ks, lane);
    return frag_tr(L + TM * LDK, n0, ks, lane);
  }

  // Fragment of columns n0 .. n0+31 at K offset ks*16 of an N-contiguous
  // (K-major) operand block: lane l gets rows (l / 32) * 8 .. +7 of column
  // n0 + l % 32, which is the layout of the MFMA's B operand and, read as
  // rows of A^T, of its A operand.
  __device__ __forceinline__ static bf16x8 frag_tr(const bf16_t* Lk, int n0, int ks, int lane) {
    // Transpose load: in each 16-lane group, source lane s names row
    // k = base + s/4 and columns 4(s%4) .. +3; lane i of the group then holds
    // rows base .. base+3 of column i.  Group g covers rows (g >> 1)*8 and
    // columns (g & 1)*16 of the 16 x 32 fragment; two loads give 8 rows.
    const int g = lane >> 4, s = lane & 15;
    const bf16_t* p = Lk + (ks * 16 + (g >> 1) * 8 + (s >> 2)) * LDN + n0 + (g & 1) * 16 + 4 * (s & 3);
    typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
    // (whole-vector casts: the two loads feed the MFMA registers directly)
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p));
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p + 4 * LDN));
    return __builtin_shufflevector(__builtin_bit_cast(bf16x4, lo), __builtin_bit_cast(bf16x4, hi), 0, 1, 2, 3, 4,
                                   5, 6, 7);
  }

  __device__ __forceinline__ static void compute(const bf16_t* L, f32x16 (&acc)[8]) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int wr = w >> 2, wc = w & 3;
#pragma unroll
    for (int ks = 0; ks < TK / 16; ++ks) {
      bf16x8 a[4], b[2];
#pragma unroll
      for (int ti = 0; ti < 4; ++ti)
        a[ti] = TA ? frag_tr(L, wr * 128 + ti * 32, ks, lane)
             : NN ? *reinterpret_cast<const bf16x8*>(L + (wr * 128 + ti * 32 + (lane & 31)) * LDK + ks * 16 +
                                                      (lane >> 5) * 8)
                  : frag_nt(L, wr * 128 + ti * 32, ks, lane);
#pragma unroll
      for (int tj = 0; tj < 2; ++tj) b[tj] = frag_b(L, wc * 64 + tj * 32, ks, lane);
#pragma unroll
      for (int ti = 0; ti < 4; ++ti)
#pragma unroll
        for (int tj = 0; tj < 2; ++tj) acc[ti * 2 + tj] = mfma(a[ti], b[tj], acc[ti * 2 + tj]);
    }
  }

  // Ends with a barrier: on return the LDS operand buffers are free.
  __device__ void run(bf16_t* lds, f32x16 (&acc)[8]) const {
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[q] = f32x16{};
    if (!NN) {  // direct loads: the next stage streams into the other buffer during this one
      const int nst = K / TK;
      const NtSrc src = nt_src();
      issue(src, 0, lds);
      __syncthreads();
      for (int st = 0; st < nst; ++st) {
        if (st + 1 < nst) issue(src, (st + 1) * TK, lds + ((st + 1) & 1) * kStageNT);
        compute(lds + (st & 1) * kStageNT, acc);
        __syncthreads();  // waits for the direct loads too
      }
      return;
    }
    uint4 ra[4], rb[4];
    const int nst = (K + TK - 1) / TK;
    load(0, ra, rb);
    store(lds, ra, rb);
    __syncthreads();
    for (int st = 0; st < nst; ++st) {
      if (st + 1 < nst) load((st + 1) * TK, ra, rb);
      compute(lds + (st & 1) * kStageElems, acc);
      if (st + 1 < nst) store(lds + ((st + 1) & 1) * kStageElems, ra, rb);
      __syncthreads();
    }
  }
};

// Round rd of the epilogue: wavefront (wr, wc) writes its accumulator tiles
// ti = 2 rd, 2 rd + 1 into buffer T + wr * 64 * LDT, whose row q is tile row
// wr*128 + rd*64 + q.
template <int RD>
__device__ __forceinline__ void spill(const f32x16 (&acc)[8], float* T) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wr = w >> 2, wc = w & 3;
  float* Tb = T + wr * 64 * LDT;
#pragma unroll
  for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
    for (int tj = 0; tj < 2; ++tj)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int q = t2 * 32 + 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
        Tb[q * LDT + wc * 64 + tj * 32 + (lane & 31)] = acc[(2 * RD + t2) * 2 + tj][i];
      }
}

// Epilogue rows of round rd for wavefront w, iteration it (0..7): 32 lanes
// per row, 8 columns per lane.  Returns the buffer row pointer; rl = tile row.
__device__ __forceinline__ const float* epi_row(const float* T, int rd, int it, int& rl) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int hb = w >> 2;
  const int q = (w & 3) * 16 + it * 2 + (lane >> 5);
  rl = hb * 128 + rd * 64 + q;
  return T + hb * 64 * LDT + q * LDT + (lane & 31) * 8;
}

// --------------------------------------------------------- epilogue helpers ---
__device__ __forceinline__ uint32_t word_of(const uint4& p, int k) {
  return k == 0 ? p.x : k == 1 ? p.y : k == 2 ? p.z : p.w;
}

// Candidate filter of the Gumbel-max draw.  With u from word w and
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

struct RowState {
  float mraw, mc, s;  // log-sum-exp: raw maximum, its scaled value, sum of exp2(x c2 - mc)
  float key;          // best Gumbel key so far
  int idx;            // its draft index
  float gval;         // target: greedy maximum (raw logit) ...
  int gidx;           // ... and its draft index
  int pad;
};
static_assert(sizeof(RowState) == sizeof(LmPartial), "partial record layout");

__device__ __forceinline__ RowState empty_state() {
  return RowState{kNegBig, kNegBig, 0.0f, -INFINITY, 0x7FFFFFFF, -INFINITY, 0x7FFFFFFF, 0};
}

__device__ __forceinline__ void state_merge(RowState& a, const RowState& b) {
  lse_merge(a.mraw, a.mc, a.s, b.mraw, b.mc, b.s);
  best_merge(a.key, a.idx, b.key, b.idx);
  best_merge(a.gval, a.gidx, b.gval, b.gidx);
}

// KL term (Eq. klv): the M best (value, draft index) pairs offered to one row
// segment (M = kLmSegM) or kept by one slice (M = kLmKlM), ordered as the
// top-K orders them (larger value first, equal values by the smaller index);
// n counts the finite values offered, so n > M means some were dropped,
// every one of them at most v[M - 1].  Only finite values take part (a token
// of zero target probability is not a member).
template <int M>
struct KlList {
  float v[M];
  int i[M];
  int n;

  __device__ __forceinline__ void init() {
#pragma unroll
    for (int j = 0; j < M; ++j) {
      v[j] = -INFINITY;
      i[j] = 0x7FFFFFFF;
    }
    n = 0;
  }
  __device__ __forceinline__ static bool beats(float a, int ia, float b, int ib) {
    return a > b || (a == b && ia < ib);
  }
  __device__ __forceinline__ void offer(float x, int idx) {
    if (!(x > -INFINITY)) return;
    ++n;
    if (!beats(x, idx, v[M - 1], i[M - 1])) return;
    v[M - 1] = x;
    i[M - 1] = idx;
#pragma unroll
    for (int j = M - 1; j > 0; --j) {  // one bubble pass keeps the list ordered
      const bool up = beats(v[j], i[j], v[j - 1], i[j - 1]);
      const float tv = v[j];
      const int ti = i[j];
      v[j] = up ? v[j - 1] : tv;
      i[j] = up ? i[j - 1] : ti;
      v[j - 1] = up ? tv : v[j - 1];
      i[j - 1] = up ? ti : i[j - 1];
    }
  }
  // an upper bound of every dropped value (-inf: nothing dropped)
  __device__ __forceinline__ float bound() const { return n > M ? v[M - 1] : -INFINITY; }
};

// Fold eight consecutive columns c .. c+7 of row r (values x; columns past
// the vocabulary hold -inf) into the running state st of one row segment.
// Every lane of a wavefront works on the same columns of a different row, so
// map lookups and Philox group changes are uniform across the wavefront.
// TARGET = false: keys of family 0 over every column.  TARGET = true: keys of
// family 1 and the greedy maximum over the mapped columns, each identified by
// its draft index; the last Philox call (group cg, words cw) is reused, and
// for an ascending map the draft indices increase along the row, so a new
// call is made once per four mapped columns.
template <bool TARGET, bool KL>
__device__ __forceinline__ void fold8(const LmFwdArgs& a, const float (&x)[8], uint32_t r, int c, int nvalid,
                                      float inv_t, float c2, RowState& st, int& cg, uint4& cw, KlList<kLmSegM>& kl) {
  float cm = x[0];
#pragma unroll
  for (int k = 1; k < 8; ++k) cm = fmaxf(cm, x[k]);
  if (cm > st.mraw) {
    const float nmc = cm * c2;
    st.s *= __builtin_amdgcn_exp2f(st.mc - nmc);
    st.mc = nmc;
    st.mraw = cm;
  }
#pragma unroll
  for (int k = 0; k < 8; ++k) st.s += __builtin_amdgcn_exp2f(fmaf(x[k], c2, -st.mc));
  if (TARGET && KL) {  // the mapped columns' logits, for the row's top-K set
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int vk = k < nvalid ? (a.inv == nullptr ? c + k : a.inv[c + k]) : -1;
      if (vk >= 0) kl.offer(x[k], vk);
    }
  }
  if (!a.sample) return;
  const float off = bound_offset(st.key);
  if (!TARGET) {
    const uint32_t c0 = (uint32_t)c >> 2;
    const uint4 p0 = philox4x32_10(c0, r, 0u, a.offset, a.k0, a.k1);
    const uint4 p1 = philox4x32_10(c0 + 1, r, 0u, a.offset, a.k0, a.k1);
    uint32_t cand = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k)
      cand |= (k < nvalid && bound_ok(x[k], word_of(k < 4 ? p0 : p1, k & 3), c2, off)) ? (1u << k) : 0u;
    if (__ballot(cand != 0u) != 0ull) {
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        if (cand & (1u << k)) {  // columns increase along the row: strict > keeps the smallest index
          const float key = gumbel_key(x[k], inv_t, word_of(k < 4 ? p0 : p1, k & 3));
          if (key > st.key) {
            st.key = key;
            st.idx = c + k;
          }
        }
      }
    }
  } else {
    int v[8];
    if (a.inv == nullptr) {
#pragma unroll
      for (int k = 0; k < 8; ++k) v[k] = k < nvalid ? c + k : -1;
    } else if (nvalid == 8) {
      load8(a.inv + c, v);
    } else {
#pragma unroll
      for (int k = 0; k < 8; ++k) v[k] = k < nvalid ? a.inv[c + k] : -1;
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      if (v[k] >= 0) {
        const int grp = v[k] >> 2;
        if (grp != cg) {
          cg = grp;
          cw = philox4x32_10((uint32_t)grp, r, 1u, a.offset, a.k0, a.k1);
        }
        const uint32_t wk = word_of(cw, v[k] & 3);
        best_merge(st.gval, st.gidx, x[k], v[k]);
        if (bound_ok(x[k], wk, c2, off)) best_merge(st.key, st.idx, gumbel_key(x[k], inv_t, wk), v[k]);
      }
    }
  }
}

// One slice of one model for rows row0 .. row0+255.  TARGET = false: draft
// logits; TARGET = true: target logits (log-sum-exp over every column, draws
// and greedy maximum over the mapped ones).  In the epilogue of each tile,
// wavefront w = (seg, hb) = (w >> 1, w & 1) and lane l take tile rows
// hb*128 + rd*64 + l (rounds rd = 0, 1) and columns seg*64 .. +63: each
// thread carries the state of two row segments across the slice's tiles, and
// the four segments of a row are merged once, at the end, through LDS.
template <bool TARGET, bool KL>
__device__ void lm_pass(const LmFwdArgs& a, int64_t row0, int slice, bf16_t* lds, float* T) {
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int hb = w & 1, seg = w >> 1;
  const int V = TARGET ? a.Vt : a.Vd;
  const int nslice = TARGET ? a.nslice_t : a.nslice_d;
  const int ntiles = (V + TN - 1) / TN;
  const int t_begin = (int)((int64_t)ntiles * slice / nslice);
  const int t_end = (int)((int64_t)ntiles * (slice + 1) / nslice);
  const float inv_t = TARGET ? a.inv_tp : a.inv_tq;
  const float c2 = inv_t * kLog2e;
  RowState st[2] = {empty_state(), empty_state()};
  KlList<kLmSegM> kl[2];
  if (TARGET && KL) {
    kl[0].init();
    kl[1].init();
  }
  Core<false> g{static_cast<const bf16_t*>(TARGET ? a.Ht : a.Hd), static_cast<const bf16_t*>(TARGET ? a.Wt : a.Wd),
                a.H, a.H, row0, a.R, 0, V, a.H};
  for (int tile = t_begin; tile < t_end; ++tile) {
    g.col0 = tile * TN;
    f32x16 acc[8];
    g.run(lds, acc);
#pragma unroll
    for (int rd = 0; rd < 2; ++rd) {
      if (rd == 0)
        spill<0>(acc, T);
      else
        spill<1>(acc, T);
      __syncthreads();
      const int64_t r = row0 + hb * 128 + rd * 64 + lane;
      if (r < a.R) {
        const float* src = T + (hb * 64 + lane) * LDT + seg * 64;
        int cg = -1;
        uint4 cw = make_uint4(0, 0, 0, 0);
#pragma unroll 1
        for (int ch = 0; ch < 8; ++ch) {
          const int c = g.col0 + seg * 64 + ch * 8;
          const int nvalid = min(8, V - c);
          if (nvalid <= 0) break;
          float x[8];
          load8(src + ch * 8, x);
          if (nvalid < 8) {
#pragma unroll
            for (int k = 0; k < 8; ++k)
              if (k >= nvalid) x[k] = -INFINITY;
          }
          fold8<TARGET, KL>(a, x, (uint32_t)r, c, nvalid, inv_t, c2, st[rd], cg, cw, kl[rd]);
        }
      }
      __syncthreads();  // the buffers are the next round's (or the next GEMM's)
    }
  }
  RowState* red = reinterpret_cast<RowState*>(T);  // [TM rows][4 segments]
  LmKlEntry* klred = reinterpret_cast<LmKlEntry*>(red + TM * 4);  // [TM rows][4 segments][kLmSegM]
  float* klbnd = reinterpret_cast<float*>(klred + TM * 4 * kLmSegM);  // [TM rows][4 segments]
#pragma unroll
  for (int rd = 0; rd < 2; ++rd) {
    const int q = (hb * 128 + rd * 64 + lane) * 4 + seg;
    red[q] = st[rd];
    if (TARGET && KL) {
#pragma unroll
      for (int j = 0; j < kLmSegM; ++j) klred[q * kLmSegM + j] = LmKlEntry{kl[rd].v[j], kl[rd].i[j]};
      klbnd[q] = kl[rd].bound();
    }
  }
  __syncthreads();
  if (TARGET && KL && threadIdx.x < TM && row0 + threadIdx.x < a.R) {
    // the slice's list: the best kLmKlM of its four segments' lists; its
    // bound covers what the segments dropped and what this merge drops
    KlList<kLmKlM> m;
    m.init();
    float bnd = -INFINITY;
#pragma unroll 1
    for (int sg = 0; sg < 4; ++sg) {
      const int q = threadIdx.x * 4 + sg;
      bnd = fmaxf(bnd, klbnd[q]);
#pragma unroll
      for (int j = 0; j < kLmSegM; ++j) {
        const LmKlEntry e = klred[q * kLmSegM + j];
        m.offer(e.val, e.idx);
      }
    }
    const int64_t row = row0 + threadIdx.x;
#pragma unroll
    for (int j = 0; j < kLmKlM; ++j) a.kl_part[row * a.kl_stride + slice * kLmKlM + j] = LmKlEntry{m.v[j], m.i[j]};
    a.kl_bound[row * a.nslice_t + slice] = fmaxf(bnd, m.bound());
  }
  if (threadIdx.x < TM && row0 + threadIdx.x < a.R) {
    RowState m = red[threadIdx.x * 4];
#pragma unroll
    for (int sg = 1; sg < 4; ++sg) state_merge(m, red[threadIdx.x * 4 + sg]);  // segments in column order
    const int col = TARGET ? slice : a.nslice_t + slice;
    a.part[(row0 + threadIdx.x) * (a.nslice_t + a.nslice_d) + col] =
        LmPartial{m.mraw, m.mc, m.s, m.key, m.idx, m.gval, m.gidx, 0};
  }
}

template <bool KL>
__global__ __launch_bounds__(kThreads, 1) void k_lm_fwd(LmFwdArgs a) {
  __shared__ __align__(16) unsigned char smem[kLdsBytes];
  bf16_t* lds = reinterpret_cast<bf16_t*>(smem);
  float* T = reinterpret_cast<float*>(smem);
  const int nrt = (int)((a.R + TM - 1) / TM);
  int rt, col;
  tile_of(blockIdx.x, nrt, a.nslice_t + a.nslice_d, rt, col);
  if (col < a.nslice_t)
    lm_pass<true, KL>(a, (int64_t)rt * TM, col, lds, T);
  else
    lm_pass<false, false>(a, (int64_t)rt * TM, col - a.nslice_t, lds, T);
}

// Inverse of the draft->target map: inv[t] = v where d2t[v] = t, else -1.
// The map must be injective: a second draft index claiming a target slot
// finds it taken (compare-and-swap against the fill value) and reports
// VSD_DEVERR_MAP_DUPLICATE instead of overwriting it.
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
  if (atomicCAS(inv + t, -1, v) != -1) report_error(err, VSD_DEVERR_MAP_DUPLICATE);
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

// The KL term of row r from its members in tk (after finish()): the draft
// logits at the members by dot products, then the row term (Eq. klv).
__device__ void lm_kl_row(const LmCombineArgs& a, const WaveTopK& tk, int64_t r, int lane) {
  const bf16_t* hd = static_cast<const bf16_t*>(a.Hd) + r * a.H;
  const bf16_t* Wd = static_cast<const bf16_t*>(a.Wd);
  const int n = min(tk.n, a.kl_k);
  float x = -INFINITY;
  for (int k = 0; k < n; ++k) {
    const int v = tk.bi[k];
    const float xk = (uint32_t)v < (uint32_t)a.Vd ? wave_dot(hd, Wd + (int64_t)v * a.H, a.H, lane) : -INFINITY;
    x = lane == k ? xk : x;
  }
  const bool mine = lane < n;
  int v = mine ? tk.bi[lane] : -1;
  v = (uint32_t)v < (uint32_t)a.Vd ? v : -1;
  const float y = mine ? tk.bv[lane] : -INFINITY;
  kl_row_term_xy(mine, v, y, x, a.kl_k, a.inv_tq, a.inv_tp, a.kl_gscale, a.kl_idx + r * a.kl_k,
                 a.kl_grad + r * a.kl_k, a.kl_row + r, lane);
}

// Offer ne (value, draft index) entries to tk, 8 per lane per round
// (non-finite values take no part).
__device__ __forceinline__ void offer_entries(WaveTopK& tk, const LmKlEntry* ent, int ne, int lane) {
  typedef __attribute__((ext_vector_type(8))) int i32x8;  // a register vector, never a private array
  for (int e0 = 0; e0 < ne; e0 += 8 * kWave) {
    float x[8];
    i32x8 ix;
    uint32_t bits = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int e = e0 + lane * 8 + k;
      const LmKlEntry en = e < ne ? ent[e] : LmKlEntry{-INFINITY, 0x7FFFFFFF};
      x[k] = en.val;
      ix[k] = en.idx;
      bits |= en.val > -INFINITY ? (1u << k) : 0u;
    }
    tk.offer8(x, 0, bits, [&](int k) { return ix[k]; }, lane);
  }
}

// Merge the slices of both models, write tokens (sampling) and the row
// statistics.  One wavefront per row.  With the KL term, the slices' lists
// are merged into the row's top-K set: exact unless some slice dropped a
// value reaching the set's K-th value; such a row is appended to kl_list
// and its term is left to k_lm_kl_redo and k_lm_kl_redo_select.
template <bool KL>
__global__ __launch_bounds__(256) void k_lm_combine(LmCombineArgs a) {
  __shared__ float kl_bv[KL ? 4 * kTopKCap : 1];
  __shared__ int kl_bi[KL ? 4 * kTopKCap : 1];
  const int lane = threadIdx.x & 63;
  const int wave = wave_id();
  const int64_t r = (int64_t)blockIdx.x * 4 + wave;
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
    if (KL) {
      if (lane < a.kl_k) {
        a.kl_idx[r * a.kl_k + lane] = -1;
        a.kl_grad[r * a.kl_k + lane] = 0.0f;
      }
      if (lane == 0) {
        a.kl_row[r] = 0.0f;
      }
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
  const float gap = lse_gap(pmraw, pt, a.inv_tp, qmraw, qt, a.inv_tq);
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
    lav[f] = log_alpha_of(xz, yz, a.inv_tq, a.inv_tp, gap);
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
  if (KL) {
    WaveTopK tk;
    tk.init(kl_bv + wave * kTopKCap, kl_bi + wave * kTopKCap, a.kl_k);
    const int ne = a.nslice_t * kLmKlM;
    offer_entries(tk, a.kl_part + r * a.kl_stride, ne, lane);
    tk.finish(lane);
    const float tau = tk.n >= a.kl_k ? tk.bv[a.kl_k - 1] : -INFINITY;
    float bmax = -INFINITY;
    for (int sl = lane; sl < a.nslice_t; sl += kWave) bmax = fmaxf(bmax, a.kl_bound[r * a.nslice_t + sl]);
    bmax = wave_max(bmax);
    // a dropped value at or above the K-th member (or any, with fewer than K
    // members) might belong to the set
    const bool redo = tk.n >= a.kl_k ? bmax >= tau : bmax > -INFINITY;
    if (redo) {
      if (lane == 0) a.kl_list[atomicAdd(a.kl_count, 1)] = (int)r;
    } else {
      lm_kl_row(a, tk, r, lane);
    }
  }
}

__global__ void k_lm_kl_reset(int32_t* count) {
  if (threadIdx.x == 0) *count = 0;
}

// Exact recompute of the rows k_lm_combine<KL> listed.  A workgroup takes
// 256 listed rows (tile row i: H_t row kl_list[row0 + i]) and one of
// kl_nslice slices of the draft vocabulary's 256-column tiles (tile column
// j: draft index v, W_t row d2t[v]).  Operands, K order and matrix-core
// arithmetic are those of the forward's target tiles, so each value equals
// the one the forward formed for (row, d2t[v]).  Each thread keeps the
// kLmRedoM best (value, v) of its row segment (64 columns of every tile),
// which holds every member of the row's top-K that lies there, since K <=
// kLmRedoM; the four segments of a row merge into the slice's record,
// written over the row's (already consumed) slice lists in kl_part.
// Workgroups past the listed rows return at once (the grid is sized for
// every row listed).
__global__ __launch_bounds__(kThreads, 1) void k_lm_kl_redo(LmCombineArgs a) {
  __shared__ __align__(16) unsigned char smem[kLdsBytes];
  // workgroup ids row tile by row tile (slices fastest): the busy ones, the
  // first ceil(n / 256) row tiles, are the lowest ids, which the dispatcher
  // deals round-robin over all the XCDs (a per-XCD regrouping as in the
  // forward would put them all on the first XCDs)
  const int n = *a.kl_count;
  const int rt = (int)(blockIdx.x / (unsigned)a.kl_nslice), sl = (int)(blockIdx.x % (unsigned)a.kl_nslice);
  const int64_t row0 = (int64_t)rt * TM;
  if (row0 >= n) return;
  bf16_t* lds = reinterpret_cast<bf16_t*>(smem);
  float* T = reinterpret_cast<float*>(smem);
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int hb = w & 1, seg = w >> 1;
  const int ntiles = (a.Vd + TN - 1) / TN;
  const int per = (ntiles + a.kl_nslice - 1) / a.kl_nslice;
  const int t_end = min(ntiles, (sl + 1) * per);
  KlList<kLmRedoM> kl[2];
  kl[0].init();
  kl[1].init();
  Core<false> g{static_cast<const bf16_t*>(a.Ht), static_cast<const bf16_t*>(a.Wt), a.H, a.H, row0, n, 0, a.Vd,
                a.H};
  g.arow = a.kl_list;
  g.brow = a.d2t;
  g.brow_n = a.Vt;
  for (int tile = sl * per; tile < t_end; ++tile) {
    g.col0 = tile * TN;
    f32x16 acc[8];
    g.run(lds, acc);
#pragma unroll
    for (int rd = 0; rd < 2; ++rd) {
      if (rd == 0)
        spill<0>(acc, T);
      else
        spill<1>(acc, T);
      __syncthreads();
      if (row0 + hb * 128 + rd * 64 + lane < n) {
        const float* src = T + (hb * 64 + lane) * LDT + seg * 64;
#pragma unroll 1
        for (int ch = 0; ch < 8; ++ch) {
          const int c = g.col0 + seg * 64 + ch * 8;
          if (c >= a.Vd) break;
          float x[8];
          load8(src + ch * 8, x);
#pragma unroll
          for (int k = 0; k < 8; ++k)
            if (c + k < a.Vd) kl[rd].offer(x[k], c + k);
        }
      }
      __syncthreads();  // the buffers are the next round's (or the next GEMM's)
    }
  }
  LmKlEntry* klred = reinterpret_cast<LmKlEntry*>(smem);  // [TM rows][4 segments][kLmRedoM]
#pragma unroll
  for (int rd = 0; rd < 2; ++rd) {
    const int q = (hb * 128 + rd * 64 + lane) * 4 + seg;
#pragma unroll
    for (int j = 0; j < kLmRedoM; ++j) klred[q * kLmRedoM + j] = LmKlEntry{kl[rd].v[j], kl[rd].i[j]};
  }
  __syncthreads();
  if (threadIdx.x < TM && row0 + threadIdx.x < n) {
    KlList<kLmRedoM> m;
    m.init();
#pragma unroll 1
    for (int e = 0; e < 4 * kLmRedoM; ++e) {
      const LmKlEntry en = klred[threadIdx.x * 4 * kLmRedoM + e];
      m.offer(en.val, en.idx);
    }
    const int64_t r = a.kl_list[row0 + threadIdx.x];
    LmKlEntry* rec = a.kl_part + r * a.kl_stride + sl * kLmRedoM;
#pragma unroll
    for (int j = 0; j < kLmRedoM; ++j) rec[j] = LmKlEntry{m.v[j], m.i[j]};
  }
}

// The KL term of each listed row from its slice records: an exact wavefront
// top-K over the records' entries, then the row term.  One wavefront per
// listed row; the grid is sized for every row listed.
__global__ __launch_bounds__(256) void k_lm_kl_redo_select(LmCombineArgs a) {
  __shared__ float kl_bv[4 * kTopKCap];
  __shared__ int kl_bi[4 * kTopKCap];
  const int lane = threadIdx.x & 63;
  const int wave = wave_id();
  const int64_t f = (int64_t)blockIdx.x * 4 + wave;
  if (f >= *a.kl_count) return;
  WaveTopK tk;
  tk.init(kl_bv + wave * kTopKCap, kl_bi + wave * kTopKCap, a.kl_k);
  const int64_t r = a.kl_list[f];
  offer_entries(tk, a.kl_part + r * a.kl_stride, a.kl_nslice * kLmRedoM, lane);
  tk.finish(lane);
  lm_kl_row(a, tk, r, lane);
}

// ----------------------------------------------------------- backward pass ---
// g for one 256x256 tile of the recomputed draft logits, written in bf16 to
// G [R, ldg] (columns [0, Vd) only).
__global__ __launch_bounds__(kThreads, 1) void k_lm_bwd_g(LmBwdArgs a) {
  __shared__ __align__(16) unsigned char smem[kLdsBytes];
  bf16_t* lds = reinterpret_cast<bf16_t*>(smem);
  float* T = reinterpret_cast<float*>(smem);
  const int lane = threadIdx.x & 63;
  const int nrt = (int)((a.R + TM - 1) / TM);
  int rt, ct;
  tile_of(blockIdx.x, nrt, (a.Vd + TN - 1) / TN, rt, ct);
  const int64_t row0 = (int64_t)rt * TM;
  const int col0 = ct * TN;
  Core<false> g{static_cast<const bf16_t*>(a.Hd), static_cast<const bf16_t*>(a.Wd), a.H, a.H, row0, a.R, col0,
                a.Vd, a.H};
  f32x16 acc[8];
  g.run(lds, acc);
  const float c2 = a.inv_tq * kLog2e;
  const float k = a.scale * a.inv_tq;
  bf16_t* G = static_cast<bf16_t*>(a.G);
#pragma unroll
  for (int rd = 0; rd < 2; ++rd) {
    if (rd == 0)
      spill<0>(acc, T);
    else
      spill<1>(acc, T);
    __syncthreads();
#pragma unroll 1
    for (int it = 0; it < 8; ++it) {
      int rl;
      const float* src = epi_row(T, rd, it, rl);
      const int64_t r = row0 + rl;
      const int c = col0 + (lane & 31) * 8;
      const int nvalid = min(8, a.Vd - c);
      if (r >= a.R || nvalid <= 0) continue;
      const float ca = a.coef_a[r], cb = a.coef_b[r];
      float gv[8];
      if (ca == 0.0f && cb == 0.0f) {
#pragma unroll
        for (int j = 0; j < 8; ++j) gv[j] = 0.0f;
      } else {
        float x[8];
        load8(src, x);
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
    __syncthreads();
  }
}

// With the KL term: g at the row's top-K members, recomputed in fp32 with the
// term's sparse gradient added, then rounded once (the entries k_lm_bwd_g
// wrote there are replaced).  One wavefront per row.
__global__ __launch_bounds__(256) void k_lm_kl_fix(LmBwdArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + wave_id();
  if (r >= a.R) return;
  const bf16_t* hd = static_cast<const bf16_t*>(a.Hd) + r * a.H;
  const bf16_t* Wd = static_cast<const bf16_t*>(a.Wd);
  const float ca = a.coef_a[r], cb = a.coef_b[r];
  const float c2 = a.inv_tq * kLog2e;
  const float k = a.scale * a.inv_tq;
  const float kab = k * (ca + cb), ka = k * ca, kb = k * cb;
  const float lse2 = a.lse_q[r] * kLog2e;
  const int zd = a.tok_d[r], zt = a.tok_t[r];
  bf16_t* G = static_cast<bf16_t*>(a.G) + r * a.ldg;
  for (int j = 0; j < a.kl_k; ++j) {
    const int v = a.kl_idx[r * a.kl_k + j];
    if ((uint32_t)v >= (uint32_t)a.Vd) continue;
    float t = 0.0f;
    if (ca != 0.0f || cb != 0.0f) {
      const float x = wave_dot(hd, Wd + (int64_t)v * a.H, a.H, lane);
      t = kab * __builtin_amdgcn_exp2f(fmaf(x, c2, -lse2));
      t -= (v == zd) ? ka : 0.0f;
      t -= (v == zt) ? kb : 0.0f;
    }
    t += a.kl_grad[r * a.kl_k + j];
    if (lane == 0) store1(G + v, t);
  }
}

// dH[R, H] = G[R, Vd] W_d[Vd, H] (bf16 in, fp32 accumulation, bf16 out):
// one 256x256 tile per workgroup, W_d's tiles read through the transpose
// load.
__global__ __launch_bounds__(kThreads, 1) void k_lm_gemm_nn(LmGemmNNArgs a) {
  __shared__ __align__(16) bf16_t lds[2 * kStageElems];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wr = w >> 2, wc = w & 3;
  const int nrt = (int)((a.M + TM - 1) / TM);
  int rt, ct;
  tile_of(blockIdx.x, nrt, (a.N + TN - 1) / TN, rt, ct);
  const int64_t row0 = (int64_t)rt * TM;
  const int n0 = ct * TN;
  Core<true> g{static_cast<const bf16_t*>(a.A), static_cast<const bf16_t*>(a.B), a.lda, a.ldb, row0, a.M, n0, a.N,
               a.K};
  f32x16 acc[8];
  g.run(lds, acc);
  bf16_t* C = static_cast<bf16_t*>(a.C);
#pragma unroll
  for (int ti = 0; ti < 4; ++ti)
#pragma unroll
    for (int tj = 0; tj < 2; ++tj)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int64_t row = row0 + wr * 128 + ti * 32 + 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
        const int col = n0 + wc * 64 + tj * 32 + (lane & 31);
        if (row < a.M && col < a.N) store1(C + row * a.ldc + col, acc[ti * 2 + tj][i]);
      }
}

// dW = A^T B (fp32): A = g [R, ldg] (K = R rows, M = V_d columns), B = H_d
// [R, H]; both K-major, staged N-contiguous and read with transpose loads.
__global__ __launch_bounds__(kThreads, 1) void k_lm_gemm_tn(LmGemmTNArgs a) {
  __shared__ __align__(16) bf16_t lds[2 * kStageElems];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wr = w >> 2, wc = w & 3;
  const int nrt = (int)((a.M + TM - 1) / TM);
  int rt, ct;
  tile_of(blockIdx.x, nrt, (a.N + TN - 1) / TN, rt, ct);
  const int64_t row0 = (int64_t)rt * TM;
  const int n0 = ct * TN;
  Core<true, true> g{static_cast<const bf16_t*>(a.A), static_cast<const bf16_t*>(a.B), a.lda, a.ldb, row0, a.M, n0,
                     a.N, a.K};
  f32x16 acc[8];
  g.run(lds, acc);
#pragma unroll
  for (int ti = 0; ti < 4; ++ti)
#pragma unroll
    for (int tj = 0; tj < 2; ++tj)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int64_t row = row0 + wr * 128 + ti * 32 + 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
        const int col = n0 + wc * 64 + tj * 32 + (lane & 31);
        if (row < a.M && col < a.N) a.C[row * a.ldc + col] = acc[ti * 2 + tj][i];
      }
}

}  // namespace

hipError_t launch_lm_inv(const int32_t* d2t, int Vd, int Vt, int32_t* inv, int32_t* err, hipStream_t s) {
  hipLaunchKernelGGL(k_lm_inv_fill, dim3((unsigned)((Vt + 255) / 256)), dim3(256), 0, s, inv, Vt);
  hipLaunchKernelGGL(k_lm_inv_scatter, dim3((unsigned)((Vd + 255) / 256)), dim3(256), 0, s, d2t, Vd, Vt, inv, err);
  return hipGetLastError();
}

hipError_t launch_lm_fwd(const LmFwdArgs& a, hipStream_t s) {
  const int64_t nrt = (a.R + TM - 1) / TM;
  const dim3 grid((unsigned)(nrt * (a.nslice_t + a.nslice_d)));
  if (a.kl_part != nullptr)
    hipLaunchKernelGGL(k_lm_fwd<true>, grid, dim3(kThreads), 0, s, a);
  else
    hipLaunchKernelGGL(k_lm_fwd<false>, grid, dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_lm_combine(const LmCombineArgs& a, hipStream_t s) {
  const dim3 grid((unsigned)((a.R + 3) / 4));
  if (a.kl_k > 0)
    hipLaunchKernelGGL(k_lm_combine<true>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(k_lm_combine<false>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_lm_kl_reset(const LmCombineArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_lm_kl_reset, dim3(1), dim3(64), 0, s, a.kl_count);
  return hipGetLastError();
}

hipError_t launch_lm_kl_redo(const LmCombineArgs& a, hipStream_t s) {
  const unsigned nrt = (unsigned)((a.R + TM - 1) / TM);
  hipLaunchKernelGGL(k_lm_kl_redo, dim3(nrt * (unsigned)a.kl_nslice), dim3(kThreads), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_lm_kl_redo_select, dim3((unsigned)((a.R + 3) / 4)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_lm_bwd(const LmBwdArgs& a, hipStream_t s) {
  const int64_t nrt = (a.R + TM - 1) / TM;
  hipLaunchKernelGGL(k_lm_bwd_g, dim3((unsigned)(nrt * ((a.Vd + TN - 1) / TN))), dim3(kThreads), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.kl_idx != nullptr) {
    hipLaunchKernelGGL(k_lm_kl_fix, dim3((unsigned)((a.R + 3) / 4)), dim3(256), 0, s, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  LmGemmNNArgs gm{a.G, a.Wd, a.dH, a.R, a.ldg, a.H, a.H, a.H, a.Vd};
  hipLaunchKernelGGL(k_lm_gemm_nn, dim3((unsigned)(nrt * ((a.H + TN - 1) / TN))), dim3(kThreads), 0, s, gm);
  e = hipGetLastError();
  if (e != hipSuccess || a.dW == nullptr) return e;
  LmGemmTNArgs tn{a.G, a.Hd, a.dW, a.Vd, a.ldg, a.H, a.H, a.H, (int32_t)a.R};
  const int64_t nvt = (a.Vd + TM - 1) / TM;
  hipLaunchKernelGGL(k_lm_gemm_tn, dim3((unsigned)(nvt * ((a.H + TN - 1) / TN))), dim3(kThreads), 0, s, tn);
  return hipGetLastError();
}

}  // namespace vsd
