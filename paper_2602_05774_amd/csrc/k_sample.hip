// E-step sampling (Alg. 1 proposal z~ ~ q and correction z' ~ p; Alg. 2
// greedy reference z-bar), one wavefront per row.
//
// Each lane walks its 8-element chunks of the row (128-bit loads), forms the
// normative Gumbel keys of both families and the raw greedy value, and keeps
// its running (value, index) maximum; lanes visit indices in increasing order
// so a strict '>' keeps the smallest index among equal values.  A butterfly
// reduction with the same tie rule yields the row's tokens, which therefore do
// not depend on the launch geometry.
#include "vsd_device.hpp"
#include "vsd_kernels.hpp"

namespace vsd {

namespace {

constexpr int kRowsPerBlock = 4;  // 256 threads = 4 wavefronts = 4 rows

template <typename T, bool MAPPED>
__global__ __launch_bounds__(256) void k_sample(SampleArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t r = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  if (r >= a.R) return;
  const int i = (int)(r % a.L);
  const int64_t path = r / a.L;  // (b*T + t)*N + s
  int d = a.L;
  if (a.depth != nullptr) {
    d = a.depth[path];
    if (d < 1 || d > a.L) {
      if (lane == 0) report_error(a.err, VSD_DEVERR_DEPTH_RANGE);
      d = 0;
    }
  }
  if (i >= d) {
    if (lane == 0) {
      a.tok_d[r] = -1;
      a.tok_t[r] = -1;
      a.tok_g[r] = -1;
    }
    return;
  }
  const T* X = static_cast<const T*>(a.X) + r * a.ld_d;
  const T* Y = static_cast<const T*>(a.Y) + r * a.ld_t;
  const uint32_t row = (uint32_t)r;

  float best_d = -INFINITY, best_t = -INFINITY, best_g = -INFINITY;
  int arg_d = 0x7FFFFFFF, arg_t = 0x7FFFFFFF, arg_g = 0x7FFFFFFF;
  bool map_bad = false;

  for (int base = lane * 8; base < a.Vd; base += 8 * kWave) {
    float x[8], y[8];
    uint32_t wd[8], wt[8];
    const bool full = base + 8 <= a.Vd;
    if (full) {
      load8(X + base, x);
      if (MAPPED) {
        int32_t t[8];
        load8(a.d2t + base, t);
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          if ((uint32_t)t[k] >= (uint32_t)a.Vt) {
            map_bad = true;
            y[k] = -INFINITY;
          } else {
            y[k] = load1(Y + t[k]);
          }
        }
      } else {
        load8(Y + base, y);
      }
      const uint32_t c0 = (uint32_t)base >> 2;
      const uint4 d0 = philox4x32_10(c0, row, 0u, a.offset, a.k0, a.k1);
      const uint4 d1 = philox4x32_10(c0 + 1, row, 0u, a.offset, a.k0, a.k1);
      const uint4 t0 = philox4x32_10(c0, row, 1u, a.offset, a.k0, a.k1);
      const uint4 t1 = philox4x32_10(c0 + 1, row, 1u, a.offset, a.k0, a.k1);
      wd[0] = d0.x; wd[1] = d0.y; wd[2] = d0.z; wd[3] = d0.w;
      wd[4] = d1.x; wd[5] = d1.y; wd[6] = d1.z; wd[7] = d1.w;
      wt[0] = t0.x; wt[1] = t0.y; wt[2] = t0.z; wt[3] = t0.w;
      wt[4] = t1.x; wt[5] = t1.y; wt[6] = t1.z; wt[7] = t1.w;
    } else {
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int v = base + k;
        x[k] = -INFINITY;
        y[k] = -INFINITY;
        wd[k] = wt[k] = 0u;
        if (v < a.Vd) {
          x[k] = load1(X + v);
          int32_t tv = v;
          if (MAPPED) tv = a.d2t[v];
          if ((uint32_t)tv >= (uint32_t)a.Vt) {
            map_bad = true;
          } else {
            y[k] = load1(Y + tv);
          }
          const uint4 pd = philox4x32_10((uint32_t)v >> 2, row, 0u, a.offset, a.k0, a.k1);
          const uint4 pt = philox4x32_10((uint32_t)v >> 2, row, 1u, a.offset, a.k0, a.k1);
          const int w = v & 3;
          wd[k] = w == 0 ? pd.x : w == 1 ? pd.y : w == 2 ? pd.z : pd.w;
          wt[k] = w == 0 ? pt.x : w == 1 ? pt.y : w == 2 ? pt.z : pt.w;
        }
      }
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int v = base + k;
      if (!full && v >= a.Vd) continue;
      const float kd = gumbel_key(x[k], a.inv_tq, wd[k]);
      if (kd > best_d) {
        best_d = kd;
        arg_d = v;
      }
      const float kt = gumbel_key(y[k], a.inv_tp, wt[k]);
      if (kt > best_t) {
        best_t = kt;
        arg_t = v;
      }
      if (y[k] > best_g) {
        best_g = y[k];
        arg_g = v;
      }
    }
  }
  if (map_bad) report_error(a.err, VSD_DEVERR_MAP_RANGE);
  wave_argmax(best_d, arg_d);
  wave_argmax(best_t, arg_t);
  wave_argmax(best_g, arg_g);
  if (lane == 0) {
    a.tok_d[r] = arg_d;
    a.tok_t[r] = arg_t;
    a.tok_g[r] = arg_g;
  }
}

template <typename T>
hipError_t launch_t(const SampleArgs& a, hipStream_t s) {
  const dim3 grid((unsigned)((a.R + kRowsPerBlock - 1) / kRowsPerBlock));
  if (a.d2t != nullptr)
    hipLaunchKernelGGL((k_sample<T, true>), grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((k_sample<T, false>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_sample(const SampleArgs& a, bool bf16, hipStream_t s) {
  return bf16 ? launch_t<bf16_t>(a, s) : launch_t<float>(a, s);
}

}  // namespace vsd
