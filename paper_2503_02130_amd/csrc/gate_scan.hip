// Gate prelude and the reverse scan of the backward.
//
//  * gate prefix: log f_t = log sigmoid(x_t), c_i = sum_{l<=i} log f_l (Sec. 3,
//    "Hardware-aware implementation"): the log sigmoid elementwise over the
//    whole part, then the scan in place, one workgroup per (batch, head) row;
//    rows of one segment (see below), or rows that do not start 16-byte
//    aligned, take one pass per row that does both.
//  * reverse scan: d(log f)_l = sum_{i>=l} (dc^q_i + dc^k_i), the chain rule
//    through c = cumsum(log f) applied to Alg. 2's dc = dc^q + dc^k, optionally
//    carried on through the gate f = sigmoid(x) (Sec. 3) in the same pass:
//    d x_l = d(log f)_l * sigmoid(-x_l).
//
// Each workgroup walks its row in segments of 8192 elements: every thread scans
// eight consecutive elements sequentially, the 1024 thread totals are scanned
// across the wave with shuffles and across the sixteen waves through LDS, and a
// running carry links the segments.  The per-thread and per-wave steps form a
// short tree, which keeps the fp32 rounding of long rows small.
#include <algorithm>
#include <cstdint>
#include <initializer_list>

#include "fox_device.h"
#include "fox_internal.h"

namespace fox {

constexpr int kScanThreads = 1024;
constexpr int kScanPerThread = 8;
constexpr int kScanSegment = kScanThreads * kScanPerThread;

// MODE 0: x = log sigmoid(a) (forward order, also stores x to aux if non-null);
//         out = the inclusive scan.
// MODE 1: x = a + b, scanned from the end of the row (reverse order); out = scan.
// MODE 2: as MODE 1, aux (if non-null) = scan, out = scan * sigmoid(-g).
// MODE 3: x = a (forward order); out = the inclusive scan.  a may be out: every
//         element is read before the barrier that precedes any store of its
//         segment, so the scan can run in place.
// VEC: every row starts 16-byte aligned (L % 4 == 0 and aligned arrays); a
// thread's eight consecutive elements then move as two 16-byte accesses per
// array instead of eight 4-byte ones (the strided 4-byte pattern touches sixteen
// cache lines per wave instruction).  The values and their order are the same.
template <int MODE, bool VEC>
__global__ __launch_bounds__(kScanThreads) void scan_rows_kernel(const float* a,
                                                                 const float* __restrict__ b,
                                                                 const float* __restrict__ g,
                                                                 float* __restrict__ aux,
                                                                 float* out, int L) {
  constexpr bool FWD = MODE == 0 || MODE == 3;  // scanned from the start of the row
  static_assert(kScanPerThread == 8, "two 16-byte accesses per thread and array");
  const size_t base = (size_t)blockIdx.x * (size_t)L;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  __shared__ float wave_total[kScanThreads / 64];
  // memory position of the thread's element e (scan order) in its row
  auto pos = [&](int p) { return (size_t)(FWD ? p : L - 1 - p); };
  float carry = 0.0f;
  for (int seg = 0; seg < L; seg += kScanSegment) {
    const int p0 = seg + threadIdx.x * kScanPerThread;
    // whole and aligned: the eight elements are memory positions i0 .. i0 + 7
    // (scan order e at i0 + e from the start of the row, at i0 + 7 - e from its end)
    const bool whole = VEC && p0 + kScanPerThread <= L;
    const size_t i0 = base + (FWD ? (size_t)p0 : (size_t)(L - kScanPerThread - p0));
    auto at = [&](int e) { return FWD ? e : kScanPerThread - 1 - e; };
    float x[kScanPerThread];
    if (whole) {
      const f32x4 a0 = *reinterpret_cast<const f32x4*>(a + i0);
      const f32x4 a1 = *reinterpret_cast<const f32x4*>(a + i0 + 4);
      const float av[8] = {a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
      if constexpr (MODE == 0) {
#pragma unroll
        for (int e = 0; e < kScanPerThread; ++e) x[e] = log_sigmoid(av[e]);
        if (aux) {
          *reinterpret_cast<f32x4*>(aux + i0) = f32x4{x[0], x[1], x[2], x[3]};
          *reinterpret_cast<f32x4*>(aux + i0 + 4) = f32x4{x[4], x[5], x[6], x[7]};
        }
      } else if constexpr (MODE == 3) {
#pragma unroll
        for (int e = 0; e < kScanPerThread; ++e) x[e] = av[e];
      } else {
        const f32x4 b0 = *reinterpret_cast<const f32x4*>(b + i0);
        const f32x4 b1 = *reinterpret_cast<const f32x4*>(b + i0 + 4);
        const float bv[8] = {b0[0], b0[1], b0[2], b0[3], b1[0], b1[1], b1[2], b1[3]};
#pragma unroll
        for (int e = 0; e < kScanPerThread; ++e) x[e] = av[at(e)] + bv[at(e)];
      }
    } else {
#pragma unroll
      for (int e = 0; e < kScanPerThread; ++e) {
        const int p = p0 + e;
        x[e] = 0.0f;
        if (p < L) {
          const size_t idx = base + pos(p);
          if (MODE == 0) {
            x[e] = log_sigmoid(a[idx]);
            if (aux) aux[idx] = x[e];
          } else if (MODE == 3) {
            x[e] = a[idx];
          } else {
            x[e] = a[idx] + b[idx];
          }
        }
      }
    }
    float run = 0.0f;
    float incl_local[kScanPerThread];
#pragma unroll
    for (int e = 0; e < kScanPerThread; ++e) {
      run += x[e];
      incl_local[e] = run;
    }
    float incl = run;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const float y = __shfl_up(incl, off);
      if (lane >= off) incl += y;
    }
    if (lane == 63) wave_total[wave] = incl;
    __syncthreads();
    float before = 0.0f, total = 0.0f;
#pragma unroll
    for (int w = 0; w < kScanThreads / 64; ++w) {
      if (w < wave) before += wave_total[w];
      total += wave_total[w];
    }
    const float excl = carry + (before + (incl - run));
    float y[kScanPerThread];
#pragma unroll
    for (int e = 0; e < kScanPerThread; ++e) y[e] = excl + incl_local[e];
    if (whole) {
      float ym[8];  // memory order
#pragma unroll
      for (int e = 0; e < kScanPerThread; ++e) ym[at(e)] = y[e];
      if constexpr (MODE == 2) {
        if (aux) {
          *reinterpret_cast<f32x4*>(aux + i0) = f32x4{ym[0], ym[1], ym[2], ym[3]};
          *reinterpret_cast<f32x4*>(aux + i0 + 4) = f32x4{ym[4], ym[5], ym[6], ym[7]};
        }
        const f32x4 g0 = *reinterpret_cast<const f32x4*>(g + i0);
        const f32x4 g1 = *reinterpret_cast<const f32x4*>(g + i0 + 4);
        const float gv[8] = {g0[0], g0[1], g0[2], g0[3], g1[0], g1[1], g1[2], g1[3]};
#pragma unroll
        for (int m = 0; m < kScanPerThread; ++m) ym[m] = ym[m] / (1.0f + expf(gv[m]));
      }
      *reinterpret_cast<f32x4*>(out + i0) = f32x4{ym[0], ym[1], ym[2], ym[3]};
      *reinterpret_cast<f32x4*>(out + i0 + 4) = f32x4{ym[4], ym[5], ym[6], ym[7]};
    } else {
#pragma unroll
      for (int e = 0; e < kScanPerThread; ++e) {
        const int p = p0 + e;
        if (p < L) {
          const size_t idx = base + pos(p);
          if (MODE == 2) {
            if (aux) aux[idx] = y[e];
            out[idx] = y[e] / (1.0f + expf(g[idx]));  // d log sigmoid(x) / dx = sigmoid(-x)
          } else {
            out[idx] = y[e];
          }
        }
      }
    }
    carry += total;
    __syncthreads();
  }
}

// rows start 16-byte aligned: L a multiple of 4 and every array aligned
static bool rows_aligned(int L, std::initializer_list<const void*> ps) {
  if (L % 4) return false;
  for (const void* p : ps)
    if (p && (reinterpret_cast<uintptr_t>(p) & 15u)) return false;
  return true;
}

// log f = log sigmoid(x) over all rows at once (16-byte accesses; the arrays
// are aligned and n a multiple of 4), into log_f if requested and into c, where
// the scan then runs in place: for long rows the transcendental work spreads
// over the whole part instead of one workgroup per row.  The values are those the scan kernel
// forms itself in MODE 0.
__global__ __launch_bounds__(256) void log_sigmoid_kernel(const float* __restrict__ x,
                                                          float* __restrict__ log_f,
                                                          float* __restrict__ c, size_t n4) {
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (size_t)gridDim.x * 256) {
    const f32x4 v = reinterpret_cast<const f32x4*>(x)[i];
    const f32x4 y = {log_sigmoid(v[0]), log_sigmoid(v[1]), log_sigmoid(v[2]), log_sigmoid(v[3])};
    if (log_f) reinterpret_cast<f32x4*>(log_f)[i] = y;
    reinterpret_cast<f32x4*>(c)[i] = y;
  }
}

hipError_t launch_gate_prefix(const float* logit, float* log_f, float* c, int rows, int L,
                              hipStream_t s) {
  const bool aligned = rows_aligned(L, {logit, log_f, c});
  if (aligned && L > kScanSegment) {
    const size_t n4 = (size_t)rows * (size_t)L / 4;
    const unsigned blocks = (unsigned)std::min<size_t>((n4 + 255) / 256, 4096);
    hipLaunchKernelGGL(log_sigmoid_kernel, dim3(blocks), dim3(256), 0, s, logit, log_f, c, n4);
    hipLaunchKernelGGL((scan_rows_kernel<3, true>), dim3(rows), dim3(kScanThreads), 0, s, c,
                       nullptr, nullptr, nullptr, c, L);
    return hipGetLastError();
  }
  // rows of one segment: one pass per row is faster than two launches
  if (aligned)
    hipLaunchKernelGGL((scan_rows_kernel<0, true>), dim3(rows), dim3(kScanThreads), 0, s, logit,
                       nullptr, nullptr, log_f, c, L);
  else
    hipLaunchKernelGGL((scan_rows_kernel<0, false>), dim3(rows), dim3(kScanThreads), 0, s, logit,
                       nullptr, nullptr, log_f, c, L);
  return hipGetLastError();
}

hipError_t launch_reverse_scan_sum(const float* a, const float* b, float* out, int rows, int L,
                                   hipStream_t s) {
  if (rows_aligned(L, {a, b, out}))
    hipLaunchKernelGGL((scan_rows_kernel<1, true>), dim3(rows), dim3(kScanThreads), 0, s, a, b,
                       nullptr, nullptr, out, L);
  else
    hipLaunchKernelGGL((scan_rows_kernel<1, false>), dim3(rows), dim3(kScanThreads), 0, s, a, b,
                       nullptr, nullptr, out, L);
  return hipGetLastError();
}

hipError_t launch_reverse_scan_gate(const float* a, const float* b, const float* logit,
                                    float* d_log_f, float* d_logit, int rows, int L,
                                    hipStream_t s) {
  if (rows_aligned(L, {a, b, logit, d_log_f, d_logit}))
    hipLaunchKernelGGL((scan_rows_kernel<2, true>), dim3(rows), dim3(kScanThreads), 0, s, a, b,
                       logit, d_log_f, d_logit, L);
  else
    hipLaunchKernelGGL((scan_rows_kernel<2, false>), dim3(rows), dim3(kScanThreads), 0, s, a, b,
                       logit, d_log_f, d_logit, L);
  return hipGetLastError();
}

}  // namespace fox
