// Gate prelude and the reverse scan of the backward.
//
//  * gate prefix: log f_t = log sigmoid(x_t), c_i = sum_{l<=i} log f_l, one
//    workgroup per (batch, head) row (Sec. 3, "Hardware-aware implementation").
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
template <int MODE>
__global__ __launch_bounds__(kScanThreads) void scan_rows_kernel(const float* __restrict__ a,
                                                                 const float* __restrict__ b,
                                                                 const float* __restrict__ g,
                                                                 float* __restrict__ aux,
                                                                 float* __restrict__ out, int L) {
  const size_t base = (size_t)blockIdx.x * (size_t)L;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  __shared__ float wave_total[kScanThreads / 64];
  float carry = 0.0f;
  for (int seg = 0; seg < L; seg += kScanSegment) {
    float run = 0.0f;
    float incl_local[kScanPerThread];
#pragma unroll
    for (int e = 0; e < kScanPerThread; ++e) {
      const int p = seg + threadIdx.x * kScanPerThread + e;
      float x = 0.0f;
      if (p < L) {
        const size_t idx = base + (size_t)(MODE == 0 ? p : L - 1 - p);
        if (MODE == 0) {
          x = log_sigmoid(a[idx]);
          if (aux) aux[idx] = x;
        } else {
          x = a[idx] + b[idx];
        }
      }
      run += x;
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
#pragma unroll
    for (int e = 0; e < kScanPerThread; ++e) {
      const int p = seg + threadIdx.x * kScanPerThread + e;
      if (p < L) {
        const size_t idx = base + (size_t)(MODE == 0 ? p : L - 1 - p);
        const float y = excl + incl_local[e];
        if (MODE == 2) {
          if (aux) aux[idx] = y;
          out[idx] = y / (1.0f + expf(g[idx]));  // d log sigmoid(x) / dx = sigmoid(-x)
        } else {
          out[idx] = y;
        }
      }
    }
    carry += total;
    __syncthreads();
  }
}

hipError_t launch_gate_prefix(const float* logit, float* log_f, float* c, int rows, int L,
                              hipStream_t s) {
  hipLaunchKernelGGL(scan_rows_kernel<0>, dim3(rows), dim3(kScanThreads), 0, s, logit, nullptr,
                     nullptr, log_f, c, L);
  return hipGetLastError();
}

hipError_t launch_reverse_scan_sum(const float* a, const float* b, float* out, int rows, int L,
                                   hipStream_t s) {
  hipLaunchKernelGGL(scan_rows_kernel<1>, dim3(rows), dim3(kScanThreads), 0, s, a, b, nullptr,
                     nullptr, out, L);
  return hipGetLastError();
}

hipError_t launch_reverse_scan_gate(const float* a, const float* b, const float* logit,
                                    float* d_log_f, float* d_logit, int rows, int L,
                                    hipStream_t s) {
  hipLaunchKernelGGL(scan_rows_kernel<2>, dim3(rows), dim3(kScanThreads), 0, s, a, b, logit,
                     d_log_f, d_logit, L);
  return hipGetLastError();
}

}  // namespace fox
