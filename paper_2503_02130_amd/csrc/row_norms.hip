// Largest row norm per (batch, head): max_t ||x_t||_2 for x [BH, L, d].  The
// gate-aware skipping entry points bound every score s q.k by
// s ||q|| ||k||, and this kernel gives them ||k||'s maximum (or ||q||'s).
//
// A workgroup takes a chunk of rows; a group of d / 8 lanes (bf16) or d / 4
// lanes (fp32) reads one row with 16-byte loads (eight rows' loads are issued
// before their sums), the row sums are DPP butterflies, the groups reduce to
// the chunk's maximum in LDS, and the chunk maxima meet in an atomic maximum on
// the float's bit pattern (non-negative floats order like their bits).  The
// result is enlarged by 2^-10 relative so that it bounds the exact norm
// despite the fp32 rounding of the sum of squares.
#include "fox_device.h"
#include "fox_internal.h"

namespace fox {

constexpr int kNormThreads = 256;
constexpr int kNormChunk = 1024;  // rows per workgroup (one atomic per chunk and head)
constexpr int kNormAhead = 8;     // rows per lane group whose loads are in flight together

__global__ void zero_kernel(float* __restrict__ out, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) out[i] = 0.0f;
}

template <typename Tt, int D>
__global__ __launch_bounds__(kNormThreads) void row_norm_max_kernel(const Tt* __restrict__ x,
                                                                    float* __restrict__ out,
                                                                    int L, int n_chunk) {
  constexpr int VEC = 16 / (int)sizeof(Tt);
  constexpr int LPR = D / VEC;                 // lanes per row
  constexpr int RPI = kNormThreads / LPR;      // rows per pass
  const int bh = blockIdx.x / n_chunk, chunk = blockIdx.x % n_chunk;
  const int tid = threadIdx.x, g = tid / LPR, lp = tid % LPR;
  const int r0 = chunk * kNormChunk, r1 = min(L, r0 + kNormChunk);
  const Tt* base = x + (size_t)bh * (size_t)L * D + lp * VEC;
  float best = 0.0f;
  for (int rb = r0 + g; rb < r1; rb += kNormAhead * RPI) {
    float ss[kNormAhead];
#pragma unroll
    for (int u = 0; u < kNormAhead; ++u) {
      const int r = min(rb + u * RPI, r1 - 1);  // rows past the chunk repeat its last row
      ss[u] = 0.0f;
      if constexpr (sizeof(Tt) == 2) {
        const bf16x8 v = *reinterpret_cast<const bf16x8*>(base + (size_t)r * D);
#pragma unroll
        for (int e = 0; e < 8; ++e) ss[u] += (float)v[e] * (float)v[e];
      } else {
        const f32x4 v = *reinterpret_cast<const f32x4*>(base + (size_t)r * D);
#pragma unroll
        for (int e = 0; e < 4; ++e) ss[u] += v[e] * v[e];
      }
    }
#pragma unroll
    for (int u = 0; u < kNormAhead; ++u) best = fmaxf(best, row_sum<LPR>(ss[u]));
  }
  __shared__ float s_best[kNormThreads / 64];
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) best = fmaxf(best, __shfl_xor(best, off));
  if ((tid & 63) == 0) s_best[tid >> 6] = best;
  __syncthreads();
  if (tid == 0) {
    float m = 0.0f;
    for (int w = 0; w < kNormThreads / 64; ++w) m = fmaxf(m, s_best[w]);
    const float nrm = sqrtf(m) * (1.0f + 0x1p-10f);
    atomicMax(reinterpret_cast<unsigned int*>(out + bh), __float_as_uint(nrm));
  }
}

template <typename Tt>
static void row_norm_t(const void* x, float* out, int BH, int L, int d, hipStream_t s) {
  const int n_chunk = (L + kNormChunk - 1) / kNormChunk;
  const dim3 grid((unsigned)BH * (unsigned)n_chunk);
  if (d == 128)
    hipLaunchKernelGGL((row_norm_max_kernel<Tt, 128>), grid, dim3(kNormThreads), 0, s,
                       (const Tt*)x, out, L, n_chunk);
  else
    hipLaunchKernelGGL((row_norm_max_kernel<Tt, 64>), grid, dim3(kNormThreads), 0, s,
                       (const Tt*)x, out, L, n_chunk);
}

hipError_t launch_row_norm_max(bool bf16_, const void* x, float* out, int BH, int L, int d,
                               hipStream_t s) {
  hipLaunchKernelGGL(zero_kernel, dim3((BH + 255) / 256), dim3(256), 0, s, out, BH);
  if (bf16_) row_norm_t<bf16>(x, out, BH, L, d, s);
  else row_norm_t<float>(x, out, BH, L, d, s);
  return hipGetLastError();
}

}  // namespace fox
