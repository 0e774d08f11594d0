// FoX (Pro) prologue and epilogue (Sec. 3 "Architecture design", Eq. shift-linear;
// appendix "Detailed FoX (Pro) layer computation").  Per head and time step t:
//
//   q_t = RMSNorm_q(q~_t)
//   k_t = RMSNorm_k(a_t k~_{t-1} + (1 - a_t) k~_t),   a_t = sigmoid(k shift logit_t)
//   v_t = b_t v~_{t-1} + (1 - b_t) v~_t,              b_t = sigmoid(v shift logit_t)
//   y_t = RMSNorm_o(o_t) o sigmoid(g_t)               (after the attention)
//
// with RMSNorm(x) = x / sqrt(mean(x^2) + eps) * w^(h) and k~_0 = v~_0 = 0.  Every
// kernel here is row-parallel and bound by HBM: LPR lanes hold one row of d
// values as 16-byte vectors, reductions over the head dimension are shuffles
// within those lanes (DPP), and a workgroup walks kProRows consecutive rows of one
// (batch, head) slice, so the neighbour rows the token shift reads come from
// the cache.  Weight gradients are summed per workgroup (through LDS) and then
// over the workgroups of a head by a second kernel: no atomics, deterministic.
#include "fox_device.h"
#include "fox_internal.h"

namespace fox {

constexpr int kProThreads = 256;
constexpr int kProRows = 256;  // rows of one (batch, head) slice per workgroup

template <typename T>
struct ProVec;
template <>
struct ProVec<bf16> {
  static constexpr int N = 8;
  using type = bf16x8;
};
template <>
struct ProVec<float> {
  static constexpr int N = 4;
  using type = f32x4;
};

template <typename T, int N = ProVec<T>::N>
__device__ __forceinline__ void load_vec(const T* p, float (&x)[N]) {
  const auto v = *reinterpret_cast<const typename ProVec<T>::type*>(p);
#pragma unroll
  for (int i = 0; i < N; ++i) x[i] = (float)v[i];
}

template <typename T, int N = ProVec<T>::N>
__device__ __forceinline__ void store_vec(T* p, const float (&x)[N]) {
  typename ProVec<T>::type v;
#pragma unroll
  for (int i = 0; i < N; ++i) v[i] = (T)x[i];
  *reinterpret_cast<typename ProVec<T>::type*>(p) = v;
}

// N consecutive fp32 weights (16-byte aligned: N is 4 or 8 and the row offset a
// multiple of N)
template <int N>
__device__ __forceinline__ void load_w(const float* p, float (&w)[N]) {
#pragma unroll
  for (int i = 0; i < N; i += 4) {
    const f32x4 v = *reinterpret_cast<const f32x4*>(p + i);
#pragma unroll
    for (int j = 0; j < 4; ++j) w[i + j] = v[j];
  }
}

__device__ __forceinline__ float sigmoid(float x) { return 1.0f / (1.0f + expf(-x)); }

// 1 / sqrt(mean of squares + eps) of one row, from each lane's partial sum of squares
template <int LPR, int D>
__device__ __forceinline__ float inv_rms(float ss, float eps) {
  return 1.0f / sqrtf(row_sum<LPR>(ss) * (1.0f / D) + eps);
}

// Weight-gradient partials: every lane's per-element sums, reduced over the
// row slots of the workgroup, go to part[D].
template <int D, int VEC, int RPP>
__device__ __forceinline__ void store_weight_partial(float (*red)[D], const float (&acc)[VEC],
                                                     int slot, int part, float* out) {
#pragma unroll
  for (int i = 0; i < VEC; ++i) red[slot][part * VEC + i] = acc[i];
  __syncthreads();
  for (int e = threadIdx.x; e < D; e += kProThreads) {
    float s = 0.0f;
#pragma unroll 8
    for (int r = 0; r < RPP; ++r) s += red[r][e];
    out[e] = s;
  }
  __syncthreads();
}

// ---------------------------------------------------------------------------
// prologue, forward
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(kProThreads) void pro_prologue_kernel(
    const T* __restrict__ qr, const T* __restrict__ kr, const T* __restrict__ vr,
    const float* __restrict__ ka, const float* __restrict__ va, const float* __restrict__ wq,
    const float* __restrict__ wk, float eps, T* __restrict__ q, T* __restrict__ k,
    T* __restrict__ v, int H, int L, int n_chunk) {
  constexpr int VEC = ProVec<T>::N, LPR = D / VEC, RPP = kProThreads / LPR;
  const int bh = (int)(blockIdx.x / n_chunk), chunk = (int)(blockIdx.x % n_chunk);
  const int part = threadIdx.x % LPR, slot = threadIdx.x / LPR;
  float wqv[VEC], wkv[VEC];
  load_w<VEC>(wq + (size_t)(bh % H) * D + part * VEC, wqv);
  load_w<VEC>(wk + (size_t)(bh % H) * D + part * VEC, wkv);
  const size_t base = (size_t)bh * L;
  const int t_end = min(L, (chunk + 1) * kProRows);
#pragma unroll 2
  for (int t = chunk * kProRows + slot; t < t_end; t += RPP) {
    const size_t row = base + t;
    const size_t off = row * D + part * VEC;
    // every load first; row t - 1 is clamped to row t at t = 0 and weighted 0
    const size_t offp = t > 0 ? off - D : off;
    float xq[VEC], xk[VEC], pk[VEC], xv[VEC], pv[VEC];
    load_vec<T>(qr + off, xq);
    load_vec<T>(kr + off, xk);
    load_vec<T>(kr + offp, pk);
    load_vec<T>(vr + off, xv);
    load_vec<T>(vr + offp, pv);
    const float a = t > 0 ? sigmoid(ka[row]) : 0.0f;
    const float a1 = 1.0f - sigmoid(ka[row]);
    const float b = t > 0 ? sigmoid(va[row]) : 0.0f;
    const float b1 = 1.0f - sigmoid(va[row]);
    sched_fence();  // keep the loads together, ahead of the arithmetic
    // q = RMSNorm_q(q~)
    float ss = 0.0f;
#pragma unroll
    for (int i = 0; i < VEC; ++i) ss += xq[i] * xq[i];
    float r = inv_rms<LPR, D>(ss, eps);
#pragma unroll
    for (int i = 0; i < VEC; ++i) xq[i] = xq[i] * r * wqv[i];
    store_vec<T>(q + off, xq);
    // k = RMSNorm_k(a k~_{t-1} + (1 - a) k~_t)
    ss = 0.0f;
#pragma unroll
    for (int i = 0; i < VEC; ++i) {
      xk[i] = a * pk[i] + a1 * xk[i];
      ss += xk[i] * xk[i];
    }
    r = inv_rms<LPR, D>(ss, eps);
#pragma unroll
    for (int i = 0; i < VEC; ++i) xk[i] = xk[i] * r * wkv[i];
    store_vec<T>(k + off, xk);
    // v = b v~_{t-1} + (1 - b) v~_t
#pragma unroll
    for (int i = 0; i < VEC; ++i) xv[i] = b * pv[i] + b1 * xv[i];
    store_vec<T>(v + off, xv);
  }
}

// ---------------------------------------------------------------------------
// prologue, backward.  For row t (n = x r the normalised row, dn = dy o w):
//   RMSNorm:     dx = r (dn - n mean(dn o n)),  dw += dy o n
//   key shift:   with s_t = a_t k~_{t-1} + (1 - a_t) k~_t and ds_t from RMSNorm_k,
//                dk~_t = (1 - a_t) ds_t + a_{t+1} ds_{t+1},
//                d(k shift logit)_t = a_t (1 - a_t) ds_t . (k~_{t-1} - k~_t)
//   value shift: the same with dv in place of ds and no normalisation.
// ds_{t+1} is recomputed from row t + 1 (the neighbour rows come from the cache).
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(kProThreads) void pro_prologue_bwd_kernel(
    const T* __restrict__ qr, const T* __restrict__ kr, const T* __restrict__ vr,
    const float* __restrict__ ka, const float* __restrict__ va, const float* __restrict__ wq,
    const float* __restrict__ wk, float eps, const T* __restrict__ dq, const T* __restrict__ dk,
    const T* __restrict__ dv, T* __restrict__ dqr, T* __restrict__ dkr, T* __restrict__ dvr,
    float* __restrict__ dka, float* __restrict__ dva, float* __restrict__ pwq,
    float* __restrict__ pwk, int H, int L, int n_chunk) {
  constexpr int VEC = ProVec<T>::N, LPR = D / VEC, RPP = kProThreads / LPR;
  __shared__ float red[RPP][D];
  const int bh = (int)(blockIdx.x / n_chunk), chunk = (int)(blockIdx.x % n_chunk);
  const int part = threadIdx.x % LPR, slot = threadIdx.x / LPR;
  float wqv[VEC], wkv[VEC], aq[VEC], ak[VEC];
  load_w<VEC>(wq + (size_t)(bh % H) * D + part * VEC, wqv);
  load_w<VEC>(wk + (size_t)(bh % H) * D + part * VEC, wkv);
#pragma unroll
  for (int i = 0; i < VEC; ++i) aq[i] = ak[i] = 0.0f;
  const size_t base = (size_t)bh * L;
  const int t_end = min(L, (chunk + 1) * kProRows);

  // RMSNorm_k backward of the key row u: s (in: the mixed row, out: n = s r),
  // g (in: dk_u) -> ds = r (g o w - n mean(g o w o n))
  auto norm_bwd = [&](float (&sn)[VEC], const float (&g)[VEC], float (&ds)[VEC]) {
    float ss = 0.0f;
#pragma unroll
    for (int i = 0; i < VEC; ++i) ss += sn[i] * sn[i];
    const float r = inv_rms<LPR, D>(ss, eps);
    float m = 0.0f;
#pragma unroll
    for (int i = 0; i < VEC; ++i) {
      sn[i] *= r;
      ds[i] = g[i] * wkv[i];
      m += ds[i] * sn[i];
    }
    m = row_sum<LPR>(m) * (1.0f / D);
#pragma unroll
    for (int i = 0; i < VEC; ++i) ds[i] = r * (ds[i] - sn[i] * m);
  };

  for (int t = chunk * kProRows + slot; t < t_end; t += RPP) {
    const size_t row = base + t;
    const size_t off = row * D + part * VEC;
    const bool first = t == 0, last = t + 1 == L;
    // every load first; the rows t - 1 and t + 1 are clamped to row t at the
    // sequence ends, where their terms are dropped
    const size_t offp = first ? off : off - D, offn = last ? off : off + D;
    float xq[VEC], gq[VEC], kp[VEC], kc[VEC], kn[VEC], gk[VEC], gkn[VEC];
    float vp[VEC], vc[VEC], gv[VEC], gvn[VEC];
    load_vec<T>(qr + off, xq);
    load_vec<T>(dq + off, gq);
    load_vec<T>(kr + offp, kp);
    load_vec<T>(kr + off, kc);
    load_vec<T>(kr + offn, kn);
    load_vec<T>(dk + off, gk);
    load_vec<T>(dk + offn, gkn);
    load_vec<T>(vr + offp, vp);
    load_vec<T>(vr + off, vc);
    load_vec<T>(dv + off, gv);
    load_vec<T>(dv + offn, gvn);
    const float a = sigmoid(ka[row]), an = sigmoid(ka[last ? row : row + 1]);
    const float b = sigmoid(va[row]), bn = sigmoid(va[last ? row : row + 1]);
    sched_fence();  // keep the loads together, ahead of the arithmetic
#pragma unroll
    for (int i = 0; i < VEC; ++i) {
      kp[i] = first ? 0.0f : kp[i];  // k~_0 = v~_0 = 0
      vp[i] = first ? 0.0f : vp[i];
    }
    // q
    {
      float ss = 0.0f;
#pragma unroll
      for (int i = 0; i < VEC; ++i) ss += xq[i] * xq[i];
      const float r = inv_rms<LPR, D>(ss, eps);
      float m = 0.0f;
#pragma unroll
      for (int i = 0; i < VEC; ++i) {
        xq[i] *= r;  // n
        aq[i] += gq[i] * xq[i];
        gq[i] *= wqv[i];  // dn
        m += gq[i] * xq[i];
      }
      m = row_sum<LPR>(m) * (1.0f / D);
#pragma unroll
      for (int i = 0; i < VEC; ++i) gq[i] = r * (gq[i] - xq[i] * m);
      store_vec<T>(dqr + off, gq);
    }
    // k: ds_t through s_t, ds_{t+1} through s_{t+1} = a_{t+1} k~_t + (1 - a_{t+1}) k~_{t+1}
    {
      float sn[VEC], ds[VEC], dsn[VEC];
#pragma unroll
      for (int i = 0; i < VEC; ++i) sn[i] = a * kp[i] + (1.0f - a) * kc[i];
      norm_bwd(sn, gk, ds);
#pragma unroll
      for (int i = 0; i < VEC; ++i) ak[i] += gk[i] * sn[i];
#pragma unroll
      for (int i = 0; i < VEC; ++i) sn[i] = an * kc[i] + (1.0f - an) * kn[i];
      norm_bwd(sn, gkn, dsn);
      float dl = 0.0f;
#pragma unroll
      for (int i = 0; i < VEC; ++i) {
        dl += ds[i] * (kp[i] - kc[i]);
        kc[i] = (1.0f - a) * ds[i] + (last ? 0.0f : an * dsn[i]);
      }
      dl = row_sum<LPR>(dl);
      store_vec<T>(dkr + off, kc);
      if (part == 0) dka[row] = a * (1.0f - a) * dl;
    }
    // v
    {
      float dl = 0.0f;
#pragma unroll
      for (int i = 0; i < VEC; ++i) {
        dl += gv[i] * (vp[i] - vc[i]);
        vc[i] = (1.0f - b) * gv[i] + (last ? 0.0f : bn * gvn[i]);
      }
      dl = row_sum<LPR>(dl);
      store_vec<T>(dvr + off, vc);
      if (part == 0) dva[row] = b * (1.0f - b) * dl;
    }
  }
  store_weight_partial<D, VEC, RPP>(red, aq, slot, part, pwq + (size_t)blockIdx.x * D);
  store_weight_partial<D, VEC, RPP>(red, ak, slot, part, pwk + (size_t)blockIdx.x * D);
}

// ---------------------------------------------------------------------------
// output norm and gate, forward (the bf16 attention forward applies it in its
// epilogue; this kernel serves the fp32 path and standalone use)
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(kProThreads) void out_gate_kernel(
    const T* __restrict__ O, const T* __restrict__ G, const float* __restrict__ wo, float eps,
    T* __restrict__ Y, int H, int L, int n_chunk) {
  constexpr int VEC = ProVec<T>::N, LPR = D / VEC, RPP = kProThreads / LPR;
  const int bh = (int)(blockIdx.x / n_chunk), chunk = (int)(blockIdx.x % n_chunk);
  const int part = threadIdx.x % LPR, slot = threadIdx.x / LPR;
  float w[VEC];
  load_w<VEC>(wo + (size_t)(bh % H) * D + part * VEC, w);
  const int t_end = min(L, (chunk + 1) * kProRows);
#pragma unroll 2
  for (int t = chunk * kProRows + slot; t < t_end; t += RPP) {
    const size_t off = ((size_t)bh * L + t) * D + part * VEC;
    float o[VEC], g[VEC];
    load_vec<T>(O + off, o);
    load_vec<T>(G + off, g);
    sched_fence();
    float ss = 0.0f;
#pragma unroll
    for (int i = 0; i < VEC; ++i) ss += o[i] * o[i];
    const float r = inv_rms<LPR, D>(ss, eps);
#pragma unroll
    for (int i = 0; i < VEC; ++i) o[i] = o[i] * r * w[i] * sigmoid(g[i]);
    store_vec<T>(Y + off, o);
  }
}

// ---------------------------------------------------------------------------
// output norm and gate, backward, fused with the attention backward's Delta:
//   u = RMSNorm_o(o), sg = sigmoid(g):  dg = dy o u o sg (1 - sg),
//   do = r (dn - n mean(dn o n)) with dn = dy o sg o w,  dw += dy o sg o n,
//   Delta = rowsum(do o o) with do rounded to the storage type as the
//   attention backward reads it.
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__(kProThreads) void out_gate_bwd_kernel(
    const T* __restrict__ O, const T* __restrict__ G, const float* __restrict__ wo, float eps,
    const T* __restrict__ dY, T* __restrict__ dO, T* __restrict__ dG, float* __restrict__ delta,
    float* __restrict__ pwo, int H, int L, int n_chunk) {
  constexpr int VEC = ProVec<T>::N, LPR = D / VEC, RPP = kProThreads / LPR;
  __shared__ float red[RPP][D];
  const int bh = (int)(blockIdx.x / n_chunk), chunk = (int)(blockIdx.x % n_chunk);
  const int part = threadIdx.x % LPR, slot = threadIdx.x / LPR;
  float w[VEC], aw[VEC];
  load_w<VEC>(wo + (size_t)(bh % H) * D + part * VEC, w);
#pragma unroll
  for (int i = 0; i < VEC; ++i) aw[i] = 0.0f;
  const int t_end = min(L, (chunk + 1) * kProRows);
#pragma unroll 2
  for (int t = chunk * kProRows + slot; t < t_end; t += RPP) {
    const size_t row = (size_t)bh * L + t;
    const size_t off = row * D + part * VEC;
    float o[VEC], g[VEC], dy[VEC], n[VEC];
    load_vec<T>(O + off, o);
    load_vec<T>(G + off, g);
    load_vec<T>(dY + off, dy);
    sched_fence();
    float ss = 0.0f;
#pragma unroll
    for (int i = 0; i < VEC; ++i) ss += o[i] * o[i];
    const float r = inv_rms<LPR, D>(ss, eps);
    float m = 0.0f;
#pragma unroll
    for (int i = 0; i < VEC; ++i) {
      const float sg = sigmoid(g[i]);
      n[i] = o[i] * r;
      const float du = dy[i] * sg;
      aw[i] += du * n[i];
      g[i] = dy[i] * n[i] * w[i] * sg * (1.0f - sg);  // dg
      dy[i] = du * w[i];                              // dn
      m += dy[i] * n[i];
    }
    store_vec<T>(dG + off, g);
    m = row_sum<LPR>(m) * (1.0f / D);
    float dl = 0.0f;
#pragma unroll
    for (int i = 0; i < VEC; ++i) {
      dy[i] = (float)(T)(r * (dy[i] - n[i] * m));
      dl += dy[i] * o[i];
    }
    store_vec<T>(dO + off, dy);
    dl = row_sum<LPR>(dl);
    if (part == 0) delta[row] = dl;
  }
  store_weight_partial<D, VEC, RPP>(red, aw, slot, part, pwo + (size_t)blockIdx.x * D);
}

// dw^(h)[e] = sum over batch rows b and chunks of part[(b H + h) n_chunk + chunk][e]:
// workgroup (h, 64 elements e); wave w sums the partials p = w, w + 4, ... in
// order (loads unrolled for memory-level parallelism), then the four waves' sums
// are added in order: a fixed order, so the result is deterministic.
constexpr int kReduceThreads = 256;
__global__ __launch_bounds__(kReduceThreads) void weight_grad_reduce_kernel(
    const float* __restrict__ part, float* __restrict__ dw, int B, int H, int n_chunk, int D) {
  const int h = (int)blockIdx.x;
  const int e = (int)blockIdx.y * 64 + (threadIdx.x & 63);
  const int w = threadIdx.x >> 6;
  const int n = B * n_chunk;
  float s = 0.0f;
#pragma unroll 8
  for (int p = w; p < n; p += kReduceThreads / 64) {
    const int b = p / n_chunk, c = p % n_chunk;
    s += part[((size_t)(b * H + h) * n_chunk + c) * D + e];
  }
  __shared__ float wsum[kReduceThreads / 64][64];
  wsum[w][threadIdx.x & 63] = s;
  __syncthreads();
  if (w == 0) {
    float t = 0.0f;
#pragma unroll
    for (int i = 0; i < kReduceThreads / 64; ++i) t += wsum[i][threadIdx.x];
    dw[(size_t)h * D + e] = t;
  }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
int pro_chunks(int L) { return (L + kProRows - 1) / kProRows; }

size_t pro_prologue_bwd_workspace_bytes(int BH, int L, int d) {
  return 2 * (size_t)BH * pro_chunks(L) * d * sizeof(float);
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

size_t bwd_pro_workspace_bytes(bool bf16_, int BH, int L, int d) {
  const size_t es = bf16_ ? 2 : 4;
  return align256(bwd_workspace_bytes(BH, L)) + align256((size_t)BH * L * d * es) +
         (size_t)BH * pro_chunks(L) * d * sizeof(float);
}

template <typename T, int D>
static void prologue_t(const void* qr, const void* kr, const void* vr, const float* ka,
                       const float* va, const float* wq, const float* wk, float eps, void* q,
                       void* k, void* v, int H, int BH, int L, hipStream_t s) {
  const int nc = pro_chunks(L);
  hipLaunchKernelGGL((pro_prologue_kernel<T, D>), dim3((unsigned)(BH * nc)), dim3(kProThreads), 0,
                     s, (const T*)qr, (const T*)kr, (const T*)vr, ka, va, wq, wk, eps, (T*)q,
                     (T*)k, (T*)v, H, L, nc);
}

hipError_t launch_pro_prologue(bool bf16_, const void* qr, const void* kr, const void* vr,
                               const float* ka, const float* va, const float* wq,
                               const float* wk, float eps, void* q, void* k, void* v, int H,
                               int BH, int L, int d, hipStream_t s) {
  if (bf16_) {
    if (d == 128) prologue_t<bf16, 128>(qr, kr, vr, ka, va, wq, wk, eps, q, k, v, H, BH, L, s);
    else prologue_t<bf16, 64>(qr, kr, vr, ka, va, wq, wk, eps, q, k, v, H, BH, L, s);
  } else {
    if (d == 128) prologue_t<float, 128>(qr, kr, vr, ka, va, wq, wk, eps, q, k, v, H, BH, L, s);
    else prologue_t<float, 64>(qr, kr, vr, ka, va, wq, wk, eps, q, k, v, H, BH, L, s);
  }
  return hipGetLastError();
}

template <typename T, int D>
static void prologue_bwd_t(const void* qr, const void* kr, const void* vr, const float* ka,
                           const float* va, const float* wq, const float* wk, float eps,
                           const void* dq, const void* dk, const void* dv, void* dqr, void* dkr,
                           void* dvr, float* dka, float* dva, float* pwq, float* pwk, int H,
                           int BH, int L, hipStream_t s) {
  const int nc = pro_chunks(L);
  hipLaunchKernelGGL((pro_prologue_bwd_kernel<T, D>), dim3((unsigned)(BH * nc)),
                     dim3(kProThreads), 0, s, (const T*)qr, (const T*)kr, (const T*)vr, ka, va,
                     wq, wk, eps, (const T*)dq, (const T*)dk, (const T*)dv, (T*)dqr, (T*)dkr,
                     (T*)dvr, dka, dva, pwq, pwk, H, L, nc);
}

hipError_t launch_pro_prologue_bwd(bool bf16_, const void* qr, const void* kr, const void* vr,
                                   const float* ka, const float* va, const float* wq,
                                   const float* wk, float eps, const void* dq, const void* dk,
                                   const void* dv, void* dqr, void* dkr, void* dvr, float* dka,
                                   float* dva, float* dwq, float* dwk, void* ws, int H, int BH,
                                   int L, int d, hipStream_t s) {
  const int nc = pro_chunks(L);
  float* pwq = static_cast<float*>(ws);
  float* pwk = pwq + (size_t)BH * nc * d;
  if (bf16_) {
    if (d == 128)
      prologue_bwd_t<bf16, 128>(qr, kr, vr, ka, va, wq, wk, eps, dq, dk, dv, dqr, dkr, dvr, dka,
                                dva, pwq, pwk, H, BH, L, s);
    else
      prologue_bwd_t<bf16, 64>(qr, kr, vr, ka, va, wq, wk, eps, dq, dk, dv, dqr, dkr, dvr, dka,
                               dva, pwq, pwk, H, BH, L, s);
  } else {
    if (d == 128)
      prologue_bwd_t<float, 128>(qr, kr, vr, ka, va, wq, wk, eps, dq, dk, dv, dqr, dkr, dvr, dka,
                                 dva, pwq, pwk, H, BH, L, s);
    else
      prologue_bwd_t<float, 64>(qr, kr, vr, ka, va, wq, wk, eps, dq, dk, dv, dqr, dkr, dvr, dka,
                                dva, pwq, pwk, H, BH, L, s);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int B = BH / H;
  const dim3 rgrid((unsigned)H, (unsigned)(d / 64));
  hipLaunchKernelGGL(weight_grad_reduce_kernel, rgrid, dim3(kReduceThreads), 0, s, pwq, dwq, B,
                     H, nc, d);
  hipLaunchKernelGGL(weight_grad_reduce_kernel, rgrid, dim3(kReduceThreads), 0, s, pwk, dwk, B,
                     H, nc, d);
  return hipGetLastError();
}

hipError_t launch_out_gate(bool bf16_, const void* o, const void* g, const float* wo, float eps,
                           void* y, int H, int BH, int L, int d, hipStream_t s) {
  const int nc = pro_chunks(L);
  const dim3 grid((unsigned)(BH * nc)), block(kProThreads);
  if (bf16_) {
    if (d == 128)
      hipLaunchKernelGGL((out_gate_kernel<bf16, 128>), grid, block, 0, s, (const bf16*)o,
                         (const bf16*)g, wo, eps, (bf16*)y, H, L, nc);
    else
      hipLaunchKernelGGL((out_gate_kernel<bf16, 64>), grid, block, 0, s, (const bf16*)o,
                         (const bf16*)g, wo, eps, (bf16*)y, H, L, nc);
  } else {
    if (d == 128)
      hipLaunchKernelGGL((out_gate_kernel<float, 128>), grid, block, 0, s, (const float*)o,
                         (const float*)g, wo, eps, (float*)y, H, L, nc);
    else
      hipLaunchKernelGGL((out_gate_kernel<float, 64>), grid, block, 0, s, (const float*)o,
                         (const float*)g, wo, eps, (float*)y, H, L, nc);
  }
  return hipGetLastError();
}

template <typename T, int D>
static void out_gate_bwd_t(const void* o, const void* g, const float* wo, float eps,
                           const void* dy, void* d_o, void* dg, float* delta, float* pwo, int H,
                           int BH, int L, hipStream_t s) {
  const int nc = pro_chunks(L);
  hipLaunchKernelGGL((out_gate_bwd_kernel<T, D>), dim3((unsigned)(BH * nc)), dim3(kProThreads),
                     0, s, (const T*)o, (const T*)g, wo, eps, (const T*)dy, (T*)d_o, (T*)dg,
                     delta, pwo, H, L, nc);
}

size_t bwd_pro_stored_workspace_bytes(int BH, int L, int d) {
  return align256(bwd_pro_workspace_bytes(true, BH, L, d)) + ds_store_bytes(BH, L);
}

hipError_t launch_bwd_pro(bool bf16_, const void* q, const void* k, const void* v, const float* c,
                          const void* o, const float* lse, const void* g, const float* wo,
                          float eps, const void* dy, void* dq, void* dk, void* dv, float* d_log_f,
                          void* dg, float* dwo, void* ws, int H, int BH, int L, int d, float scale,
                          hipStream_t s, bool keep_ds) {
  const int nc = pro_chunks(L);
  const size_t es = bf16_ ? 2 : 4;
  char* w = static_cast<char*>(ws);
  float* delta = reinterpret_cast<float*>(w);
  float* dcq = delta + (size_t)BH * L;
  float* dck = dcq + (size_t)BH * L;
  void* d_o = w + align256(bwd_workspace_bytes(BH, L));
  float* pwo = reinterpret_cast<float*>(static_cast<char*>(d_o) + align256((size_t)BH * L * d * es));
  if (bf16_) {
    if (d == 128) out_gate_bwd_t<bf16, 128>(o, g, wo, eps, dy, d_o, dg, delta, pwo, H, BH, L, s);
    else out_gate_bwd_t<bf16, 64>(o, g, wo, eps, dy, d_o, dg, delta, pwo, H, BH, L, s);
  } else {
    if (d == 128) out_gate_bwd_t<float, 128>(o, g, wo, eps, dy, d_o, dg, delta, pwo, H, BH, L, s);
    else out_gate_bwd_t<float, 64>(o, g, wo, eps, dy, d_o, dg, delta, pwo, H, BH, L, s);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(weight_grad_reduce_kernel, dim3((unsigned)H, (unsigned)(d / 64)),
                     dim3(kReduceThreads), 0, s, pwo, dwo, BH / H, H, nc, d);
  e = hipGetLastError();
  const GateSpec gs = gate_array(c);
  if (keep_ds) {
    void* dss = w + align256(bwd_pro_workspace_bytes(true, BH, L, d));
    if (e == hipSuccess)
      e = launch_bwd_dkdv_store(q, k, v, gs, lse, d_o, delta, dk, dv, dck, dss, nullptr, BH, L, d,
                                scale, s);
    if (e == hipSuccess) e = launch_bwd_dq_stored(k, dss, nullptr, dq, dcq, BH, L, d, scale, s);
  } else {
    if (e == hipSuccess)
      e = launch_bwd_dkdv(bf16_, q, k, v, gs, lse, d_o, delta, dk, dv, dck, BH, L, d, scale, s);
    if (e == hipSuccess)
      e = launch_bwd_dq(bf16_, q, k, v, gs, lse, d_o, delta, dq, dcq, BH, L, d, scale, s);
  }
  if (e == hipSuccess) e = launch_reverse_scan_sum(dcq, dck, d_log_f, BH, L, s);
  return e;
}

}  // namespace fox
