// One decode step of Forgetting Attention: Eq. fot-weight evaluated for the last
// position T of a sequence whose keys and values sit in a cache.
//
//     c_T   = c_{T-1} + log sigmoid(x_new)           (c_0 = 0)
//     s_j   = s q.k_j + c_T - c_j,   j = 1..T         (key T is the new token)
//     o     = sum_j softmax(s)_j v_j,  lse = log sum_j exp(s_j)
//
// The step streams K and V once from HBM (the bound), so the kernel is built for
// bandwidth: the T keys of each (batch, head) are split across workgroups, a
// group of D/8 (bf16) lanes reads one key's row with 16-byte loads so that a
// wave reads consecutive rows, several keys per lane group are loaded before
// any is used, and every lane group keeps its own running (max, sum, output).
// Workgroups are ordered split-major, most recent keys first, so that work is
// spread over all XCDs also when gate-aware skipping (below) keeps only the
// recent splits of every sequence.
// The lane groups of a workgroup merge through LDS into one partial per split;
// a small second kernel merges the splits (log-sum-exp merge) and appends c_T
// to the prefix cache.  Entry T-1 of that cache is never read: every workgroup
// derives c_T itself, so the write cannot race with the readers.
#include <mutex>

#include "fox_device.h"
#include "fox_internal.h"

namespace fox {

constexpr int kDecThreads = 256;
constexpr int kDecUnroll = 4;
// A split is skipped when its scores provably lie this far (base 2) below the
// new token's own score: 150 makes its merge weight exp2(m_split - M) an exact
// fp32 zero, and 10 more absorb the rounding of the bound itself.
constexpr float kSkipMargin = 160.0f;

static int decode_keys_per_split(int BH, int T) {
  // The largest split (fewer partials) that still gives >= 2048 workgroups.
  for (int ks = 1024; ks >= 256; ks >>= 1) {
    const long long wgs = (long long)BH * ((T + ks - 1) / ks);
    if (wgs >= 2048) return ks;
  }
  return 256;
}

int decode_num_splits(int BH, int T) {
  const int ks = decode_keys_per_split(BH, T);
  return (T + ks - 1) / ks;
}

size_t decode_workspace_bytes(int BH, int T, int d) {
  return (size_t)BH * (size_t)decode_num_splits(BH, T) * (size_t)(d + 2) * sizeof(float);
}

template <typename Tt>
struct Vec16;
template <>
struct Vec16<bf16> {
  typedef bf16x8 type;
  static constexpr int N = 8;
};
template <>
struct Vec16<float> {
  typedef f32x4 type;
  static constexpr int N = 4;
};

// FIXED: gate = b [H] (fixed gates, c_T - c_j = (T - 1 - j) log sigmoid(b));
// otherwise gate = the prefix cache [BH, T] and x_new the new token's gate logit.
// SKIP: knorm [BH] bounds the key norms; a split that cannot contribute (its
// merge weight would be an exact zero) writes an empty partial without reading
// its keys, which leaves the result bit for bit as without skipping.
template <typename Tt, int D, bool FIXED, bool SKIP>
__global__ __launch_bounds__(kDecThreads) void decode_split_kernel(
    const Tt* __restrict__ q, const Tt* __restrict__ kc, const Tt* __restrict__ vc,
    const float* __restrict__ gate, const float* __restrict__ x_new,
    const float* __restrict__ knorm, float* __restrict__ part, int H, int T, int keys_per_split,
    int n_split, float scale_log2) {
  typedef typename Vec16<Tt>::type VT;
  constexpr int VEC = Vec16<Tt>::N;
  constexpr int LPK = D / VEC;                // lanes per key
  constexpr int KPI = kDecThreads / LPK;      // keys per workgroup pass
  __shared__ float s_acc[KPI][D];
  __shared__ float s_m[KPI], s_l[KPI];

  const int tid = threadIdx.x;
  const int g = tid / LPK, lp = tid % LPK;
  // split-major, most recent split first: the splits that gate-aware skipping
  // keeps (the recent ones) are spread over all XCDs and dispatched first
  const int n_bh = (int)(gridDim.x / n_split);
  const int bh = blockIdx.x % n_bh, split = n_split - 1 - (int)(blockIdx.x / n_bh);
  const size_t head = (size_t)bh * (size_t)T;
  const int kbeg = split * keys_per_split;
  const int kend = min(T, kbeg + keys_per_split);
  float cT = 0.0f, lf = 0.0f;
  if constexpr (FIXED) {
    lf = log_sigmoid(gate[bh % H]);
  } else {
    cT = (T >= 2 ? gate[head + T - 2] : 0.0f) + log_sigmoid(x_new[bh]);
  }

  float qv[VEC], acc[VEC];
  {
    const VT qq = *reinterpret_cast<const VT*>(q + (size_t)bh * D + lp * VEC);
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      qv[e] = (float)qq[e] * scale_log2;
      acc[e] = 0.0f;
    }
  }
  float m = -INFINITY, l = 0.0f;
  const Tt* kh = kc + head * D + lp * VEC;
  const Tt* vh = vc + head * D + lp * VEC;

  if constexpr (SKIP) {
    // Every score of the split is at most ||s log2(e) q|| max||k|| minus the
    // decay to the split's last key (c decreases along the sequence), while the
    // merged maximum is at least the new token's own score.  The butterfly sums
    // below give bitwise the same value in every lane, so the decision is
    // uniform across the workgroup.
    float qq = 0.0f, dot = 0.0f;
    const VT kl = *reinterpret_cast<const VT*>(kh + (size_t)(T - 1) * D);
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      qq += qv[e] * qv[e];
      dot += qv[e] * (float)kl[e];
    }
#pragma unroll
    for (int off = 1; off < LPK; off <<= 1) {
      qq += __shfl_xor(qq, off);
      dot += __shfl_xor(dot, off);
    }
    const int jl = kend - 1;  // the split's last (least decayed) key
    float decay = 0.0f;       // (c_jl - c_T) log2(e) >= 0
    if (jl != T - 1) {
      if constexpr (FIXED) decay = (float)(jl - (T - 1)) * lf * kLog2e;
      else decay = (gate[head + jl] - cT) * kLog2e;
    }
    const float bound = sqrtf(qq) * knorm[bh] - decay;
    if (bound < dot - kSkipMargin) {
      float* out = part + ((size_t)bh * n_split + split) * (D + 2);
      for (int dd = tid; dd < D; dd += kDecThreads) out[2 + dd] = 0.0f;
      if (tid == 0) {
        out[0] = -INFINITY;
        out[1] = 0.0f;
      }
      return;
    }
  }

  for (int base = kbeg; base < kend; base += KPI * kDecUnroll) {
    VT kr[kDecUnroll], vr[kDecUnroll];
    float cj[kDecUnroll];
#pragma unroll
    for (int u = 0; u < kDecUnroll; ++u) {
      const int key = base + u * KPI + g;
      if (key < kend) {
        kr[u] = __builtin_nontemporal_load(reinterpret_cast<const VT*>(kh + (size_t)key * D));
        vr[u] = __builtin_nontemporal_load(reinterpret_cast<const VT*>(vh + (size_t)key * D));
        if constexpr (FIXED) cj[u] = (float)(key - (T - 1)) * lf * kLog2e;
        else cj[u] = key == T - 1 ? 0.0f : (gate[head + key] - cT) * kLog2e;
      } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          kr[u][e] = (Tt)0.0f;
          vr[u][e] = (Tt)0.0f;
        }
        cj[u] = INFINITY;
      }
    }
    float sv[kDecUnroll];
    float mu = -INFINITY;
#pragma unroll
    for (int u = 0; u < kDecUnroll; ++u) {
      float dot = 0.0f;
#pragma unroll
      for (int e = 0; e < VEC; ++e) dot += qv[e] * (float)kr[u][e];
#pragma unroll
      for (int off = 1; off < LPK; off <<= 1) dot += __shfl_xor(dot, off);
      sv[u] = dot - cj[u];
      mu = fmaxf(mu, sv[u]);
    }
    const float m_new = fmaxf(m, mu);
    // A lane group with no key yet keeps m = -inf; a finite reference keeps the
    // exponents below free of (-inf) - (-inf).
    const float m_ref = m_new == -INFINITY ? 0.0f : m_new;
    const float alpha = exp2_fast(m - m_ref);
    l *= alpha;
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[e] *= alpha;
#pragma unroll
    for (int u = 0; u < kDecUnroll; ++u) {
      const float p = exp2_fast(sv[u] - m_ref);
      l += p;
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc[e] += p * (float)vr[u][e];
    }
    m = m_new;
  }

#pragma unroll
  for (int e = 0; e < VEC; ++e) s_acc[g][lp * VEC + e] = acc[e];
  if (lp == 0) {
    s_m[g] = m;
    s_l[g] = l;
  }
  __syncthreads();
  float M = -INFINITY;
  for (int i = 0; i < KPI; ++i) M = fmaxf(M, s_m[i]);
  float* out = part + ((size_t)bh * n_split + split) * (D + 2);
  for (int dd = tid; dd < D; dd += kDecThreads) {
    float o = 0.0f;
    for (int i = 0; i < KPI; ++i) o += s_acc[i][dd] * exp2_fast(s_m[i] - M);
    out[2 + dd] = o;
  }
  if (tid == 0) {
    float Ls = 0.0f;
    for (int i = 0; i < KPI; ++i) Ls += s_l[i] * exp2_fast(s_m[i] - M);
    out[0] = M;
    out[1] = Ls;
  }
}

template <typename Tt, int D>
__global__ __launch_bounds__(D) void decode_combine_kernel(
    const float* __restrict__ part, float* __restrict__ cc, const float* __restrict__ x_new,
    Tt* __restrict__ o, float* __restrict__ lse, int T, int n_split) {
  const int bh = blockIdx.x, tid = threadIdx.x;
  const float* p = part + (size_t)bh * n_split * (D + 2);
  float M = -INFINITY;
  for (int s = 0; s < n_split; ++s) M = fmaxf(M, p[(size_t)s * (D + 2)]);
  float Ls = 0.0f, acc = 0.0f;
  for (int s = 0; s < n_split; ++s) {
    const float* ps = p + (size_t)s * (D + 2);
    const float w = exp2_fast(ps[0] - M);
    Ls += ps[1] * w;
    acc += ps[2 + tid] * w;
  }
  o[(size_t)bh * D + tid] = (Tt)(acc / Ls);
  if (tid == 0) {
    lse[bh] = kLn2 * (M + log2f(Ls));
    if (cc) {  // append c_T to the prefix cache (data-dependent gates)
      const size_t head = (size_t)bh * (size_t)T;
      cc[head + T - 1] = (T >= 2 ? cc[head + T - 2] : 0.0f) + log_sigmoid(x_new[bh]);
    }
  }
}

template <typename Tt, int D, bool FIXED, bool SKIP>
static hipError_t launch_decode_t(const void* q, const void* k_cache, const void* v_cache,
                                  const float* gate, int H, float* c_cache, const float* logit_new,
                                  const float* knorm, void* o, float* lse, void* ws, int BH, int T,
                                  float scale, hipStream_t s) {
  const int ks = decode_keys_per_split(BH, T);
  const int n_split = (T + ks - 1) / ks;
  float* part = static_cast<float*>(ws);
  hipLaunchKernelGGL((decode_split_kernel<Tt, D, FIXED, SKIP>),
                     dim3((unsigned)n_split * (unsigned)BH), dim3(kDecThreads), 0, s,
                     (const Tt*)q, (const Tt*)k_cache, (const Tt*)v_cache, gate, logit_new, knorm,
                     part, H, T, ks, n_split, scale * kLog2e);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((decode_combine_kernel<Tt, D>), dim3(BH), dim3(D), 0, s, part, c_cache,
                     logit_new, (Tt*)o, lse, T, n_split);
  return hipGetLastError();
}

template <bool FIXED, bool SKIP>
static hipError_t decode_dispatch(bool bf16_, const void* q, const void* k_cache,
                                  const void* v_cache, const float* gate, int H, float* c_cache,
                                  const float* logit_new, const float* knorm, void* o, float* lse,
                                  void* ws, int BH, int T, int d, float scale, hipStream_t s) {
  if (bf16_) {
    return d == 128 ? launch_decode_t<bf16, 128, FIXED, SKIP>(q, k_cache, v_cache, gate, H,
                                                              c_cache, logit_new, knorm, o, lse,
                                                              ws, BH, T, scale, s)
                    : launch_decode_t<bf16, 64, FIXED, SKIP>(q, k_cache, v_cache, gate, H,
                                                             c_cache, logit_new, knorm, o, lse,
                                                             ws, BH, T, scale, s);
  }
  return d == 128 ? launch_decode_t<float, 128, FIXED, SKIP>(q, k_cache, v_cache, gate, H,
                                                             c_cache, logit_new, knorm, o, lse,
                                                             ws, BH, T, scale, s)
                  : launch_decode_t<float, 64, FIXED, SKIP>(q, k_cache, v_cache, gate, H,
                                                            c_cache, logit_new, knorm, o, lse,
                                                            ws, BH, T, scale, s);
}

hipError_t launch_decode(bool bf16_, const void* q, const void* k_cache, const void* v_cache,
                         float* c_cache, const float* logit_new, void* o, float* lse, void* ws,
                         int BH, int T, int d, float scale, hipStream_t s) {
  return decode_dispatch<false, false>(bf16_, q, k_cache, v_cache, c_cache, 1, c_cache, logit_new,
                                       nullptr, o, lse, ws, BH, T, d, scale, s);
}

// ---------------------------------------------------------------------------
// The decode step without a caller workspace: the split partials live in a
// file-scope device array, `scratch`, of kDecodeScratchBytes (every device the
// library runs on holds its own copy, loaded with the code object, until the
// process ends).  In host code the name `scratch` is only a host-side stand-in;
// the device address comes from hipGetSymbolAddress, taken once per device with
// that device current and kept in scratch_ptr[].  The partials are fully
// written by the split kernel before the combine kernel reads them (skipped
// splits write empty partials), so nothing needs clearing between calls; calls
// that overlap on one device share the array and race.
// ---------------------------------------------------------------------------
static __device__ __align__(256) float scratch[kDecodeScratchBytes / sizeof(float)];

namespace {
constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void* scratch_ptr[kMaxDevices] = {};

hipError_t device_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (!scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    scratch_ptr[dev] = p;
  }
  *out = scratch_ptr[dev];
  return hipSuccess;
}
}  // namespace

hipError_t launch_decode_noalloc(bool bf16_, const void* q, const void* k_cache,
                                 const void* v_cache, float* c_cache, const float* logit_new,
                                 void* o, float* lse, int BH, int T, int d, float scale,
                                 hipStream_t s) {
  if (decode_workspace_bytes(BH, T, d) > kDecodeScratchBytes) return hipErrorInvalidValue;
  void* ws = nullptr;
  hipError_t e = device_scratch(&ws);
  if (e != hipSuccess) return e;
  return decode_dispatch<false, false>(bf16_, q, k_cache, v_cache, c_cache, 1, c_cache, logit_new,
                                       nullptr, o, lse, ws, BH, T, d, scale, s);
}

hipError_t launch_decode_skip(bool bf16_, const void* q, const void* k_cache, const void* v_cache,
                              float* c_cache, const float* logit_new, const float* k_norm_max,
                              void* o, float* lse, void* ws, int BH, int T, int d, float scale,
                              hipStream_t s) {
  return decode_dispatch<false, true>(bf16_, q, k_cache, v_cache, c_cache, 1, c_cache, logit_new,
                                      k_norm_max, o, lse, ws, BH, T, d, scale, s);
}

hipError_t launch_decode_fixed(bool bf16_, const void* q, const void* k_cache, const void* v_cache,
                               const float* bias, int H, void* o, float* lse, void* ws, int BH,
                               int T, int d, float scale, hipStream_t s,
                               const float* k_norm_max) {
  if (k_norm_max)
    return decode_dispatch<true, true>(bf16_, q, k_cache, v_cache, bias, H, nullptr, nullptr,
                                       k_norm_max, o, lse, ws, BH, T, d, scale, s);
  return decode_dispatch<true, false>(bf16_, q, k_cache, v_cache, bias, H, nullptr, nullptr,
                                      nullptr, o, lse, ws, BH, T, d, scale, s);
}

}  // namespace fox
