// C ABI of the Forgetting Attention library: argument validation on the host,
// then kernel launches on the caller's stream.  Nothing here allocates device
// memory or synchronises.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <initializer_list>

#include "fox.h"
#include "fox_internal.h"

namespace {

constexpr long long kMaxElems = 1LL << 40;        // per tensor
constexpr long long kMaxWorkgroups = 1LL << 22;   // 256-thread workgroups per launch

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

fox_status_t check_dims(int B, int H, int L, int d) {
  if (B <= 0 || H <= 0 || L <= 0 || d <= 0) return FOX_ERR_SHAPE;
  const long long bh = (long long)B * H;
  if (bh > (1LL << 30)) return FOX_ERR_SHAPE;
  if (bh * L > (1LL << 31) - 1) return FOX_ERR_SHAPE;          // row index fits in int
  if (bh * L * d > kMaxElems) return FOX_ERR_SHAPE;
  if ((long long)L * d * 4 >= (1LL << 31)) return FOX_ERR_SHAPE;  // one head addressed in 32 bits
  if (bh * ((L + 63) / 64) > kMaxWorkgroups) return FOX_ERR_SHAPE;
  return FOX_OK;
}

fox_status_t check_dtype_d(int dtype, int d) {
  if (dtype != FOX_DTYPE_F32 && dtype != FOX_DTYPE_BF16) return FOX_ERR_UNSUPPORTED;
  if (d != 64 && d != 128) return FOX_ERR_UNSUPPORTED;
  return FOX_OK;
}

fox_status_t launch_status(hipError_t e) { return e == hipSuccess ? FOX_OK : FOX_ERR_HIP; }

fox_status_t check_projection(int dtype, int B, int L, int H, int M) {
  if (B <= 0 || L <= 0 || H <= 0 || M <= 0) return FOX_ERR_SHAPE;
  const long long n = (long long)B * L;
  if (n > (1LL << 31) - 1 || (long long)B * H * L > (1LL << 31) - 1) return FOX_ERR_SHAPE;
  if (n * M > kMaxElems) return FOX_ERR_SHAPE;
  if (dtype != FOX_DTYPE_F32 && dtype != FOX_DTYPE_BF16) return FOX_ERR_UNSUPPORTED;
  if (H > 64 || M % 8 != 0) return FOX_ERR_UNSUPPORTED;
  return FOX_OK;
}

bool valid_eps(float eps) { return isfinite(eps) && eps >= 0.0f; }

bool all_aligned16(std::initializer_list<const void*> ps) {
  for (const void* p : ps)
    if (!aligned16(p)) return false;
  return true;
}

bool all_set(std::initializer_list<const void*> ps) {
  for (const void* p : ps)
    if (!p) return false;
  return true;
}

}  // namespace

extern "C" {

const char* fox_status_string(fox_status_t status) {
  switch (status) {
    case FOX_OK: return "FOX_OK";
    case FOX_ERR_NULL: return "FOX_ERR_NULL: a required pointer is NULL";
    case FOX_ERR_SHAPE: return "FOX_ERR_SHAPE: sizes must be positive and within limits";
    case FOX_ERR_UNSUPPORTED: return "FOX_ERR_UNSUPPORTED: dtype must be f32/bf16, head dim 64/128";
    case FOX_ERR_ALIGN: return "FOX_ERR_ALIGN: device pointers must be 16-byte aligned";
    case FOX_ERR_WORKSPACE: return "FOX_ERR_WORKSPACE: workspace missing or too small";
    case FOX_ERR_HIP: return "FOX_ERR_HIP: the HIP runtime reported a launch error";
    case FOX_ERR_VALUE: return "FOX_ERR_VALUE: a scalar argument is out of range (eps: finite, >= 0)";
    case FOX_ERR_TOO_LARGE:
      return "FOX_ERR_TOO_LARGE: the shape needs more scratch than fox_attn_decode_noalloc holds "
             "(64 MiB of split partials); use fox_attn_decode with a workspace";
    default: return "unknown fox status";
  }
}

int fox_version(void) { return 100; }

fox_status_t fox_gate_prefix(const float* gate_logit, float* log_f, float* c, int B, int H, int L,
                    hipStream_t stream) {
  if (!gate_logit || !c) return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, L, 1);
  if (st) return st;
  if (!aligned16(gate_logit) || !aligned16(c) || (log_f && !aligned16(log_f))) return FOX_ERR_ALIGN;
  return launch_status(fox::launch_gate_prefix(gate_logit, log_f, c, B * H, L,
                                               static_cast<hipStream_t>(stream)));
}

fox_status_t fox_attn_fwd(fox_dtype_t dtype, const void* q, const void* k, const void* v, const float* c, void* o,
                 float* lse, int B, int H, int L, int d, float scale, hipStream_t stream) {
  if (!q || !k || !v || !c || !o || !lse) return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, L, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(c) || !aligned16(o) ||
      !aligned16(lse))
    return FOX_ERR_ALIGN;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (dtype == FOX_DTYPE_BF16)
    return launch_status(fox::launch_fwd_bf16(q, k, v, fox::gate_array(c), o, lse, B * H, L, d, scale, s));
  return launch_status(fox::launch_fwd_f32((const float*)q, (const float*)k, (const float*)v,
                                           fox::gate_array(c), (float*)o, lse, B * H, L, d, scale,
                                           s));
}

size_t fox_attn_bwd_workspace_bytes(fox_dtype_t dtype, int B, int H, int L, int d) {
  if (check_dims(B, H, L, d) || check_dtype_d(dtype, d)) return 0;
  return fox::bwd_workspace_bytes(B * H, L);
}

fox_status_t fox_attn_bwd(fox_dtype_t dtype, const void* q, const void* k, const void* v, const float* c,
                 const void* o, const float* lse, const void* d_o, void* dq, void* dk, void* dv,
                 float* d_log_f, void* workspace, size_t workspace_bytes, int B, int H, int L,
                 int d, float scale, hipStream_t stream) {
  if (!q || !k || !v || !c || !o || !lse || !d_o || !dq || !dk || !dv || !d_log_f)
    return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, L, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(c) || !aligned16(o) ||
      !aligned16(lse) || !aligned16(d_o) || !aligned16(dq) || !aligned16(dk) || !aligned16(dv) ||
      !aligned16(d_log_f))
    return FOX_ERR_ALIGN;
  if (!workspace || workspace_bytes < fox::bwd_workspace_bytes(B * H, L)) return FOX_ERR_WORKSPACE;
  if (!aligned16(workspace)) return FOX_ERR_ALIGN;
  return launch_status(fox::launch_bwd(dtype == FOX_DTYPE_BF16, q, k, v, c, o, lse, d_o, dq, dk,
                                       dv, d_log_f, workspace, B * H, L, d, scale,
                                       static_cast<hipStream_t>(stream)));
}

size_t fox_attn_bwd_stored_workspace_bytes(fox_dtype_t dtype, int B, int H, int L, int d) {
  if (check_dims(B, H, L, d) || check_dtype_d(dtype, d) || dtype != FOX_DTYPE_BF16) return 0;
  return fox::bwd_stored_workspace_bytes(B * H, L);
}

fox_status_t fox_attn_bwd_stored(fox_dtype_t dtype, const void* q, const void* k, const void* v, const float* c,
                        const void* o, const float* lse, const void* d_o, void* dq, void* dk,
                        void* dv, float* d_log_f, void* workspace, size_t workspace_bytes, int B,
                        int H, int L, int d, float scale, hipStream_t stream) {
  if (!q || !k || !v || !c || !o || !lse || !d_o || !dq || !dk || !dv || !d_log_f)
    return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, L, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (dtype != FOX_DTYPE_BF16) return FOX_ERR_UNSUPPORTED;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(c) || !aligned16(o) ||
      !aligned16(lse) || !aligned16(d_o) || !aligned16(dq) || !aligned16(dk) || !aligned16(dv) ||
      !aligned16(d_log_f))
    return FOX_ERR_ALIGN;
  if (!workspace || workspace_bytes < fox::bwd_stored_workspace_bytes(B * H, L))
    return FOX_ERR_WORKSPACE;
  if (!aligned16(workspace)) return FOX_ERR_ALIGN;
  return launch_status(fox::launch_bwd_stored(q, k, v, c, o, lse, d_o, dq, dk, dv, d_log_f,
                                              workspace, B * H, L, d, scale,
                                              static_cast<hipStream_t>(stream)));
}

fox_status_t fox_attn_bwd_delta(fox_dtype_t dtype, const void* o, const void* d_o, float* delta, int B, int H,
                       int L, int d, hipStream_t stream) {
  if (!o || !d_o || !delta) return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, L, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (!aligned16(o) || !aligned16(d_o) || !aligned16(delta)) return FOX_ERR_ALIGN;
  return launch_status(fox::launch_bwd_delta(dtype == FOX_DTYPE_BF16, o, d_o, delta, B * H, L, d,
                                             static_cast<hipStream_t>(stream)));
}

fox_status_t fox_attn_bwd_dkdv(fox_dtype_t dtype, const void* q, const void* k, const void* v, const float* c,
                      const float* lse, const void* d_o, const float* delta, void* dk, void* dv,
                      float* dc_k, int B, int H, int L, int d, float scale, hipStream_t stream) {
  if (!q || !k || !v || !c || !lse || !d_o || !delta || !dk || !dv || !dc_k) return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, L, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(c) || !aligned16(lse) ||
      !aligned16(d_o) || !aligned16(delta) || !aligned16(dk) || !aligned16(dv) ||
      !aligned16(dc_k))
    return FOX_ERR_ALIGN;
  return launch_status(fox::launch_bwd_dkdv(dtype == FOX_DTYPE_BF16, q, k, v, fox::gate_array(c), lse, d_o, delta,
                                            dk, dv, dc_k, B * H, L, d, scale,
                                            static_cast<hipStream_t>(stream)));
}

fox_status_t fox_attn_bwd_dq(fox_dtype_t dtype, const void* q, const void* k, const void* v, const float* c,
                    const float* lse, const void* d_o, const float* delta, void* dq, float* dc_q,
                    int B, int H, int L, int d, float scale, hipStream_t stream) {
  if (!q || !k || !v || !c || !lse || !d_o || !delta || !dq || !dc_q) return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, L, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(c) || !aligned16(lse) ||
      !aligned16(d_o) || !aligned16(delta) || !aligned16(dq) || !aligned16(dc_q))
    return FOX_ERR_ALIGN;
  return launch_status(fox::launch_bwd_dq(dtype == FOX_DTYPE_BF16, q, k, v, fox::gate_array(c), lse, d_o, delta,
                                          dq, dc_q, B * H, L, d, scale,
                                          static_cast<hipStream_t>(stream)));
}

size_t fox_attn_bwd_ds_store_bytes(fox_dtype_t dtype, int B, int H, int L, int d) {
  if (check_dims(B, H, L, d) || check_dtype_d(dtype, d) || dtype != FOX_DTYPE_BF16) return 0;
  return fox::ds_store_bytes(B * H, L);
}

fox_status_t fox_attn_bwd_dkdv_store(fox_dtype_t dtype, const void* q, const void* k, const void* v,
                            const float* c, const float* lse, const void* d_o,
                            const float* delta, void* dk, void* dv, float* dc_k, void* ds_store,
                            size_t ds_store_bytes, int B, int H, int L, int d, float scale,
                            hipStream_t stream) {
  if (!q || !k || !v || !c || !lse || !d_o || !delta || !dk || !dv || !dc_k) return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, L, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (dtype != FOX_DTYPE_BF16) return FOX_ERR_UNSUPPORTED;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(c) || !aligned16(lse) ||
      !aligned16(d_o) || !aligned16(delta) || !aligned16(dk) || !aligned16(dv) ||
      !aligned16(dc_k))
    return FOX_ERR_ALIGN;
  if (!ds_store || ds_store_bytes < fox::ds_store_bytes(B * H, L)) return FOX_ERR_WORKSPACE;
  if (!aligned16(ds_store)) return FOX_ERR_ALIGN;
  return launch_status(fox::launch_bwd_dkdv_store(q, k, v, fox::gate_array(c), lse, d_o, delta,
                                                  dk, dv, dc_k, ds_store, nullptr, B * H, L, d,
                                                  scale, static_cast<hipStream_t>(stream)));
}

fox_status_t fox_attn_bwd_dq_stored(fox_dtype_t dtype, const void* k, const void* ds_store, size_t ds_store_bytes,
                           void* dq, float* dc_q, int B, int H, int L, int d, float scale,
                           hipStream_t stream) {
  if (!k || !dq || !dc_q) return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, L, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (dtype != FOX_DTYPE_BF16) return FOX_ERR_UNSUPPORTED;
  if (!aligned16(k) || !aligned16(dq) || !aligned16(dc_q)) return FOX_ERR_ALIGN;
  if (!ds_store || ds_store_bytes < fox::ds_store_bytes(B * H, L)) return FOX_ERR_WORKSPACE;
  if (!aligned16(ds_store)) return FOX_ERR_ALIGN;
  return launch_status(fox::launch_bwd_dq_stored(k, ds_store, nullptr, dq, dc_q, B * H, L, d,
                                                 scale, static_cast<hipStream_t>(stream)));
}

fox_status_t fox_dlogf_from_dc(const float* dc_q, const float* dc_k, float* d_log_f, int B, int H, int L,
                      hipStream_t stream) {
  if (!dc_q || !dc_k || !d_log_f) return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, L, 1);
  if (st) return st;
  if (!aligned16(dc_q) || !aligned16(dc_k) || !aligned16(d_log_f)) return FOX_ERR_ALIGN;
  return launch_status(fox::launch_reverse_scan_sum(dc_q, dc_k, d_log_f, B * H, L,
                                                    static_cast<hipStream_t>(stream)));
}

fox_status_t fox_dlogit_from_dc(const float* dc_q, const float* dc_k, const float* gate_logit,
                       float* d_log_f, float* d_logit, int B, int H, int L, hipStream_t stream) {
  if (!dc_q || !dc_k || !gate_logit || !d_logit) return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, L, 1);
  if (st) return st;
  if (!aligned16(dc_q) || !aligned16(dc_k) || !aligned16(gate_logit) || !aligned16(d_logit) ||
      (d_log_f && !aligned16(d_log_f)))
    return FOX_ERR_ALIGN;
  return launch_status(fox::launch_reverse_scan_gate(dc_q, dc_k, gate_logit, d_log_f, d_logit,
                                                     B * H, L, static_cast<hipStream_t>(stream)));
}

size_t fox_attn_decode_workspace_bytes(fox_dtype_t dtype, int B, int H, int T, int d) {
  if (check_dims(B, H, T, d) || check_dtype_d(dtype, d)) return 0;
  return fox::decode_workspace_bytes(B * H, T, d);
}

fox_status_t fox_attn_decode(fox_dtype_t dtype, const void* q, const void* k_cache, const void* v_cache,
                    float* c_cache, const float* gate_logit_new, void* o, float* lse,
                    void* workspace, size_t workspace_bytes, int B, int H, int T, int d,
                    float scale, hipStream_t stream) {
  if (!q || !k_cache || !v_cache || !c_cache || !gate_logit_new || !o || !lse)
    return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, T, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(c_cache) ||
      !aligned16(gate_logit_new) || !aligned16(o) || !aligned16(lse))
    return FOX_ERR_ALIGN;
  if (!workspace || workspace_bytes < fox::decode_workspace_bytes(B * H, T, d))
    return FOX_ERR_WORKSPACE;
  if (!aligned16(workspace)) return FOX_ERR_ALIGN;
  return launch_status(fox::launch_decode(dtype == FOX_DTYPE_BF16, q, k_cache, v_cache, c_cache,
                                          gate_logit_new, o, lse, workspace, B * H, T, d, scale,
                                          static_cast<hipStream_t>(stream)));
}

fox_status_t fox_attn_decode_noalloc(fox_dtype_t dtype, const void* q, const void* k_cache,
                                     const void* v_cache, float* c_cache,
                                     const float* gate_logit_new, void* o, float* lse, int B,
                                     int H, int T, int d, float scale, hipStream_t stream) {
  if (!q || !k_cache || !v_cache || !c_cache || !gate_logit_new || !o || !lse)
    return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, T, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(c_cache) ||
      !aligned16(gate_logit_new) || !aligned16(o) || !aligned16(lse))
    return FOX_ERR_ALIGN;
  if (fox::decode_workspace_bytes(B * H, T, d) > fox::kDecodeScratchBytes)
    return FOX_ERR_TOO_LARGE;
  return launch_status(fox::launch_decode_noalloc(dtype == FOX_DTYPE_BF16, q, k_cache, v_cache,
                                                  c_cache, gate_logit_new, o, lse, B * H, T, d,
                                                  scale, stream));
}

// ------------------------------------------------------- gate-aware skipping
fox_status_t fox_row_norm_max(fox_dtype_t dtype, const void* x, float* out, int B, int H, int L, int d,
                     hipStream_t stream) {
  if (!x || !out) return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, L, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (!aligned16(x) || !aligned16(out)) return FOX_ERR_ALIGN;
  return launch_status(fox::launch_row_norm_max(dtype == FOX_DTYPE_BF16, x, out, B * H, L, d,
                                                static_cast<hipStream_t>(stream)));
}

fox_status_t fox_attn_fwd_skip(fox_dtype_t dtype, const void* q, const void* k, const void* v, const float* c,
                      const float* q_norm_max, const float* k_norm_max, void* o, float* lse,
                      int B, int H, int L, int d, float scale, hipStream_t stream) {
  if (!q || !k || !v || !c || !q_norm_max || !k_norm_max || !o || !lse) return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, L, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(c) ||
      !aligned16(q_norm_max) || !aligned16(k_norm_max) || !aligned16(o) || !aligned16(lse))
    return FOX_ERR_ALIGN;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (dtype == FOX_DTYPE_BF16)
    return launch_status(fox::launch_fwd_bf16(q, k, v, fox::gate_array(c), o, lse, B * H, L, d,
                                              scale, s, q_norm_max, k_norm_max));
  return launch_status(fox::launch_fwd_f32((const float*)q, (const float*)k, (const float*)v,
                                           fox::gate_array(c), (float*)o, lse, B * H, L, d, scale,
                                           s));
}

fox_status_t fox_attn_bwd_skip(fox_dtype_t dtype, const void* q, const void* k, const void* v, const float* c,
                      const void* o, const float* lse, const void* d_o, const float* q_norm_max,
                      const float* k_norm_max, void* dq, void* dk, void* dv, float* d_log_f,
                      void* workspace, size_t workspace_bytes, int B, int H, int L, int d,
                      float scale, hipStream_t stream) {
  if (!q || !k || !v || !c || !o || !lse || !d_o || !q_norm_max || !k_norm_max || !dq || !dk ||
      !dv || !d_log_f)
    return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, L, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(c) || !aligned16(o) ||
      !aligned16(lse) || !aligned16(d_o) || !aligned16(q_norm_max) || !aligned16(k_norm_max) ||
      !aligned16(dq) || !aligned16(dk) || !aligned16(dv) || !aligned16(d_log_f))
    return FOX_ERR_ALIGN;
  if (!workspace || workspace_bytes < fox::bwd_workspace_bytes(B * H, L)) return FOX_ERR_WORKSPACE;
  if (!aligned16(workspace)) return FOX_ERR_ALIGN;
  const bool bf = dtype == FOX_DTYPE_BF16;
  return launch_status(fox::launch_bwd(bf, q, k, v, c, o, lse, d_o, dq, dk, dv, d_log_f,
                                       workspace, B * H, L, d, scale,
                                       static_cast<hipStream_t>(stream), bf ? q_norm_max : nullptr,
                                       bf ? k_norm_max : nullptr));
}

fox_status_t fox_attn_bwd_skip_stored(fox_dtype_t dtype, const void* q, const void* k, const void* v,
                             const float* c, const void* o, const float* lse, const void* d_o,
                             const float* q_norm_max, const float* k_norm_max, void* dq, void* dk,
                             void* dv, float* d_log_f, void* workspace, size_t workspace_bytes,
                             int B, int H, int L, int d, float scale, hipStream_t stream) {
  if (!all_set({q, k, v, c, o, lse, d_o, q_norm_max, k_norm_max, dq, dk, dv, d_log_f}))
    return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, L, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (dtype != FOX_DTYPE_BF16) return FOX_ERR_UNSUPPORTED;
  if (!all_aligned16({q, k, v, c, o, lse, d_o, q_norm_max, k_norm_max, dq, dk, dv, d_log_f}))
    return FOX_ERR_ALIGN;
  if (!workspace || workspace_bytes < fox::bwd_stored_workspace_bytes(B * H, L))
    return FOX_ERR_WORKSPACE;
  if (!aligned16(workspace)) return FOX_ERR_ALIGN;
  return launch_status(fox::launch_bwd_stored(q, k, v, c, o, lse, d_o, dq, dk, dv, d_log_f,
                                              workspace, B * H, L, d, scale,
                                              static_cast<hipStream_t>(stream), q_norm_max,
                                              k_norm_max));
}

fox_status_t fox_attn_decode_skip(fox_dtype_t dtype, const void* q, const void* k_cache, const void* v_cache,
                         float* c_cache, const float* gate_logit_new, const float* k_norm_max,
                         void* o, float* lse, void* workspace, size_t workspace_bytes, int B,
                         int H, int T, int d, float scale, hipStream_t stream) {
  if (!q || !k_cache || !v_cache || !c_cache || !gate_logit_new || !k_norm_max || !o || !lse)
    return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, T, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(c_cache) ||
      !aligned16(gate_logit_new) || !aligned16(k_norm_max) || !aligned16(o) || !aligned16(lse))
    return FOX_ERR_ALIGN;
  if (!workspace || workspace_bytes < fox::decode_workspace_bytes(B * H, T, d))
    return FOX_ERR_WORKSPACE;
  if (!aligned16(workspace)) return FOX_ERR_ALIGN;
  return launch_status(fox::launch_decode_skip(dtype == FOX_DTYPE_BF16, q, k_cache, v_cache,
                                               c_cache, gate_logit_new, k_norm_max, o, lse,
                                               workspace, B * H, T, d, scale,
                                               static_cast<hipStream_t>(stream)));
}

// ---------------------------------------------------------------- fixed gates
fox_status_t fox_fixed_gate_init(float* gate_bias, int H, float t_min, float t_max) {
  if (!gate_bias) return FOX_ERR_NULL;
  if (H <= 0 || !(t_min > 0.0f) || !(t_max >= t_min) || !isfinite(t_max)) return FOX_ERR_SHAPE;
  for (int h = 0; h < H; ++h) {
    const double frac = H > 1 ? (double)h / (double)(H - 1) : 0.0;
    const double T = exp(log((double)t_min) + (log((double)t_max) - log((double)t_min)) * frac);
    // sigmoid(b) = exp(-1/T)  <=>  b = log(e^{-1/T} / (1 - e^{-1/T}))
    gate_bias[h] = (float)(-1.0 / T - log(-expm1(-1.0 / T)));
  }
  return FOX_OK;
}

fox_status_t fox_attn_fwd_fixed_gate(fox_dtype_t dtype, const void* q, const void* k, const void* v,
                            const float* gate_bias, void* o, float* lse, int B, int H, int L, int d,
                            float scale, hipStream_t stream) {
  if (!q || !k || !v || !gate_bias || !o || !lse) return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, L, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(gate_bias) || !aligned16(o) ||
      !aligned16(lse))
    return FOX_ERR_ALIGN;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const fox::GateSpec g = fox::gate_fixed(gate_bias, H);
  if (dtype == FOX_DTYPE_BF16)
    return launch_status(fox::launch_fwd_bf16(q, k, v, g, o, lse, B * H, L, d, scale, s));
  return launch_status(fox::launch_fwd_f32((const float*)q, (const float*)k, (const float*)v, g,
                                           (float*)o, lse, B * H, L, d, scale, s));
}

size_t fox_attn_bwd_fixed_gate_workspace_bytes(fox_dtype_t dtype, int B, int H, int L, int d) {
  if (check_dims(B, H, L, d) || check_dtype_d(dtype, d)) return 0;
  return fox::bwd_fixed_workspace_bytes(B * H, L);
}

fox_status_t fox_attn_bwd_fixed_gate(fox_dtype_t dtype, const void* q, const void* k, const void* v,
                            const float* gate_bias, const void* o, const float* lse,
                            const void* d_o, void* dq, void* dk, void* dv, float* d_gate_bias,
                            void* workspace, size_t workspace_bytes, int B, int H, int L, int d,
                            float scale, hipStream_t stream) {
  if (!q || !k || !v || !gate_bias || !o || !lse || !d_o || !dq || !dk || !dv)
    return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, L, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(gate_bias) || !aligned16(o) ||
      !aligned16(lse) || !aligned16(d_o) || !aligned16(dq) || !aligned16(dk) || !aligned16(dv) ||
      (d_gate_bias && !aligned16(d_gate_bias)))
    return FOX_ERR_ALIGN;
  if (!workspace || workspace_bytes < fox::bwd_fixed_workspace_bytes(B * H, L))
    return FOX_ERR_WORKSPACE;
  if (!aligned16(workspace)) return FOX_ERR_ALIGN;
  return launch_status(fox::launch_bwd_fixed(dtype == FOX_DTYPE_BF16, q, k, v, gate_bias, H, o,
                                             lse, d_o, dq, dk, dv, d_gate_bias, workspace, B * H,
                                             L, d, scale, static_cast<hipStream_t>(stream)));
}

size_t fox_attn_bwd_fixed_gate_stored_workspace_bytes(fox_dtype_t dtype, int B, int H, int L, int d) {
  if (check_dims(B, H, L, d) || check_dtype_d(dtype, d) || dtype != FOX_DTYPE_BF16) return 0;
  return fox::bwd_fixed_stored_workspace_bytes(B * H, L);
}

// fox_attn_bwd_fixed_gate_stored and its skipping twin (norms non-NULL)
static fox_status_t bwd_fixed_stored(fox_dtype_t dtype, const void* q, const void* k, const void* v,
                            const float* gate_bias, const void* o, const float* lse,
                            const void* d_o, const float* q_norm_max, const float* k_norm_max,
                            void* dq, void* dk, void* dv, float* d_gate_bias, void* workspace,
                            size_t workspace_bytes, int B, int H, int L, int d, float scale,
                            hipStream_t stream) {
  fox_status_t st = check_dims(B, H, L, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (dtype != FOX_DTYPE_BF16) return FOX_ERR_UNSUPPORTED;
  if (!all_aligned16({q, k, v, gate_bias, o, lse, d_o, dq, dk, dv}) ||
      (q_norm_max && !all_aligned16({q_norm_max, k_norm_max})) ||
      (d_gate_bias && !aligned16(d_gate_bias)))
    return FOX_ERR_ALIGN;
  if (!workspace || workspace_bytes < fox::bwd_fixed_stored_workspace_bytes(B * H, L))
    return FOX_ERR_WORKSPACE;
  if (!aligned16(workspace)) return FOX_ERR_ALIGN;
  return launch_status(fox::launch_bwd_fixed_stored(q, k, v, gate_bias, H, o, lse, d_o, dq, dk,
                                                    dv, d_gate_bias, workspace, B * H, L, d,
                                                    scale, static_cast<hipStream_t>(stream),
                                                    q_norm_max, k_norm_max));
}

fox_status_t fox_attn_bwd_fixed_gate_stored(fox_dtype_t dtype, const void* q, const void* k, const void* v,
                                   const float* gate_bias, const void* o, const float* lse,
                                   const void* d_o, void* dq, void* dk, void* dv,
                                   float* d_gate_bias, void* workspace, size_t workspace_bytes,
                                   int B, int H, int L, int d, float scale, hipStream_t stream) {
  if (!all_set({q, k, v, gate_bias, o, lse, d_o, dq, dk, dv})) return FOX_ERR_NULL;
  return bwd_fixed_stored(dtype, q, k, v, gate_bias, o, lse, d_o, nullptr, nullptr, dq, dk, dv,
                          d_gate_bias, workspace, workspace_bytes, B, H, L, d, scale, stream);
}

fox_status_t fox_attn_bwd_fixed_gate_skip_stored(fox_dtype_t dtype, const void* q, const void* k, const void* v,
                                        const float* gate_bias, const void* o, const float* lse,
                                        const void* d_o, const float* q_norm_max,
                                        const float* k_norm_max, void* dq, void* dk, void* dv,
                                        float* d_gate_bias, void* workspace,
                                        size_t workspace_bytes, int B, int H, int L, int d,
                                        float scale, hipStream_t stream) {
  if (!all_set({q, k, v, gate_bias, o, lse, d_o, q_norm_max, k_norm_max, dq, dk, dv}))
    return FOX_ERR_NULL;
  return bwd_fixed_stored(dtype, q, k, v, gate_bias, o, lse, d_o, q_norm_max, k_norm_max, dq, dk,
                          dv, d_gate_bias, workspace, workspace_bytes, B, H, L, d, scale, stream);
}

fox_status_t fox_attn_decode_fixed_gate(fox_dtype_t dtype, const void* q, const void* k_cache,
                               const void* v_cache, const float* gate_bias, void* o, float* lse,
                               void* workspace, size_t workspace_bytes, int B, int H, int T, int d,
                               float scale, hipStream_t stream) {
  if (!q || !k_cache || !v_cache || !gate_bias || !o || !lse) return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, T, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(gate_bias) ||
      !aligned16(o) || !aligned16(lse))
    return FOX_ERR_ALIGN;
  if (!workspace || workspace_bytes < fox::decode_workspace_bytes(B * H, T, d))
    return FOX_ERR_WORKSPACE;
  if (!aligned16(workspace)) return FOX_ERR_ALIGN;
  return launch_status(fox::launch_decode_fixed(dtype == FOX_DTYPE_BF16, q, k_cache, v_cache,
                                                gate_bias, H, o, lse, workspace, B * H, T, d, scale,
                                                static_cast<hipStream_t>(stream)));
}

fox_status_t fox_attn_fwd_fixed_gate_skip(fox_dtype_t dtype, const void* q, const void* k, const void* v,
                                 const float* gate_bias, const float* q_norm_max,
                                 const float* k_norm_max, void* o, float* lse, int B, int H, int L,
                                 int d, float scale, hipStream_t stream) {
  if (!all_set({q, k, v, gate_bias, q_norm_max, k_norm_max, o, lse})) return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, L, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (!all_aligned16({q, k, v, gate_bias, q_norm_max, k_norm_max, o, lse})) return FOX_ERR_ALIGN;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const fox::GateSpec g = fox::gate_fixed(gate_bias, H);
  if (dtype == FOX_DTYPE_BF16)
    return launch_status(
        fox::launch_fwd_bf16(q, k, v, g, o, lse, B * H, L, d, scale, s, q_norm_max, k_norm_max));
  return launch_status(fox::launch_fwd_f32((const float*)q, (const float*)k, (const float*)v, g,
                                           (float*)o, lse, B * H, L, d, scale, s));
}

fox_status_t fox_attn_bwd_fixed_gate_skip(fox_dtype_t dtype, const void* q, const void* k, const void* v,
                                 const float* gate_bias, const void* o, const float* lse,
                                 const void* d_o, const float* q_norm_max,
                                 const float* k_norm_max, void* dq, void* dk, void* dv,
                                 float* d_gate_bias, void* workspace, size_t workspace_bytes,
                                 int B, int H, int L, int d, float scale, hipStream_t stream) {
  if (!all_set({q, k, v, gate_bias, o, lse, d_o, q_norm_max, k_norm_max, dq, dk, dv}))
    return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, L, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (!all_aligned16({q, k, v, gate_bias, o, lse, d_o, q_norm_max, k_norm_max, dq, dk, dv}) ||
      (d_gate_bias && !aligned16(d_gate_bias)))
    return FOX_ERR_ALIGN;
  if (!workspace || workspace_bytes < fox::bwd_fixed_workspace_bytes(B * H, L))
    return FOX_ERR_WORKSPACE;
  if (!aligned16(workspace)) return FOX_ERR_ALIGN;
  const bool bf = dtype == FOX_DTYPE_BF16;
  return launch_status(fox::launch_bwd_fixed(bf, q, k, v, gate_bias, H, o, lse, d_o, dq, dk, dv,
                                             d_gate_bias, workspace, B * H, L, d, scale,
                                             static_cast<hipStream_t>(stream),
                                             bf ? q_norm_max : nullptr, bf ? k_norm_max : nullptr));
}

fox_status_t fox_attn_decode_fixed_gate_skip(fox_dtype_t dtype, const void* q, const void* k_cache,
                                    const void* v_cache, const float* gate_bias,
                                    const float* k_norm_max, void* o, float* lse, void* workspace,
                                    size_t workspace_bytes, int B, int H, int T, int d,
                                    float scale, hipStream_t stream) {
  if (!all_set({q, k_cache, v_cache, gate_bias, k_norm_max, o, lse})) return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, T, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (!all_aligned16({q, k_cache, v_cache, gate_bias, k_norm_max, o, lse})) return FOX_ERR_ALIGN;
  if (!workspace || workspace_bytes < fox::decode_workspace_bytes(B * H, T, d))
    return FOX_ERR_WORKSPACE;
  if (!aligned16(workspace)) return FOX_ERR_ALIGN;
  return launch_status(fox::launch_decode_fixed(dtype == FOX_DTYPE_BF16, q, k_cache, v_cache,
                                                gate_bias, H, o, lse, workspace, B * H, T, d,
                                                scale, static_cast<hipStream_t>(stream),
                                                k_norm_max));
}

// ---------------------------------------------------------------------------
// FoX (Pro) prologue and epilogue
// ---------------------------------------------------------------------------
fox_status_t fox_pro_prologue(fox_dtype_t dtype, const void* q_raw, const void* k_raw, const void* v_raw,
                     const float* k_shift_logit, const float* v_shift_logit,
                     const float* q_norm_weight, const float* k_norm_weight, float eps, void* q,
                     void* k, void* v, int B, int H, int L, int d, hipStream_t stream) {
  if (!all_set({q_raw, k_raw, v_raw, k_shift_logit, v_shift_logit, q_norm_weight, k_norm_weight,
                q, k, v}))
    return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, L, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (!valid_eps(eps)) return FOX_ERR_VALUE;
  if (!all_aligned16({q_raw, k_raw, v_raw, k_shift_logit, v_shift_logit, q_norm_weight,
                      k_norm_weight, q, k, v}))
    return FOX_ERR_ALIGN;
  return launch_status(fox::launch_pro_prologue(
      dtype == FOX_DTYPE_BF16, q_raw, k_raw, v_raw, k_shift_logit, v_shift_logit, q_norm_weight,
      k_norm_weight, eps, q, k, v, H, B * H, L, d, static_cast<hipStream_t>(stream)));
}

size_t fox_pro_prologue_bwd_workspace_bytes(fox_dtype_t dtype, int B, int H, int L, int d) {
  if (check_dims(B, H, L, d) || check_dtype_d(dtype, d)) return 0;
  return fox::pro_prologue_bwd_workspace_bytes(B * H, L, d);
}

fox_status_t fox_pro_prologue_bwd(fox_dtype_t dtype, const void* q_raw, const void* k_raw, const void* v_raw,
                         const float* k_shift_logit, const float* v_shift_logit,
                         const float* q_norm_weight, const float* k_norm_weight, float eps,
                         const void* dq, const void* dk, const void* dv, void* dq_raw,
                         void* dk_raw, void* dv_raw, float* dk_shift_logit,
                         float* dv_shift_logit, float* dq_norm_weight, float* dk_norm_weight,
                         void* workspace, size_t workspace_bytes, int B, int H, int L, int d,
                         hipStream_t stream) {
  if (!all_set({q_raw, k_raw, v_raw, k_shift_logit, v_shift_logit, q_norm_weight, k_norm_weight,
                dq, dk, dv, dq_raw, dk_raw, dv_raw, dk_shift_logit, dv_shift_logit,
                dq_norm_weight, dk_norm_weight}))
    return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, L, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (!valid_eps(eps)) return FOX_ERR_VALUE;
  if (!all_aligned16({q_raw, k_raw, v_raw, k_shift_logit, v_shift_logit, q_norm_weight,
                      k_norm_weight, dq, dk, dv, dq_raw, dk_raw, dv_raw, dk_shift_logit,
                      dv_shift_logit, dq_norm_weight, dk_norm_weight}))
    return FOX_ERR_ALIGN;
  if (!workspace || workspace_bytes < fox::pro_prologue_bwd_workspace_bytes(B * H, L, d))
    return FOX_ERR_WORKSPACE;
  if (!aligned16(workspace)) return FOX_ERR_ALIGN;
  return launch_status(fox::launch_pro_prologue_bwd(
      dtype == FOX_DTYPE_BF16, q_raw, k_raw, v_raw, k_shift_logit, v_shift_logit, q_norm_weight,
      k_norm_weight, eps, dq, dk, dv, dq_raw, dk_raw, dv_raw, dk_shift_logit, dv_shift_logit,
      dq_norm_weight, dk_norm_weight, workspace, H, B * H, L, d,
      static_cast<hipStream_t>(stream)));
}

fox_status_t fox_pro_output_gate(fox_dtype_t dtype, const void* o, const void* g_logit,
                        const float* o_norm_weight, float eps, void* y, int B, int H, int L,
                        int d, hipStream_t stream) {
  if (!all_set({o, g_logit, o_norm_weight, y})) return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, L, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (!valid_eps(eps)) return FOX_ERR_VALUE;
  if (!all_aligned16({o, g_logit, o_norm_weight, y})) return FOX_ERR_ALIGN;
  return launch_status(fox::launch_out_gate(dtype == FOX_DTYPE_BF16, o, g_logit, o_norm_weight,
                                            eps, y, H, B * H, L, d,
                                            static_cast<hipStream_t>(stream)));
}

fox_status_t fox_attn_fwd_pro(fox_dtype_t dtype, const void* q, const void* k, const void* v, const float* c,
                     const void* g_logit, const float* o_norm_weight, float eps, void* o,
                     float* lse, void* y, int B, int H, int L, int d, float scale, hipStream_t stream) {
  if (!all_set({q, k, v, c, g_logit, o_norm_weight, o, lse, y})) return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, L, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (!valid_eps(eps)) return FOX_ERR_VALUE;
  if (!all_aligned16({q, k, v, c, g_logit, o_norm_weight, o, lse, y})) return FOX_ERR_ALIGN;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (dtype == FOX_DTYPE_BF16)
    return launch_status(fox::launch_fwd_bf16_out_gate(q, k, v, c, o, lse, g_logit,
                                                       o_norm_weight, eps, y, H, B * H, L, d,
                                                       scale, s));
  hipError_t e = fox::launch_fwd_f32((const float*)q, (const float*)k, (const float*)v,
                                     fox::gate_array(c), (float*)o, lse, B * H, L, d, scale, s);
  if (e == hipSuccess)
    e = fox::launch_out_gate(false, o, g_logit, o_norm_weight, eps, y, H, B * H, L, d, s);
  return launch_status(e);
}

size_t fox_attn_bwd_pro_workspace_bytes(fox_dtype_t dtype, int B, int H, int L, int d) {
  if (check_dims(B, H, L, d) || check_dtype_d(dtype, d)) return 0;
  return fox::bwd_pro_workspace_bytes(dtype == FOX_DTYPE_BF16, B * H, L, d);
}

// fox_attn_bwd_pro and fox_attn_bwd_pro_stored: the same checks, the attention
// backward recomputing or keeping dS.
static fox_status_t attn_bwd_pro(bool keep_ds, fox_dtype_t dtype, const void* q, const void* k, const void* v,
                        const float* c, const void* o, const float* lse, const void* g_logit,
                        const float* o_norm_weight, float eps, const void* dy, void* dq,
                        void* dk, void* dv, float* d_log_f, void* dg_logit, float* do_norm_weight,
                        void* workspace, size_t workspace_bytes, int B, int H, int L, int d,
                        float scale, hipStream_t stream) {
  if (!all_set({q, k, v, c, o, lse, g_logit, o_norm_weight, dy, dq, dk, dv, d_log_f, dg_logit,
                do_norm_weight}))
    return FOX_ERR_NULL;
  fox_status_t st = check_dims(B, H, L, d);
  if (st) return st;
  st = check_dtype_d(dtype, d);
  if (st) return st;
  if (!valid_eps(eps)) return FOX_ERR_VALUE;
  if (!all_aligned16({q, k, v, c, o, lse, g_logit, o_norm_weight, dy, dq, dk, dv, d_log_f,
                      dg_logit, do_norm_weight}))
    return FOX_ERR_ALIGN;
  const bool bf = dtype == FOX_DTYPE_BF16;
  if (keep_ds && !bf) return FOX_ERR_UNSUPPORTED;
  const size_t need = keep_ds ? fox::bwd_pro_stored_workspace_bytes(B * H, L, d)
                              : fox::bwd_pro_workspace_bytes(bf, B * H, L, d);
  if (!workspace || workspace_bytes < need) return FOX_ERR_WORKSPACE;
  if (!aligned16(workspace)) return FOX_ERR_ALIGN;
  return launch_status(fox::launch_bwd_pro(bf, q, k, v, c, o, lse, g_logit, o_norm_weight, eps,
                                           dy, dq, dk, dv, d_log_f, dg_logit, do_norm_weight,
                                           workspace, H, B * H, L, d, scale,
                                           static_cast<hipStream_t>(stream), keep_ds));
}

fox_status_t fox_attn_bwd_pro(fox_dtype_t dtype, const void* q, const void* k, const void* v, const float* c,
                     const void* o, const float* lse, const void* g_logit,
                     const float* o_norm_weight, float eps, const void* dy, void* dq, void* dk,
                     void* dv, float* d_log_f, void* dg_logit, float* do_norm_weight,
                     void* workspace, size_t workspace_bytes, int B, int H, int L, int d,
                     float scale, hipStream_t stream) {
  return attn_bwd_pro(false, dtype, q, k, v, c, o, lse, g_logit, o_norm_weight, eps, dy, dq, dk,
                      dv, d_log_f, dg_logit, do_norm_weight, workspace, workspace_bytes, B, H, L,
                      d, scale, stream);
}

size_t fox_attn_bwd_pro_stored_workspace_bytes(fox_dtype_t dtype, int B, int H, int L, int d) {
  if (check_dims(B, H, L, d) || check_dtype_d(dtype, d) || dtype != FOX_DTYPE_BF16) return 0;
  return fox::bwd_pro_stored_workspace_bytes(B * H, L, d);
}

fox_status_t fox_attn_bwd_pro_stored(fox_dtype_t dtype, const void* q, const void* k, const void* v,
                            const float* c, const void* o, const float* lse, const void* g_logit,
                            const float* o_norm_weight, float eps, const void* dy, void* dq,
                            void* dk, void* dv, float* d_log_f, void* dg_logit,
                            float* do_norm_weight, void* workspace, size_t workspace_bytes, int B,
                            int H, int L, int d, float scale, hipStream_t stream) {
  return attn_bwd_pro(true, dtype, q, k, v, c, o, lse, g_logit, o_norm_weight, eps, dy, dq, dk,
                      dv, d_log_f, dg_logit, do_norm_weight, workspace, workspace_bytes, B, H, L,
                      d, scale, stream);
}

fox_status_t fox_gate_projection(fox_dtype_t dtype, const void* x, const float* w_f, const float* b_f,
                        float* gate_logit, int B, int L, int H, int M, hipStream_t stream) {
  if (!all_set({x, w_f, gate_logit})) return FOX_ERR_NULL;
  fox_status_t st = check_projection(dtype, B, L, H, M);
  if (st) return st;
  if (!all_aligned16({x, w_f, gate_logit})) return FOX_ERR_ALIGN;
  return launch_status(fox::launch_gate_proj_fwd(dtype == FOX_DTYPE_BF16, x, w_f, b_f, gate_logit,
                                                 B * L, L, H, M,
                                                 static_cast<hipStream_t>(stream)));
}

size_t fox_gate_projection_bwd_workspace_bytes(fox_dtype_t dtype, int B, int L, int H, int M) {
  if (check_projection(dtype, B, L, H, M)) return 0;
  return fox::gate_proj_bwd_workspace_bytes(B * L, H, M);
}

fox_status_t fox_gate_projection_bwd(fox_dtype_t dtype, const void* x, const float* w_f, const float* d_logit,
                            void* dx, float* dw_f, float* db_f, void* workspace,
                            size_t workspace_bytes, int B, int L, int H, int M, hipStream_t stream) {
  if (!all_set({x, w_f, d_logit, dw_f})) return FOX_ERR_NULL;
  fox_status_t st = check_projection(dtype, B, L, H, M);
  if (st) return st;
  if (!all_aligned16({x, w_f, d_logit, dw_f}) || (dx && !aligned16(dx))) return FOX_ERR_ALIGN;
  if (!workspace || workspace_bytes < fox::gate_proj_bwd_workspace_bytes(B * L, H, M))
    return FOX_ERR_WORKSPACE;
  if (!aligned16(workspace)) return FOX_ERR_ALIGN;
  return launch_status(fox::launch_gate_proj_bwd(dtype == FOX_DTYPE_BF16, x, w_f, d_logit, dx,
                                                 dw_f, db_f, workspace, B, L, H, M,
                                                 static_cast<hipStream_t>(stream)));
}

}  // extern "C"
