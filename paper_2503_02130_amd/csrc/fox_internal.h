// Host-side launchers shared between the C ABI and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>

namespace fox {

// The forget gates as the attention kernels see them: the prefix array c
// [BH, L] (data-dependent gates) or one bias per head, b [H] (fixed gates,
// f_t = sigmoid(b)); bh % H selects a row's head.
struct GateSpec {
  const float* ptr;
  bool fixed;
  int H;
};
inline GateSpec gate_array(const float* c) { return GateSpec{c, false, 1}; }
inline GateSpec gate_fixed(const float* bias, int H) { return GateSpec{bias, true, H}; }

// Inclusive prefix sums over rows of length L (one workgroup per row).
hipError_t launch_gate_prefix(const float* logit, float* log_f, float* c, int rows, int L,
                              hipStream_t s);
// out_l = sum_{i>=l} (a_i + b_i) per row: the chain rule through c = cumsum(log f).
hipError_t launch_reverse_scan_sum(const float* a, const float* b, float* out, int rows, int L,
                                   hipStream_t s);
// d(log f) (optional) and d(logit) = d(log f) * sigmoid(-logit) in one reverse scan.
hipError_t launch_reverse_scan_gate(const float* a, const float* b, const float* logit,
                                    float* d_log_f, float* d_logit, int rows, int L,
                                    hipStream_t s);

// q_norm_max / k_norm_max [BH] (both or neither): exact gate-aware skipping of
// key tiles whose contribution is an fp32 zero.
hipError_t launch_fwd_bf16(const void* q, const void* k, const void* v, GateSpec g, void* o,
                           float* lse, int BH, int L, int d, float scale, hipStream_t s,
                           const float* q_norm_max = nullptr, const float* k_norm_max = nullptr);
hipError_t launch_fwd_f32(const float* q, const float* k, const float* v, GateSpec g, float* o,
                          float* lse, int BH, int L, int d, float scale, hipStream_t s);

// Workspace layout of the backward: delta, dc_q, dc_k, each [BH, L] fp32.
size_t bwd_workspace_bytes(int BH, int L);
hipError_t launch_bwd_delta(bool bf16, const void* o, const void* d_o, float* delta, int BH,
                            int L, int d, hipStream_t s);
hipError_t launch_bwd_dkdv(bool bf16, const void* q, const void* k, const void* v, GateSpec g,
                           const float* lse, const void* d_o, const float* delta, void* dk,
                           void* dv, float* dck, int BH, int L, int d, float scale, hipStream_t s,
                           const float* q_norm_max = nullptr, const float* k_norm_max = nullptr);
hipError_t launch_bwd_dq(bool bf16, const void* q, const void* k, const void* v, GateSpec g,
                         const float* lse, const void* d_o, const float* delta, void* dq,
                         float* dcq, int BH, int L, int d, float scale, hipStream_t s,
                         const float* q_norm_max = nullptr, const float* k_norm_max = nullptr);
hipError_t launch_bwd(bool bf16, const void* q, const void* k, const void* v, const float* c,
                      const void* o, const float* lse, const void* d_o, void* dq, void* dk,
                      void* dv, float* d_log_f, void* ws, int BH, int L, int d, float scale,
                      hipStream_t s, const float* q_norm_max = nullptr,
                      const float* k_norm_max = nullptr);
// The backward that keeps dS (bf16 only): the workspace above, aligned to 256
// bytes, then the stored dS, 16 KB per (128-key block, 64-query tile) pair of
// the causal order and head.  The dK/dV pass writes it, the dQ pass reads it
// instead of recomputing S and dP.
// With skipping (q_norm_max / k_norm_max given) the dK/dV pass also records,
// after the stored dS, how many query tiles each key block stored, and the dQ
// pass reads only those.
size_t bwd_stored_workspace_bytes(int BH, int L);
size_t ds_store_bytes(int BH, int L);  // the stored dS alone
hipError_t launch_bwd_dkdv_store(const void* q, const void* k, const void* v, GateSpec g,
                                 const float* lse, const void* d_o, const float* delta, void* dk,
                                 void* dv, float* dck, void* ds_store, int* ds_tiles, int BH,
                                 int L, int d, float scale, hipStream_t s,
                                 const float* q_norm_max = nullptr,
                                 const float* k_norm_max = nullptr);
hipError_t launch_bwd_dq_stored(const void* k, const void* ds_store, const int* ds_tiles,
                                void* dq, float* dcq, int BH, int L, int d, float scale,
                                hipStream_t s);
hipError_t launch_bwd_stored(const void* q, const void* k, const void* v, const float* c,
                             const void* o, const float* lse, const void* d_o, void* dq, void* dk,
                             void* dv, float* d_log_f, void* ws, int BH, int L, int d, float scale,
                             hipStream_t s, const float* q_norm_max = nullptr,
                             const float* k_norm_max = nullptr);
// Fixed gates keeping dS: the fixed-gate workspace, aligned, then the stored tail.
size_t bwd_fixed_stored_workspace_bytes(int BH, int L);
hipError_t launch_bwd_fixed_stored(const void* q, const void* k, const void* v,
                                   const float* bias, int H, const void* o, const float* lse,
                                   const void* d_o, void* dq, void* dk, void* dv, float* d_bias,
                                   void* ws, int BH, int L, int d, float scale, hipStream_t s,
                                   const float* q_norm_max = nullptr,
                                   const float* k_norm_max = nullptr);
// Fixed gates: workspace delta, dc_q, dc_k, d(log f), each [BH, L] fp32; the bias
// gradient d_bias [H] (may be NULL) = sigmoid(-b) * sum over rows and t of d(log f).
size_t bwd_fixed_workspace_bytes(int BH, int L);
hipError_t launch_bwd_fixed(bool bf16, const void* q, const void* k, const void* v,
                            const float* bias, int H, const void* o, const float* lse,
                            const void* d_o, void* dq, void* dk, void* dv, float* d_bias, void* ws,
                            int BH, int L, int d, float scale, hipStream_t s,
                            const float* q_norm_max = nullptr, const float* k_norm_max = nullptr);

// out[bh] = max_t ||x[bh, t, :]||_2, enlarged by 2^-10 relative (an upper bound).
hipError_t launch_row_norm_max(bool bf16, const void* x, float* out, int BH, int L, int d,
                               hipStream_t s);

int decode_num_splits(int BH, int T);
size_t decode_workspace_bytes(int BH, int T, int d);
// the allocation-free decode: its split partials in a file-scope device array of
// this many bytes (per device); shapes needing more are rejected
constexpr size_t kDecodeScratchBytes = size_t(64) << 20;
hipError_t launch_decode_noalloc(bool bf16, const void* q, const void* k_cache,
                                 const void* v_cache, float* c_cache, const float* logit_new,
                                 void* o, float* lse, int BH, int T, int d, float scale,
                                 hipStream_t s);
hipError_t launch_decode(bool bf16, const void* q, const void* k_cache, const void* v_cache,
                         float* c_cache, const float* logit_new, void* o, float* lse, void* ws,
                         int BH, int T, int d, float scale, hipStream_t s);
// Exact gate-aware skipping (k_norm_max [BH] from launch_row_norm_max over the
// whole cache): a split whose every score lies more than 160 (base 2) below the
// new token's own score is not read; its merge weight would underflow to 0.
hipError_t launch_decode_skip(bool bf16, const void* q, const void* k_cache, const void* v_cache,
                              float* c_cache, const float* logit_new, const float* k_norm_max,
                              void* o, float* lse, void* ws, int BH, int T, int d, float scale,
                              hipStream_t s);
// Fixed gates: no prefix cache; bias [H]; with k_norm_max, exact skipping as above.
hipError_t launch_decode_fixed(bool bf16, const void* q, const void* k_cache, const void* v_cache,
                               const float* bias, int H, void* o, float* lse, void* ws, int BH,
                               int T, int d, float scale, hipStream_t s,
                               const float* k_norm_max = nullptr);

// FoX (Pro) prologue and epilogue (pro_fusions.hip).  Weights [H, d] fp32; shift
// logits [BH, L] fp32; everything else [BH, L, d] in the storage type.
int pro_chunks(int L);
size_t pro_prologue_bwd_workspace_bytes(int BH, int L, int d);
size_t bwd_pro_workspace_bytes(bool bf16, int BH, int L, int d);
hipError_t launch_pro_prologue(bool bf16, const void* qr, const void* kr, const void* vr,
                               const float* ka, const float* va, const float* wq,
                               const float* wk, float eps, void* q, void* k, void* v, int H,
                               int BH, int L, int d, hipStream_t s);
hipError_t launch_pro_prologue_bwd(bool bf16, const void* qr, const void* kr, const void* vr,
                                   const float* ka, const float* va, const float* wq,
                                   const float* wk, float eps, const void* dq, const void* dk,
                                   const void* dv, void* dqr, void* dkr, void* dvr, float* dka,
                                   float* dva, float* dwq, float* dwk, void* ws, int H, int BH,
                                   int L, int d, hipStream_t s);
hipError_t launch_out_gate(bool bf16, const void* o, const void* g, const float* wo, float eps,
                           void* y, int H, int BH, int L, int d, hipStream_t s);
// bf16 forward with the output norm and gate in its epilogue (writes O, LSE and y)
hipError_t launch_fwd_bf16_out_gate(const void* q, const void* k, const void* v, const float* c,
                                    void* o, float* lse, const void* g, const float* wo,
                                    float eps, void* y, int H, int BH, int L, int d, float scale,
                                    hipStream_t s);
// backward of attention + output norm and gate: the norm/gate backward writes dO
// and Delta into the workspace, then the attention backward stages run
// keep_ds (bf16 only): the attention backward keeps dS, in a workspace of
// bwd_pro_stored_workspace_bytes (the one above, aligned, then the stored dS).
size_t bwd_pro_stored_workspace_bytes(int BH, int L, int d);
hipError_t launch_bwd_pro(bool bf16, const void* q, const void* k, const void* v, const float* c,
                          const void* o, const float* lse, const void* g, const float* wo,
                          float eps, const void* dy, void* dq, void* dk, void* dv, float* d_log_f,
                          void* dg, float* dwo, void* ws, int H, int BH, int L, int d, float scale,
                          hipStream_t s, bool keep_ds = false);

// Forget-gate projection (gate_proj.hip): x [N = B L, M] (bf16 or fp32, M % 8 == 0),
// w_f [H, M] fp32 (H <= 64), bias [H] (may be NULL), logits [B, H, L] fp32.
int gate_proj_chunk_tokens(int N, int H, int M);
size_t gate_proj_bwd_workspace_bytes(int N, int H, int M);  // the dw_f partials
hipError_t launch_gate_proj_fwd(bool bf16, const void* x, const float* w, const float* bias,
                                float* logit, int N, int L, int H, int M, hipStream_t s);
// dx (may be NULL) in x's type; dw [H, M]; db [H] (may be NULL)
hipError_t launch_gate_proj_bwd(bool bf16, const void* x, const float* w, const float* d_logit,
                                void* dx, float* dw, float* db, void* ws, int B, int L, int H,
                                int M, hipStream_t s);

}  // namespace fox
