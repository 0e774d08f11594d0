/*
 * fox.h -- C ABI of the Forgetting Attention library for AMD Instinct MI355X (gfx950).
 *
 * Forgetting Attention (Forgetting Transformer, arXiv 2503.02130, Sec. 3,
 * Eq. fot-weight / fot-matrix) computes, for every (batch, head) slice,
 *
 *     o_i = sum_{j<=i} exp(s q_i.k_j + c_i - c_j) v_j / sum_{j<=i} exp(s q_i.k_j + c_i - c_j)
 *
 * with the forget gate f_t = sigmoid(logit_t), the prefix vector
 * c_i = sum_{l<=i} log f_l (inclusive), and the scale s (the paper always
 * scales q.k by 1/sqrt(d), footnote of Eq. attn-softmax; the scale multiplies
 * q.k only, never c_i - c_j).
 *
 * Conventions shared by every entry point
 *   - Layout: q, k, v, o, dO, dq, dk, dv are contiguous [B, H, L, d] (d innermost);
 *     gate logits, log f, c, lse, d(log f) are contiguous [B, H, L] fp32.  The
 *     decode cache is [B, H, T, d]; its prefix vector [B, H, T] fp32.
 *   - dtype: FOX_DTYPE_BF16 (bf16 storage, fp32 accumulation, MFMA) or
 *     FOX_DTYPE_F32 (fp32 storage and arithmetic).  Head dim d is 64 or 128.
 *   - Pointers are device pointers owned by the caller; every device pointer
 *     must be 16-byte aligned.  The library allocates no device memory and
 *     keeps no state between calls; workspaces are caller-provided and their
 *     contents are undefined on entry and exit.
 *   - stream is a hipStream_t (NULL = the default stream).  Every call only
 *     enqueues work on that stream and returns; the library never synchronises.
 *     Calls on different streams are independent.
 *   - Errors: arguments are validated on the host before anything is enqueued;
 *     a failed validation returns a non-zero fox_status_t and launches nothing.
 *     A failed kernel launch returns FOX_ERR_HIP.  Faults during execution
 *     surface at the caller's next synchronisation.
 *   - Causal only (the paper considers causal sequence modelling only, Sec. 2).
 *   - Gate logits must be finite (then log f is finite and c_i - c_j is defined).
 *   - Backward families: every backward (plain, exact skipping, fixed gates, FoX
 *     Pro) recomputes P in its dQ half within an O(B H L) workspace; its *_stored
 *     twin (bf16 only) keeps dS in an O(B H L^2) workspace instead, which is
 *     faster at long L and gives the same dK, dV bit for bit.
 */
#ifndef FOX_H_
#define FOX_H_

#include <stddef.h>

/* hipStream_t (the stream every entry point enqueues on) */
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FOX_DTYPE_F32 = 0,
  FOX_DTYPE_BF16 = 1,
  /* not a dtype: makes the enum as wide as an int, so that any int a caller
     passes is a representable value and is rejected by the range check */
  FOX_DTYPE_MAX_ENUM = 0x7FFFFFFF
} fox_dtype_t;

typedef enum {
  FOX_OK = 0,
  FOX_ERR_NULL = 1,         /* a required pointer is NULL                         */
  FOX_ERR_SHAPE = 2,        /* B, H, L (or T) not positive, or sizes overflow      */
  FOX_ERR_UNSUPPORTED = 3,  /* unsupported dtype or head dim                       */
  FOX_ERR_ALIGN = 4,        /* a pointer is not 16-byte aligned                    */
  FOX_ERR_WORKSPACE = 5,    /* workspace missing or smaller than required          */
  FOX_ERR_HIP = 6,          /* the HIP runtime reported an error at launch         */
  FOX_ERR_VALUE = 7,        /* a scalar argument out of range (eps: finite, >= 0)  */
  FOX_ERR_TOO_LARGE = 8,    /* the shape needs more scratch than the allocation-free
                               entry point holds                                   */
  FOX_STATUS_MAX_ENUM = 0x7FFFFFFF  /* not a status: keeps the enum int-sized        */
} fox_status_t;

/* Human-readable name of a status code.  Never returns NULL. */
const char* fox_status_string(fox_status_t status);

/* Library version as major*10000 + minor*100 + patch. */
int fox_version(void);

/*
 * Gate prelude (Sec. 3: f_t = sigmoid(w_f^T x_t + b_f); "Hardware-aware
 * implementation": c_i = sum_{l=1}^{i} log f_l, stored in HBM).
 *
 *   gate_logit [B,H,L] fp32 in   the pre-sigmoid gate logits x_t
 *   log_f      [B,H,L] fp32 out  log f_t = log sigmoid(x_t); may be NULL
 *   c          [B,H,L] fp32 out  inclusive prefix sum of log f along t
 */
fox_status_t fox_gate_prefix(const float* gate_logit, float* log_f, float* c,
                    int B, int H, int L, hipStream_t stream);

/*
 * Forward pass (Alg. 1 of the appendix "Hardware-aware implementation of
 * Forgetting Attention": O = softmax(s Q K^T + D) V with D_ij = c_i - c_j for
 * j <= i and -inf above the diagonal, plus the row logsumexp).
 *
 *   q, k, v [B,H,L,d] dtype in
 *   c       [B,H,L]   fp32  in   prefix vector from fox_gate_prefix
 *   o       [B,H,L,d] dtype out
 *   lse     [B,H,L]   fp32  out  natural-log logsumexp of row i of s Q K^T + D
 *   scale   the factor s on q.k (1/sqrt(d) in the paper)
 */
fox_status_t fox_attn_fwd(fox_dtype_t dtype, const void* q, const void* k, const void* v, const float* c,
                 void* o, float* lse, int B, int H, int L, int d, float scale, hipStream_t stream);

/* Bytes of workspace fox_attn_bwd needs for this shape (0 on invalid arguments). */
size_t fox_attn_bwd_workspace_bytes(fox_dtype_t dtype, int B, int H, int L, int d);

/*
 * Backward pass (Alg. 2 of the same appendix): the gradients of
 * sum(O o dO) with respect to q, k, v and log f.  The paper returns
 * dc = dc^q + dc^k (dc^q += rowsum(dS), dc^k -= colsum(dS)); this entry
 * point carries the chain rule through c = cumsum(log f) one step further:
 * d(log f)_l = sum_{i>=l} dc_i.
 *
 *   q, k, v, o, d_o  [B,H,L,d] dtype in  (o and lse from fox_attn_fwd)
 *   c                [B,H,L]   fp32  in
 *   lse              [B,H,L]   fp32  in
 *   dq, dk, dv       [B,H,L,d] dtype out (fully overwritten)
 *   d_log_f          [B,H,L]   fp32  out (fully overwritten)
 *   workspace        device buffer of at least fox_attn_bwd_workspace_bytes()
 */
fox_status_t fox_attn_bwd(fox_dtype_t dtype, const void* q, const void* k, const void* v, const float* c,
                 const void* o, const float* lse, const void* d_o,
                 void* dq, void* dk, void* dv, float* d_log_f,
                 void* workspace, size_t workspace_bytes,
                 int B, int H, int L, int d, float scale, hipStream_t stream);

/*
 * The same backward (Alg. 2) trading memory for the recomputation in the dQ
 * half: the dK/dV pass also writes the bf16 dS it forms, and the dQ pass reads
 * it instead of recomputing S, P and dP (dQ = s dS K, dc^q = rowsum(dS)).  The
 * workspace grows with L^2: 16 KB per (128-key block, 64-query tile) pair of the
 * causal order, per (b, h), plus 4 bytes per (b, h, key block): about B H L^2
 * bytes, 8.7 GB at B = 2, H = 16, L = 16384 (fox_attn_bwd needs 12 B H L bytes).  bf16 only (FOX_ERR_UNSUPPORTED
 * for fp32).  Arguments, outputs and errors as for fox_attn_bwd; the workspace is
 * at least fox_attn_bwd_stored_workspace_bytes() (0 for fp32 or invalid
 * arguments).  Results agree with fox_attn_bwd to rounding (the two dQ halves sum
 * the same bf16 dS in different orders); dc^q and dc^k remain the row and
 * column sums of one matrix.
 */
size_t fox_attn_bwd_stored_workspace_bytes(fox_dtype_t dtype, int B, int H, int L, int d);
fox_status_t fox_attn_bwd_stored(fox_dtype_t dtype, const void* q, const void* k, const void* v, const float* c,
                        const void* o, const float* lse, const void* d_o,
                        void* dq, void* dk, void* dv, float* d_log_f,
                        void* workspace, size_t workspace_bytes,
                        int B, int H, int L, int d, float scale, hipStream_t stream);

/*
 * fox_attn_bwd_stored in stages: it is exactly
 *     fox_attn_bwd_delta -> fox_attn_bwd_dkdv_store -> fox_attn_bwd_dq_stored
 *     -> fox_dlogf_from_dc
 * with delta, dc_q, dc_k and the stored dS carved from its workspace.
 *
 * fox_attn_bwd_ds_store_bytes: bytes of the stored dS (0 for fp32 or invalid
 *   arguments).
 * fox_attn_bwd_dkdv_store: fox_attn_bwd_dkdv (same arguments and outputs, bit for
 *   bit the same dK, dV, dc_k) that also writes dS, bf16, into ds_store (device,
 *   at least fox_attn_bwd_ds_store_bytes(), 16-byte aligned; caller-owned, layout
 *   private to the library, fully rewritten where the dQ stage reads it).
 * fox_attn_bwd_dq_stored: dQ (overwritten) and dc_q = rowsum(dS) [B,H,L] fp32
 *   (overwritten) from k [B,H,L,d] and the ds_store written by
 *   fox_attn_bwd_dkdv_store for the same shape.
 * bf16 only: FOX_ERR_UNSUPPORTED for fp32.
 */
size_t fox_attn_bwd_ds_store_bytes(fox_dtype_t dtype, int B, int H, int L, int d);
fox_status_t fox_attn_bwd_dkdv_store(fox_dtype_t dtype, const void* q, const void* k, const void* v,
                            const float* c, const float* lse, const void* d_o,
                            const float* delta, void* dk, void* dv, float* dc_k,
                            void* ds_store, size_t ds_store_bytes,
                            int B, int H, int L, int d, float scale, hipStream_t stream);
fox_status_t fox_attn_bwd_dq_stored(fox_dtype_t dtype, const void* k, const void* ds_store, size_t ds_store_bytes,
                           void* dq, float* dc_q, int B, int H, int L, int d, float scale,
                           hipStream_t stream);

/*
 * The backward pass in stages, for callers that schedule them themselves (for
 * instance dK/dV and dQ on two streams).  fox_attn_bwd is exactly
 *     fox_attn_bwd_delta -> fox_attn_bwd_dkdv -> fox_attn_bwd_dq -> fox_dlogf_from_dc
 * with delta, dc_q and dc_k carved from its workspace.
 *
 * fox_attn_bwd_delta: delta_i = sum_d dO_id O_id (Alg. 2, the preprocessing
 *   rowsum(dO o O), one value per row).  o, d_o [B,H,L,d] dtype; delta [B,H,L] fp32 out.
 * fox_attn_bwd_dkdv: dK, dV (dtype, overwritten) and dc_k = -colsum(dS) [B,H,L]
 *   fp32 (overwritten), the key-side half of Alg. 2.
 * fox_attn_bwd_dq: dQ (dtype, overwritten) and dc_q = rowsum(dS) [B,H,L] fp32
 *   (overwritten), the query-side half of Alg. 2.
 * fox_dlogf_from_dc: d(log f)_l = sum_{i>=l} (dc_q_i + dc_k_i), the chain rule
 *   through c = cumsum(log f) (Alg. 2 returns dc = dc^q + dc^k); [B,H,L] fp32.
 * Both halves form P and dS from the same expression (bf16 dtype: P rounded to
 * bf16 before dS = P o (dP - delta), and dc summed over dS rounded to bf16, the
 * values the dQ and dK products take), so that dc_q and dc_k are the row and
 * column sums of one matrix and sum(dc) = d(log f)_1 = 0 holds to fp32 rounding.
 * Inputs as for fox_attn_bwd.
 */
fox_status_t fox_attn_bwd_delta(fox_dtype_t dtype, const void* o, const void* d_o, float* delta,
                       int B, int H, int L, int d, hipStream_t stream);
fox_status_t fox_attn_bwd_dkdv(fox_dtype_t dtype, const void* q, const void* k, const void* v, const float* c,
                      const float* lse, const void* d_o, const float* delta,
                      void* dk, void* dv, float* dc_k,
                      int B, int H, int L, int d, float scale, hipStream_t stream);
fox_status_t fox_attn_bwd_dq(fox_dtype_t dtype, const void* q, const void* k, const void* v, const float* c,
                    const float* lse, const void* d_o, const float* delta,
                    void* dq, float* dc_q,
                    int B, int H, int L, int d, float scale, hipStream_t stream);
fox_status_t fox_dlogf_from_dc(const float* dc_q, const float* dc_k, float* d_log_f,
                      int B, int H, int L, hipStream_t stream);

/*
 * Gate backward (Sec. 3: f_t = sigmoid(x_t), so d log f_t / d x_t = 1 - f_t =
 * sigmoid(-x_t)), fused into the reverse scan of fox_dlogf_from_dc:
 *     d(log f)_l = sum_{i>=l} (dc_q_i + dc_k_i),   d x_l = d(log f)_l * sigmoid(-x_l).
 *
 *   dc_q, dc_k  [B,H,L] fp32 in   from fox_attn_bwd_dq / fox_attn_bwd_dkdv
 *   gate_logit  [B,H,L] fp32 in   the logits x_t given to fox_gate_prefix
 *   d_log_f     [B,H,L] fp32 out  may be NULL
 *   d_logit     [B,H,L] fp32 out  the gradient with respect to the gate logits
 */
fox_status_t fox_dlogit_from_dc(const float* dc_q, const float* dc_k, const float* gate_logit,
                       float* d_log_f, float* d_logit, int B, int H, int L, hipStream_t stream);

/* Bytes of workspace fox_attn_decode needs for this shape (0 on invalid arguments). */
size_t fox_attn_decode_workspace_bytes(fox_dtype_t dtype, int B, int H, int T, int d);

/*
 * One decode step: Eq. fot-weight evaluated for the last position i = T of a
 * sequence whose keys/values 1..T sit in a cache (the paper's outlook mentions
 * KV caches, Sec. 6).  The new token attends to every cached key including
 * itself.
 *
 *   q              [B,H,d]   dtype in   query of the new token
 *   k_cache,v_cache[B,H,T,d] dtype in   slot T-1 already holds the new token's k, v
 *   c_cache        [B,H,T]   fp32 in/out  entries 0..T-2 are read (c_1..c_{T-1});
 *                                       entry T-1 is written with
 *                                       c_T = c_{T-1} + log sigmoid(gate_logit_new)
 *                                       (c_0 = 0 when T = 1) and never read
 *   gate_logit_new [B,H]     fp32 in
 *   o              [B,H,d]   dtype out
 *   lse            [B,H]     fp32 out  natural-log logsumexp of the new row
 *   workspace      device buffer of at least fox_attn_decode_workspace_bytes()
 */
fox_status_t fox_attn_decode(fox_dtype_t dtype, const void* q, const void* k_cache, const void* v_cache,
                    float* c_cache, const float* gate_logit_new, void* o, float* lse,
                    void* workspace, size_t workspace_bytes,
                    int B, int H, int T, int d, float scale, hipStream_t stream);

/*
 * fox_attn_decode for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation.  It takes
 * no workspace; the split partials live in a file-scope device array of 64 MiB
 * that the library holds on every device it runs on until the process ends.  No
 * call allocates or frees anything (the array's device address is looked up once
 * per device, on the first call with that device current).
 *
 *   Arguments, outputs and results as for fox_attn_decode (bit for bit: the same
 *   kernels, the same split plan).
 *   Limit: shapes whose partials exceed the array, i.e. whenever
 *   fox_attn_decode_workspace_bytes() > 64 MiB (for example B*H = 1024 heads at
 *   d = 128 with T above 129024), return FOX_ERR_TOO_LARGE and launch nothing.
 *   Calls that overlap on one device (different streams, or host threads) share
 *   the array and race: serialise them.  Each call overwrites every partial it
 *   reads, so nothing carries over from an earlier call.
 */
fox_status_t fox_attn_decode_noalloc(fox_dtype_t dtype, const void* q, const void* k_cache,
                                     const void* v_cache, float* c_cache,
                                     const float* gate_logit_new, void* o, float* lse,
                                     int B, int H, int T, int d, float scale, hipStream_t stream);

/*
 * Gate-aware exact skipping (the paper's outlook, Sec. 6: forget gates could
 * prune computation).  D_ij = c_i - c_j <= 0 falls monotonically with the
 * distance i - j, and s q.k <= s ||q|| ||k||, so a whole block of keys can be
 * shown to contribute an exact fp32 zero.  Such blocks are not read; the
 * results are bit for bit those of the entry points without skipping.
 *
 * fox_row_norm_max: out[b,h] = max_t ||x[b,h,t,:]||_2 (fp32 [B,H]), enlarged by
 *   2^-10 relative so that it bounds the exact norm.  x [B,H,L,d] dtype.
 * fox_attn_decode_skip: fox_attn_decode with k_norm_max [B,H] fp32, an upper
 *   bound of ||k_j|| over the whole cache (fox_row_norm_max over k_cache, or
 *   maintained as keys are appended: max(old, ||k_new||)).  A split of keys is
 *   skipped when all its scores lie more than 160 (base 2) below the new
 *   token's own score, which makes its merge weight an exact zero.
 */
/*
 * fox_attn_fwd_skip / fox_attn_bwd_skip: fox_attn_fwd / fox_attn_bwd with
 *   q_norm_max, k_norm_max [B,H] fp32 (fox_row_norm_max of q and k).  With
 *   Qmax, Kmax the bounds, P_ij < exp(2 s Qmax Kmax + c_i - c_j) relative to the
 *   row maximum (forward) or exp(-LSE_i) (backward), so a tile pair whose
 *   closest query/key pair puts this below 2^-160 is skipped.  bf16 only; the
 *   fp32 path runs dense.  Workspace as fox_attn_bwd.
 */
fox_status_t fox_row_norm_max(fox_dtype_t dtype, const void* x, float* out, int B, int H, int L, int d,
                     hipStream_t stream);
fox_status_t fox_attn_fwd_skip(fox_dtype_t dtype, const void* q, const void* k, const void* v, const float* c,
                      const float* q_norm_max, const float* k_norm_max, void* o, float* lse,
                      int B, int H, int L, int d, float scale, hipStream_t stream);
fox_status_t fox_attn_bwd_skip(fox_dtype_t dtype, const void* q, const void* k, const void* v, const float* c,
                      const void* o, const float* lse, const void* d_o, const float* q_norm_max,
                      const float* k_norm_max, void* dq, void* dk, void* dv, float* d_log_f,
                      void* workspace, size_t workspace_bytes, int B, int H, int L, int d,
                      float scale, hipStream_t stream);
/* fox_attn_bwd_skip keeping dS (as fox_attn_bwd_stored; bf16 only): the dK/dV pass
 * stores the dS of the tiles it computes and the dQ pass reads only those.  Workspace:
 * at least fox_attn_bwd_stored_workspace_bytes().  Results are bitwise those of
 * fox_attn_bwd_stored. */
fox_status_t fox_attn_bwd_skip_stored(fox_dtype_t dtype, const void* q, const void* k, const void* v,
                             const float* c, const void* o, const float* lse, const void* d_o,
                             const float* q_norm_max, const float* k_norm_max, void* dq, void* dk,
                             void* dv, float* d_log_f, void* workspace, size_t workspace_bytes,
                             int B, int H, int L, int d, float scale, hipStream_t stream);
fox_status_t fox_attn_decode_skip(fox_dtype_t dtype, const void* q, const void* k_cache, const void* v_cache,
                         float* c_cache, const float* gate_logit_new, const float* k_norm_max,
                         void* o, float* lse, void* workspace, size_t workspace_bytes, int B,
                         int H, int T, int d, float scale, hipStream_t stream);

/*
 * Fixed (data-independent) forget gates: f_t^(h) = sigmoid(b^(h)) for every t
 * (Sec. 3, "Connection to ALiBi": ALiBi with slope -log sigmoid(b^(h))).  The
 * kernels form c_i - c_j = (i - j) log sigmoid(b^(h)) from the positions, so no
 * prefix array exists; everything else is as in the entry points above.
 *
 * fox_fixed_gate_init: the appendix "Data-independent forget gate
 *   initialization": with T(b) = 1 / (-log sigmoid(b)), head h = 0..H-1 gets
 *   T(b^(h)) = exp(log T_min + (log T_max - log T_min) h / (H - 1)) (H = 1: T_min).
 *   gate_bias is HOST memory [H] fp32 (out).  Requires 0 < t_min <= t_max.
 *   No device work.
 * fox_attn_fwd_fixed_gate: O, LSE as fox_attn_fwd; gate_bias [H] fp32 device.
 * fox_attn_bwd_fixed_gate: dq, dk, dv as fox_attn_bwd, and the gradient of the
 *   biases d_gate_bias [H] fp32 (may be NULL for a gate that is not trained):
 *   d b^(h) = sigmoid(-b^(h)) * sum over batch and t of d(log f)_t^(h).
 *   workspace: at least fox_attn_bwd_fixed_gate_workspace_bytes().
 * fox_attn_decode_fixed_gate: one decode step as fox_attn_decode, without a
 *   prefix cache; workspace: fox_attn_decode_workspace_bytes().
 */
fox_status_t fox_fixed_gate_init(float* gate_bias, int H, float t_min, float t_max);
fox_status_t fox_attn_fwd_fixed_gate(fox_dtype_t dtype, const void* q, const void* k, const void* v,
                            const float* gate_bias, void* o, float* lse, int B, int H, int L, int d,
                            float scale, hipStream_t stream);
size_t fox_attn_bwd_fixed_gate_workspace_bytes(fox_dtype_t dtype, int B, int H, int L, int d);
fox_status_t fox_attn_bwd_fixed_gate(fox_dtype_t dtype, const void* q, const void* k, const void* v,
                            const float* gate_bias, const void* o, const float* lse,
                            const void* d_o, void* dq, void* dk, void* dv, float* d_gate_bias,
                            void* workspace, size_t workspace_bytes, int B, int H, int L, int d,
                            float scale, hipStream_t stream);
/* fox_attn_bwd_fixed_gate keeping dS (as fox_attn_bwd_stored; bf16 only), and
 * fox_attn_bwd_fixed_gate_skip keeping dS (bitwise the results of
 * fox_attn_bwd_fixed_gate_stored).  Workspace: at least
 * fox_attn_bwd_fixed_gate_stored_workspace_bytes() (0 for fp32 or invalid
 * arguments), about B H L^2 bytes.  dK and dV are bit for bit those of
 * fox_attn_bwd_fixed_gate; dQ and the bias gradient agree to rounding. */
size_t fox_attn_bwd_fixed_gate_stored_workspace_bytes(fox_dtype_t dtype, int B, int H, int L, int d);
fox_status_t fox_attn_bwd_fixed_gate_stored(fox_dtype_t dtype, const void* q, const void* k, const void* v,
                                   const float* gate_bias, const void* o, const float* lse,
                                   const void* d_o, void* dq, void* dk, void* dv,
                                   float* d_gate_bias, void* workspace, size_t workspace_bytes,
                                   int B, int H, int L, int d, float scale, hipStream_t stream);
fox_status_t fox_attn_bwd_fixed_gate_skip_stored(fox_dtype_t dtype, const void* q, const void* k, const void* v,
                                        const float* gate_bias, const void* o, const float* lse,
                                        const void* d_o, const float* q_norm_max,
                                        const float* k_norm_max, void* dq, void* dk, void* dv,
                                        float* d_gate_bias, void* workspace,
                                        size_t workspace_bytes, int B, int H, int L, int d,
                                        float scale, hipStream_t stream);
fox_status_t fox_attn_decode_fixed_gate(fox_dtype_t dtype, const void* q, const void* k_cache,
                               const void* v_cache, const float* gate_bias, void* o, float* lse,
                               void* workspace, size_t workspace_bytes, int B, int H, int T, int d,
                               float scale, hipStream_t stream);

/*
 * Fixed gates with exact gate-aware skipping: the entry points above with the
 * row-norm bounds of fox_attn_fwd_skip / fox_attn_bwd_skip / fox_attn_decode_skip
 * (q_norm_max, k_norm_max [B,H] fp32 from fox_row_norm_max; the decode needs
 * only k_norm_max over the cache).  c_i - c_j = (i - j) log sigmoid(b^(h)) makes
 * the decay of a tile pair a function of its distance alone, so a strongly
 * forgetting head keeps only a band of tiles near the diagonal.  The results are
 * bit for bit those of the fixed-gate entry points without skipping.  The forward
 * and backward skip in bf16 (fp32 runs dense); the decode skips in both dtypes.
 * Workspaces as the entry points without skipping.
 */
fox_status_t fox_attn_fwd_fixed_gate_skip(fox_dtype_t dtype, const void* q, const void* k, const void* v,
                                 const float* gate_bias, const float* q_norm_max,
                                 const float* k_norm_max, void* o, float* lse, int B, int H, int L,
                                 int d, float scale, hipStream_t stream);
fox_status_t fox_attn_bwd_fixed_gate_skip(fox_dtype_t dtype, const void* q, const void* k, const void* v,
                                 const float* gate_bias, const void* o, const float* lse,
                                 const void* d_o, const float* q_norm_max,
                                 const float* k_norm_max, void* dq, void* dk, void* dv,
                                 float* d_gate_bias, void* workspace, size_t workspace_bytes,
                                 int B, int H, int L, int d, float scale, hipStream_t stream);
fox_status_t fox_attn_decode_fixed_gate_skip(fox_dtype_t dtype, const void* q, const void* k_cache,
                                    const void* v_cache, const float* gate_bias,
                                    const float* k_norm_max, void* o, float* lse, void* workspace,
                                    size_t workspace_bytes, int B, int H, int T, int d,
                                    float scale, hipStream_t stream);

/*
 * FoX (Pro) prologue and epilogue (Sec. 3 "Architecture design", Eq. shift-linear;
 * appendix "Detailed FoX (Pro) layer computation").  Per head h and time t, from
 * the raw projections q~ = W_q x, k~ = W_k x, v~ = W_v x (already split into
 * heads, [B,H,L,d] in dtype) and the shift logits w_k^T x_t, w_v^T x_t ([B,H,L]
 * fp32, one per head and token):
 *     q_t = RMSNorm_q(q~_t)
 *     k_t = RMSNorm_k(a_t k~_{t-1} + (1 - a_t) k~_t),   a_t = sigmoid(k_shift_logit_t)
 *     v_t = b_t v~_{t-1} + (1 - b_t) v~_t,              b_t = sigmoid(v_shift_logit_t)
 * with k~_0 = v~_0 = 0 (the first token mixes with zeros), and after the attention
 *     y_t = RMSNorm_o(o_t) o sigmoid(g_t),   g = W_g x ([B,H,L,d] in dtype).
 * RMSNorm(x) = x / sqrt(mean over d of x^2 + eps) * w^(h), with per-head weights
 * [H,d] fp32 (a weight shared by all heads, as in the paper's runs, is H equal
 * rows).  eps must be finite and >= 0 (else FOX_ERR_VALUE).  The projections
 * and W_o are ordinary matrix products and not part of this library.  Outputs
 * must not alias inputs (rows t - 1 and t + 1 are read while row t is written).
 *
 * fox_pro_prologue: q, k, v for the attention entry points.
 * fox_pro_prologue_bwd: from dq, dk, dv (of the attention backward) the
 *   gradients of the raw projections (dtype), of the shift logits ([B,H,L]
 *   fp32) and of the QK-norm weights ([H,d] fp32, summed over batch and time).
 *   workspace: at least fox_pro_prologue_bwd_workspace_bytes().
 * fox_pro_output_gate: y from an attention output o (standalone epilogue).
 * fox_attn_fwd_pro: fox_attn_fwd followed by the output norm and gate: writes
 *   o and lse (the backward needs them) and y.  bf16 applies the norm and gate
 *   in the attention kernel's epilogue, to o as rounded to bf16; fp32 runs the
 *   standalone epilogue kernel after the attention.
 * fox_attn_bwd_pro: gradients of sum(y o dy): dq, dk, dv, d_log_f as
 *   fox_attn_bwd, the gate-logit gradient dg_logit (dtype, [B,H,L,d]) and the
 *   output-norm weight gradient do_norm_weight ([H,d] fp32).  The norm/gate
 *   backward also forms dO (rounded to dtype) and Delta_i = rowsum(dO o O) for
 *   the attention backward, in the workspace: at least
 *   fox_attn_bwd_pro_workspace_bytes().
 */
fox_status_t fox_pro_prologue(fox_dtype_t dtype, const void* q_raw, const void* k_raw, const void* v_raw,
                     const float* k_shift_logit, const float* v_shift_logit,
                     const float* q_norm_weight, const float* k_norm_weight, float eps, void* q,
                     void* k, void* v, int B, int H, int L, int d, hipStream_t stream);
size_t fox_pro_prologue_bwd_workspace_bytes(fox_dtype_t dtype, int B, int H, int L, int d);
fox_status_t fox_pro_prologue_bwd(fox_dtype_t dtype, const void* q_raw, const void* k_raw, const void* v_raw,
                         const float* k_shift_logit, const float* v_shift_logit,
                         const float* q_norm_weight, const float* k_norm_weight, float eps,
                         const void* dq, const void* dk, const void* dv, void* dq_raw,
                         void* dk_raw, void* dv_raw, float* dk_shift_logit,
                         float* dv_shift_logit, float* dq_norm_weight, float* dk_norm_weight,
                         void* workspace, size_t workspace_bytes, int B, int H, int L, int d,
                         hipStream_t stream);
fox_status_t fox_pro_output_gate(fox_dtype_t dtype, const void* o, const void* g_logit,
                        const float* o_norm_weight, float eps, void* y, int B, int H, int L,
                        int d, hipStream_t stream);
fox_status_t fox_attn_fwd_pro(fox_dtype_t dtype, const void* q, const void* k, const void* v, const float* c,
                     const void* g_logit, const float* o_norm_weight, float eps, void* o,
                     float* lse, void* y, int B, int H, int L, int d, float scale, hipStream_t stream);
size_t fox_attn_bwd_pro_workspace_bytes(fox_dtype_t dtype, int B, int H, int L, int d);
fox_status_t fox_attn_bwd_pro(fox_dtype_t dtype, const void* q, const void* k, const void* v, const float* c,
                     const void* o, const float* lse, const void* g_logit,
                     const float* o_norm_weight, float eps, const void* dy, void* dq, void* dk,
                     void* dv, float* d_log_f, void* dg_logit, float* do_norm_weight,
                     void* workspace, size_t workspace_bytes, int B, int H, int L, int d,
                     float scale, hipStream_t stream);

/*
 * fox_attn_bwd_pro with the attention backward keeping dS, as
 * fox_attn_bwd_stored does: bf16 only (FOX_ERR_UNSUPPORTED for fp32); the
 * workspace is at least fox_attn_bwd_pro_stored_workspace_bytes() (0 for fp32
 * or invalid arguments), about B H L^2 bytes.  Arguments, outputs and errors
 * otherwise as for fox_attn_bwd_pro; dK, dV and the gate and norm-weight
 * gradients are bit for bit the same, dQ and d(log f) agree to rounding.
 */
size_t fox_attn_bwd_pro_stored_workspace_bytes(fox_dtype_t dtype, int B, int H, int L, int d);
fox_status_t fox_attn_bwd_pro_stored(fox_dtype_t dtype, const void* q, const void* k, const void* v,
                            const float* c, const void* o, const float* lse, const void* g_logit,
                            const float* o_norm_weight, float eps, const void* dy, void* dq,
                            void* dk, void* dv, float* d_log_f, void* dg_logit,
                            float* do_norm_weight, void* workspace, size_t workspace_bytes,
                            int B, int H, int L, int d, float scale, hipStream_t stream);

/*
 * The forget-gate projection (Sec. 3, gate definition: f_t = sigmoid(w_f^T x_t
 * + b_f), one w_f and b_f per head): the logits that fox_gate_prefix and
 * fox_dlogit_from_dc take, from the layer input.
 *
 *   x          [B,L,M] dtype in   layer input, M contiguous; M a multiple of 8
 *   w_f        [H,M]   fp32  in   one weight row per head (H <= 64)
 *   b_f        [H]     fp32  in   per-head bias; may be NULL (no bias)
 *   gate_logit [B,H,L] fp32  out  gate_logit[b,h,t] = w_f[h] . x[b,t] + b_f[h]
 *
 * The products run on bf16 MFMA with fp32 accumulation; fp32 operands enter as
 * a pair of bf16 (hi + lo, within 2^-16 relative), so each product is within
 * 4 * 2^-16 of exact and the result close to an fp32 dot product (measured
 * relative L2 error near 2e-6 for either dtype).  Values must be finite and below 3.38e38 in
 * magnitude (the bf16 range).  H > 64 or M % 8 != 0: FOX_ERR_UNSUPPORTED.
 */
fox_status_t fox_gate_projection(fox_dtype_t dtype, const void* x, const float* w_f, const float* b_f,
                        float* gate_logit, int B, int L, int H, int M, hipStream_t stream);

/* Bytes of workspace fox_gate_projection_bwd needs (0 on invalid arguments). */
size_t fox_gate_projection_bwd_workspace_bytes(fox_dtype_t dtype, int B, int L, int H, int M);

/*
 * Backward of fox_gate_projection: the gradients of sum(gate_logit * d_logit).
 *
 *   x, w_f     as for fox_gate_projection                     in
 *   d_logit    [B,H,L] fp32  in   e.g. from fox_dlogit_from_dc
 *   dx         [B,L,M] dtype out  sum_h d_logit[b,h,t] w_f[h]; may be NULL (not needed)
 *   dw_f       [H,M]   fp32  out  sum_{b,t} d_logit[b,h,t] x[b,t] (overwritten, not accumulated)
 *   db_f       [H]     fp32  out  sum_{b,t} d_logit[b,h,t]; may be NULL
 *   workspace  device buffer of at least fox_gate_projection_bwd_workspace_bytes()
 *              (per-chunk partials of dw_f, summed in a fixed order: results are
 *              deterministic)
 */
fox_status_t fox_gate_projection_bwd(fox_dtype_t dtype, const void* x, const float* w_f, const float* d_logit,
                            void* dx, float* dw_f, float* db_f, void* workspace,
                            size_t workspace_bytes, int B, int L, int H, int M, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* FOX_H_ */
