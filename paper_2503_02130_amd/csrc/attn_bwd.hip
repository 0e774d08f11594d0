// Forgetting Attention backward pass (appendix, Alg. 2).
//
// With P = exp(S - LSE) recomputed from the saved logsumexp,
//     dV = P^T dO,  dP = dO V^T,  dS = P o (dP - Delta),  Delta_i = rowsum(dO_i o O_i),
//     dQ = s dS K,  dK = s dS^T Q,  dc^q_i = rowsum_i(dS),  dc^k_j = -colsum_j(dS),
// and d(log f)_l = sum_{i>=l} (dc^q_i + dc^k_i), the chain rule through
// c = cumsum(log f).  The paper computes dK, dV, dc^k and dQ, dc^q in two kernels;
// this file does the same, which keeps every accumulation in one workgroup's
// registers (no atomics, deterministic results):
//
//   delta kernel   Delta_i from the stored O (bf16 or fp32) and dO.
//   dq kernel      query-stationary: 32 queries per wave; S^T = K Q^T and
//                  dP^T = V dO^T on MFMA, dS^T in registers, dQ^T += K^T dS^T with
//                  K^T taken from the row-major LDS tile by transposing reads;
//                  dc^q from in-register row sums.
//   dkdv kernel    key-stationary: 32 keys per wave; S = Q K^T and dP = dO V^T,
//                  then dV^T += dO^T P and dK^T += Q^T dS, the transposed
//                  operands again by transposing reads; dc^k from in-register sums.
//   reverse scan   (gate_scan.hip) turns dc^q + dc^k into d(log f).
//
// The backward that keeps dS replaces the dq kernel: the dkdv kernel's STORE
// instantiation also writes the bf16 dS it forms, and the stored-dS dq kernel
// streams it from HBM (dQ^T += K^T dS^T, dc^q = rowsum) instead of recomputing
// S, P and dP.
//
// The forget-gate bias is formed relative to c_ref (the first query of the
// block for dq, the first key of the block for dkdv), exactly as in the forward:
//     log2 P_ij = s log2(e) q_i.k_j + log2(e) ((c_i - c_ref) - LSE_i) - log2(e) (c_j - c_ref).
#include <cstddef>
#include <type_traits>

#include "fox_device.h"
#include "fox_internal.h"

namespace fox {

size_t bwd_workspace_bytes(int BH, int L) { return (size_t)3 * BH * (size_t)L * sizeof(float); }

// ---------------------------------------------------------------------------
// Delta_i = sum_d dO_id * O_id.  LPR lanes share a row, one 16-byte piece of O
// and of dO each; a lane group takes kDeltaRows rows (one workgroup pass apart)
// and issues all of their loads before it reduces any (rows past the end load
// the last row and store nothing).  Each row's sum has the same order for any
// kDeltaRows.
// ---------------------------------------------------------------------------
constexpr int kDeltaRows = 4;
template <typename T, int D>
__global__ __launch_bounds__(256) void bwd_delta_kernel(const T* __restrict__ O,
                                                        const T* __restrict__ dO,
                                                        float* __restrict__ delta, size_t rows) {
  constexpr int VEC = 16 / sizeof(T);
  constexpr int LPR = D / VEC;     // lanes per row
  constexpr int RPP = 256 / LPR;   // rows per workgroup pass
  typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
  const int part = threadIdx.x % LPR;
  const size_t row0 = (size_t)blockIdx.x * (RPP * kDeltaRows) + threadIdx.x / LPR;
  u32x4_t ov[kDeltaRows], gv[kDeltaRows];
#pragma unroll
  for (int r = 0; r < kDeltaRows; ++r) {
    const size_t row = min(row0 + (size_t)r * RPP, rows - 1);
    ov[r] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(O + row * D + part * VEC));
    gv[r] = *reinterpret_cast<const u32x4_t*>(dO + row * D + part * VEC);
  }
#pragma unroll
  for (int r = 0; r < kDeltaRows; ++r) {
    const size_t row = row0 + (size_t)r * RPP;
    T o[VEC], g[VEC];
    __builtin_memcpy(o, &ov[r], 16);
    __builtin_memcpy(g, &gv[r], 16);
    float acc = 0.0f;
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc += (float)o[e] * (float)g[e];
#pragma unroll
    for (int off = 1; off < LPR; off <<= 1) acc += __shfl_xor(acc, off);
    if (row < rows && part == 0) delta[row] = acc;
  }
}

// ---------------------------------------------------------------------------
// bf16 dq kernel: 128 queries per workgroup (4 waves x 32), 64-key tiles
// double-buffered in LDS through DMA loads, diagonal tile first.  The tile loop
// is unrolled by two so every LDS address is a per-lane base plus an immediate.
// ---------------------------------------------------------------------------
constexpr int kBwdThreads = 256;
constexpr int kDqWaves = 4;
constexpr int kDqBM = 32 * kDqWaves;
constexpr int kDqBN = 64;
// Both backward kernels form P from the same expression, so that their bf16
// roundings of P agree bit for bit and dc^q, dc^k are the row and column sums of
// one matrix: the bias is taken relative to the prefix value at the start of the
// key's aligned block of kRefBlock keys, the query's part
// ((c_i - c_ref) - LSE_i) / s seeds the S accumulator, the key's part
// (c_j - c_ref) log2(e) is subtracted in the exponent.
constexpr int kRefBlock = 128;
// Gate-aware skipping: with Qmax, Kmax bounding the row norms, every
// P_ij = exp(s q_i.k_j + c_i - c_j - LSE_i) is below exp(2 s Qmax Kmax + c_i - c_j)
// (LSE_i >= s q_i.k_i >= -s Qmax Kmax).  A (query tile, key tile) pair whose
// closest query and key give log2 of that bound below -kSkipMargin produces an
// exact fp32 zero everywhere (150 for the underflow, 10 for the rounding of the
// bound), and since c falls along the sequence so do all pairs further apart:
// the tile loops stop there, bit for bit as without skipping.
constexpr float kSkipMargin = 160.0f;

// ---------------------------------------------------------------------------
// Stored dS, for the backward that keeps dS instead of recomputing it in the
// dQ pass.  For each (b, h), one 16 KB slot per pair (128-key block nb, 64-query
// tile qt) that the causal order reaches (qt >= 2 nb), block-major.  A slot
// holds the bf16 dS of the block's keys and the tile's queries in the register
// layout of the dK/dV kernel's G waves: [32-key pair 4][32-query half qb 2]
// [16-query chunk c 2][lane 64][8 bf16], where lane = 32 h + the key within the
// pair and element 4 g2 + jj is query 16 c + 8 g2 + 4 h + jj of the half.
// ---------------------------------------------------------------------------
constexpr int kDsSlotBytes = 16384;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
__host__ __device__ inline int ds_query_tiles(int L) { return (L + 63) / 64; }
__host__ __device__ inline int ds_key_blocks(int L) { return (L + 127) / 128; }
__host__ __device__ inline size_t ds_slots_per_head(int L) {
  const size_t nq = (size_t)ds_query_tiles(L), nk = (size_t)ds_key_blocks(L);
  return nk * nq - nk * (nk - 1);
}
// slot of (key block nb, query tile qt >= 2 nb) within its head
__host__ __device__ inline size_t ds_slot(int L, int nb, int qt) {
  return (size_t)nb * (size_t)ds_query_tiles(L) - (size_t)nb * (size_t)(nb - 1) +
         (size_t)(qt - 2 * nb);
}
static_assert(kRefBlock % kDqBN == 0, "a dq key tile lies in one reference block");

template <int D>
struct DqSmem {
  bf16 k[2][kDqBN * D];
  bf16 v[2][kDqBN * D];
  float c[2][kDqBN];
  float cref[2];  // the tile's reference prefix value
  int skip[2];    // the tile and every earlier one contribute exact zeros
};

// Occupancy: two waves per SIMD at D = 128; three at D = 64 (168 VGPRs; measured
// 11 % faster than two).
template <int D, bool FIXED, bool SKIP>
__global__ __launch_bounds__(kBwdThreads) __attribute__((amdgpu_waves_per_eu(D == 64 ? 3 : 2)))
void bwd_dq_bf16_kernel(const bf16* __restrict__ Q, const bf16* __restrict__ K,
                        const bf16* __restrict__ V, const float* __restrict__ gate,
                        const float* __restrict__ qnorm, const float* __restrict__ knorm,
                        const float* __restrict__ LSE, const bf16* __restrict__ dO,
                        const float* __restrict__ delta, bf16* __restrict__ dQ,
                        float* __restrict__ dcq, int BH, int H, int L, int n_mblk, float scale,
                        float scale_log2) {
  constexpr int TILE = kDqBN * D;
  constexpr int NDMA = TILE * 2 / 1024 / kDqWaves;
  __shared__ __attribute__((aligned(16))) DqSmem<D> sm;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = lane >> 5, col = lane & 31;
  // heads fastest; rotated over the XCDs when skipping (see the forward kernel)
  const int row = (int)(blockIdx.x / BH);
  const int bh = SKIP ? (int)((blockIdx.x + row) % BH) : (int)(blockIdx.x % BH);
  const int mblk = n_mblk - 1 - row;
  const int q0 = mblk * kDqBM;
  const size_t head = (size_t)bh * (size_t)L;
  const GateRow<FIXED> gr(gate, bh, H, head);
  const int qw0 = q0 + wave * 32;
  const int qi = qw0 + col;
  const bool q_valid = qi < L;
  const uint32_t head_bytes = (uint32_t)L * D * 2;
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(K + head * D, head_bytes);
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(V + head * D, head_bytes);
  const uint32_t dma_off = tile_dma_offset<D, kDqWaves>(wave, lane);
  int roff[D / 16];
  tile_row_offsets<D>(roff, col, h);
  int toff[2][D / 32];
  tile_tr_offsets<D>(toff, lane);

  bf16x8 qf[D / 16], dof[D / 16];
#pragma unroll
  for (int s = 0; s < D / 16; ++s) {
    if (q_valid) {
      qf[s] = *reinterpret_cast<const bf16x8*>(Q + (head + qi) * D + 16 * s + 8 * h);
      dof[s] = *reinterpret_cast<const bf16x8*>(dO + (head + qi) * D + 16 * s + 8 * h);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        qf[s][e] = to_bf16(0.0f);
        dof[s][e] = to_bf16(0.0f);
      }
    }
  }
  float cq = 0.0f;  // c_i itself (prefix array only)
  if constexpr (!FIXED) cq = q_valid ? gr.c[qi] : 0.0f;
  const float lse_q = q_valid ? LSE[head + qi] : 0.0f;
  const float dlt = q_valid ? delta[head + qi] : 0.0f;

  f32x16 dqacc[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) dqacc[db][r] = 0.0f;
  float dcq_part = 0.0f;

  const int kend = min(L, q0 + kDqBM);
  const int t_last = (kend + kDqBN - 1) / kDqBN - 1;
  const int t_diag = qw0 / kDqBN;

  const float inv_scale = 1.0f / scale;
  const float skip_norm = SKIP ? 2.0f * scale * qnorm[bh] * knorm[bh] : 0.0f;
  // Wave 0 loads the next tile's prefix values (one key per lane, and the
  // tile's reference value) before its share of the tile DMA and turns them
  // into the LDS row terms only after the current tile's body: memory
  // operations complete in order, so a wait for them issued right away, or
  // for loads issued after the DMA, would also wait for the DMA.
  const float c_q0 = gr.raw(q0);
  float craw = 0.0f, crefreg = 0.0f;
  auto issue_tile = [&](int kt, auto bufc) {
    constexpr int B = decltype(bufc)::value;
    const uint32_t base = (uint32_t)kt * kDqBN * D * 2;
    if (wave == 0) {
      const int key = kt * kDqBN + lane;
      crefreg = gr.raw(kt * kDqBN / kRefBlock * kRefBlock);
      craw = key < L ? gr.raw(key) : 0.0f;
    }
#pragma unroll
    for (int i = 0; i < NDMA; ++i) {
      const int wslot = (i * kDqWaves + wave) * 512;
      const uint32_t voff = dma_off + uniform_u32(base + i * tile_dma_stride<kDqWaves>());
      dma16(rk, &sm.k[B][wslot], voff);
      dma16(rv, &sm.v[B][wslot], voff);
    }
  };
  auto store_c = [&](int kt, auto bufc) {
    constexpr int B = decltype(bufc)::value;
    if (wave == 0) {
      const int key = kt * kDqBN + lane;
      const int kref = kt * kDqBN / kRefBlock * kRefBlock;
      sm.c[B][lane] = key < L ? gr.diff_raw(key, craw, kref, crefreg) * kLog2e : INFINITY;
      if (lane == 0) sm.cref[B] = crefreg;
      // the tile's last key against the block's first query
      if (SKIP && lane == kDqBN - 1)
        sm.skip[B] = key < L && kLog2e * (skip_norm + gr.diff_raw(q0, c_q0, key, craw)) < -kSkipMargin;
    }
  };

  // LDS operand addresses: a few opaque per-lane registers plus immediates.
  // Reads through them (and the transposing reads in assembly) are not taken
  // for possible readers of the tile that is loading by DMA meanwhile, so the
  // compiler adds no wait for that DMA before them; they only ever read the
  // other buffer.  The V tiles sit at a fixed distance from the K tiles.
  constexpr int kVOff = 2 * 2 * TILE;  // bytes from sm.k[0] to sm.v[0]
  static_assert(offsetof(DqSmem<D>, v) - offsetof(DqSmem<D>, k) == (size_t)kVOff,
                "V tiles follow the K tiles");
  const lds_byte* ka_at[D / 16];
#pragma unroll
  for (int s = 0; s < D / 16; ++s) ka_at[s] = lds_opaque(lds_ptr(&sm.k[0][0]) + 2 * roff[s]);
  uint32_t taddr[2][D / 32];
#pragma unroll
  for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
      taddr[k2][db] = (uint32_t)(uintptr_t)lds_opaque(lds_ptr(&sm.k[0][0]) + 2 * toff[k2][db]);
  const lds_byte* c_at = lds_opaque(lds_ptr(&sm.c[0][4 * h]));
  const lds_byte* cref_at = lds_opaque(lds_ptr(&sm.cref[0]));

  auto tile_body = [&](int j, auto bufc, auto masked) {
    constexpr int B = decltype(bufc)::value;
    constexpr bool MASK = decltype(masked)::value;
    const int key0 = j * kDqBN;
    const float dref = FIXED ? gr.diff(qi, key0 / kRefBlock * kRefBlock)
                             : cq - *(const lds_f32_t*)(cref_at + 4 * B);
    const float bq = q_valid ? (dref - lse_q) * inv_scale : -INFINITY;
    static_for<2>([&](auto kbc) {
      constexpr int kb = decltype(kbc)::value;
      f32x16 sacc, pacc;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        sacc[r] = bq;
        pacc[r] = 0.0f;
      }
      {
        bf16x8 ka[D / 16];
#pragma unroll
        for (int s = 0; s < D / 16; ++s)
          ka[s] = *(const lds_bf16x8_t*)(ka_at[s] + 2 * (B * TILE + kb * 32 * D));
        sched_fence();
#pragma unroll
        for (int s = 0; s < D / 16; ++s) sacc = mfma32(ka[s], qf[s], sacc);
      }
      {
        bf16x8 va[D / 16];
#pragma unroll
        for (int s = 0; s < D / 16; ++s)
          va[s] = *(const lds_bf16x8_t*)(ka_at[s] + kVOff + 2 * (B * TILE + kb * 32 * D));
        sched_fence();
#pragma unroll
        for (int s = 0; s < D / 16; ++s) pacc = mfma32(va[s], dof[s], pacc);
      }
      float pv[16];
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 ck4 = *(const lds_f32x4_t*)(c_at + 4 * (B * kDqBN + kb * 32 + 8 * g));
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          float p = exp2_fast(sacc[4 * g + jj] * scale_log2 - ck4[jj]);
          if (MASK && key0 + kb * 32 + 8 * g + 4 * h + jj > qi) p = 0.0f;
          pv[4 * g + jj] = p;
        }
      }
      // P rounded to bf16 exactly as the dkdv kernel sees it
#pragma unroll
      for (int r = 0; r < 16; r += 2) round_bf16_pair(pv[r], pv[r + 1]);
      float dsv[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        dsv[r] = pv[r] * (pacc[r] - dlt);
      }
      static_for<2>([&](auto cc) {
        constexpr int c = decltype(cc)::value;
        constexpr int OFF = 2 * (B * TILE + (2 * kb + c) * 16 * D);
        const bf16x8 dsb = pack8(&dsv[8 * c]);
        // dc^q and dc^k sum the bf16 dS the products use: row and column sums of one matrix
        dcq_part = sum8_bf16(dsb, dcq_part);
        bf16x4 t[2 * (D / 32)];
        static_for<D / 32>([&](auto dbc) {
          constexpr int db = decltype(dbc)::value;
          t[2 * db] = ds_read_tr_asm<OFF>(taddr[0][db]);
          t[2 * db + 1] = ds_read_tr_asm<OFF>(taddr[1][db]);
        });
        lds_wait<0>(t);
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
          dqacc[db] = mfma32(cat4(t[2 * db], t[2 * db + 1]), dsb, dqacc[db]);
      });
    });
  };

  // returns true when tile j and all earlier tiles can be skipped
  auto step = [&](int j, auto bufc) {
    constexpr int B = decltype(bufc)::value;
    wait_all_memory();
    __syncthreads();  // tile j is in LDS; every wave is done with tile j + 1
    if (SKIP && sm.skip[B]) return true;
    if (j > 0) issue_tile(j - 1, std::integral_constant<int, 1 - B>());
    if (j == t_diag) {
      tile_body(j, bufc, std::true_type());
    } else if (j < t_diag) {
      tile_body(j, bufc, std::false_type());
    }
    if (j > 0) store_c(j - 1, std::integral_constant<int, 1 - B>());
    return false;
  };

  issue_tile(t_last, std::integral_constant<int, 0>());
  store_c(t_last, std::integral_constant<int, 0>());
  for (int j = t_last; j >= 0; j -= 2) {
    if (step(j, std::integral_constant<int, 0>())) break;
    if (j > 0 && step(j - 1, std::integral_constant<int, 1>())) break;
  }

  const float dcq_tot = wave_sum_pair(dcq_part);
  if (q_valid) {
    bf16* out = dQ + (head + qi) * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        bf16x4 w;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) w[jj] = to_bf16(dqacc[db][4 * g + jj] * scale);
        *reinterpret_cast<bf16x4*>(out + db * 32 + 8 * g + 4 * h) = w;
      }
    }
    if (h == 0) dcq[head + qi] = dcq_tot;
  }
}

// ---------------------------------------------------------------------------
// bf16 dkdv kernel, split into two wave roles.  Eight waves per workgroup own
// 128 keys as four pairs of 32; both waves of a pair run on the same SIMD.
//   P wave (waves 0-3): K rows in registers; for query tile t computes
//          S = Q K^T, P = exp(S - LSE) with the gate bias and the mask, stores P
//          (bf16) in LDS, and accumulates dV^T += dO^T P.
//   G wave (waves 4-7): V rows in registers; one tile behind, for tile t - 1
//          computes dP = dO V^T, reads P back, dS = P o (dP - Delta),
//          dc^k -= colsum(dS) and accumulates dK^T += Q^T dS.
// Each wave holds one D x 32 accumulator, so two waves fit on a SIMD, and the
// two roles never wait for each other inside a tile: Q / dO tiles, their row
// statistics and P are triple-buffered (tile t + 1 loads by DMA while P works
// on t and G on t - 1), with one barrier per tile of 64 queries.  The P waves
// issue all of the DMA, so the G waves never wait for vector memory.  Every LDS
// operand address is one of a few opaque per-lane registers plus an immediate:
// plain reads come from the tile the role multiplies from the left (Q for P,
// dO for G) and transposing reads from the other one, so both roles share the
// same sixteen address registers, and the loop is unrolled by three so the
// buffer index is part of the immediate.
// ---------------------------------------------------------------------------
constexpr int kKvWaves = 8;
constexpr int kKvThreads = 64 * kKvWaves;
constexpr int kKvPairs = kKvWaves / 2;
constexpr int kKvBN = 32 * kKvPairs;  // keys per workgroup
static_assert(kKvBN == kRefBlock, "a dkdv workgroup's keys form one reference block");
template <int D>
constexpr int kv_bm() { return 64; }  // queries per tile

template <int D>
struct KvSmem {
  static constexpr int BM = kv_bm<D>();
  bf16 q[3][BM * D];
  bf16 g[3][BM * D];
  bf16x8 p[3][kKvPairs][BM / 16][64];  // P of each pair: [16-query chunk][lane], bf16 x 8
  float bq[3][BM];  // ((c_i - c_ref) - LSE_i) / s of each query row
  float dl[3][BM];  // Delta_i
  float raw[2][3][BM];  // c_i, LSE_i, Delta_i of the next tiles as loaded (two tiles ahead)
  int skip[3];          // the query tile and every later one contribute exact zeros
};

template <int D, bool FIXED, bool SKIP, bool STORE = false>
__global__ __launch_bounds__(kKvThreads) void bwd_dkdv_bf16_kernel(
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V,
    const float* __restrict__ gate, const float* __restrict__ qnorm,
    const float* __restrict__ knorm, const float* __restrict__ LSE, const bf16* __restrict__ dO,
    const float* __restrict__ delta, bf16* __restrict__ dK, bf16* __restrict__ dV,
    float* __restrict__ dck, bf16x8* __restrict__ ds_store, int* __restrict__ ds_tiles, int BH,
    int H, int L, float scale, float scale_log2) {
  static_assert(!STORE || (kv_bm<D>() == 64 && kKvBN == 128 && kKvPairs == 4),
                "the stored-dS slot layout");
  constexpr int kKvBM = kv_bm<D>();
  constexpr int NQB = kKvBM / 32;  // 32-query sub-blocks per tile
  constexpr int TILE = kKvBM * D;
  constexpr int NDMA = TILE * 2 / 1024 / kKvWaves;
  static_assert(NDMA >= 1 && 2 * NDMA * kKvPairs * 1024 == TILE * 2,
                "the P waves' DMA loads cover a tile exactly");
  __shared__ __attribute__((aligned(16))) KvSmem<D> sm;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = lane >> 5, col = lane & 31;
  const bool pwave = wave < kKvPairs;  // role
  const int pair = wave % kKvPairs;
  const int nblk = (int)(blockIdx.x / BH);  // key block 0 has the most work: first
  // heads fastest; rotated over the XCDs when skipping (see the forward kernel)
  const int bh = SKIP ? (int)((blockIdx.x + nblk) % BH) : (int)(blockIdx.x % BH);
  const int k0 = nblk * kKvBN;
  const size_t head = (size_t)bh * (size_t)L;
  const GateRow<FIXED> gr(gate, bh, H, head);  // reference: c at k0
  const float* Lh = LSE + head;
  const float* Dh = delta + head;
  const int kw0 = k0 + pair * 32;
  const int kj = kw0 + col;
  const bool k_valid = kj < L;
  const uint32_t head_bytes = (uint32_t)L * D * 2;
  const __amdgpu_buffer_rsrc_t rq = make_rsrc(Q + head * D, head_bytes);
  const __amdgpu_buffer_rsrc_t rg = make_rsrc(dO + head * D, head_bytes);
  const uint32_t dma_off = tile_dma_offset<D, kKvPairs>(pair, lane);
  int roff[D / 16];
  tile_row_offsets<D>(roff, col, h);
  int toff[2][D / 32];
  tile_tr_offsets<D>(toff, lane);
  const lds_byte* plain_base = pwave ? lds_ptr(&sm.q[0][0]) : lds_ptr(&sm.g[0][0]);
  const lds_byte* tr_base = pwave ? lds_ptr(&sm.g[0][0]) : lds_ptr(&sm.q[0][0]);
  const lds_byte* pa[D / 16];
#pragma unroll
  for (int s = 0; s < D / 16; ++s) pa[s] = lds_opaque(plain_base + 2 * roff[s]);
  const lds_byte* ta_[2][D / 32];
#pragma unroll
  for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
    for (int db = 0; db < D / 32; ++db) ta_[k2][db] = lds_opaque(tr_base + 2 * toff[k2][db]);
  const lds_byte* p_at = lds_opaque(lds_ptr(&sm.p[0][pair][0][lane]));
  const lds_byte* row_at = lds_opaque(lds_ptr(&sm.bq[0][4 * h]));
  constexpr int kPBuf = kKvPairs * (kKvBM / 16) * 64 * 16;  // bytes of one P buffer
  constexpr int kDlOff = 3 * kKvBM * 4;                      // bytes from bq to dl
  // plain operand s of 32-row block qb of buffer B; transposing operand of
  // 16-row chunk ch, head-dim block db
  auto plain_op = [&](int s, int boff) { return *(const lds_bf16x8_t*)(pa[s] + boff); };
  uint32_t taddr[2][D / 32];  // the same as 32-bit addresses for the assembly reads
#pragma unroll
  for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
    for (int db = 0; db < D / 32; ++db) taddr[k2][db] = (uint32_t)(uintptr_t)ta_[k2][db];
  constexpr int NR = 2 * (D / 32);  // transposing reads per 16-query chunk
  // transposing operands of 16-query chunk CH of buffer B, read by inline assembly
  auto read_tr = [&](auto bufc, auto chc, bf16x4 (&t)[NR]) {
    constexpr int OFF = 2 * (decltype(bufc)::value * TILE + decltype(chc)::value * 16 * D);
    static_for<D / 32>([&](auto dbc) {
      constexpr int DB = decltype(dbc)::value;
      t[2 * DB] = ds_read_tr_asm<OFF>(taddr[0][DB]);
      t[2 * DB + 1] = ds_read_tr_asm<OFF>(taddr[1][DB]);
    });
  };

  // P waves hold K rows, G waves hold V rows
  bf16x8 kvf[D / 16];
  {
    const bf16* src = (pwave ? K : V) + (head + kj) * D;
#pragma unroll
    for (int s = 0; s < D / 16; ++s) {
      if (k_valid) {
        kvf[s] = *reinterpret_cast<const bf16x8*>(src + 16 * s + 8 * h);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) kvf[s][e] = to_bf16(0.0f);
      }
    }
  }
  const float ck2 = k_valid ? gr.diff(kj, k0) * kLog2e : INFINITY;

  f32x16 acc[D / 32];  // dV^T (P waves) or dK^T (G waves)
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[db][r] = 0.0f;
  float dck_part = 0.0f;

  const int t_first = k0 / kKvBM;
  int n_tiles = (L + kKvBM - 1) / kKvBM - t_first;  // lowered by gate-aware skipping
  const float skip_norm = SKIP ? 2.0f * scale * qnorm[bh] * knorm[bh] : 0.0f;
  const int k_last = min(L, k0 + kKvBN) - 1;  // the block's least decayed key
  const int t_diag = kw0 / kKvBM;  // tile holding this pair's diagonal

  // per query row of a tile: ((c_i - c_ref) - LSE_i) / s and Delta_i
  const float inv_scale = 1.0f / scale;
  // The rows' c, LSE and Delta reach LDS by DMA two tiles ahead (wave 0, one
  // row per lane; rows past L read as zero), and wave 0 converts them
  // LDS to LDS one tile ahead: no register holds them across a tile and no
  // wait for them ever waits for a tile's DMA.
  const float c_k0 = gr.raw(k0), c_klast = gr.raw(k_last);
  const __amdgpu_buffer_rsrc_t rsc = make_rsrc(FIXED ? Lh : gate + head, (uint32_t)L * 4);
  const __amdgpu_buffer_rsrc_t rsl = make_rsrc(Lh, (uint32_t)L * 4);
  const __amdgpu_buffer_rsrc_t rsd = make_rsrc(Dh, (uint32_t)L * 4);
  auto issue_stats = [&](int qt, int rb) {
    if (wave == 0) {
      const uint32_t off = ((uint32_t)qt * kKvBM + lane) * 4;
      if constexpr (!FIXED) dma4(rsc, &sm.raw[rb][0][0], off);
      dma4(rsl, &sm.raw[rb][1][0], off);
      dma4(rsd, &sm.raw[rb][2][0], off);
    }
  };
  auto convert_stats = [&](int qt, int rb, auto bufc) {
    constexpr int B = decltype(bufc)::value;
    if (wave == 0 && lane < kKvBM) {
      const int qq = qt * kKvBM + lane;
      const float cr = FIXED ? 0.0f : sm.raw[rb][0][lane];
      sm.bq[B][lane] = qq < L ? (gr.diff_raw(qq, cr, k0, c_k0) - sm.raw[rb][1][lane]) * inv_scale
                              : -INFINITY;
      sm.dl[B][lane] = qq < L ? sm.raw[rb][2][lane] : 0.0f;
      // the tile's first query against the block's last key
      if (SKIP && lane == 0)
        sm.skip[B] = kLog2e * (skip_norm + gr.diff_raw(qq, cr, k_last, c_klast)) < -kSkipMargin;
    }
  };
  auto issue_tile = [&](int qt, auto bufc) {
    constexpr int B = decltype(bufc)::value;
    const uint32_t base = (uint32_t)qt * kKvBM * D * 2;
    if (pwave) {
#pragma unroll
      for (int i = 0; i < 2 * NDMA; ++i) {
        const int wslot = (i * kKvPairs + pair) * 512;
        const uint32_t voff = dma_off + uniform_u32(base + i * tile_dma_stride<kKvPairs>());
        dma16(rq, &sm.q[B][wslot], voff);
        dma16(rg, &sm.g[B][wslot], voff);
      }
    }
  };

  // P wave on tile qt held in buffer B
  auto p_tile = [&](int qt, auto bufc, auto masked) {
    constexpr int B = decltype(bufc)::value;
    constexpr bool MASK = decltype(masked)::value;
    const int qs0 = qt * kKvBM;
    static_for<NQB>([&](auto qbc) {
      constexpr int qb = decltype(qbc)::value;
      bf16x8 qa[D / 16];
#pragma unroll
      for (int s = 0; s < D / 16; ++s)
        qa[s] = plain_op(s, 2 * (B * TILE + qb * 32 * D));
      // the accumulator starts at the query's row term divided by s
      f32x16 sacc;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 bq4 = *(const lds_f32x4_t*)(row_at + 4 * (B * kKvBM + qb * 32 + 8 * g));
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) sacc[4 * g + jj] = bq4[jj];
      }
#pragma unroll
      for (int s = 0; s < D / 16; ++s) sacc = mfma32(qa[s], kvf[s], sacc);
      // the dO^T operands of the first chunk load while P is formed (the
      // skipping kernel, short of registers, reads them just before use)
      bf16x4 tr[NR];
      if constexpr (!SKIP) read_tr(bufc, std::integral_constant<int, 2 * qb>(), tr);
      float pv[16];
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int ql = qb * 32 + 8 * g + 4 * h;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          float p = exp2_fast(sacc[4 * g + jj] * scale_log2 - ck2);
          if (MASK && kj > qs0 + ql + jj) p = 0.0f;
          pv[4 * g + jj] = p;
        }
      }
      static_for<2>([&](auto cc) {
        constexpr int c = decltype(cc)::value;
        const bf16x8 pb = pack8(&pv[8 * c]);
        *(lds_bf16x8_t*)(p_at + B * kPBuf + (2 * qb + c) * 1024) = pb;
        if constexpr (SKIP) read_tr(bufc, std::integral_constant<int, 2 * qb + c>(), tr);
        lds_wait<SKIP ? 0 : 1>(tr);  // the store may stay in flight
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
          acc[db] = mfma32(cat4(tr[2 * db], tr[2 * db + 1]), pb, acc[db]);
        if constexpr (!SKIP && c == 0) read_tr(bufc, std::integral_constant<int, 2 * qb + 1>(), tr);
      });
    });
  };
  // STORE: the G waves also write their bf16 dS, as packed for the dK MFMA, to
  // this block's run of stored slots (16 KB per 64-query tile, from tile t_first
  // on), for the dQ pass; non-temporal stores, the reader comes after the kernel.
  const __amdgpu_buffer_rsrc_t rds = make_rsrc(
      STORE ? ds_store + ((size_t)bh * ds_slots_per_head(L) + ds_slot(L, nblk, t_first)) *
                             (kDsSlotBytes / 16)
            : ds_store,
      STORE ? (uint32_t)(ds_query_tiles(L) - t_first) * kDsSlotBytes : 0u);
  const int lane16 = lane * 16;
  // G wave on tile qt held in buffer B (its P was stored in the same buffer slot)
  auto g_tile = [&](int qt, auto bufc) {
    constexpr int B = decltype(bufc)::value;
    static_for<NQB>([&](auto qbc) {
      constexpr int qb = decltype(qbc)::value;
      bf16x8 ga[D / 16];
#pragma unroll
      for (int s = 0; s < D / 16; ++s)
        ga[s] = plain_op(s, 2 * (B * TILE + qb * 32 * D));
      f32x16 pacc;
#pragma unroll
      for (int r = 0; r < 16; ++r) pacc[r] = 0.0f;
#pragma unroll
      for (int s = 0; s < D / 16; ++s) pacc = mfma32(ga[s], kvf[s], pacc);
      // the Q^T operands of the first chunk load while dS is formed
      bf16x4 tr[NR];
      if constexpr (!SKIP) read_tr(bufc, std::integral_constant<int, 2 * qb>(), tr);
      static_for<2>([&](auto cc) {
        constexpr int c = decltype(cc)::value;
        const bf16x8 pb = *(const lds_bf16x8_t*)(p_at + B * kPBuf + (2 * qb + c) * 1024);
        float dsv[8];
#pragma unroll
        for (int g2 = 0; g2 < 2; ++g2) {
          const f32x4 dl4 = *(const lds_f32x4_t*)(row_at + kDlOff + 4 * (B * kKvBM + qb * 32 + 8 * (2 * c + g2)));
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) {
            dsv[4 * g2 + jj] = to_f32(pb[4 * g2 + jj]) * (pacc[8 * c + 4 * g2 + jj] - dl4[jj]);
          }
        }
        const bf16x8 dsb = pack8(dsv);
        dck_part = sum8_bf16(dsb, dck_part);  // the column sums of the bf16 dS (see the dq kernel)
        if constexpr (STORE)
          __builtin_amdgcn_raw_buffer_store_b128(
              __builtin_bit_cast(u32x4, dsb), rds, lane16,
              (int)uniform_u32((uint32_t)(qt - t_first) * kDsSlotBytes + (uint32_t)pair * 4096u) +
                  (2 * qb + c) * 1024,
              kNonTemporal);
        if constexpr (SKIP) read_tr(bufc, std::integral_constant<int, 2 * qb + c>(), tr);
        lds_wait<0>(tr);
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
          acc[db] = mfma32(cat4(tr[2 * db], tr[2 * db + 1]), dsb, acc[db]);
        if constexpr (!SKIP && c == 0) read_tr(bufc, std::integral_constant<int, 2 * qb + 1>(), tr);
      });
    });
  };

  // iteration it: the P wave works on tile it (buffer it % 3), the G wave on tile
  // it - 1 (buffer (it - 1) % 3), and tile it + 1 loads into buffer (it + 1) % 3
  auto step = [&](int it, auto bufc) {
    constexpr int B = decltype(bufc)::value;
    constexpr int BN = (B + 1) % 3, BP = (B + 2) % 3;
    // The P waves issue every DMA of the loop and wait for it here; the G waves
    // wait for their LDS operations only (with the stored-dS backward their
    // vector memory counter also counts their dS stores, which need no wait).
    if (pwave) wait_all_memory();
    else wait_lds();
    __syncthreads();  // tile it and P of tile it - 1 are in LDS
    // tile it and all later ones add exact zeros: the G waves finish tile it - 1
    if (SKIP && it < n_tiles && sm.skip[B]) n_tiles = it;
    if (it + 1 < n_tiles) issue_tile(t_first + it + 1, std::integral_constant<int, BN>());
    if (it + 2 < n_tiles) issue_stats(t_first + it + 2, it & 1);
    if (pwave) {
      const int qt = t_first + it;
      if (it < n_tiles) {
        if (qt == t_diag) p_tile(qt, bufc, std::true_type());
        else if (qt > t_diag) p_tile(qt, bufc, std::false_type());
      }
    } else {
      const int qt = t_first + it - 1;
      if (it >= 1 && it <= n_tiles && qt >= t_diag) g_tile(qt, std::integral_constant<int, BP>());
    }
    if (it + 1 < n_tiles) convert_stats(t_first + it + 1, (it + 1) & 1, std::integral_constant<int, BN>());
  };

  issue_stats(t_first, 0);
  if (1 < n_tiles) issue_stats(t_first + 1, 1);
  issue_tile(t_first, std::integral_constant<int, 0>());
  wait_all_memory();  // wave 0's own DMA of the first tile's rows
  convert_stats(t_first, 0, std::integral_constant<int, 0>());
  // the three steps run unconditionally (a step past the last tile only meets
  // the barrier): with steps skipped by branches the accumulators were copied
  // at the loop's back edge, about 20 VALU instructions per P-wave tile
  for (int it = 0; it <= n_tiles; it += 3) {
    step(it, std::integral_constant<int, 0>());
    step(it + 1, std::integral_constant<int, 1>());
    step(it + 2, std::integral_constant<int, 2>());
  }

  if (k_valid) {
    bf16* out = (pwave ? dV : dK) + (head + kj) * D;
    const float f = pwave ? 1.0f : scale;
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        bf16x4 w;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) w[jj] = to_bf16(acc[db][4 * g + jj] * f);
        *reinterpret_cast<bf16x4*>(out + db * 32 + 8 * g + 4 * h) = w;
      }
    }
  }
  if (!pwave) {
    const float dck_tot = wave_sum_pair(dck_part);
    if (k_valid && h == 0) dck[head + kj] = -dck_tot;
  }
  // the number of query tiles whose dS this block stored (the rest are zeros)
  if constexpr (STORE && SKIP)
    if (tid == 0) ds_tiles[(size_t)bh * ds_key_blocks(L) + nblk] = n_tiles;
}

// ---------------------------------------------------------------------------
// dQ from the stored dS: dQ = s dS K and dc^q = rowsum(dS) over the bf16 dS the
// dK/dV kernel wrote.  Eight waves own 256 queries (four 64-query tiles, two
// 32-query halves each); stages of 64 keys (half a stored block) load K and the
// four tiles' dS by DMA, triple-buffered (two stages in flight, 156 KB of LDS),
// one barrier per stage.  Each wave
// accumulates dQ^T = K^T dS^T: the A operand is K transposed out of the LDS
// tile, the B operand dS^T comes out of the stored layout by transposing reads
// (lane = query, eight keys in the contraction order of the A operand).  A tile
// skips the stages wholly above its diagonal; those slots were never written.
// HBM-bound: every stored dS byte is read once, by non-temporal DMA, which
// leaves the caches to the K tiles that neighbouring workgroups re-read.
// ---------------------------------------------------------------------------
constexpr int kDsWaves = 8;
constexpr int kDsThreads = 64 * kDsWaves;
constexpr int kDsBM = 32 * kDsWaves;  // queries per workgroup
constexpr int kDsBN = 64;             // keys per stage
constexpr int kDsTiles = kDsBM / 64;  // query tiles per workgroup
constexpr int kDsStageBytes = kDsSlotBytes / 2;  // one tile's dS for one stage
// In LDS each 1 KB stored chunk takes 1152 bytes, so that the two 16-query
// chunks of a half fall 128 bytes apart modulo the 256-byte bank row, and inside
// a chunk the slot of lane 32 + k moves to position (32 + k) ^ 4: the 16 slots a
// transposing read touches then sit in 16 distinct bank groups for any 32 lanes.
constexpr int kDsChunkLds = 1152;
constexpr int kDsStageLds = (kDsStageBytes / 1024) * kDsChunkLds;
__device__ __forceinline__ int ds_lds_pos(int slot) { return slot ^ ((slot >> 5) << 2); }

template <int D>
struct DsSmem {
  bf16 k[3][kDsBN * D];
  bf16x8 ds[3][kDsTiles][kDsStageLds / 16];
};

template <int D, bool SKIP>
__global__ __launch_bounds__(kDsThreads) void bwd_dq_stored_kernel(
    const bf16* __restrict__ K, const bf16x8* __restrict__ ds_store,
    const int* __restrict__ ds_tiles, bf16* __restrict__ dQ, float* __restrict__ dcq, int BH,
    int L, int n_mblk, float scale) {
  constexpr int TILE = kDsBN * D;
  constexpr int NDMA = TILE * 2 / 1024 / kDsWaves;
  static_assert(NDMA >= 1, "every wave issues at least one K DMA load per stage");
  __shared__ __attribute__((aligned(16))) DsSmem<D> sm;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = lane >> 5, col = lane & 31;
  const int row = (int)(blockIdx.x / BH);
  // heads fastest; rotated over the XCDs when skipping, whose work per head
  // depends on its gates (see the forward kernel)
  const int bh = SKIP ? (int)((blockIdx.x + row) % BH) : (int)(blockIdx.x % BH);
  const int mblk = n_mblk - 1 - row;  // the longest rows first
  const int q0 = mblk * kDsBM;
  const int qt0 = q0 / 64;
  const int my_t = wave >> 1, qb = wave & 1;  // this wave's tile and half
  const int qt = qt0 + my_t;
  const int qi = qt * 64 + qb * 32 + col;
  const bool q_valid = qi < L;
  const int n_qt = ds_query_tiles(L);
  const size_t head = (size_t)bh * (size_t)L;
  const size_t head_slot = (size_t)bh * ds_slots_per_head(L);
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(K + head * D, (uint32_t)L * D * 2);
  const uint32_t dma_off = tile_dma_offset<D, kDsWaves>(wave, lane);

  // A operand: transposing reads of the K tile (tile_tr_offsets); B operand:
  // in group g16 = lane / 16, lane j16 reads, for the 4 x 16 block of keys
  // (rows) by the group's 16 queries (columns), key row j16 / 4 and queries
  // 4 (j16 % 4) .. +3, which sit in one 8-byte half of one stored lane slot.
  int toff[2][D / 32];
  tile_tr_offsets<D>(toff, lane);
  uint32_t taddr[2][D / 32];
#pragma unroll
  for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
      taddr[k2][db] = (uint32_t)(uintptr_t)lds_opaque(lds_ptr(&sm.k[0][0]) + 2 * toff[k2][db]);
  const int g16 = lane >> 4, j16 = lane & 15, cg = j16 & 3;
  const uint32_t ds_addr = (uint32_t)(uintptr_t)lds_opaque(
      lds_ptr(&sm.ds[0][my_t][0]) + (2 * qb + (g16 & 1)) * kDsChunkLds +
      ds_lds_pos((cg & 1) * 32 + 4 * (g16 >> 1) + (j16 >> 2)) * 16 + (cg >> 1) * 8);
  // buffer 2 lies beyond the 16-bit reach of an LDS immediate offset: own base
  const uint32_t ds_addr2 = (uint32_t)(uintptr_t)lds_opaque(
      (const lds_byte*)(uintptr_t)(ds_addr + 2 * (uint32_t)sizeof(sm.ds[0])));
  const uint32_t ds_src = (uint32_t)ds_lds_pos(lane) * 16;  // DMA: stored slot of LDS position lane

  f32x16 dqacc[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) dqacc[db][r] = 0.0f;
  float dcq_part = 0.0f;

  const int n_st = (min(L, q0 + kDsBM) + kDsBN - 1) / kDsBN;
  // SKIP: key block nb stored the query tiles below cut(nb) = 2 nb + its tile
  // count, the others being exact zeros; cut never decreases with nb (c never
  // increases), so the blocks this workgroup needs start at the first nb with
  // cut(nb) > qt0 (a binary search; block qt0 / 2 holds the diagonal, stored).
  const int* tiles_row = SKIP ? ds_tiles + (size_t)bh * ds_key_blocks(L) : nullptr;
  auto cut = [&](int nb) { return SKIP ? 2 * nb + tiles_row[nb] : n_qt; };
  int j_first = 0;
  if constexpr (SKIP) {
    int lo = 0, hi = qt0 / 2;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (cut(mid) > qt0) hi = mid;
      else lo = mid + 1;
    }
    j_first = 2 * lo;
  }
  // stage j's DMA into buffer B; returns the number of loads this wave issued
  auto issue = [&](int j, auto bufc) -> int {
    constexpr int B = decltype(bufc)::value;
    const uint32_t base = (uint32_t)j * TILE * 2;
#pragma unroll
    for (int i = 0; i < NDMA; ++i)
      dma16(rk, &sm.k[B][(i * kDsWaves + wave) * 512],
            dma_off + uniform_u32(base + i * tile_dma_stride<kDsWaves>()));
    // the tiles on or below the diagonal of stage j: slots of key block j / 2
    const int nb = j >> 1;
    const int t_lo = max(0, j - qt0), t_hi = min(min(kDsTiles, n_qt - qt0), cut(nb) - qt0);
    if (t_lo < t_hi) {
      const __amdgpu_buffer_rsrc_t rs = make_rsrc(
          ds_store + (head_slot + ds_slot(L, nb, qt0 + t_lo)) * (kDsSlotBytes / 16),
          (uint32_t)(t_hi - t_lo) * kDsSlotBytes);
      for (int t = t_lo; t < t_hi; ++t)
        dma16_nt(rs, &sm.ds[B][t][wave * (kDsChunkLds / 16)],
                 ds_src + uniform_u32((uint32_t)(t - t_lo) * kDsSlotBytes +
                                      (uint32_t)(j & 1) * kDsStageBytes + (uint32_t)wave * 1024));
      return NDMA + (t_hi - t_lo);
    }
    return NDMA;
  };
  auto body = [&](auto bufc) {
    constexpr int B = decltype(bufc)::value;
    static_for<kDsBN / 16>([&](auto sc) {
      constexpr int S = decltype(sc)::value;  // 16-key step: pair S / 2, keys 16 (S % 2) ..
      constexpr int DOFF = (B == 2 ? 0 : B * (int)sizeof(sm.ds[0])) + (S / 2) * 4 * kDsChunkLds +
                           (S % 2) * 256;
      const uint32_t dbase = B == 2 ? ds_addr2 : ds_addr;
      constexpr int KOFF = 2 * (B * TILE + S * 16 * D);
      bf16x4 t[2 * (D / 32) + 2];
      t[0] = ds_read_tr_asm<DOFF>(dbase);
      t[1] = ds_read_tr_asm<DOFF + 128>(dbase);
      static_for<D / 32>([&](auto dbc) {
        constexpr int db = decltype(dbc)::value;
        t[2 + 2 * db] = ds_read_tr_asm<KOFF>(taddr[0][db]);
        t[3 + 2 * db] = ds_read_tr_asm<KOFF>(taddr[1][db]);
      });
      lds_wait<0>(t);
      const bf16x8 dsb = cat4(t[0], t[1]);
      dcq_part = sum8_bf16(dsb, dcq_part);
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
        dqacc[db] = mfma32(cat4(t[2 + 2 * db], t[3 + 2 * db]), dsb, dqacc[db]);
    });
  };

  // tile qt takes part in stage j when it lies on or below the diagonal and
  // (skipping) its dS for the stage's block was stored
  auto active = [&](int j) { return qt >= j && qt < n_qt && (!SKIP || qt < cut(j >> 1)); };
  // Three buffers: stages j + 1 and j + 2 load while stage j is used.  Before
  // stage j is read, the wave waits until only its loads of stage j + 1 (the
  // newest issued) are outstanding; the barrier then shows every wave's part of
  // stage j and that every wave is done reading stage j - 1, whose buffer stage
  // j + 2 fills.  The body's LDS reads are complete when it returns.
  static_assert(NDMA + kDsTiles < 16, "loads per stage fit the vmcnt immediate");
  int newest = -1, pending = 0;  // the newest issued stage, this wave's loads for it
  auto wait_stage = [&](int j) {
    if (newest <= j) {
      wait_all_memory();
      return;
    }
    switch (pending) {
      case 0: wait_vmem<0>(); break;
      case 1: wait_vmem<1>(); break;
      case 2: wait_vmem<2>(); break;
      case 3: wait_vmem<3>(); break;
      case 4: wait_vmem<4>(); break;
      case 5: wait_vmem<5>(); break;
      default: wait_vmem<NDMA + kDsTiles>(); break;
    }
  };
  // every step runs (a step past the last stage only meets the barrier) so that
  // no copies of the accumulators appear at the unrolled loop's back edge
  auto step = [&](int j, auto bufc) {
    constexpr int B = decltype(bufc)::value;
    wait_stage(j);
    barrier_no_fence();
    if (j + 2 < n_st) {
      pending = issue(j + 2, std::integral_constant<int, (B + 2) % 3>());
      newest = j + 2;
    }
    if (j < n_st && active(j)) body(bufc);
  };
  if (j_first < n_st) {
    pending = issue(j_first, std::integral_constant<int, 0>());
    newest = j_first;
  }
  if (j_first + 1 < n_st) {
    pending = issue(j_first + 1, std::integral_constant<int, 1>());
    newest = j_first + 1;
  }
  for (int j = j_first; j < n_st; j += 3) {
    step(j, std::integral_constant<int, 0>());
    step(j + 1, std::integral_constant<int, 1>());
    step(j + 2, std::integral_constant<int, 2>());
  }

  const float dcq_tot = wave_sum_pair(dcq_part);
  if (q_valid) {
    bf16* out = dQ + (head + qi) * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        bf16x4 w;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) w[jj] = to_bf16(dqacc[db][4 * g + jj] * scale);
        *reinterpret_cast<bf16x4*>(out + db * 32 + 8 * g + 4 * h) = w;
      }
    }
    if (h == 0) dcq[head + qi] = dcq_tot;
  }
}

// ---------------------------------------------------------------------------
// fp32 kernels: G = D/32 lanes per row, each lane owning 32 head dims.
// ---------------------------------------------------------------------------
constexpr int kF32Threads = 256;
constexpr int kF32Tile = 32;

template <int D, bool FIXED>
__global__ __launch_bounds__(kF32Threads) void bwd_dq_f32_kernel(
    const float* __restrict__ Q, const float* __restrict__ K, const float* __restrict__ V,
    const float* __restrict__ gate, const float* __restrict__ LSE, const float* __restrict__ dO,
    const float* __restrict__ delta, float* __restrict__ dQ, float* __restrict__ dcq, int H,
    int L, int n_blk, float scale, float scale_log2) {
  constexpr int G = D / 32;
  constexpr int RPW = kF32Threads / G;
  __shared__ float ks[kF32Tile][D + 1];
  __shared__ float vs[kF32Tile][D + 1];
  __shared__ float cks[kF32Tile];
  const int tid = threadIdx.x, sub = tid % G;
  const int bh = (int)(blockIdx.x / n_blk);
  const size_t head = (size_t)bh * (size_t)L;
  const int q0 = (int)(blockIdx.x % n_blk) * RPW;
  const int qi = q0 + tid / G;
  const bool q_valid = qi < L;
  const GateRow<FIXED> gr(gate, bh, H, head);
  float qv[32], gv[32], acc[32];
#pragma unroll
  for (int e = 0; e < 32; ++e) {
    qv[e] = q_valid ? Q[(head + qi) * D + sub * 32 + e] : 0.0f;
    gv[e] = q_valid ? dO[(head + qi) * D + sub * 32 + e] : 0.0f;
    acc[e] = 0.0f;
  }
  const float cq = q_valid ? gr.diff(qi, q0) : 0.0f;
  const float lq = q_valid ? LSE[head + qi] : INFINITY;
  const float dlt = q_valid ? delta[head + qi] : 0.0f;
  float dc = 0.0f;
  const int kend = min(L, q0 + RPW);
  for (int key0 = 0; key0 < kend; key0 += kF32Tile) {
    __syncthreads();
    for (int i = tid; i < kF32Tile * D; i += kF32Threads) {
      const int r = i / D, e = i % D, key = key0 + r;
      ks[r][e] = key < L ? K[(head + key) * D + e] : 0.0f;
      vs[r][e] = key < L ? V[(head + key) * D + e] : 0.0f;
    }
    if (tid < kF32Tile) {
      const int key = key0 + tid;
      cks[tid] = key < L ? gr.diff(key, q0) : INFINITY;
    }
    __syncthreads();
    for (int j = 0; j < kF32Tile; ++j) {
      float s = 0.0f, dp = 0.0f;
#pragma unroll
      for (int e = 0; e < 32; ++e) {
        s += qv[e] * ks[j][sub * 32 + e];
        dp += gv[e] * vs[j][sub * 32 + e];
      }
#pragma unroll
      for (int off = 1; off < G; off <<= 1) {
        s += __shfl_xor(s, off);
        dp += __shfl_xor(dp, off);
      }
      float p = exp2_fast(s * scale_log2 + ((cq - cks[j]) - lq) * kLog2e);
      if (key0 + j > qi) p = 0.0f;
      const float ds = p * (dp - dlt);
      dc += ds;
#pragma unroll
      for (int e = 0; e < 32; ++e) acc[e] += ds * ks[j][sub * 32 + e];
    }
  }
  if (q_valid) {
#pragma unroll
    for (int e = 0; e < 32; ++e) dQ[(head + qi) * D + sub * 32 + e] = acc[e] * scale;
    if (sub == 0) dcq[head + qi] = dc;
  }
}

template <int D, bool FIXED>
__global__ __launch_bounds__(kF32Threads) void bwd_dkdv_f32_kernel(
    const float* __restrict__ Q, const float* __restrict__ K, const float* __restrict__ V,
    const float* __restrict__ gate, const float* __restrict__ LSE, const float* __restrict__ dO,
    const float* __restrict__ delta, float* __restrict__ dK, float* __restrict__ dV,
    float* __restrict__ dck, int H, int L, int n_blk, float scale, float scale_log2) {
  constexpr int G = D / 32;
  constexpr int RPW = kF32Threads / G;
  __shared__ float qs[kF32Tile][D + 1];
  __shared__ float gs[kF32Tile][D + 1];
  __shared__ float cqs[kF32Tile];
  __shared__ float lqs[kF32Tile];
  __shared__ float dls[kF32Tile];
  const int tid = threadIdx.x, sub = tid % G;
  const int bh = (int)(blockIdx.x / n_blk);
  const size_t head = (size_t)bh * (size_t)L;
  const int k0 = (int)(blockIdx.x % n_blk) * RPW;
  const int kj = k0 + tid / G;
  const bool k_valid = kj < L;
  const GateRow<FIXED> gr(gate, bh, H, head);
  float kv[32], vv[32], ak[32], av[32];
#pragma unroll
  for (int e = 0; e < 32; ++e) {
    kv[e] = k_valid ? K[(head + kj) * D + sub * 32 + e] : 0.0f;
    vv[e] = k_valid ? V[(head + kj) * D + sub * 32 + e] : 0.0f;
    ak[e] = 0.0f;
    av[e] = 0.0f;
  }
  const float ck = k_valid ? gr.diff(kj, k0) : -INFINITY;
  float dc = 0.0f;
  for (int qs0 = k0; qs0 < L; qs0 += kF32Tile) {
    __syncthreads();
    for (int i = tid; i < kF32Tile * D; i += kF32Threads) {
      const int r = i / D, e = i % D, qq = qs0 + r;
      qs[r][e] = qq < L ? Q[(head + qq) * D + e] : 0.0f;
      gs[r][e] = qq < L ? dO[(head + qq) * D + e] : 0.0f;
    }
    if (tid < kF32Tile) {
      const int qq = qs0 + tid;
      cqs[tid] = qq < L ? gr.diff(qq, k0) : 0.0f;
      lqs[tid] = qq < L ? LSE[head + qq] : INFINITY;
      dls[tid] = qq < L ? delta[head + qq] : 0.0f;
    }
    __syncthreads();
    for (int i = 0; i < kF32Tile; ++i) {
      float s = 0.0f, dp = 0.0f;
#pragma unroll
      for (int e = 0; e < 32; ++e) {
        s += kv[e] * qs[i][sub * 32 + e];
        dp += vv[e] * gs[i][sub * 32 + e];
      }
#pragma unroll
      for (int off = 1; off < G; off <<= 1) {
        s += __shfl_xor(s, off);
        dp += __shfl_xor(dp, off);
      }
      float p = exp2_fast(s * scale_log2 + ((cqs[i] - ck) - lqs[i]) * kLog2e);
      if (kj > qs0 + i || !k_valid) p = 0.0f;
      const float ds = p * (dp - dls[i]);
      dc -= ds;
#pragma unroll
      for (int e = 0; e < 32; ++e) {
        av[e] += p * gs[i][sub * 32 + e];
        ak[e] += ds * qs[i][sub * 32 + e];
      }
    }
  }
  if (k_valid) {
#pragma unroll
    for (int e = 0; e < 32; ++e) {
      dK[(head + kj) * D + sub * 32 + e] = ak[e] * scale;
      dV[(head + kj) * D + sub * 32 + e] = av[e];
    }
    if (sub == 0) dck[head + kj] = dc;
  }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
template <typename T>
static hipError_t launch_delta(const T* o, const T* g, float* delta, int BH, int L, int d,
                               hipStream_t s) {
  const size_t rows = (size_t)BH * (size_t)L;
  const int lpr = d / (16 / (int)sizeof(T));
  const size_t per_block = (size_t)(256 / lpr) * kDeltaRows;
  const dim3 grid((unsigned)((rows + per_block - 1) / per_block));
  if (d == 128) {
    hipLaunchKernelGGL((bwd_delta_kernel<T, 128>), grid, dim3(256), 0, s, o, g, delta, rows);
  } else {
    hipLaunchKernelGGL((bwd_delta_kernel<T, 64>), grid, dim3(256), 0, s, o, g, delta, rows);
  }
  return hipGetLastError();
}

hipError_t launch_bwd_delta(bool bf16_, const void* o, const void* d_o, float* delta, int BH,
                            int L, int d, hipStream_t s) {
  return bf16_ ? launch_delta((const bf16*)o, (const bf16*)d_o, delta, BH, L, d, s)
               : launch_delta((const float*)o, (const float*)d_o, delta, BH, L, d, s);
}

template <int D, bool FIXED>
static void dkdv_t(bool bf16_, const void* q, const void* k, const void* v, GateSpec g,
                   const float* lse, const void* d_o, const float* delta, void* dk, void* dv,
                   float* dck, int BH, int L, float scale, hipStream_t s, const float* qn,
                   const float* kn) {
  const float sl2 = scale * kLog2e;
  if (bf16_) {
    const dim3 grid((unsigned)((L + kKvBN - 1) / kKvBN) * (unsigned)BH);
    if (qn)
      hipLaunchKernelGGL((bwd_dkdv_bf16_kernel<D, FIXED, true>), grid, dim3(kKvThreads), 0, s,
                         (const bf16*)q, (const bf16*)k, (const bf16*)v, g.ptr, qn, kn, lse,
                         (const bf16*)d_o, delta, (bf16*)dk, (bf16*)dv, dck, nullptr, nullptr, BH, g.H, L, scale,
                         sl2);
    else
    hipLaunchKernelGGL((bwd_dkdv_bf16_kernel<D, FIXED, false>), grid, dim3(kKvThreads), 0, s,
                       (const bf16*)q, (const bf16*)k, (const bf16*)v, g.ptr, qn, kn, lse,
                       (const bf16*)d_o, delta, (bf16*)dk, (bf16*)dv, dck, nullptr, nullptr, BH, g.H, L, scale,
                       sl2);
  } else {
    const int rpw = kF32Threads / (D / 32);
    const int n_blk = (L + rpw - 1) / rpw;
    const dim3 grid((unsigned)n_blk * (unsigned)BH);
    hipLaunchKernelGGL((bwd_dkdv_f32_kernel<D, FIXED>), grid, dim3(kF32Threads), 0, s,
                       (const float*)q, (const float*)k, (const float*)v, g.ptr, lse,
                       (const float*)d_o, delta, (float*)dk, (float*)dv, dck, g.H, L, n_blk,
                       scale, sl2);
  }
}

hipError_t launch_bwd_dkdv(bool bf16_, const void* q, const void* k, const void* v, GateSpec g,
                           const float* lse, const void* d_o, const float* delta, void* dk,
                           void* dv, float* dck, int BH, int L, int d, float scale,
                           hipStream_t s, const float* qn, const float* kn) {
  if (d == 128) {
    if (g.fixed)
      dkdv_t<128, true>(bf16_, q, k, v, g, lse, d_o, delta, dk, dv, dck, BH, L, scale, s, qn, kn);
    else
      dkdv_t<128, false>(bf16_, q, k, v, g, lse, d_o, delta, dk, dv, dck, BH, L, scale, s, qn, kn);
  } else {
    if (g.fixed)
      dkdv_t<64, true>(bf16_, q, k, v, g, lse, d_o, delta, dk, dv, dck, BH, L, scale, s, qn, kn);
    else
      dkdv_t<64, false>(bf16_, q, k, v, g, lse, d_o, delta, dk, dv, dck, BH, L, scale, s, qn, kn);
  }
  return hipGetLastError();
}

template <int D, bool FIXED>
static void dq_t(bool bf16_, const void* q, const void* k, const void* v, GateSpec g,
                 const float* lse, const void* d_o, const float* delta, void* dq, float* dcq,
                 int BH, int L, float scale, hipStream_t s, const float* qn, const float* kn) {
  const float sl2 = scale * kLog2e;
  if (bf16_) {
    const int n_mblk = (L + kDqBM - 1) / kDqBM;
    const dim3 grid((unsigned)n_mblk * (unsigned)BH);
    if (qn)
      hipLaunchKernelGGL((bwd_dq_bf16_kernel<D, FIXED, true>), grid, dim3(kBwdThreads), 0, s,
                         (const bf16*)q, (const bf16*)k, (const bf16*)v, g.ptr, qn, kn, lse,
                         (const bf16*)d_o, delta, (bf16*)dq, dcq, BH, g.H, L, n_mblk, scale, sl2);
    else
    hipLaunchKernelGGL((bwd_dq_bf16_kernel<D, FIXED, false>), grid, dim3(kBwdThreads), 0, s,
                       (const bf16*)q, (const bf16*)k, (const bf16*)v, g.ptr, qn, kn, lse,
                       (const bf16*)d_o, delta, (bf16*)dq, dcq, BH, g.H, L, n_mblk, scale, sl2);
  } else {
    const int rpw = kF32Threads / (D / 32);
    const int n_blk = (L + rpw - 1) / rpw;
    const dim3 grid((unsigned)n_blk * (unsigned)BH);
    hipLaunchKernelGGL((bwd_dq_f32_kernel<D, FIXED>), grid, dim3(kF32Threads), 0, s,
                       (const float*)q, (const float*)k, (const float*)v, g.ptr, lse,
                       (const float*)d_o, delta, (float*)dq, dcq, g.H, L, n_blk, scale, sl2);
  }
}

hipError_t launch_bwd_dq(bool bf16_, const void* q, const void* k, const void* v, GateSpec g,
                         const float* lse, const void* d_o, const float* delta, void* dq,
                         float* dcq, int BH, int L, int d, float scale, hipStream_t s,
                         const float* qn, const float* kn) {
  if (d == 128) {
    if (g.fixed)
      dq_t<128, true>(bf16_, q, k, v, g, lse, d_o, delta, dq, dcq, BH, L, scale, s, qn, kn);
    else
      dq_t<128, false>(bf16_, q, k, v, g, lse, d_o, delta, dq, dcq, BH, L, scale, s, qn, kn);
  } else {
    if (g.fixed)
      dq_t<64, true>(bf16_, q, k, v, g, lse, d_o, delta, dq, dcq, BH, L, scale, s, qn, kn);
    else
      dq_t<64, false>(bf16_, q, k, v, g, lse, d_o, delta, dq, dcq, BH, L, scale, s, qn, kn);
  }
  return hipGetLastError();
}

static hipError_t launch_bwd_stages(bool bf16_, const void* q, const void* k, const void* v,
                                    GateSpec g, const void* o, const float* lse, const void* d_o,
                                    void* dq, void* dk, void* dv, float* d_log_f, float* ws,
                                    int BH, int L, int d, float scale, hipStream_t s,
                                    const float* qn = nullptr, const float* kn = nullptr) {
  float* delta = ws;
  float* dcq = delta + (size_t)BH * L;
  float* dck = dcq + (size_t)BH * L;
  hipError_t e = launch_bwd_delta(bf16_, o, d_o, delta, BH, L, d, s);
  if (e == hipSuccess)
    e = launch_bwd_dkdv(bf16_, q, k, v, g, lse, d_o, delta, dk, dv, dck, BH, L, d, scale, s, qn,
                        kn);
  if (e == hipSuccess)
    e = launch_bwd_dq(bf16_, q, k, v, g, lse, d_o, delta, dq, dcq, BH, L, d, scale, s, qn, kn);
  if (e == hipSuccess) e = launch_reverse_scan_sum(dcq, dck, d_log_f, BH, L, s);
  return e;
}

hipError_t launch_bwd(bool bf16_, const void* q, const void* k, const void* v, const float* c,
                      const void* o, const float* lse, const void* d_o, void* dq, void* dk,
                      void* dv, float* d_log_f, void* ws, int BH, int L, int d, float scale,
                      hipStream_t s, const float* q_norm_max, const float* k_norm_max) {
  return launch_bwd_stages(bf16_, q, k, v, gate_array(c), o, lse, d_o, dq, dk, dv, d_log_f,
                           static_cast<float*>(ws), BH, L, d, scale, s, q_norm_max, k_norm_max);
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

size_t ds_store_bytes(int BH, int L) {
  return (size_t)BH * ds_slots_per_head(L) * (size_t)kDsSlotBytes;
}

// the stored dS, then (skipping) the stored tile count of each key block
static size_t stored_tail_bytes(int BH, int L) {
  return ds_store_bytes(BH, L) + (size_t)BH * ds_key_blocks(L) * sizeof(int);
}

size_t bwd_stored_workspace_bytes(int BH, int L) {
  return align256(bwd_workspace_bytes(BH, L)) + stored_tail_bytes(BH, L);
}

template <int D, bool FIXED, bool SKIP>
static void dkdv_store_t(const void* q, const void* k, const void* v, GateSpec g,
                         const float* lse, const void* d_o, const float* delta, void* dk,
                         void* dv, float* dck, void* ds_store, int* ds_tiles, int BH, int L,
                         float scale, hipStream_t s, const float* qn, const float* kn) {
  const dim3 grid((unsigned)((L + kKvBN - 1) / kKvBN) * (unsigned)BH);
  hipLaunchKernelGGL((bwd_dkdv_bf16_kernel<D, FIXED, SKIP, true>), grid, dim3(kKvThreads), 0, s,
                     (const bf16*)q, (const bf16*)k, (const bf16*)v, g.ptr, qn, kn, lse,
                     (const bf16*)d_o, delta, (bf16*)dk, (bf16*)dv, dck, (bf16x8*)ds_store,
                     ds_tiles, BH, g.H, L, scale, scale * kLog2e);
}

template <int D>
static void dkdv_store_d(const void* q, const void* k, const void* v, GateSpec g,
                         const float* lse, const void* d_o, const float* delta, void* dk,
                         void* dv, float* dck, void* ds_store, int* ds_tiles, int BH, int L,
                         float scale, hipStream_t s, const float* qn, const float* kn) {
  if (g.fixed) {
    if (qn)
      dkdv_store_t<D, true, true>(q, k, v, g, lse, d_o, delta, dk, dv, dck, ds_store, ds_tiles,
                                  BH, L, scale, s, qn, kn);
    else
      dkdv_store_t<D, true, false>(q, k, v, g, lse, d_o, delta, dk, dv, dck, ds_store, ds_tiles,
                                   BH, L, scale, s, qn, kn);
  } else {
    if (qn)
      dkdv_store_t<D, false, true>(q, k, v, g, lse, d_o, delta, dk, dv, dck, ds_store, ds_tiles,
                                   BH, L, scale, s, qn, kn);
    else
      dkdv_store_t<D, false, false>(q, k, v, g, lse, d_o, delta, dk, dv, dck, ds_store, ds_tiles,
                                    BH, L, scale, s, qn, kn);
  }
}

hipError_t launch_bwd_dkdv_store(const void* q, const void* k, const void* v, GateSpec g,
                                 const float* lse, const void* d_o, const float* delta, void* dk,
                                 void* dv, float* dck, void* ds_store, int* ds_tiles, int BH,
                                 int L, int d, float scale, hipStream_t s, const float* qn,
                                 const float* kn) {
  if (d == 128)
    dkdv_store_d<128>(q, k, v, g, lse, d_o, delta, dk, dv, dck, ds_store, ds_tiles, BH, L, scale,
                      s, qn, kn);
  else
    dkdv_store_d<64>(q, k, v, g, lse, d_o, delta, dk, dv, dck, ds_store, ds_tiles, BH, L, scale,
                     s, qn, kn);
  return hipGetLastError();
}

template <int D, bool SKIP>
static void dq_stored_t(const void* k, const void* ds_store, const int* ds_tiles, void* dq,
                        float* dcq, int BH, int L, float scale, hipStream_t s) {
  const int n_mblk = (L + kDsBM - 1) / kDsBM;
  const dim3 grid((unsigned)n_mblk * (unsigned)BH);
  hipLaunchKernelGGL((bwd_dq_stored_kernel<D, SKIP>), grid, dim3(kDsThreads), 0, s,
                     (const bf16*)k, (const bf16x8*)ds_store, ds_tiles, (bf16*)dq, dcq, BH, L,
                     n_mblk, scale);
}

hipError_t launch_bwd_dq_stored(const void* k, const void* ds_store, const int* ds_tiles,
                                void* dq, float* dcq, int BH, int L, int d, float scale,
                                hipStream_t s) {
  if (d == 128) {
    if (ds_tiles) dq_stored_t<128, true>(k, ds_store, ds_tiles, dq, dcq, BH, L, scale, s);
    else dq_stored_t<128, false>(k, ds_store, ds_tiles, dq, dcq, BH, L, scale, s);
  } else {
    if (ds_tiles) dq_stored_t<64, true>(k, ds_store, ds_tiles, dq, dcq, BH, L, scale, s);
    else dq_stored_t<64, false>(k, ds_store, ds_tiles, dq, dcq, BH, L, scale, s);
  }
  return hipGetLastError();
}

// delta -> dK/dV storing dS -> dQ from it -> d(log f), with delta, dc_q, dc_k at
// the start of ws and the stored dS (and tile counts) at `tail`
static hipError_t launch_bwd_stored_stages(const void* q, const void* k, const void* v,
                                           GateSpec g, const void* o, const float* lse,
                                           const void* d_o, void* dq, void* dk, void* dv,
                                           float* d_log_f, float* ws, char* tail, int BH, int L,
                                           int d, float scale, hipStream_t s, const float* qn,
                                           const float* kn) {
  float* delta = ws;
  float* dcq = delta + (size_t)BH * L;
  float* dck = dcq + (size_t)BH * L;
  void* dss = tail;
  int* tiles = qn ? reinterpret_cast<int*>(tail + ds_store_bytes(BH, L)) : nullptr;
  hipError_t e = launch_bwd_delta(true, o, d_o, delta, BH, L, d, s);
  if (e == hipSuccess)
    e = launch_bwd_dkdv_store(q, k, v, g, lse, d_o, delta, dk, dv, dck, dss, tiles, BH, L, d,
                              scale, s, qn, kn);
  if (e == hipSuccess) e = launch_bwd_dq_stored(k, dss, tiles, dq, dcq, BH, L, d, scale, s);
  if (e == hipSuccess) e = launch_reverse_scan_sum(dcq, dck, d_log_f, BH, L, s);
  return e;
}

hipError_t launch_bwd_stored(const void* q, const void* k, const void* v, const float* c,
                             const void* o, const float* lse, const void* d_o, void* dq, void* dk,
                             void* dv, float* d_log_f, void* ws, int BH, int L, int d, float scale,
                             hipStream_t s, const float* q_norm_max, const float* k_norm_max) {
  return launch_bwd_stored_stages(q, k, v, gate_array(c), o, lse, d_o, dq, dk, dv, d_log_f,
                                  static_cast<float*>(ws),
                                  static_cast<char*>(ws) + align256(bwd_workspace_bytes(BH, L)),
                                  BH, L, d, scale, s, q_norm_max, k_norm_max);
}

// d b^(h) = sigmoid(-b^(h)) * sum over the rows of head h and all t of d(log f):
// one workgroup per head, a tree sum over its B rows of length L.
constexpr int kBiasThreads = 256;
__global__ __launch_bounds__(kBiasThreads) void fixed_bias_grad_kernel(
    const float* __restrict__ dlf, const float* __restrict__ bias, float* __restrict__ dbias,
    int B, int H, int L) {
  const int h = blockIdx.x;
  float acc = 0.0f;
  for (int b = 0; b < B; ++b) {
    const float* row = dlf + ((size_t)b * H + h) * (size_t)L;
    for (int t = threadIdx.x; t < L; t += kBiasThreads) acc += row[t];
  }
  __shared__ float part[kBiasThreads / 64];
  for (int off = 32; off >= 1; off >>= 1) acc += __shfl_xor(acc, off);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    float tot = 0.0f;
    for (int w = 0; w < kBiasThreads / 64; ++w) tot += part[w];
    dbias[h] = tot / (1.0f + expf(bias[h]));  // times sigmoid(-b)
  }
}

size_t bwd_fixed_workspace_bytes(int BH, int L) { return 16 * (size_t)BH * (size_t)L; }

hipError_t launch_bwd_fixed(bool bf16_, const void* q, const void* k, const void* v,
                            const float* bias, int H, const void* o, const float* lse,
                            const void* d_o, void* dq, void* dk, void* dv, float* d_bias, void* ws,
                            int BH, int L, int d, float scale, hipStream_t s,
                            const float* q_norm_max, const float* k_norm_max) {
  float* w = static_cast<float*>(ws);
  float* dlf = w + 3 * (size_t)BH * L;
  hipError_t e = launch_bwd_stages(bf16_, q, k, v, gate_fixed(bias, H), o, lse, d_o, dq, dk, dv,
                                   dlf, w, BH, L, d, scale, s, q_norm_max, k_norm_max);
  if (e == hipSuccess && d_bias) {
    hipLaunchKernelGGL(fixed_bias_grad_kernel, dim3(H), dim3(kBiasThreads), 0, s, dlf, bias,
                       d_bias, BH / H, H, L);
    e = hipGetLastError();
  }
  return e;
}

size_t bwd_fixed_stored_workspace_bytes(int BH, int L) {
  return align256(bwd_fixed_workspace_bytes(BH, L)) + stored_tail_bytes(BH, L);
}

hipError_t launch_bwd_fixed_stored(const void* q, const void* k, const void* v,
                                   const float* bias, int H, const void* o, const float* lse,
                                   const void* d_o, void* dq, void* dk, void* dv, float* d_bias,
                                   void* ws, int BH, int L, int d, float scale, hipStream_t s,
                                   const float* q_norm_max, const float* k_norm_max) {
  float* w = static_cast<float*>(ws);
  float* dlf = w + 3 * (size_t)BH * L;
  hipError_t e = launch_bwd_stored_stages(
      q, k, v, gate_fixed(bias, H), o, lse, d_o, dq, dk, dv, dlf, w,
      static_cast<char*>(ws) + align256(bwd_fixed_workspace_bytes(BH, L)), BH, L, d, scale, s,
      q_norm_max, k_norm_max);
  if (e == hipSuccess && d_bias) {
    hipLaunchKernelGGL(fixed_bias_grad_kernel, dim3(H), dim3(kBiasThreads), 0, s, dlf, bias,
                       d_bias, BH / H, H, L);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace fox
