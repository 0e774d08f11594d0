// Forgetting Attention forward pass (appendix, Alg. 1): O = softmax(s Q K^T + D) V
// with D_ij = c_i - c_j (j <= i), plus the natural-log row logsumexp.
//
// bf16 kernel (MFMA, gfx950)
//   * A workgroup owns 128 query rows of one (batch, head): four waves of 32 rows,
//     two workgroups per CU.  Key/value tiles of 64 rows are double-buffered in
//     LDS and move there with buffer loads that write LDS directly (no registers,
//     no VALU); out-of-range rows of a ragged last tile read as zero.  The next
//     tile's loads are in flight while the current tile is used.
//   * LDS rows are stored with an XOR swizzle of their 16-byte chunks so that the
//     32 rows touched by one MFMA operand read fall in different banks.
//   * Each wave computes S^T = K Q^T (keys on MFMA rows, its 32 queries on
//     columns), so every lane owns one query: the softmax statistics are per lane
//     and only the two half-waves holding the same query exchange values.
//   * The forget-gate bias is applied in registers, as in the paper (D is never
//     materialised), in base 2 and relative to c_ref, the prefix value of the
//     block's first query: u_ij = s log2(e) q_i.k_j - log2(e) (c_j - c_ref).  The
//     row term c_i shifts a whole softmax row and cancels; it only enters the
//     logsumexp: LSE_i = (c_i - c_ref) + ln2 (m_i + log2 l_i).  Keeping the c
//     differences small keeps them exact in fp32 even where |c| is 1e4-1e5.
//     The key term enters through the accumulator: each S tile starts from
//     (c_ref - c_j) / s, so the MFMA chain adds it and one fma per score gives
//     u_ij - m_i.
//   * P^T (accumulator layout) is the B operand of O^T += V^T P^T.  The V^T
//     A operand comes straight from the row-major V tile through transposing LDS
//     reads; keys are consumed in the order the accumulator layout holds them, a
//     permutation of the contraction index applied identically to both operands.
//   * Key tiles are visited from the diagonal backwards, so the row maximum of
//     the diagonal tile (the first one visited) is a good reference for all
//     later tiles: they are exponentiated against it without a maximum search.
//     Only when some score exceeds the reference by more than the slack (then a
//     lane's tile sum of P exceeds 2^8) is the tile maximum taken and O and l
//     rescaled.  Exponents up to 8 are absorbed by bf16 P and the fp32 sums.
//   * l sums P after its rounding to bf16 (v_dot2_f32_bf16 against ones), the
//     same values the P V product uses.
//   * Causal structure: tiles after a wave's last query are skipped and only the
//     tile holding its diagonal applies the mask.  Query blocks are dispatched
//     longest-first with heads fastest, so a head's blocks share an XCD's L2
//     whenever the head count is a multiple of 8.
//
// fp32 kernel: a straightforward vector-ALU kernel (D/32 lanes per query row,
// keys staged through LDS 32 at a time).  It favours accuracy over speed: the
// bias c_i - c_j is formed in natural-log units before the change to base 2, so
// the row maximum stays small and the logsumexp carries no cancellation even
// when c changes by thousands within a block.
#include <type_traits>

#include "fox_device.h"
#include "fox_internal.h"

namespace fox {

constexpr int kFwdWaves = 4;
constexpr int kFwdThreads = 64 * kFwdWaves;
constexpr int kFwdBM = 32 * kFwdWaves;  // query rows per workgroup
constexpr int kFwdBN = 64;              // keys per tile
constexpr float kRescaleSlack = 8.0f;   // log2 headroom before O and l are rescaled
constexpr float kRescaleSum = 256.0f;  // 2^slack: a lane's tile sum above it triggers a rescale
// Gate-aware skipping: a key tile is dropped when every P it could produce lies
// below 2^-160 relative to the row maximum (150 for an exact fp32 zero, 10 more
// for the rounding of the bound).
constexpr float kSkipMargin = 160.0f;

template <int D>
struct FwdSmem {
  bf16 k[2][kFwdBN * D];
  bf16 v[2][kFwdBN * D];
  float c[2][kFwdBN];
};

// SKIP: qnorm, knorm [BH] bound the row norms of Q and K.  For a query block
// starting at q0 and a key tile ending at jl, every score is at most
// s Qmax Kmax + (c_i - c_j) <= s Qmax Kmax + (c_q0 - c_jl), and every row
// maximum is at least the diagonal score s q_i.k_i >= -s Qmax Kmax, so once
// log2(e) (2 s Qmax Kmax + c_q0 - c_jl) < -kSkipMargin the tile (and, as c
// falls along the sequence, every earlier tile) adds exact zeros: the loop
// stops there and the results equal the dense kernel's bit for bit.
//
// OUTG: the FoX (Pro) output norm and gate in the epilogue (appendix, FoX (Pro)
// layer computation): y = RMSNorm(o) o sigmoid(g) per query row, from the row
// as rounded to bf16 for O (the backward normalises the stored O the same way).
// A lane holds half of its row; the other half is in lane l ^ 32.
//
// Occupancy: two waves per SIMD at D = 128 (about 240 VGPRs); at D = 64 the
// kernel fits 128 VGPRs and runs four (the LDS would allow four workgroups per
// CU; measured 3 % faster than three).
template <int D, bool FIXED, bool SKIP, bool OUTG = false>
__global__ __launch_bounds__(kFwdThreads) __attribute__((amdgpu_waves_per_eu(D == 64 ? 4 : 2)))
void fwd_bf16_kernel(const bf16* __restrict__ Q, const bf16* __restrict__ K,
                     const bf16* __restrict__ V, const float* __restrict__ gate,
                     const float* __restrict__ qnorm, const float* __restrict__ knorm,
                     bf16* __restrict__ O, float* __restrict__ LSE, int BH, int H, int L,
                     int n_mblk, float scale_log2, OutGateArgs og) {
  constexpr int TILE = kFwdBN * D;                         // bf16 elements per tile
  constexpr int NDMA = TILE * 2 / 1024 / kFwdWaves;        // 1 KB DMA loads per wave per tile
  __shared__ __attribute__((aligned(16))) FwdSmem<D> sm;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = lane >> 5, col = lane & 31;
  // heads fastest (a head's blocks on one XCD, sharing its L2); with skipping the
  // work per head depends on its gates, so the heads rotate over the XCDs
  const int row = (int)(blockIdx.x / BH);
  const int bh = SKIP ? (int)((blockIdx.x + row) % BH) : (int)(blockIdx.x % BH);
  const int mblk = n_mblk - 1 - row;
  const int q0 = mblk * kFwdBM;
  const size_t head = (size_t)bh * (size_t)L;
  const bf16* Qh = Q + head * D;
  const GateRow<FIXED> gr(gate, bh, H, head);  // c_i - c_j; the reference is c at q0
  const int qw0 = q0 + wave * 32;
  const int qi = qw0 + col;
  const bool q_valid = qi < L;
  const uint32_t head_bytes = (uint32_t)L * D * 2;
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(K + head * D, head_bytes);
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(V + head * D, head_bytes);

  const uint32_t dma_off = tile_dma_offset<D, kFwdWaves>(wave, lane);
  int koff[D / 16];
  tile_row_offsets<D>(koff, col, h);
  int voff[2][D / 32];
  tile_tr_offsets<D>(voff, lane);
  uint32_t vaddr[2][D / 32];  // byte addresses of the transposing reads in V buffer 0
#pragma unroll
  for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
    for (int db = 0; db < D / 32; ++db) vaddr[k2][db] = lds_addr(&sm.v[0][0]) + 2 * voff[k2][db];

  bf16x8 qf[D / 16];
#pragma unroll
  for (int s = 0; s < D / 16; ++s) {
    if (q_valid) {
      qf[s] = *reinterpret_cast<const bf16x8*>(Qh + (size_t)qi * D + 16 * s + 8 * h);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) qf[s][e] = to_bf16(0.0f);
    }
  }
  f32x16 oacc[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[db][r] = 0.0f;
  float m_used = -INFINITY, l_run = 0.0f;
  const float inv_scale = kLog2e / scale_log2;  // 1 / s

  const int kend = min(L, q0 + kFwdBM);
  const int t_last = (kend + kFwdBN - 1) / kFwdBN - 1;
  const int t_diag = qw0 / kFwdBN;  // tile holding this wave's diagonal
  // skip test in the units of the stored key terms ((c_q0 - c_j) / s)
  const float skip_norm = SKIP ? 2.0f * qnorm[bh] * knorm[bh] : 0.0f;

  // wave 0 stages the key terms of the next tile: the prefix values are loaded
  // with the tile's DMA and converted after the tile body, so that waiting for
  // them never waits for the DMA (memory operations complete in order)
  const float c_q0 = gr.raw(q0);
  float craw = 0.0f;
  int ckey = 0;
  auto issue_tile = [&](int kt, auto bufc) {
    constexpr int B = decltype(bufc)::value;
    const uint32_t base = (uint32_t)kt * kFwdBN * D * 2;
#pragma unroll
    for (int i = 0; i < NDMA; ++i) {
      const int wslot = (i * kFwdWaves + wave) * 512;  // bf16 elements of this wave's 1 KB
      const uint32_t voff = dma_off + uniform_u32(base + i * tile_dma_stride<kFwdWaves>());
      dma16(rk, &sm.k[B][wslot], voff);
      dma16(rv, &sm.v[B][wslot], voff);
    }
    if (wave == 0) {
      ckey = kt * kFwdBN + lane;
      if (ckey < L) craw = gr.raw(ckey);
    }
  };
  auto store_c = [&](auto bufc) {
    constexpr int B = decltype(bufc)::value;
    if (wave == 0)
      sm.c[B][lane] = ckey < L ? gr.diff_raw(q0, c_q0, ckey, craw) * inv_scale : -INFINITY;
  };

  auto tile_body = [&](int j, auto bufc, auto masked) {
    constexpr int B = decltype(bufc)::value;
    constexpr bool MASK = decltype(masked)::value;
    const bf16* kt_ = sm.k[B];
    const bf16* vt_ = sm.v[B];
    const float* ct_ = sm.c[B];
    const int key0 = j * kFwdBN;
    // u = log2(e) (s q.k - (c_j - c_ref)) - m: the accumulator starts at the key's
    // bias divided by s, so the MFMA chain adds it and one fma per score remains
    const float m_sub = MASK ? 0.0f : m_used;
    float u[32];
    bf16x8 pb[4];
    float psum_fast = 0.0f;
    if constexpr (!MASK) {
      // unmasked tiles: the scale, exponentials and row sums of keys 0..31 are
      // scheduled between the MFMAs of keys 32..63 (one wave overlaps the two)
      bf16x8 ka0[D / 16], ka1[D / 16];
      f32x16 acc0, acc1;
#pragma unroll
      for (int s = 0; s < D / 16; ++s) ka0[s] = *reinterpret_cast<const bf16x8*>(kt_ + koff[s]);
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 ck4 = *reinterpret_cast<const f32x4*>(ct_ + 8 * g + 4 * h);
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) acc0[4 * g + jj] = ck4[jj];
      }
      sched_fence();
#pragma unroll
      for (int s = 0; s < D / 16; ++s) acc0 = mfma32(ka0[s], qf[s], acc0);
#pragma unroll
      for (int s = 0; s < D / 16; ++s)
        ka1[s] = *reinterpret_cast<const bf16x8*>(kt_ + 32 * D + koff[s]);
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 ck4 = *reinterpret_cast<const f32x4*>(ct_ + 32 + 8 * g + 4 * h);
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) acc1[4 * g + jj] = ck4[jj];
      }
      sched_fence();
#pragma unroll
      for (int r = 0; r < 16; ++r) u[r] = acc0[r] * scale_log2 - m_sub;
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        float pv[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) pv[i] = exp2_fast(u[8 * c + i]);
        pb[c] = pack8(pv);
        psum_fast = sum8_bf16(pb[c], psum_fast);
      }
#pragma unroll
      for (int s = 0; s < D / 16; ++s) acc1 = mfma32(ka1[s], qf[s], acc1);
#pragma unroll
      for (int i = 0; i < D / 16; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);
      }
      sched_fence();
#pragma unroll
      for (int r = 0; r < 16; ++r) u[16 + r] = acc1[r] * scale_log2 - m_sub;
#pragma unroll
      for (int c = 2; c < 4; ++c) {
        float pv[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) pv[i] = exp2_fast(u[8 * c + i]);
        pb[c] = pack8(pv);
        psum_fast = sum8_bf16(pb[c], psum_fast);
      }
    } else {  // the diagonal tile: plain order, then the causal mask
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        bf16x8 ka[D / 16];
#pragma unroll
        for (int s = 0; s < D / 16; ++s)
          ka[s] = *reinterpret_cast<const bf16x8*>(kt_ + kb * 32 * D + koff[s]);
        f32x16 acc;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x4 ck4 = *reinterpret_cast<const f32x4*>(ct_ + kb * 32 + 8 * g + 4 * h);
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) acc[4 * g + jj] = ck4[jj];
        }
        sched_fence();
#pragma unroll
        for (int s = 0; s < D / 16; ++s) acc = mfma32(ka[s], qf[s], acc);
#pragma unroll
        for (int g = 0; g < 4; ++g) {
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) {
            float x = acc[4 * g + jj] * scale_log2 - m_sub;
            if (MASK && key0 + kb * 32 + 8 * g + 4 * h + jj > qi) x = -INFINITY;
            u[kb * 16 + 4 * g + jj] = x;
          }
        }
      }
    }
    // rescale O and l by 2^-shift and take u relative to the new maximum
    auto rescale = [&](float shift) {
      const float alpha = exp2_fast(-shift);
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < D / 32; ++db) oacc[db] *= alpha;
#pragma unroll
      for (int r = 0; r < 32; ++r) u[r] -= shift;
    };
    auto tile_max = [&]() {
      float mt = u[0];
#pragma unroll
      for (int r = 1; r < 32; ++r) mt = fmaxf(mt, u[r]);
      return wave_max_pair(mt);
    };
    auto exponentiate = [&]() {
      float psum = 0.0f;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        float pv[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) pv[i] = exp2_fast(u[8 * c + i]);
        pb[c] = pack8(pv);
        psum = sum8_bf16(pb[c], psum);
      }
      return psum;
    };
    float psum;
    if (MASK) {
      // the diagonal tile is the first one a wave visits (O and l are still zero):
      // its row maximum becomes the reference
      const float mt = tile_max();
#pragma unroll
      for (int r = 0; r < 32; ++r) u[r] -= mt;
      m_used = mt;
      psum = exponentiate();
    } else {
      // no maximum: the scores were exponentiated against the running one above;
      // only if some score exceeds it by more than the slack (the lane's sum then
      // exceeds 2^slack) find the tile maximum, rescale and exponentiate again
      psum = psum_fast;
      if (__any(q_valid && psum > kRescaleSum)) {
        const float shift = fmaxf(tile_max(), 0.0f);
        rescale(shift);
        m_used += shift;
        psum = exponentiate();
      }
    }
    l_run += psum;
    // O^T += V^T P^T over the four 16-key chunks; the V^T operands of chunk c + 1
    // are read while chunk c is multiplied
    constexpr int NR = 2 * (D / 32);  // transposing reads per chunk
    bf16x4 tv[2][NR];
    auto read_v = [&](auto cc, bf16x4 (&t)[NR]) {
      constexpr int C = decltype(cc)::value;
      static_for<D / 32>([&](auto dbc) {
        constexpr int DB = decltype(dbc)::value;
        t[2 * DB] = ds_read_tr_asm<(B * TILE + C * 16 * D) * 2>(vaddr[0][DB]);
        t[2 * DB + 1] = ds_read_tr_asm<(B * TILE + C * 16 * D) * 2>(vaddr[1][DB]);
      });
    };
    read_v(std::integral_constant<int, 0>(), tv[0]);
    static_for<4>([&](auto cc) {
      constexpr int C = decltype(cc)::value;
      if constexpr (C + 1 < 4) {
        read_v(std::integral_constant<int, C + 1>(), tv[(C + 1) % 2]);
        lds_wait<NR>(tv[C % 2]);
      } else {
        lds_wait<0>(tv[C % 2]);
      }
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
        oacc[db] = mfma32(cat4(tv[C % 2][2 * db], tv[C % 2][2 * db + 1]), pb[C], oacc[db]);
    });
  };

  // returns true when tile j and all earlier tiles can be skipped
  auto step = [&](int j, auto bufc) {
    constexpr int B = decltype(bufc)::value;
    wait_all_memory();
    __syncthreads();  // tile j is in LDS; every wave is done with tile j + 1
    if constexpr (SKIP) {
      // the tile's last key is the least decayed one (full tiles only: the
      // diagonal region never passes the test)
      if (j < t_last && scale_log2 * (skip_norm + sm.c[B][kFwdBN - 1]) < -kSkipMargin)
        return true;
    }
    if (j > 0) issue_tile(j - 1, std::integral_constant<int, 1 - B>());
    if (j == t_diag) {
      tile_body(j, bufc, std::true_type());
    } else if (j < t_diag) {
      tile_body(j, bufc, std::false_type());
    }
    if (j > 0) store_c(std::integral_constant<int, 1 - B>());
    return false;
  };

  issue_tile(t_last, std::integral_constant<int, 0>());
  store_c(std::integral_constant<int, 0>());
  for (int j = t_last; j >= 0; j -= 2) {
    if (step(j, std::integral_constant<int, 0>())) break;
    if (j > 0 && step(j - 1, std::integral_constant<int, 1>())) break;
  }

  const float l_tot = wave_sum_pair(l_run);
  if constexpr (OUTG) {
    const float inv = 1.0f / l_tot;
    bf16x4 ob[D / 32][4];
    float ss = 0.0f;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          ob[db][g][jj] = to_bf16(oacc[db][4 * g + jj] * inv);
          const float x = to_f32(ob[db][g][jj]);
          ss += x * x;
        }
    ss += __shfl_xor(ss, 32);
    if (q_valid) {
      const float r = 1.0f / sqrtf(ss * (1.0f / D) + og.eps);
      const size_t roff = (head + (size_t)qi) * D;
      const float* w = og.w + (size_t)(bh % og.heads) * D;
#pragma unroll
      for (int db = 0; db < D / 32; ++db) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int e = db * 32 + 8 * g + 4 * h;
          *reinterpret_cast<bf16x4*>(O + roff + e) = ob[db][g];
          const bf16x4 gv = *reinterpret_cast<const bf16x4*>(og.g + roff + e);
          const f32x4 wv = *reinterpret_cast<const f32x4*>(w + e);
          bf16x4 y;
#pragma unroll
          for (int jj = 0; jj < 4; ++jj)
            y[jj] = to_bf16(to_f32(ob[db][g][jj]) * r * wv[jj] /
                            (1.0f + expf(-to_f32(gv[jj]))));
          *reinterpret_cast<bf16x4*>(og.y + roff + e) = y;
        }
      }
      if (h == 0) LSE[head + qi] = gr.diff(qi, q0) + kLn2 * (m_used + log2f(l_tot));
    }
  } else if (q_valid) {
    const float inv = 1.0f / l_tot;
    bf16* orow = O + (head + (size_t)qi) * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        bf16x4 w;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) w[jj] = to_bf16(oacc[db][4 * g + jj] * inv);
        *reinterpret_cast<bf16x4*>(orow + db * 32 + 8 * g + 4 * h) = w;
      }
    }
    if (h == 0) LSE[head + qi] = gr.diff(qi, q0) + kLn2 * (m_used + log2f(l_tot));
  }
}

// ---------------------------------------------------------------------------
// fp32 forward: G = D/32 lanes per query row, each lane owning 32 head dims.
// ---------------------------------------------------------------------------
constexpr int kF32Threads = 256;
constexpr int kF32BN = 32;

template <int D, bool FIXED>
__global__ __launch_bounds__(kF32Threads) void fwd_f32_kernel(
    const float* __restrict__ Q, const float* __restrict__ K, const float* __restrict__ V,
    const float* __restrict__ gate, float* __restrict__ O, float* __restrict__ LSE, int H, int L,
    int n_blk, float scale_log2) {
  constexpr int G = D / 32;
  constexpr int RPW = kF32Threads / G;  // query rows per workgroup
  __shared__ float ks[kF32BN][D + 1];
  __shared__ float vs[kF32BN][D + 1];
  __shared__ float cks[kF32BN];
  const int tid = threadIdx.x;
  const int sub = tid % G;
  const int bh = (int)(blockIdx.x / n_blk);
  const size_t head = (size_t)bh * (size_t)L;
  const int q0 = (int)(blockIdx.x % n_blk) * RPW;
  const int qi = q0 + tid / G;
  const bool q_valid = qi < L;
  const GateRow<FIXED> gr(gate, bh, H, head);
  const float cq = q_valid ? gr.diff(qi, q0) : 0.0f;
  float qv[32], ov[32];
#pragma unroll
  for (int e = 0; e < 32; ++e) {
    qv[e] = q_valid ? Q[(head + qi) * D + sub * 32 + e] : 0.0f;
    ov[e] = 0.0f;
  }
  float m_run = -INFINITY, l_run = 0.0f;
  const int kend = min(L, q0 + RPW);
  for (int key0 = 0; key0 < kend; key0 += kF32BN) {
    __syncthreads();
    for (int i = tid; i < kF32BN * D; i += kF32Threads) {
      const int r = i / D, e = i % D, key = key0 + r;
      ks[r][e] = key < L ? K[(head + key) * D + e] : 0.0f;
      vs[r][e] = key < L ? V[(head + key) * D + e] : 0.0f;
    }
    if (tid < kF32BN) {
      const int key = key0 + tid;
      cks[tid] = key < L ? gr.diff(key, q0) : INFINITY;
    }
    __syncthreads();
    float sc[kF32BN];
    float mt = -INFINITY;
#pragma unroll
    for (int j = 0; j < kF32BN; ++j) {
      float part = 0.0f;
#pragma unroll
      for (int e = 0; e < 32; ++e) part += qv[e] * ks[j][sub * 32 + e];
#pragma unroll
      for (int off = 1; off < G; off <<= 1) part += __shfl_xor(part, off);
      float x = part * scale_log2 + (cq - cks[j]) * kLog2e;
      if (key0 + j > qi) x = -INFINITY;
      sc[j] = x;
      mt = fmaxf(mt, x);
    }
    // Key 0 lies in the first tile and is never masked, so m_new is finite.
    const float m_new = fmaxf(m_run, mt);
    const float alpha = exp2_fast(m_run - m_new);
    l_run *= alpha;
#pragma unroll
    for (int e = 0; e < 32; ++e) ov[e] *= alpha;
#pragma unroll
    for (int j = 0; j < kF32BN; ++j) {
      const float p = exp2_fast(sc[j] - m_new);
      l_run += p;
#pragma unroll
      for (int e = 0; e < 32; ++e) ov[e] += p * vs[j][sub * 32 + e];
    }
    m_run = m_new;
  }
  if (q_valid) {
    const float inv = 1.0f / l_run;
#pragma unroll
    for (int e = 0; e < 32; ++e) O[(head + qi) * D + sub * 32 + e] = ov[e] * inv;
    if (sub == 0) LSE[head + qi] = kLn2 * (m_run + log2f(l_run));
  }
}

template <int D, bool FIXED, bool SKIP>
static void fwd_bf16_t(const void* q, const void* k, const void* v, GateSpec g,
                       const float* qn, const float* kn, void* o, float* lse, int BH, int L,
                       float sl2, hipStream_t s) {
  const int n_mblk = (L + kFwdBM - 1) / kFwdBM;
  const dim3 grid((unsigned)n_mblk * (unsigned)BH);
  hipLaunchKernelGGL((fwd_bf16_kernel<D, FIXED, SKIP>), grid, dim3(kFwdThreads), 0, s,
                     (const bf16*)q, (const bf16*)k, (const bf16*)v, g.ptr, qn, kn, (bf16*)o, lse,
                     BH, g.H, L, n_mblk, sl2, OutGateArgs{});
}

template <int D, bool FIXED>
static void fwd_bf16_s(const void* q, const void* k, const void* v, GateSpec g,
                       const float* qn, const float* kn, void* o, float* lse, int BH, int L,
                       float sl2, hipStream_t s) {
  if (qn) fwd_bf16_t<D, FIXED, true>(q, k, v, g, qn, kn, o, lse, BH, L, sl2, s);
  else fwd_bf16_t<D, FIXED, false>(q, k, v, g, qn, kn, o, lse, BH, L, sl2, s);
}

hipError_t launch_fwd_bf16(const void* q, const void* k, const void* v, GateSpec g, void* o,
                           float* lse, int BH, int L, int d, float scale, hipStream_t s,
                           const float* q_norm_max, const float* k_norm_max) {
  const float sl2 = scale * kLog2e;
  const float* qn = q_norm_max;
  const float* kn = k_norm_max;
  if (d == 128) {
    if (g.fixed) fwd_bf16_s<128, true>(q, k, v, g, qn, kn, o, lse, BH, L, sl2, s);
    else fwd_bf16_s<128, false>(q, k, v, g, qn, kn, o, lse, BH, L, sl2, s);
  } else {
    if (g.fixed) fwd_bf16_s<64, true>(q, k, v, g, qn, kn, o, lse, BH, L, sl2, s);
    else fwd_bf16_s<64, false>(q, k, v, g, qn, kn, o, lse, BH, L, sl2, s);
  }
  return hipGetLastError();
}

template <int D>
static void fwd_bf16_outg_t(const void* q, const void* k, const void* v, const float* c, void* o,
                            float* lse, OutGateArgs og, int BH, int L, float sl2, hipStream_t s) {
  const int n_mblk = (L + kFwdBM - 1) / kFwdBM;
  const dim3 grid((unsigned)n_mblk * (unsigned)BH);
  hipLaunchKernelGGL((fwd_bf16_kernel<D, false, false, true>), grid, dim3(kFwdThreads), 0, s,
                     (const bf16*)q, (const bf16*)k, (const bf16*)v, c, nullptr, nullptr,
                     (bf16*)o, lse, BH, 1, L, n_mblk, sl2, og);
}

hipError_t launch_fwd_bf16_out_gate(const void* q, const void* k, const void* v, const float* c,
                                    void* o, float* lse, const void* g, const float* wo,
                                    float eps, void* y, int H, int BH, int L, int d, float scale,
                                    hipStream_t s) {
  const OutGateArgs og{static_cast<const bf16*>(g), wo, eps, static_cast<bf16*>(y), H};
  if (d == 128) fwd_bf16_outg_t<128>(q, k, v, c, o, lse, og, BH, L, scale * kLog2e, s);
  else fwd_bf16_outg_t<64>(q, k, v, c, o, lse, og, BH, L, scale * kLog2e, s);
  return hipGetLastError();
}

template <int D, bool FIXED>
static void fwd_f32_t(const float* q, const float* k, const float* v, GateSpec g, float* o,
                      float* lse, int BH, int L, float sl2, hipStream_t s) {
  const int rpw = kF32Threads / (D / 32);
  const int n_blk = (L + rpw - 1) / rpw;
  const dim3 grid((unsigned)n_blk * (unsigned)BH);
  hipLaunchKernelGGL((fwd_f32_kernel<D, FIXED>), grid, dim3(kF32Threads), 0, s, q, k, v, g.ptr,
                     o, lse, g.H, L, n_blk, sl2);
}

hipError_t launch_fwd_f32(const float* q, const float* k, const float* v, GateSpec g, float* o,
                          float* lse, int BH, int L, int d, float scale, hipStream_t s) {
  const float sl2 = scale * kLog2e;
  if (d == 128) {
    if (g.fixed) fwd_f32_t<128, true>(q, k, v, g, o, lse, BH, L, sl2, s);
    else fwd_f32_t<128, false>(q, k, v, g, o, lse, BH, L, sl2, s);
  } else {
    if (g.fixed) fwd_f32_t<64, true>(q, k, v, g, o, lse, BH, L, sl2, s);
    else fwd_f32_t<64, false>(q, k, v, g, o, lse, BH, L, sl2, s);
  }
  return hipGetLastError();
}

}  // namespace fox
