// Device-side helpers shared by the Forgetting Attention kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4_t;

namespace fox {

// Arguments of the FoX (Pro) output norm and gate fused into a forward epilogue:
// gate logits g [BH, L, D] bf16, per-head weights w [heads, D] fp32, RMSNorm eps,
// output y [BH, L, D] bf16.
struct OutGateArgs {
  const bf16* g;
  const float* w;
  float eps;
  bf16* y;
  int heads;
};

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// 2^x on the transcendental unit (v_exp_f32); exp2(-inf) = 0.
__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// One 32x32x16 bf16 MFMA: C[32x32] += A[32x16] * B[16x32], fp32 accumulation.
//
// Operand layout (wave64, lane l, h = l / 32): lane l supplies row (l % 32) of A
// and column (l % 32) of B, eight contraction elements each; lanes h = 0 and
// h = 1 supply complementary halves of the 16-element contraction.  Both
// operands use the same element-to-k assignment, so any consistent permutation
// of the contraction index gives the same product.
//
// Result layout: lane l holds column (l % 32) of C; its register r holds row
//     row(r, h) = 8 * (r / 4) + 4 * h + (r % 4),   r = 0..15.
__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ int mfma_row(int r, int h) { return 8 * (r >> 2) + 4 * h + (r & 3); }

// Round-to-nearest-even fp32 -> bf16 (the hardware conversion on gfx950).
__device__ __forceinline__ bf16 to_bf16(float x) { return (bf16)x; }
__device__ __forceinline__ float to_f32(bf16 x) { return (float)x; }

// Round two floats to bf16 (round to nearest even) and back, converting them as
// one packed pair (one v_cvt_pk_bf16_f32 instead of one per value).
__device__ __forceinline__ void round_bf16_pair(float& a, float& b) {
  const bf16x2 v = {to_bf16(a), to_bf16(b)};
  uint32_t w = __builtin_bit_cast(uint32_t, v);
  asm volatile("" : "+v"(w));  // keep the pair packed in one register
  a = __uint_as_float(w << 16);
  b = __uint_as_float(w & 0xffff0000u);
}

// Eight consecutive accumulator registers (starting at r0) packed to bf16 as one
// MFMA operand: register r0+i becomes element i.
__device__ __forceinline__ bf16x8 pack8(const float* p) {
  bf16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = to_bf16(p[i]);
  return r;
}

// acc + the sum of eight bf16 values (v_dot2_f32_bf16 against (1, 1): two
// elements per instruction, fp32 accumulation).
__device__ __forceinline__ float sum8_bf16(const bf16x8& v, float acc) {
  const bf16x2 one = {(bf16)1.0f, (bf16)1.0f};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const bf16x2 pair = {v[2 * i], v[2 * i + 1]};
    acc = __builtin_amdgcn_fdot2_f32_bf16(pair, one, acc, false);
  }
  return acc;
}

// x from another lane of the same DPP row (16 lanes), selected by a DPP control
template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

// Sum over aligned groups of LPR lanes (8, 16 or 32), every lane receiving its
// group's sum: lane ^ 1 and lane ^ 2 (quad permutes), then the mirrored lane
// within 8 (the other quad) and within 16 (the other half), then lane ^ 16.
template <int LPR>
__device__ __forceinline__ float row_sum(float x) {
  static_assert(LPR == 8 || LPR == 16 || LPR == 32, "rows span 8, 16 or 32 lanes");
  x += dpp<0xB1>(x);   // quad_perm [1,0,3,2]
  x += dpp<0x4E>(x);   // quad_perm [2,3,0,1]
  x += dpp<0x141>(x);  // row_half_mirror
  if constexpr (LPR >= 16) x += dpp<0x140>(x);  // row_mirror
  if constexpr (LPR == 32) x += __shfl_xor(x, 16);
  return x;
}

// Combine a value with the one held by lane l ^ 32 (v_permlane32_swap on gfx950:
// the swap of the two half-waves leaves lane l holding both x_l and x_{l^32}).
__device__ __forceinline__ float wave_max_pair(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float wave_sum_pair(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Keep the compiler from moving instructions across this point (used to issue
// a batch of operand loads before the MFMAs that consume them).
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }

// log sigmoid(x) = min(x, 0) - log1p(exp(-|x|)), overflow-free for any finite x.
__device__ __forceinline__ float log_sigmoid(float x) {
  return fminf(x, 0.0f) - log1pf(expf(-fabsf(x)));
}

// ---------------------------------------------------------------------------
// The forget gates of one (batch, head) row, used only through differences of
// the prefix values, c_i - c_j (0-based positions).  Data-dependent gates pass
// the array c of fox_gate_prefix; a gate fixed per head, f_t = sigmoid(b)
// (the ALiBi form of Sec. 3), passes the biases b [H] and gets
// c_i - c_j = (i - j) log sigmoid(b) straight from the indices.
// ---------------------------------------------------------------------------
template <bool FIXED>
struct GateRow;
template <>
struct GateRow<false> {
  const float* c;
  __device__ GateRow(const float* gate, int /*bh*/, int /*H*/, size_t row)
      : c(gate + row) {}
  __device__ float diff(int i, int j) const { return c[i] - c[j]; }
  // the same difference split into loads (issued early) and arithmetic (later)
  __device__ float raw(int j) const { return c[j]; }
  __device__ float diff_raw(int, float ci, int, float cj) const { return ci - cj; }
};
template <>
struct GateRow<true> {
  float lf;
  __device__ GateRow(const float* gate, int bh, int H, size_t /*row*/)
      : lf(log_sigmoid(gate[bh % H])) {}
  // The slope passes through an empty asm at each use: otherwise the compiler
  // hoists products of it out of the tile loops and the kernels run out of
  // registers.
  __device__ float slope() const {
    float x = lf;
    asm volatile("" : "+v"(x));
    return x;
  }
  __device__ float diff(int i, int j) const { return (float)(i - j) * slope(); }
  __device__ float raw(int) const { return 0.0f; }
  __device__ float diff_raw(int i, float, int j, float) const { return (float)(i - j) * slope(); }
};

// ---------------------------------------------------------------------------
// Global -> LDS without registers (buffer_load ... lds).  One instruction moves
// 16 bytes per lane: lane l's bytes land at lds_wave_base + 16 * l, whatever
// global offset the lane asked for, and offsets at or beyond the resource's
// byte count read as zero (the hardware range check), which pads ragged tiles.
// ---------------------------------------------------------------------------
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  // word 3 = 0x00020000: 32-bit data format, the raw-buffer setting for gfx9-family parts
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           0x00020000);
}

constexpr int kNonTemporal = 2;  // cache policy of a buffer instruction: non-temporal

__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t rsrc, void* lds_wave_base,
                                      uint32_t voffset) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void_t*)lds_wave_base, 16, voffset, 0, 0, 0);
}

// The same for data read once: non-temporal, so that it does not displace what
// the caches hold for reuse.
__device__ __forceinline__ void dma16_nt(__amdgpu_buffer_rsrc_t rsrc, void* lds_wave_base,
                                         uint32_t voffset) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void_t*)lds_wave_base, 16, voffset, 0, 0,
                                           kNonTemporal);
}

// The same with 4 bytes per lane: lane l's dword lands at lds_wave_base + 4 * l.
__device__ __forceinline__ void dma4(__amdgpu_buffer_rsrc_t rsrc, void* lds_wave_base,
                                     uint32_t voffset) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void_t*)lds_wave_base, 4, voffset, 0, 0, 0);
}

// Workgroup barrier without the memory fence of __syncthreads() (which waits for
// every outstanding memory operation of the wave).  The caller must first wait
// for whatever other waves read after the barrier: its LDS writes (lgkmcnt) and
// its DMA into LDS (vmcnt).
__device__ __forceinline__ void barrier_no_fence() { asm volatile("s_barrier" ::: "memory"); }

// Wait until at most N vector-memory operations of this wave are outstanding
// (loads complete in order, so all but the last N issued are done); the LDS
// and export counts are left at their maxima (no wait).
template <int N>
__device__ __forceinline__ void wait_vmem() {
  static_assert(N >= 0 && N < 16, "vmcnt immediate");
  __builtin_amdgcn_s_waitcnt(0x0F70 | N);
}

// Wait until every outstanding memory operation of this wave (including the
// LDS-bound buffer loads above) has completed.
__device__ __forceinline__ void wait_all_memory() { __builtin_amdgcn_s_waitcnt(0); }
// Wait until every LDS operation of this wave has completed (s_waitcnt with
// lgkmcnt = 0 and the vector-memory and export counts at their maxima, which
// wait for nothing).
__device__ __forceinline__ void wait_lds() { __builtin_amdgcn_s_waitcnt(0xC07F); }

// Transposing LDS read (ds_read_b64_tr_b16).  Within each group of 16 lanes,
// lane j supplies the address of 4 consecutive bf16 in row (j / 4) of a 4 x 16
// block, columns 4 * (j % 4) .. +3; lane i of the group receives column i of the
// block, i.e. the 4 values of rows 0..3 in that column.
__device__ __forceinline__ bf16x4 lds_read_tr16(const bf16* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)p);
}

// LDS pointers with explicit address space (32-bit), for kernels whose LDS use
// exceeds the 64 KB reach of an instruction's immediate offset.
typedef __attribute__((address_space(3))) char lds_byte;
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8_t;
typedef __attribute__((address_space(3))) f32x4 lds_f32x4_t;
typedef __attribute__((address_space(3))) float lds_f32_t;

template <typename T>
__device__ __forceinline__ const lds_byte* lds_ptr(const T* generic) {
  return (const lds_byte*)generic;
}
// The same address, opaque to the compiler: accesses through it compile to this
// register plus an immediate offset instead of a precomputed register per
// access (which spills once the constant offsets pass 64 KB).
__device__ __forceinline__ const lds_byte* lds_opaque(const lds_byte* p) {
  asm volatile("" : "+v"(p));
  return p;
}

// Compile-time loop: f(std::integral_constant<int, I>()) for I = 0 .. N-1.
template <typename F, int... Is>
__device__ __forceinline__ void static_for_seq(F&& f, std::integer_sequence<int, Is...>) {
  (f(std::integral_constant<int, Is>()), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_seq(f, std::make_integer_sequence<int, N>());
}

// 32-bit LDS address of a shared-memory object.
template <typename T>
__device__ __forceinline__ uint32_t lds_addr(const T* p) {
  return (uint32_t)(uintptr_t)(const lds_byte*)p;
}

// The transposing read (ds_read_b64_tr_b16, see lds_read_tr16) at byte address
// base + OFF, issued as inline assembly.  Through the compiler builtin every such
// read first waits for all of the wave's outstanding LDS DMA (the compiler cannot
// tell the buffers apart), which would stall each tile on the next tile's loads;
// the tiles read here are never a DMA target while they are read.  The results
// are valid only after lds_wait() (LDS operations complete in order).
template <int OFF>
__device__ __forceinline__ bf16x4 ds_read_tr_asm(uint32_t base) {
  bf16x4 r;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(base), "i"(OFF));
  return r;
}
// Wait until at most N LDS operations of the wave are outstanding; the values
// are tied to the wait so that their users come after it.
template <int N>
__device__ __forceinline__ void lds_wait(bf16x4 (&r)[4]) {
  asm volatile("s_waitcnt lgkmcnt(%4)"
               : "+v"(r[0]), "+v"(r[1]), "+v"(r[2]), "+v"(r[3])
               : "i"(N));
}
template <int N>
__device__ __forceinline__ void lds_wait(bf16x4 (&r)[8]) {
  asm volatile("s_waitcnt lgkmcnt(%8)"
               : "+v"(r[0]), "+v"(r[1]), "+v"(r[2]), "+v"(r[3]), "+v"(r[4]), "+v"(r[5]),
                 "+v"(r[6]), "+v"(r[7])
               : "i"(N));
}
// The same for any number of reads: the wait, then each value passes through
// an empty asm that comes after it (volatile asm statements keep their order).
template <int N, int M>
__device__ __forceinline__ void lds_wait(bf16x4 (&r)[M]) {
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"i"(N));
#pragma unroll
  for (int i = 0; i < M; ++i) asm volatile("" : "+v"(r[i]));
}
__device__ __forceinline__ bf16x8 cat4(const bf16x4& lo, const bf16x4& hi) {
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// ---------------------------------------------------------------------------
// Swizzled LDS tiles: a [rows][D] bf16 tile stores the 16-byte chunk c of row r
// at chunk position c ^ f(r).  Two access patterns must be free of bank
// conflicts, whether the LDS serves 128 or 256 bytes per cycle:
//   * plain 16-byte operand reads: 8 (or 16) consecutive rows, same chunk;
//   * transposing reads: 4 consecutive rows (aligned to 4), 2 (or 4)
//     consecutive chunks (aligned).
// With r = (r3 r2 r1 r0) the masks below are linear maps chosen so that both
// sets of rows/chunks land on distinct chunk positions modulo 8 and 16:
//   D = 128 (16 chunks per row): f = r2 | r1 << 1 | r0 << 2 | (r3^r1^r0) << 3
//   D = 64  ( 8 chunks per row): f = r2 | (r0^r3) << 1 | r1 << 2
// ---------------------------------------------------------------------------
template <int D>
__device__ __forceinline__ int swz_chunk(int r, int c) {
  const int r0 = r & 1, r1 = (r >> 1) & 1, r2 = (r >> 2) & 1, r3 = (r >> 3) & 1;
  const int f = D == 128 ? (r2 | (r1 << 1) | (r0 << 2) | ((r3 ^ r1 ^ r0) << 3))
                         : (r2 | ((r0 ^ r3) << 1) | (r1 << 2));
  return c ^ f;
}

// Global byte offset (relative to the tile's first row) of the 16-byte chunk a
// wave's first DMA load moves for this lane: load i of wave w fills LDS slots
// [(i * NWAVES + w) * 64, +64), and slot s holds logical chunk swz(r, s % CPR) of
// row r = s / CPR.  One load covers NWAVES * 64 / CPR rows, a whole number of the
// swizzle's 16-row periods, so load i moves the chunks of load 0 shifted by
// i * tile_dma_stride<NWAVES>() bytes: one register per lane serves every load.
template <int D, int NWAVES>
__device__ __forceinline__ uint32_t tile_dma_offset(int wave, int lane) {
  static_assert((NWAVES * 64 / (D / 8)) % 16 == 0, "a DMA load covers whole 16-row periods");
  const int slot = wave * 64 + lane;
  const int r = slot / (D / 8);
  return (uint32_t)(r * D * 2 + swz_chunk<D>(r, slot % (D / 8)) * 16);
}
template <int NWAVES>
constexpr uint32_t tile_dma_stride() { return NWAVES * 64 * 16; }

// A wave-uniform value the compiler keeps in a scalar register and does not
// reassociate with per-lane terms (so no per-load sum is hoisted into a vector
// register).
__device__ __forceinline__ uint32_t uniform_u32(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_readfirstlane((int)x);
}

// Element offsets of a lane's plain MFMA-operand reads from a swizzled tile:
// row `row` (the lane's M or N index), contraction chunk 2s+h (elements 16s+8h..+7).
template <int D>
__device__ __forceinline__ void tile_row_offsets(int (&off)[D / 16], int row, int h) {
#pragma unroll
  for (int s = 0; s < D / 16; ++s) off[s] = row * D + swz_chunk<D>(row, 2 * s + h) * 8;
}

// Element offsets of a lane's transposing reads from a swizzled tile, giving the
// A operand X^T (rows = head dims, contraction = tile rows) of a 32x32x16 MFMA:
// for 16-row chunk 0, half k2 (rows 8*k2 + 4*h + 0..3) and 32-dim block db.  Add
// 16 * D * chunk for later chunks (the swizzle depends on the row modulo 16).
template <int D>
__device__ __forceinline__ void tile_tr_offsets(int (&off)[2][D / 32], int lane) {
  const int g16 = lane >> 4, j16 = lane & 15;
#pragma unroll
  for (int k2 = 0; k2 < 2; ++k2) {
    const int r = 8 * k2 + 4 * (g16 >> 1) + (j16 >> 2);
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
      const int e = db * 32 + 16 * (g16 & 1) + 4 * (j16 & 3);
      off[k2][db] = r * D + swz_chunk<D>(r, e >> 3) * 8 + (e & 7);
    }
  }
}

// The A operand X^T[db block][16-row chunk c] from a swizzled tile.
template <int D>
__device__ __forceinline__ bf16x8 tile_tr_operand(const bf16* tile, const int (&off)[2][D / 32],
                                                  int c, int db) {
  const bf16x4 lo = lds_read_tr16(tile + c * 16 * D + off[0][db]);
  const bf16x4 hi = lds_read_tr16(tile + c * 16 * D + off[1][db]);
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

}  // namespace fox
