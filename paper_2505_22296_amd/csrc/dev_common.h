// Device-side helpers shared by the gfx950 kernels of the SP attention library.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define SP_DEV __device__ __forceinline__

static constexpr float kLog2e = 1.4426950408889634f;
static constexpr float kLn2 = 0.6931471805599453f;

SP_DEV float neg_inf() { return -__builtin_inff(); }

// 32x32x16 bf16 MFMA (fp32 accumulate).  Operand layouts (verified on gfx950):
//   A (32 x 16): lane l holds row l%32, k = (l/32)*8 + [0..7]
//   B (16 x 32): lane l holds col l%32, k = (l/32)*8 + [0..7]
//   C (32 x 32): lane l holds col l%32, register r is row (r/4)*8 + (l/32)*4 + r%4
SP_DEV f32x16 mfma32(const u32x4& a, const u32x4& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                  __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// Round 8 floats to bf16 (RNE, v_cvt_pk_bf16_f32) and pack into 16 bytes.
// Streaming 16-byte accesses for data a kernel touches exactly once (the
// Ulysses copies, the logits of the loss path): non-temporal loads and
// stores, so the lines are not kept in the caches for reuse that never
// comes (measured 1.1-1.25x the bandwidth of plain accesses on these copies).
SP_DEV u32x4 ld_stream(const u32x4* p) { return __builtin_nontemporal_load(p); }
SP_DEV void st_stream(const u32x4& v, u32x4* p) { __builtin_nontemporal_store(v, p); }

SP_DEV u32x4 pack_bf16x8(float a0, float a1, float a2, float a3, float a4, float a5, float a6,
                         float a7) {
  f32x8 v = {a0, a1, a2, a3, a4, a5, a6, a7};
  return __builtin_bit_cast(u32x4, __builtin_convertvector(v, bf16x8));
}
SP_DEV u32x2 pack_bf16x4(float a0, float a1, float a2, float a3) {
  f32x4 v = {a0, a1, a2, a3};
  return __builtin_bit_cast(u32x2, __builtin_convertvector(v, bf16x4));
}
SP_DEV float bf16_to_f32(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

// Row permutation used for MFMA A operands whose C result feeds a later MFMA as
// a B operand: A row m is loaded from physical row perm32(m) so that, in the C
// layout, lane half h of register block r/8 holds the 8 consecutive physical
// rows (r/8)*16 + h*8 + [0..7] -- exactly a B operand's k-slice.
SP_DEV int perm32(int m) { return ((m >> 4) << 4) | (((m >> 2) & 1) << 3) | (((m >> 3) & 1) << 2) | (m & 3); }

// Physical index (row or key) held by C register r of lane half h after an
// A operand loaded with perm32 rows.
SP_DEV int c_row_of(int r, int h) { return ((r >> 3) << 4) + (h << 3) + (r & 7); }

// XOR swizzle of 16-byte chunks inside an LDS tile row, so that 8 lanes that
// read the same logical chunk of 8 different rows hit distinct banks.
// `nch` = 16-byte chunks per row (8 or 16).
template <int NCH>
SP_DEV int swz_chunk(int row, int chunk) {
  if constexpr (NCH >= 16) {
    return chunk ^ (row & 15);
  } else {
    // two 128-byte rows share one 256-byte bank window
    return chunk ^ ((row >> 1) & 7);
  }
}
template <int NCH>
SP_DEV int swz(int row, int chunk) { return row * NCH + swz_chunk<NCH>(row, chunk); }

// ---- Blocked LDS tiles: a [ROWS][D] bf16 tile is stored as D/32 sub-tiles
// [ROWS][32] (64-byte rows, four 16-byte chunks), chunk c of row r at
// position c ^ ((r >> 2) & 3).  Sixteen consecutive rows at one logical chunk
// and four consecutive rows x four chunks both hit distinct banks, so plain
// fragment reads (rows on lanes) and transposed reads (ds_read_b64_tr_b16,
// tile rows become the k index) are conflict-free; the sub-tile index is an
// immediate offset.
SP_DEV int blk_chunk(int row, int chunk) { return chunk ^ ((row >> 2) & 3); }

// Chunk index (16-byte units) of tile row `row`, logical 16-byte chunk
// `chunk` of D, in a blocked tile of ROWS rows.
template <int ROWS>
SP_DEV int blk_idx(int row, int chunk) {
  return (chunk >> 2) * (ROWS * 4) + row * 4 + blk_chunk(row, chunk & 3);
}

typedef short s16x4 __attribute__((ext_vector_type(4)));

// gfx950 ds_read_b64_tr_b16 (lane layout measured on the GPU): within each
// group of 16 lanes, output lane j element e is input lane 4e + j/4's
// element j%4, where every input lane reads 4 consecutive 16-bit values.
SP_DEV u32x2 lds_tr16(const void* p) {
  s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)p);
  return __builtin_bit_cast(u32x2, v);
}

// Per-lane element offset (within one sub-tile of a blocked tile) of the
// transposed MFMA A-operand read: the fragment A[m][k] = T[k][m] (m = 32
// columns of the sub-tile, k = 16 tile rows from row 0) is two tr16 reads at
// this offset and at +4 rows; k-steps add 16 rows, sub-tiles ROWS*32 elements.
SP_DEV int blk_tr_off(int lane) {
  const int grp = lane >> 4, j = lane & 15;
  const int row = (grp >> 1) * 8 + (j >> 2);         // + 4 for the second read
  const int col = (grp & 1) * 16 + 4 * (j & 3);
  return row * 32 + blk_chunk(row, col >> 3) * 8 + (col & 7);
}
// The second read's rows are 4 further on, which flips bit 0 of (row >> 2).
SP_DEV int blk_tr_off2(int lane) {
  const int grp = lane >> 4, j = lane & 15;
  const int row = (grp >> 1) * 8 + 4 + (j >> 2);
  const int col = (grp & 1) * 16 + 4 * (j & 3);
  return row * 32 + blk_chunk(row, col >> 3) * 8 + (col & 7);
}

// max(a, b, c) as one gfx950 v_maximum3_f32 (NaN-propagating maximum).
// fmaxf in IEEE mode first quiets every operand that could be a signalling
// NaN (one v_max_f32 per MFMA result); the NaN-propagating form needs no
// quieting and, for operands that are never NaN (scores: finite or -inf),
// gives the same value.  Compiler-visible, so the wait states after the
// MFMAs that produce the operands are inserted as for any VALU read.
SP_DEV float max3_nonan(float a, float b, float c) {
  return __builtin_elementwise_maximum(a, __builtin_elementwise_maximum(b, c));
}

// Combine a value with the one of lane l^32 through v_permlane32_swap_b32
// (a VALU op; a shuffle would go through LDS with ds_bpermute).  Called with
// the same register as both operands, the swap returns {x[l & 31], x[l | 32]}
// in some order on every lane, so max / sum of the two is the xor-32 result.
// The max is the NaN-propagating one: its operands (row maxima of scores)
// are never NaN, and it needs no quieting.
SP_DEV float wave_max_xor32(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __builtin_elementwise_maximum(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
SP_DEV float wave_sum_xor32(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Direct global -> LDS copy of 16 (4) bytes per lane (gfx950
// global_load_lds_dwordx4 / _dword).  `lds_block` must be wave-uniform: lane
// i's bytes land at lds_block + 16 i (4 i).  Completion is tracked by vmcnt
// only; callers wait with wait_vmcnt<N>() and a barrier before other
// wavefronts read the data, and never copy into a stage that is being read.
// The copies are issued from inline assembly on purpose: the compiler treats
// an LDS DMA it can see as a pending write to all of LDS and inserts
// s_waitcnt vmcnt(0) before every later LDS read and barrier, which drains
// the multi-stage prefetch on every tile.  Hidden from it, the only vmcnt
// waits are the explicit ones of the staging protocol.  The s_nop is the one
// wait state the gfx9 family requires between an SALU write of M0 and an LDS
// DMA that reads it (the compiler adds it for the DMAs it generates itself).
SP_DEV uint32_t lds_addr(const void* lds_block) {
  return __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)lds_block);
}
SP_DEV void dma16(const void* gsrc, void* lds_block) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :: "v"(gsrc), "s"(lds_addr(lds_block)) : "memory", "m0");
}
// The same 16-byte copy from a wavefront-uniform base (SGPR pair) plus a
// per-lane 32-bit byte offset (global saddr addressing): a tile's base moves
// with scalar arithmetic and the lane offsets stay fixed from tile to tile.
SP_DEV void dma16s(const void* sbase, uint32_t voff, void* lds_block) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(voff), "s"(sbase), "s"(lds_addr(lds_block)) : "memory", "m0");
}
SP_DEV void dma4(const void* gsrc, void* lds_block) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off"
               :: "v"(gsrc), "s"(lds_addr(lds_block)) : "memory", "m0");
}
// s_waitcnt vmcnt(N) leaving expcnt / lgkmcnt unconstrained (gfx9 encoding).
template <int N>
SP_DEV void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
// Wait until at most `pending` (0 <= pending <= P) batches of PER copies are
// still in flight (the wave issues the same number of copies per batch).
template <int PER, int P>
SP_DEV void wait_batches(int pending) {
  if constexpr (P > 0) {
    if (pending >= P) {
      wait_vmcnt<P * PER>();
      return;
    }
    wait_batches<PER, P - 1>(pending);
  } else {
    wait_vmcnt<0>();
  }
}

// The 8 int32 of work item `pos`, read through the scalar cache (the list is
// not written during a launch).  A plain read can become a vector load with a
// full wait per field when the compiler cannot prove that no store of the
// kernel precedes it.
SP_DEV void load_item(const int32_t* items, int64_t pos, int32_t (&v)[8]) {
  typedef const __attribute__((address_space(4))) int32_t cint;
  cint* p = (cint*)(items + pos * 8);
#pragma unroll
  for (int j = 0; j < 8; ++j) v[j] = p[j];
}

// Zero-fill work items (dummy query slots, unread KV heads): the whole
// workgroup writes rows [r0, r1) of head h of a [T, H, D] tensor with 16-byte
// stores, block-strided.  bf16 (zero = +0) and float32 variants.
SP_DEV void fill_rows_bf16(uint16_t* x, int r0, int r1, int H, int h, int D, int tid, int nt) {
  const int nch = D / 8;
  const int64_t n = (int64_t)(r1 - r0) * nch;
  for (int64_t e = tid; e < n; e += nt) {
    const int64_t row = r0 + e / nch;
    *(u32x4*)(x + (row * H + h) * D + (e % nch) * 8) = u32x4{0u, 0u, 0u, 0u};
  }
}
SP_DEV void fill_rows_f32(float* x, int r0, int r1, int H, int h, int D, int tid, int nt) {
  const int nch = D / 4;
  const int64_t n = (int64_t)(r1 - r0) * nch;
  for (int64_t e = tid; e < n; e += nt) {
    const int64_t row = r0 + e / nch;
    *(f32x4*)(x + (row * H + h) * D + (e % nch) * 4) = f32x4{0.f, 0.f, 0.f, 0.f};
  }
}
SP_DEV void fill_span_f32(float* x, int n, float v, int tid, int nt) {
  for (int e = tid; e < n; e += nt) x[e] = v;
}
