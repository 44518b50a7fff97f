// HBM-bound kernels of the SP attention library (gfx950):
//   * Ulysses pack / unpack with dummy-head zero fill (Listing 1 pad/unpad
//     around the all-to-all layout of Section 4), and the summing unpack of
//     GQA K/V gradients replicated to several ranks,
//   * the log-sum-exp merge of two partial attention results (ring combine,
//     Section 2.1),
//   * fills, bf16 casts, the backward's row dot D_i = dO_i . O_i, and the
//     GQA reduction of per-query-head dK/dV partials.
// All accesses are 16-byte vectors; consecutive lanes touch consecutive
// 16-byte chunks of a row.
#include <algorithm>

#include "dev_common.h"
#include "launch.h"

namespace spk {

static constexpr int kBlock = 256;
static constexpr int kMaxBlocks = 256 * 32;  // grid-stride beyond this

static inline int grid_for(int64_t n_threads) {
  int64_t b = (n_threads + kBlock - 1) / kBlock;
  if (b < 1) b = 1;
  return (int)(b > kMaxBlocks ? kMaxBlocks : b);
}

// ---------------------------------------------------------------- pack
// The copies run one (destination slot or head) per grid row (blockIdx.y),
// so the head map is read once per block at a uniform index; inside a block
// thread e of the row handles 16-byte chunks e, e + kBlock, ... of the
// T x nch (row, chunk) plane with 32-bit index arithmetic, streaming loads
// issued before streaming stores.  Rows are 16 * nch bytes apart on both sides (whole cache
// lines for D = 64 and 128).  Planes past 2^31 chunks take 64-bit indices.
static constexpr int kPer = 4;  // 16-byte chunks per thread

template <typename I>
SP_DEV void plane_index(I e, int nch, int lg, I& t, int& c) {
  if (lg >= 0) {
    t = e >> lg;
    c = (int)(e & (I)(nch - 1));
  } else {
    t = e / nch;
    c = (int)(e % nch);
  }
}

static inline int log2_or_neg(int n) {
  return (n > 0 && (n & (n - 1)) == 0) ? __builtin_ctz(n) : -1;
}

// dst[j, t, h, c] = src[t, map[j*Hd + h], c] or 0 (blockIdx.y = j*Hd + h).
template <typename I>
__global__ __launch_bounds__(kBlock) void pack_kernel(const u32x4* __restrict__ src,
                                                      u32x4* __restrict__ dst, PackArgs a,
                                                      int lg) {
  const int slot = blockIdx.y;
  const int j = slot / a.Hd, h = slot - j * a.Hd;
  const int g = a.map[slot];
  const I n = (I)a.T * a.nch;
  const I e0 = (I)blockIdx.x * (kBlock * kPer) + threadIdx.x;
  u32x4 v[kPer];
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const I e = e0 + (I)k * kBlock;
    v[k] = u32x4{0u, 0u, 0u, 0u};
    if (g >= 0 && e < n) {
      I t;
      int c;
      plane_index<I>(e, a.nch, lg, t, c);
      v[k] = ld_stream(&src[(t * a.Hs + g) * a.nch + c]);
    }
  }
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const I e = e0 + (I)k * kBlock;
    if (e < n) {
      I t;
      int c;
      plane_index<I>(e, a.nch, lg, t, c);
      st_stream(v[k], &dst[(((I)j * a.T + t) * a.Hd + h) * a.nch + c]);
    }
  }
}

// dst[t, g, c] = src[j, t, h, c] with map[g] = j*Hs + h (blockIdx.y = g).
template <typename I>
__global__ __launch_bounds__(kBlock) void unpack_kernel(const u32x4* __restrict__ src,
                                                        u32x4* __restrict__ dst, PackArgs a,
                                                        int lg) {
  const int g = blockIdx.y;
  const int s = a.map[g];
  const int j = s / a.Hs, h = s - j * a.Hs;
  const I n = (I)a.T * a.nch;
  const I e0 = (I)blockIdx.x * (kBlock * kPer) + threadIdx.x;
  u32x4 v[kPer];
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const I e = e0 + (I)k * kBlock;
    if (e < n) {
      I t;
      int c;
      plane_index<I>(e, a.nch, lg, t, c);
      v[k] = ld_stream(&src[(((I)j * a.T + t) * a.Hs + h) * a.nch + c]);
    }
  }
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const I e = e0 + (I)k * kBlock;
    if (e < n) {
      I t;
      int c;
      plane_index<I>(e, a.nch, lg, t, c);
      st_stream(v[k], &dst[(t * a.Hd + g) * a.nch + c]);
    }
  }
}

// dst[t, g, c] = sum over the slots s = j*Hs + h listed for g (ascending) of
// src[j, t, h, c]: eight bf16 per 16-byte chunk, summed in float32 one slot
// at a time, rounded once to bf16 (nearest-even); no slot gives +0
// (blockIdx.y = g).  Each thread has two chunks of the plane in flight and,
// per chunk, up to eight slots' loads before the additions.
template <typename I>
__global__ __launch_bounds__(kBlock) void unpack_add_kernel(const u32x4* __restrict__ src,
                                                            u32x4* __restrict__ dst,
                                                            PackAddArgs a, int lg) {
  constexpr int P = 2, NS = 8;
  const int g = blockIdx.y;
  const int i0 = a.start[g], i1 = a.start[g + 1];
  const I n = (I)a.T * a.nch;
  const I e0 = (I)blockIdx.x * (kBlock * P) + threadIdx.x;
  auto add = [](float* acc, const u32x4& v) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      acc[2 * k] += __uint_as_float(v[k] << 16);
      acc[2 * k + 1] += __uint_as_float(v[k] & 0xffff0000u);
    }
  };
  float acc[P][8];
  I t[P];
  int c[P];
#pragma unroll
  for (int p = 0; p < P; ++p) {
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[p][i] = 0.f;
    plane_index<I>(e0 + (I)p * kBlock, a.nch, lg, t[p], c[p]);
  }
  for (int b = i0; b < i1; b += NS) {
    u32x4 v[P][NS];
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      if (b + k < i1) {
        const int s = a.slot[b + k];
        const int j = s / a.Hs, h = s - j * a.Hs;
#pragma unroll
        for (int p = 0; p < P; ++p)
          if (e0 + (I)p * kBlock < n)
            v[p][k] = ld_stream(&src[(((I)j * a.T + t[p]) * a.Hs + h) * a.nch + c[p]]);
      }
    }
#pragma unroll
    for (int k = 0; k < NS; ++k)
      if (b + k < i1)
#pragma unroll
        for (int p = 0; p < P; ++p)
          if (e0 + (I)p * kBlock < n) add(acc[p], v[p][k]);
  }
#pragma unroll
  for (int p = 0; p < P; ++p)
    if (e0 + (I)p * kBlock < n)
      st_stream(pack_bf16x8(acc[p][0], acc[p][1], acc[p][2], acc[p][3], acc[p][4], acc[p][5],
                            acc[p][6], acc[p][7]),
                &dst[(t[p] * a.Hd + g) * a.nch + c[p]]);
}

// 32-bit indices when every chunk index of both tensors (plus a block's
// overshoot) fits; x blocks of the grid must fit as well.
static inline bool fits32(int64_t chunks) { return chunks + kBlock * kPer < ((int64_t)1 << 31); }
static inline bool grid_ok(int64_t blocks) { return blocks <= 0x7fffffff; }

hipError_t launch_pack(const void* src, void* dst, const PackArgs& a, hipStream_t st) {
  const int64_t n = (int64_t)a.T * a.nch;
  if (n == 0) return hipSuccess;
  const int64_t bx = (n + kBlock * kPer - 1) / (kBlock * kPer);
  if (!grid_ok(bx)) return hipErrorInvalidValue;
  const dim3 grid((unsigned)bx, a.sp * a.Hd);
  const int lg = log2_or_neg(a.nch);
  if (fits32(std::max((int64_t)a.Hs, (int64_t)a.sp * a.Hd) * n))
    return sp_launch(kKPack, pack_kernel<int>, grid, dim3(kBlock), st, (const u32x4*)src,
                     (u32x4*)dst, a, lg);
  return sp_launch(kKPack, pack_kernel<int64_t>, grid, dim3(kBlock), st, (const u32x4*)src,
                   (u32x4*)dst, a, lg);
}

hipError_t launch_unpack_add(const void* src, void* dst, const PackAddArgs& a, hipStream_t st) {
  const int64_t n = (int64_t)a.T * a.nch;
  if (n == 0) return hipSuccess;
  const int64_t bx = (n + kBlock * 2 - 1) / (kBlock * 2);
  if (!grid_ok(bx)) return hipErrorInvalidValue;
  const dim3 grid((unsigned)bx, a.Hd);
  const int lg = log2_or_neg(a.nch);
  if (fits32(std::max((int64_t)a.sp * a.Hs, (int64_t)a.Hd) * n))
    return sp_launch(kKUnpackAdd, unpack_add_kernel<int>, grid, dim3(kBlock), st,
                     (const u32x4*)src, (u32x4*)dst, a, lg);
  return sp_launch(kKUnpackAdd, unpack_add_kernel<int64_t>, grid, dim3(kBlock), st,
                   (const u32x4*)src, (u32x4*)dst, a, lg);
}

hipError_t launch_unpack(const void* src, void* dst, const PackArgs& a, hipStream_t st) {
  const int64_t n = (int64_t)a.T * a.nch;
  if (n == 0) return hipSuccess;
  const int64_t bx = (n + kBlock * kPer - 1) / (kBlock * kPer);
  if (!grid_ok(bx)) return hipErrorInvalidValue;
  const dim3 grid((unsigned)bx, a.Hd);
  const int lg = log2_or_neg(a.nch);
  if (fits32(std::max((int64_t)a.sp * a.Hs, (int64_t)a.Hd) * n))
    return sp_launch(kKUnpack, unpack_kernel<int>, grid, dim3(kBlock), st, (const u32x4*)src,
                     (u32x4*)dst, a, lg);
  return sp_launch(kKUnpack, unpack_kernel<int64_t>, grid, dim3(kBlock), st, (const u32x4*)src,
                   (u32x4*)dst, a, lg);
}

// ---------------------------------------------------------------- merge
// Each group of D/8 consecutive lanes (a power of two dividing 64) owns one
// (t, h) row, so the in-place LSE update happens after every lane of the row
// has read it (same wavefront, program order).
SP_DEV void merge_weights(float la, float lb, float& wa, float& wb, float& L) {
  float m = fmaxf(la, lb);
  if (m == neg_inf()) {
    wa = 0.f; wb = 0.f; L = neg_inf();
    return;
  }
  float ea = expf(la - m), eb = expf(lb - m);  // exp(-inf) = 0
  float s = ea + eb;
  L = m + logf(s);
  float inv = 1.f / s;
  wa = ea * inv;
  wb = eb * inv;
}

template <bool PART_BF16>
__global__ __launch_bounds__(kBlock) void merge_kernel(float* __restrict__ o_acc,
                                                       float* __restrict__ lse_acc,
                                                       const void* __restrict__ o_part,
                                                       const float* __restrict__ lse_part,
                                                       uint16_t* __restrict__ o_out, int T, int H,
                                                       int D) {
  const int n8 = D >> 3;
  const int64_t n = (int64_t)T * H * n8;
  for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < n;
       e += (int64_t)gridDim.x * kBlock) {
    int c = (int)(e % n8);
    int64_t row = e / n8;  // t*H + h
    int h = (int)(row % H);
    int t = (int)(row / H);
    int64_t li = (int64_t)h * T + t;
    float la = lse_acc[li], lb = lse_part[li];
    float wa, wb, L;
    merge_weights(la, lb, wa, wb, L);
    float4* oa = (float4*)(o_acc + row * D + c * 8);
    float4 a0 = oa[0], a1 = oa[1];
    float b[8];
    if constexpr (PART_BF16) {
      u32x4 pv = ((const u32x4*)o_part)[row * n8 + c];
      for (int i = 0; i < 4; ++i) {
        b[2 * i] = __uint_as_float(pv[i] << 16);
        b[2 * i + 1] = __uint_as_float(pv[i] & 0xffff0000u);
      }
    } else {
      const float4* pb = (const float4*)((const float*)o_part + row * D + c * 8);
      float4 p0 = pb[0], p1 = pb[1];
      b[0] = p0.x; b[1] = p0.y; b[2] = p0.z; b[3] = p0.w;
      b[4] = p1.x; b[5] = p1.y; b[6] = p1.z; b[7] = p1.w;
    }
    float r[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
    for (int i = 0; i < 8; ++i) r[i] = wa * r[i] + wb * b[i];
    oa[0] = make_float4(r[0], r[1], r[2], r[3]);
    oa[1] = make_float4(r[4], r[5], r[6], r[7]);
    if (o_out) ((u32x4*)o_out)[row * n8 + c] = pack_bf16x8(r[0], r[1], r[2], r[3], r[4], r[5], r[6], r[7]);
    if (c == 0) lse_acc[li] = L;
  }
}

hipError_t launch_merge(float* o_acc, float* lse_acc, const void* o_part, bool part_bf16,
                        const float* lse_part, int T, int H, int D, void* o_out, hipStream_t st) {
  int64_t n = (int64_t)T * H * (D / 8);
  if (n == 0) return hipSuccess;
  // keep whole rows inside one wavefront: the grid-stride step must be a
  // multiple of the row's lane count, which kBlock * grid already is.
  if (part_bf16)
    return sp_launch(kKMerge, merge_kernel<true>, dim3(grid_for(n)), dim3(kBlock), st, o_acc,
                     lse_acc, o_part, lse_part, (uint16_t*)o_out, T, H, D);
  return sp_launch(kKMerge, merge_kernel<false>, dim3(grid_for(n)), dim3(kBlock), st, o_acc,
                   lse_acc, o_part, lse_part, (uint16_t*)o_out, T, H, D);
}

// ---------------------------------------------------------------- fills
// Fill heads [h0, h1) of every row of a [T, H, D] bf16 tensor with zero.
__global__ __launch_bounds__(kBlock) void zero_heads_bf16_kernel(u32x4* __restrict__ x, int T,
                                                                 int H, int nch, int h0, int h1) {
  const int per_row = (h1 - h0) * nch;
  const int64_t n = (int64_t)T * per_row;
  for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < n;
       e += (int64_t)gridDim.x * kBlock) {
    int t = (int)(e / per_row);
    int w = (int)(e % per_row);
    x[((int64_t)t * H + h0) * nch + w] = u32x4{0u, 0u, 0u, 0u};
  }
}

hipError_t launch_zero_heads_bf16(void* x, int T, int H, int D, int h0, int h1, hipStream_t st) {
  if (h1 <= h0 || T == 0) return hipSuccess;
  int64_t n = (int64_t)T * (h1 - h0) * (D / 8);
  hipLaunchKernelGGL(zero_heads_bf16_kernel, dim3(grid_for(n)), dim3(kBlock), 0, st, (u32x4*)x, T,
                     H, D / 8, h0, h1);
  return hipGetLastError();
}

__global__ __launch_bounds__(kBlock) void fill_f32_kernel(float* __restrict__ x, int64_t n,
                                                          float v) {
  for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < n;
       e += (int64_t)gridDim.x * kBlock)
    x[e] = v;
}

hipError_t launch_fill_f32(float* x, int64_t n, float v, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_f32_kernel, dim3(grid_for(n)), dim3(kBlock), 0, st, x, n, v);
  return hipGetLastError();
}

// Fill heads [h0, h1) of a float32 [T, H, D] tensor with zero (o_acc dummies).
__global__ __launch_bounds__(kBlock) void zero_heads_f32_kernel(float4* __restrict__ x, int T, int H,
                                                                int n4, int h0, int h1) {
  const int per_row = (h1 - h0) * n4;
  const int64_t n = (int64_t)T * per_row;
  for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < n;
       e += (int64_t)gridDim.x * kBlock) {
    int t = (int)(e / per_row);
    int w = (int)(e % per_row);
    x[((int64_t)t * H + h0) * n4 + w] = make_float4(0.f, 0.f, 0.f, 0.f);
  }
}

hipError_t launch_zero_heads_f32(float* x, int T, int H, int D, int h0, int h1, hipStream_t st) {
  if (h1 <= h0 || T == 0) return hipSuccess;
  int64_t n = (int64_t)T * (h1 - h0) * (D / 4);
  hipLaunchKernelGGL(zero_heads_f32_kernel, dim3(grid_for(n)), dim3(kBlock), 0, st, (float4*)x, T,
                     H, D / 4, h0, h1);
  return hipGetLastError();
}

__global__ __launch_bounds__(kBlock) void f32_to_bf16_kernel(const float* __restrict__ s,
                                                             uint16_t* __restrict__ d, int64_t n) {
  const int64_t n8 = n >> 3;
  for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < n8;
       e += (int64_t)gridDim.x * kBlock) {
    const float4* p = (const float4*)(s + e * 8);
    float4 a = p[0], b = p[1];
    ((u32x4*)d)[e] = pack_bf16x8(a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w);
  }
  // tail (n % 8) handled by the first threads
  int64_t tail0 = n8 * 8;
  int64_t t = tail0 + (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (t < n) {
    f32x2 v = {s[t], 0.f};
    bf16x2 r = __builtin_convertvector(v, bf16x2);
    d[t] = (uint16_t)(__builtin_bit_cast(uint32_t, r) & 0xffffu);
  }
}

hipError_t launch_f32_to_bf16(const float* s, void* d, int64_t n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(f32_to_bf16_kernel, dim3(grid_for((n + 7) / 8)), dim3(kBlock), 0, st, s,
                     (uint16_t*)d, n);
  return hipGetLastError();
}

// ---------------------------------------------------------------- row dot
// neg_d[y][t] = -sum_d dO[t][y][d] * O[t][y][d]  (float32, -D of the
// backward), y < nh, t < T;
// lse2[y][t] = LSE[y][t] * log2(e) (+inf where LSE = -inf: rows without keys).
template <int D>
__global__ __launch_bounds__(kBlock) void rowdot_kernel(const uint16_t* __restrict__ o,
                                                        const uint16_t* __restrict__ dout,
                                                        const float* __restrict__ lse,
                                                        float* __restrict__ neg_d,
                                                        float* __restrict__ lse2, int T, int H,
                                                        int nh) {
  constexpr int NC = D / 8;  // lanes per row
  const int64_t rows = (int64_t)T * nh;
  const int64_t gid = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  const int64_t row = gid / NC;
  const int c = (int)(gid % NC);
  float s = 0.f;
  int t = 0, y = 0;
  if (row < rows) {
    y = (int)(row % nh);
    t = (int)(row / nh);
    int64_t off = ((int64_t)t * H + y) * D + c * 8;
    u32x4 va = *(const u32x4*)(o + off);
    u32x4 vb = *(const u32x4*)(dout + off);
    for (int i = 0; i < 4; ++i) {
      s += __uint_as_float(va[i] << 16) * __uint_as_float(vb[i] << 16);
      s += __uint_as_float(va[i] & 0xffff0000u) * __uint_as_float(vb[i] & 0xffff0000u);
    }
  }
  for (int m = NC / 2; m >= 1; m >>= 1) s += __shfl_xor(s, m);
  if (row < rows && c == 0) {
    const int64_t i = (int64_t)y * T + t;
    neg_d[i] = -s;
    const float l = lse[i];
    lse2[i] = (l == neg_inf()) ? __builtin_inff() : l * kLog2e;
  }
}

hipError_t launch_rowdot(const void* o, const void* dout, const float* lse, float* neg_d,
                         float* lse2, int T, int H, int nh, int D, hipStream_t st) {
  int64_t n = (int64_t)T * nh * (D / 8);
  if (n == 0) return hipSuccess;
  int grid = (int)((n + kBlock - 1) / kBlock);
  if (D == 128)
    hipLaunchKernelGGL(rowdot_kernel<128>, dim3(grid), dim3(kBlock), 0, st, (const uint16_t*)o,
                       (const uint16_t*)dout, lse, neg_d, lse2, T, H, nh);
  else
    hipLaunchKernelGGL(rowdot_kernel<64>, dim3(grid), dim3(kBlock), 0, st, (const uint16_t*)o,
                       (const uint16_t*)dout, lse, neg_d, lse2, T, H, nh);
  return hipGetLastError();
}

// ------------------------------------------------------- GQA dK/dV reduce
// out[t][kv][d] = bf16( sum_{y in heads of kv} part[y][t][d] ), ascending y;
// dK (blockIdx.y = 0) and dV (blockIdx.y = 1) in one launch.
__global__ __launch_bounds__(kBlock) void reduce_kv_kernel(const float* __restrict__ part_k,
                                                           const float* __restrict__ part_v,
                                                           uint16_t* __restrict__ dk,
                                                           uint16_t* __restrict__ dv,
                                                           ReduceArgs a) {
  const float* part = blockIdx.y ? part_v : part_k;
  uint16_t* out = blockIdx.y ? dv : dk;
  const int n8 = a.D >> 3;
  const int64_t n = (int64_t)a.T * a.Hkv * n8;
  for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < n;
       e += (int64_t)gridDim.x * kBlock) {
    int c = (int)(e % n8);
    int64_t r = e / n8;
    int kv = (int)(r % a.Hkv);
    int t = (int)(r / a.Hkv);
    float s[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    int y0 = a.head_lo[kv], y1 = a.head_hi[kv];
    for (int y = y0; y < y1; ++y) {
      const float4* p = (const float4*)(part + ((int64_t)y * a.T + t) * a.D + c * 8);
      float4 u = p[0], w = p[1];
      s[0] += u.x; s[1] += u.y; s[2] += u.z; s[3] += u.w;
      s[4] += w.x; s[5] += w.y; s[6] += w.z; s[7] += w.w;
    }
    ((u32x4*)out)[e] = pack_bf16x8(s[0], s[1], s[2], s[3], s[4], s[5], s[6], s[7]);
  }
}

hipError_t launch_reduce_kv(const float* part_k, const float* part_v, void* dk, void* dv,
                            const ReduceArgs& a, hipStream_t st) {
  int64_t n = (int64_t)a.T * a.Hkv * (a.D / 8);
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(reduce_kv_kernel, dim3(grid_for(n), 2), dim3(kBlock), 0, st, part_k, part_v,
                     (uint16_t*)dk, (uint16_t*)dv, a);
  return hipGetLastError();
}

}  // namespace spk
