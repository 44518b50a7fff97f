// Attention backward for one SP rank's real heads on gfx950 (deterministic:
// no atomics).  P is recomputed from the forward's LSE; with
// D_i = dO_i . O_i (precomputed per row):
//   dP = dO V^T,  dS = P (dP - D),  dQ = scale dS K,
//   dK = scale dS^T Q,  dV = P^T dO.
//
// dq kernel (query-stationary): workgroup = 128 query rows of one head,
//   wavefront w owns 32 rows; per 32-key tile (K, V row-major and K^T staged
//   in LDS):
//     S^T = K Q^T, dP^T = V dO^T     (Q, dO rows kept as B operands)
//     dS^T = P^T (dP^T - D)          (row statistics are per lane)
//     dQ^T += K^T dS^T               (dS^T C registers used directly as B)
// dk/dv kernel (key-stationary): workgroup = 128 keys of one KV head and
//   one query head, wavefront w owns 32 keys (K, V rows as B operands in
//   registers); per 32-row query chunk (Q, dO row-major and Q^T, dO^T
//   staged in LDS):
//     S = Q K^T, dP = dO V^T          (Q, dO rows loaded in perm32 order)
//     dS = P (dP - D)
//     dV^T += dO^T P, dK^T += Q^T dS (P, dS C registers used directly as B)
//   With one query head per KV head the results are written as bf16; under
//   GQA each query head writes a float32 partial that a reduction kernel
//   sums over the group in ascending head order.
#include "dev_common.h"
#include "launch.h"

namespace spk {

namespace {

constexpr int NT = 256;

// 4-chunk rows (32 bf16) share a 256-byte bank window in groups of four.
SP_DEV int swz4(int row, int chunk) { return row * 4 + (chunk ^ ((row >> 2) & 3)); }

// ------------------------------------------------------------------- dQ
template <int D>
__global__ __launch_bounds__(NT, 2) void attn_dq_kernel(DqArgs a) {
  constexpr int BN = kDqBN;    // 32 keys per tile
  constexpr int KS = D / 16;
  constexpr int DB = D / 32;
  constexpr int KCH = D / 8;
  constexpr int RLD = BN * KCH / NT;  // chunks per thread for a [32][D] tile
  constexpr int TLD = D * 4 / NT;     // chunks per thread for a [D][32] tile
  static_assert(RLD * NT == BN * KCH && TLD * NT == D * 4, "tile/threads mismatch");

  __shared__ u32x4 sK[2][BN * KCH];
  __shared__ u32x4 sV[2][BN * KCH];
  __shared__ u32x4 sKt[2][D * 4];

  const int32_t* it = a.items + (int64_t)blockIdx.x * kItemInts;
  const int q0 = it[0], q1 = it[1], k0 = it[2], k1 = it[3], delta = it[4], head = it[5],
            kvh = it[6];
  const int tid = threadIdx.x;
  const int w = tid >> 6, lane = tid & 63, hh = lane >> 5, l32 = lane & 31;
  const int row = q0 + w * 32 + l32;
  const bool row_ok = row < q1;
  const int lrow = row_ok ? row : q0;

  u32x4 qf[KS], df[KS];
  {
    const int64_t off = ((int64_t)lrow * a.H + head) * D + hh * 8;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      qf[s] = *(const u32x4*)(a.q + off + s * 16);
      df[s] = *(const u32x4*)(a.dout + off + s * 16);
    }
  }
  const float lse = a.lse[(int64_t)head * a.T_q + lrow];
  const float l2 = (lse == neg_inf()) ? __builtin_inff() : lse * kLog2e;
  const float drow = a.delta[(int64_t)head * a.T_q + lrow];
  const float c2 = a.scale_log2;

  f32x16 acc[DB];
#pragma unroll
  for (int d = 0; d < DB; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[d][r] = 0.f;

  const int kt_first = k0 & ~7;
  const int n_tiles = (k1 > k0) ? (k1 - kt_first + BN - 1) / BN : 0;

  u32x4 stK[RLD], stV[RLD], stT[TLD];
  auto load_tile = [&](int kt) {
#pragma unroll
    for (int i = 0; i < RLD; ++i) {
      int c = tid + i * NT;
      int r = c / KCH, cc = c % KCH;
      int key = kt + r;
      stK[i] = u32x4{0u, 0u, 0u, 0u};
      stV[i] = u32x4{0u, 0u, 0u, 0u};
      if (key < k1) {
        int64_t off = ((int64_t)key * a.Hkv + kvh) * D + cc * 8;
        stK[i] = *(const u32x4*)(a.k + off);
        stV[i] = *(const u32x4*)(a.v + off);
      }
    }
#pragma unroll
    for (int i = 0; i < TLD; ++i) {
      int c = tid + i * NT;
      int d = c / 4, cc = c % 4;
      stT[i] = *(const u32x4*)(a.kt + ((int64_t)kvh * D + d) * a.Tkp + kt + cc * 8);
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int i = 0; i < RLD; ++i) {
      int c = tid + i * NT;
      int idx = swz<KCH>(c / KCH, c % KCH);
      sK[buf][idx] = stK[i];
      sV[buf][idx] = stV[i];
    }
#pragma unroll
    for (int i = 0; i < TLD; ++i) {
      int c = tid + i * NT;
      sKt[buf][swz4(c / 4, c % 4)] = stT[i];
    }
  };

  if (n_tiles > 0) {
    load_tile(kt_first);
    store_tile(0);
  }
  __syncthreads();

  const int prow = perm32(l32);
  int buf = 0;
  for (int n = 0; n < n_tiles; ++n) {
    const int kt = kt_first + n * BN;
    if (n + 1 < n_tiles) load_tile(kt + BN);

    f32x16 s, dp;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      s[r] = 0.f;
      dp[r] = 0.f;
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      int idx = swz<KCH>(prow, ks * 2 + hh);
      s = mfma32(sK[buf][idx], qf[ks], s);
      dp = mfma32(sV[buf][idx], df[ks], dp);
    }
    const bool need_mask = (kt < k0) || (kt + BN > k1) || (a.causal && kt + BN - 1 > q0 + delta);
    float ds[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[r], c2, -l2));
      if (need_mask) {
        int key = kt + c_row_of(r, hh);
        bool ok = key >= k0 && key < k1 && (!a.causal || key <= row + delta);
        p = ok ? p : 0.f;
      }
      ds[r] = p * (dp[r] - drow);
    }
    u32x4 b0 = pack_bf16x8(ds[0], ds[1], ds[2], ds[3], ds[4], ds[5], ds[6], ds[7]);
    u32x4 b1 = pack_bf16x8(ds[8], ds[9], ds[10], ds[11], ds[12], ds[13], ds[14], ds[15]);
#pragma unroll
    for (int d = 0; d < DB; ++d) {
      acc[d] = mfma32(sKt[buf][swz4(d * 32 + l32, hh)], b0, acc[d]);
      acc[d] = mfma32(sKt[buf][swz4(d * 32 + l32, 2 + hh)], b1, acc[d]);
    }

    if (n + 1 < n_tiles) store_tile(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }

  if (!row_ok) return;
  const float sc = a.scale;
  const int64_t base = ((int64_t)row * a.H + head) * D + hh * 4;
#pragma unroll
  for (int d = 0; d < DB; ++d)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float x0 = acc[d][j * 4] * sc, x1 = acc[d][j * 4 + 1] * sc;
      float x2 = acc[d][j * 4 + 2] * sc, x3 = acc[d][j * 4 + 3] * sc;
      if (a.dq_acc) {
        float4* p = (float4*)(a.dq_acc + base + d * 32 + j * 8);
        float4 o = *p;
        *p = make_float4(o.x + x0, o.y + x1, o.z + x2, o.w + x3);
      } else {
        *(u32x2*)(a.dq + base + d * 32 + j * 8) = pack_bf16x4(x0, x1, x2, x3);
      }
    }
}

// ---------------------------------------------------------------- dK / dV
template <int D>
__global__ __launch_bounds__(NT, 1) void attn_dkdv_kernel(DkdvArgs a) {
  constexpr int BQ = kDkdvBQ;  // 32 query rows per chunk
  constexpr int KS = D / 16;
  constexpr int DB = D / 32;
  constexpr int KCH = D / 8;
  constexpr int RLD = BQ * KCH / NT;
  constexpr int TLD = D * 4 / NT;
  static_assert(RLD * NT == BQ * KCH && TLD * NT == D * 4, "tile/threads mismatch");

  __shared__ u32x4 sQ[2][BQ * KCH];
  __shared__ u32x4 sO[2][BQ * KCH];   // dO rows
  __shared__ u32x4 sQt[2][D * 4];
  __shared__ u32x4 sOt[2][D * 4];     // dO^T
  __shared__ float sL[2][BQ];         // LSE * log2(e) (+inf for rows without keys)
  __shared__ float sD[2][BQ];         // D_i

  const int32_t* it = a.items + (int64_t)blockIdx.x * kItemInts;
  const int k0 = it[0], k1 = it[1], qb = it[2], qe = it[3], delta = it[4], head = it[5],
            kvh = it[6];
  const int tid = threadIdx.x;
  const int w = tid >> 6, lane = tid & 63, hh = lane >> 5, l32 = lane & 31;
  const int key = k0 + w * 32 + l32;  // this lane's key (column of S)
  const bool key_ok = key < k1;

  // K, V rows as B operands (col = key, k = dims).
  u32x4 kf[KS], vf[KS];
  {
    const int64_t off = ((int64_t)(key_ok ? key : k0) * a.Hkv + kvh) * D + hh * 8;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      kf[s] = *(const u32x4*)(a.k + off + s * 16);
      vf[s] = *(const u32x4*)(a.v + off + s * 16);
      if (!key_ok) {
        kf[s] = u32x4{0u, 0u, 0u, 0u};
        vf[s] = u32x4{0u, 0u, 0u, 0u};
      }
    }
  }
  f32x16 dk[DB], dv[DB];
#pragma unroll
  for (int d = 0; d < DB; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      dk[d][r] = 0.f;
      dv[d][r] = 0.f;
    }
  const float c2 = a.scale_log2;

  const int qc_first = qb & ~7;
  const int n_chunks = (qe > qb) ? (qe - qc_first + BQ - 1) / BQ : 0;

  u32x4 stQ[RLD], stO[RLD], stQt[TLD], stOt[TLD];
  float stL = 0.f;
  auto load_chunk = [&](int qc) {
#pragma unroll
    for (int i = 0; i < RLD; ++i) {
      int c = tid + i * NT;
      int r = c / KCH, cc = c % KCH;
      int rr = qc + r;
      stQ[i] = u32x4{0u, 0u, 0u, 0u};
      stO[i] = u32x4{0u, 0u, 0u, 0u};
      if (rr < a.T_q) {
        int64_t off = ((int64_t)rr * a.H + head) * D + cc * 8;
        stQ[i] = *(const u32x4*)(a.q + off);
        stO[i] = *(const u32x4*)(a.dout + off);
      }
    }
#pragma unroll
    for (int i = 0; i < TLD; ++i) {
      int c = tid + i * NT;
      int d = c / 4, cc = c % 4;
      int64_t off = ((int64_t)head * D + d) * a.Tqp + qc + cc * 8;
      stQt[i] = *(const u32x4*)(a.qt + off);
      stOt[i] = *(const u32x4*)(a.dot + off);
    }
    if (tid < 2 * BQ) {
      int rr = qc + (tid & (BQ - 1));
      if (tid < BQ) {
        float l = rr < a.T_q ? a.lse[(int64_t)head * a.T_q + rr] : neg_inf();
        stL = (l == neg_inf()) ? __builtin_inff() : l * kLog2e;
      } else {
        stL = rr < a.T_q ? a.delta[(int64_t)head * a.T_q + rr] : 0.f;
      }
    }
  };
  auto store_chunk = [&](int buf) {
#pragma unroll
    for (int i = 0; i < RLD; ++i) {
      int c = tid + i * NT;
      int idx = swz<KCH>(c / KCH, c % KCH);
      sQ[buf][idx] = stQ[i];
      sO[buf][idx] = stO[i];
    }
#pragma unroll
    for (int i = 0; i < TLD; ++i) {
      int c = tid + i * NT;
      int idx = swz4(c / 4, c % 4);
      sQt[buf][idx] = stQt[i];
      sOt[buf][idx] = stOt[i];
    }
    if (tid < BQ) sL[buf][tid] = stL;
    else if (tid < 2 * BQ) sD[buf][tid - BQ] = stL;
  };

  if (n_chunks > 0) {
    load_chunk(qc_first);
    store_chunk(0);
  }
  __syncthreads();

  const int prow = perm32(l32);
  int buf = 0;
  for (int n = 0; n < n_chunks; ++n) {
    const int qc = qc_first + n * BQ;
    if (n + 1 < n_chunks) load_chunk(qc + BQ);

    f32x16 s, dp;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      s[r] = 0.f;
      dp[r] = 0.f;
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      int idx = swz<KCH>(prow, ks * 2 + hh);
      s = mfma32(sQ[buf][idx], kf[ks], s);
      dp = mfma32(sO[buf][idx], vf[ks], dp);
    }
    // chunk needs masking if it straddles the item's row range, the key
    // tile's end, or the causal diagonal of this wavefront's keys
    const int wk0 = k0 + w * 32;
    const bool need_mask = (qc < qb) || (qc + BQ > qe) || (wk0 + 32 > k1) ||
                           (a.causal && wk0 + 31 > qc + delta);
    float p[16], ds[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int lr = c_row_of(r, hh);
      float pv = __builtin_amdgcn_exp2f(__builtin_fmaf(s[r], c2, -sL[buf][lr]));
      if (need_mask) {
        int rr = qc + lr;
        bool ok = rr >= qb && rr < qe && key_ok && (!a.causal || key <= rr + delta);
        pv = ok ? pv : 0.f;
      }
      p[r] = pv;
      ds[r] = pv * (dp[r] - sD[buf][lr]);
    }
    u32x4 pb0 = pack_bf16x8(p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7]);
    u32x4 pb1 = pack_bf16x8(p[8], p[9], p[10], p[11], p[12], p[13], p[14], p[15]);
    u32x4 db0 = pack_bf16x8(ds[0], ds[1], ds[2], ds[3], ds[4], ds[5], ds[6], ds[7]);
    u32x4 db1 = pack_bf16x8(ds[8], ds[9], ds[10], ds[11], ds[12], ds[13], ds[14], ds[15]);
#pragma unroll
    for (int d = 0; d < DB; ++d) {
      const int r0 = swz4(d * 32 + l32, hh), r1 = swz4(d * 32 + l32, 2 + hh);
      dv[d] = mfma32(sOt[buf][r0], pb0, dv[d]);
      dv[d] = mfma32(sOt[buf][r1], pb1, dv[d]);
      dk[d] = mfma32(sQt[buf][r0], db0, dk[d]);
      dk[d] = mfma32(sQt[buf][r1], db1, dk[d]);
    }

    if (n + 1 < n_chunks) store_chunk(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }

  if (!key_ok) return;
  const float sc = a.scale;
#pragma unroll
  for (int d = 0; d < DB; ++d)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int dim = d * 32 + j * 8 + hh * 4;
      float k0v = dk[d][j * 4] * sc, k1v = dk[d][j * 4 + 1] * sc;
      float k2v = dk[d][j * 4 + 2] * sc, k3v = dk[d][j * 4 + 3] * sc;
      if (a.direct) {
        const int64_t off = ((int64_t)key * a.Hkv + kvh) * D + dim;
        *(u32x2*)(a.dk + off) = pack_bf16x4(k0v, k1v, k2v, k3v);
        *(u32x2*)(a.dv + off) = pack_bf16x4(dv[d][j * 4], dv[d][j * 4 + 1], dv[d][j * 4 + 2],
                                            dv[d][j * 4 + 3]);
      } else {
        const int64_t off = ((int64_t)head * a.T_k + key) * D + dim;
        *(float4*)(a.part_k + off) = make_float4(k0v, k1v, k2v, k3v);
        *(float4*)(a.part_v + off) =
            make_float4(dv[d][j * 4], dv[d][j * 4 + 1], dv[d][j * 4 + 2], dv[d][j * 4 + 3]);
      }
    }
}

}  // namespace

hipError_t launch_attn_dq(const DqArgs& a, int n_items, int D, hipStream_t st) {
  if (n_items <= 0) return hipSuccess;
  if (D == 128) return sp_launch(kKDq, attn_dq_kernel<128>, dim3(n_items), dim3(NT), st, a);
  return sp_launch(kKDq, attn_dq_kernel<64>, dim3(n_items), dim3(NT), st, a);
}

hipError_t launch_attn_dkdv(const DkdvArgs& a, int n_items, int D, hipStream_t st) {
  if (n_items <= 0) return hipSuccess;
  if (D == 128) return sp_launch(kKDkdv, attn_dkdv_kernel<128>, dim3(n_items), dim3(NT), st, a);
  return sp_launch(kKDkdv, attn_dkdv_kernel<64>, dim3(n_items), dim3(NT), st, a);
}

}  // namespace spk
