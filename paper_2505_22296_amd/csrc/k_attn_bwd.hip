// Attention backward for one SP rank's real heads on gfx950 (deterministic:
// no atomics).  P is recomputed from the forward's LSE; with
// D_i = dO_i . O_i (precomputed per row and stored negated):
//   dP = dO V^T,  dS = P (dP - D),  dQ = scale dS K,
//   dK = scale dS^T Q,  dV = P^T dO.
//
// dq kernel (query-stationary): workgroup = 256 query rows of one head,
//   wavefront w owns 32 rows; per 32-key tile (K, V staged in LDS):
//     S^T = K Q^T, dP^T = V dO^T     (Q, dO rows kept as B operands)
//     dS^T = P^T (dP^T - D)          (row statistics are per lane)
//     dQ^T += K^T dS^T               (K^T by transposing LDS reads; dS^T C
//                                     registers used directly as B)
// dk/dv kernel (key-stationary): workgroup = 128 keys of one KV head and one
//   query head, 4 wavefront pairs of 32 keys (K resp. V rows as B operands
//   in registers); per 32-row query chunk, visited last to first (Q, dO
//   staged in LDS), the pair's P-wavefront computes
//     S = Q K^T, P, dV^T += dO^T P    (dO^T by transposing LDS reads)
//   and hands P to the pair's dS-wavefront, which computes
//     dP = dO V^T, dS = P (dP - D), dK^T += Q^T dS
//   (Q, dO rows loaded in perm32 order, so P / dS C registers are used
//   directly as B operands).  With one query head per KV head the results
//   are written as bf16; under GQA each query head writes a float32 partial
//   that a reduction kernel sums over the group in ascending head order.
#include "dev_common.h"
#include "launch.h"

namespace spk {

namespace {

constexpr int NT = 256;

// ------------------------------------------------------------------- dQ
// Workgroup = NWQ wavefronts = 32*NWQ query rows of one head.  LDS stage:
// K and V tiles [32 keys][D] in the blocked layout of dev_common.h (K^T
// fragments are transposing reads of the K tile), filled by DMA in 1 KB
// blocks spread over the wavefronts; NSTQ tiles resident, barrier every
// TPBQ tiles.
constexpr int NWQ = kDqWaves, NTQ = 64 * NWQ, NSTQ = kDqStages, TPBQ = kDqTilesPerSync;
static_assert(kDqBM == 32 * NWQ && NSTQ % TPBQ == 0 && NSTQ >= 2 * TPBQ, "dq tiling");

template <int D>
struct DqStage {
  static constexpr int BN = kDqBN;
  static constexpr int SUB = BN * 4;             // chunks per sub-tile [BN][32]
  static constexpr int RB = BN * (D / 8) / 64;   // 1 KB blocks of a tile
  static constexpr int NB = 2 * RB;
  static constexpr int NBW = (NB + NWQ - 1) / NWQ;  // blocks per wavefront (tail ones junk)
  static constexpr int OFF_V = RB * 64, STAGE = NB * 64;
  static constexpr int JUNK = NSTQ * STAGE, SMEM = JUNK + 64;
  // 0 = K, 1 = V, 2 = unused slot (copied to the junk block)
  static SP_DEV int kind(int b) { return b < RB ? 0 : b < NB ? 1 : 2; }
};

template <int D>
__global__ __launch_bounds__(NTQ, 1) void attn_dq_kernel(DqArgs a) {
  using S = DqStage<D>;
  constexpr int BN = S::BN, KS = D / 16, DB = D / 32;
  constexpr int NBW = S::NBW, STAGE = S::STAGE, SUB = S::SUB;

  __shared__ u32x4 smem[S::SMEM];

  const int32_t* it = a.items + (int64_t)blockIdx.x * kItemInts;
  const int q0 = it[0], q1 = it[1], k0 = it[2], k1 = it[3], delta = it[4], head = it[5],
            kvh = it[6];
  const int tid = threadIdx.x;
  if (it[7] == kItemFillQ) {  // dummy slot of a bf16 dQ: +0
    fill_rows_bf16(a.dq, q0, q1, a.H, head, D, tid, NTQ);
    return;
  }
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63, hh = lane >> 5, l32 = lane & 31;
  const int row = q0 + w * 32 + l32;
  const bool row_ok = row < q1;
  const int lrow = row_ok ? row : q0;
  const int wave_rows = min(32, q1 - q0 - w * 32);
  const int wave_kmax = wave_rows <= 0 ? -1
                        : a.causal     ? min(k1, q0 + w * 32 + wave_rows + delta)
                                       : k1;

  u32x4 qf[KS], df[KS];
  {
    const int64_t qoff = ((int64_t)lrow * a.H + head) * D + hh * 8;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      qf[s] = *(const u32x4*)(a.q + qoff + s * 16);
      df[s] = *(const u32x4*)(a.dout + qoff + s * 16);
    }
  }
  const float lse = a.lse[(int64_t)head * a.T_q + lrow];
  const float l2 = (lse == neg_inf()) ? __builtin_inff() : lse * kLog2e;
  const float ndrow = a.neg_d[(int64_t)head * a.T_q + lrow];
  const float c2 = a.scale_log2;
  // -D of the lane's row in every C register (the lane's row is fixed for
  // the item): the accumulator input of each tile's first dP MFMA
  f32x16 ndv;
#pragma unroll
  for (int r = 0; r < 16; ++r) ndv[r] = ndrow;

  f32x16 acc[DB];
#pragma unroll
  for (int d = 0; d < DB; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[d][r] = 0.f;

  const int kt_first = k0 & ~7;
  const int n_tiles = (k1 > k0) ? (k1 - kt_first + BN - 1) / BN : 0;

  // Per-lane, tile-independent element offsets of this wavefront's DMA blocks
  // w + NWQ*j (the block kinds are wave-uniform; K and V share shape and
  // source row stride).
  const int kstride = a.Hkv * D;
  int off[NBW], key_of[NBW];
#pragma unroll
  for (int j = 0; j < NBW; ++j) {
    const int b = w + NWQ * j;
    const int k = S::kind(b);
    const int t = (k == 1 ? b - S::RB : k == 0 ? b : 0) * 64 + lane;
    const int ts = t % SUB, r = ts / 4;
    key_of[j] = r;
    off[j] = 2 * (r * kstride + (t / SUB) * 32 + blk_chunk(r, ts % 4) * 8);  // bytes
  }
  const uint16_t* kbase = a.k + (int64_t)kvh * D;
  const uint16_t* vbase = a.v + (int64_t)kvh * D;
  auto issue = [&](int n) {
    const int kt = kt_first + n * BN;
    u32x4* stg = smem + (n % NSTQ) * STAGE;
    const int64_t rowoff = (int64_t)kt * kstride;
    auto copy = [&](int j, int o) {
      const int b = w + NWQ * j;
      const int k = S::kind(b);
      dma16s((k == 1 ? vbase : kbase) + rowoff, o, k == 2 ? smem + S::JUNK : stg + b * 64);
    };
    if (kt + BN <= k1) {
#pragma unroll
      for (int j = 0; j < NBW; ++j) copy(j, off[j]);
    } else {  // keys past k1 (masked) are clamped to k1-1
#pragma unroll
      for (int j = 0; j < NBW; ++j)
        copy(j, off[j] + 2 * (min(kt + key_of[j], k1 - 1) - kt - key_of[j]) * kstride);
    }
  };
  // lane-constant LDS offsets of the fragments (see the forward kernel)
  const int kr = perm32(l32);
  const int kf0 = kr * 4 + blk_chunk(kr, hh), kf1 = kr * 4 + blk_chunk(kr, 2 + hh);
  const int kt0 = blk_tr_off(lane), kt1 = blk_tr_off2(lane);

  for (int n = 0; n < NSTQ - TPBQ && n < n_tiles; ++n) issue(n);

  for (int n0 = 0; n0 < n_tiles; n0 += NSTQ) {
#pragma unroll
    for (int u = 0; u < NSTQ; ++u) {
      const int n = n0 + u;
      if (n >= n_tiles) break;
      if (u % TPBQ == 0) {
        // tiles n .. n+TPBQ-1 landed; the stages of tiles n-TPBQ .. n-1 are
        // free and receive tiles n+NSTQ-TPBQ ..
        const int issued = min(n_tiles, n + NSTQ - TPBQ);
        wait_batches<NBW, NSTQ - 2 * TPBQ>(issued - min(n_tiles, n + TPBQ));
        __syncthreads();
#pragma unroll
        for (int t = 0; t < TPBQ; ++t)
          if (n + NSTQ - TPBQ + t < n_tiles) issue(n + NSTQ - TPBQ + t);
      }
      const int kt = kt_first + n * BN;
      if (kt >= wave_kmax) continue;  // wholly past this wavefront's rows
      const u32x4* stg = smem + u * STAGE;

      // K and V fragments of the tile, all read before the first MFMA
      u32x4 kfr[KS], vfr[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int fo = (ks >> 1) * SUB + ((ks & 1) ? kf1 : kf0);
        kfr[ks] = stg[fo];
        vfr[ks] = stg[S::OFF_V + fo];
      }
      __builtin_amdgcn_sched_barrier(0);
      f32x16 s, dp = ndv;  // dP starts from -D, so the MFMAs leave dP - D
#pragma unroll
      for (int r = 0; r < 16; ++r) s[r] = 0.f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        s = mfma32(kfr[ks], qf[ks], s);
        dp = mfma32(vfr[ks], df[ks], dp);
      }
      // K^T fragments of the dQ product, read while dS is formed
      const uint16_t* stg16 = (const uint16_t*)stg;
      u32x4 ktr[DB * 2];
#pragma unroll
      for (int d = 0; d < DB; ++d)
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const int o = d * SUB * 8 + ks * 16 * 32;
          const u32x2 lo = lds_tr16(stg16 + kt0 + o), hi = lds_tr16(stg16 + kt1 + o);
          ktr[d * 2 + ks] = u32x4{lo[0], lo[1], hi[0], hi[1]};
        }
      __builtin_amdgcn_sched_barrier(0);
      const bool need_mask = (kt < k0) | (kt + BN > k1) | (a.causal & (kt + BN - 1 > q0 + w * 32 + delta));
      if (need_mask) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          int key = kt + c_row_of(r, hh);
          bool ok = key >= k0 && key < k1 && (!a.causal || key <= row + delta);
          s[r] = ok ? s[r] : neg_inf();
        }
      }
      float ds[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[r], c2, -l2));
        ds[r] = p * dp[r];
      }
      u32x4 b0 = pack_bf16x8(ds[0], ds[1], ds[2], ds[3], ds[4], ds[5], ds[6], ds[7]);
      u32x4 b1 = pack_bf16x8(ds[8], ds[9], ds[10], ds[11], ds[12], ds[13], ds[14], ds[15]);
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int d = 0; d < DB; ++d) acc[d] = mfma32(ktr[d * 2 + ks], ks ? b1 : b0, acc[d]);
      __builtin_amdgcn_s_setprio(0);
    }
  }

  if (!row_ok) return;
  const float sc = a.scale;
  const int64_t base = ((int64_t)row * a.H + head) * D + hh * 4;
  if (a.dq_acc) {  // ring: accumulate; the last chunk emits bf16 instead
    // every accumulator value is loaded before the first store: the stores
    // (through dq or dq_acc) could alias later loads for all the compiler
    // knows, which would serialize one memory round trip per 16 bytes
    float4 old[DB * 4];
#pragma unroll
    for (int i = 0; i < DB * 4; ++i)
      old[i] = a.dq_init ? make_float4(0.f, 0.f, 0.f, 0.f)
                         : *(const float4*)(a.dq_acc + base + (i >> 2) * 32 + (i & 3) * 8);
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float4 o = old[d * 4 + j];
        const float4 t = make_float4(o.x + acc[d][j * 4] * sc, o.y + acc[d][j * 4 + 1] * sc,
                                     o.z + acc[d][j * 4 + 2] * sc, o.w + acc[d][j * 4 + 3] * sc);
        if (a.dq)
          *(u32x2*)(a.dq + base + d * 32 + j * 8) = pack_bf16x4(t.x, t.y, t.z, t.w);
        else
          *(float4*)(a.dq_acc + base + d * 32 + j * 8) = t;
      }
  } else {
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        *(u32x2*)(a.dq + base + d * 32 + j * 8) =
            pack_bf16x4(acc[d][j * 4] * sc, acc[d][j * 4 + 1] * sc, acc[d][j * 4 + 2] * sc,
                        acc[d][j * 4 + 3] * sc);
  }
}

// ---------------------------------------------------------------- dK / dV
// Workgroup = 8 wavefronts = 4 pairs; pair p owns keys k0 + 32p .. +32.
// Per 32-row query chunk the pair splits the work: its P-wavefront (w < 4)
// computes S = Q K^T, P and dV^T += dO^T P and hands P to its partner through
// LDS (fp16: P lies in [0, 1]); the dS-wavefront (w >= 4) computes
// dP = dO V^T, dS = P (dP - D) and dK^T += Q^T dS.  S is evaluated once per
// pair (8*D MFMA work per pair instead of 10*D for separate dK and dV
// kernels, which would each recompute S) and the Q / dO chunk tiles are
// staged once for both gradients.
// Chunks go in groups of TPBF between barriers: in group g the
// P-wavefronts work on group g, the dS-wavefronts on group g-1 (whose P is
// complete), while group g+1 is copied in; stages hold three groups and the
// P exchange has one slot per stage, so the loop unrolled over three groups
// addresses both with immediate offsets.
constexpr int NPF = kDkdvWaves / 2;  // wavefront pairs per workgroup
constexpr int TPBF = 2;              // chunks per group (barrier interval)
constexpr int NSTF = 3 * TPBF;       // resident chunks
constexpr int NXF = NSTF;            // P exchange slots (one per stage)
static_assert(kDkdvBN == 32 * NPF, "dkdv tiling");

template <int D>
struct DkdvStage {
  static constexpr int BQ = kDkdvBQ;
  static constexpr int SUB = BQ * 4;            // chunks per sub-tile [BQ][32]
  static constexpr int RB = BQ * (D / 8) / 64;  // 1 KB blocks of a tile
  static constexpr int NB = 2 * RB;             // Q, dO
  static constexpr int NBW = (NB + 2 * NPF - 1) / (2 * NPF);
  static constexpr int OFF_O = RB * 64, OFF_LD = NB * 64, STAGE = OFF_LD + 16;
  static constexpr int XSLOT = NPF * 128;       // per pair: 2 x 16 bytes x 64 lanes
  static constexpr int OFF_X = NSTF * STAGE, JUNK = OFF_X + NXF * XSLOT, SMEM = JUNK + 64;
  static SP_DEV int kind(int b) { return b < RB ? 0 : b < NB ? 1 : 2; }
};

template <int D, bool PWAVE>
SP_DEV void dkdv_body(const DkdvArgs& a, const int32_t (&it)[kItemInts], u32x4* smem, int w,
                      int lane) {
  using S = DkdvStage<D>;
  constexpr int BQ = S::BQ, KS = D / 16, DB = D / 32, SUB = S::SUB, NBW = S::NBW;
  constexpr int STAGE = S::STAGE;
  const int k0 = it[0], k1 = it[1], qb = it[2], qe = it[3], delta = it[4], head = it[5],
            kvh = it[6];
  const int hh = lane >> 5, l32 = lane & 31;
  const int pr = PWAVE ? w : w - NPF;  // pair index
  const int wk0 = k0 + pr * 32;
  const int key = wk0 + l32;
  const bool key_ok = key < k1;
  const int qc_first = qb & ~7;
  const int n_chunks = (qe > qb) ? (qe - qc_first + BQ - 1) / BQ : 0;
  const int n_groups = (n_chunks + TPBF - 1) / TPBF;
  const int qc_last = qc_first + (n_chunks - 1) * BQ;
  const int Tq1 = a.T_q - 1;
  const int hstride = a.H * D;
  const uint16_t* qh = a.q + (int64_t)head * D;
  const uint16_t* oh = a.dout + (int64_t)head * D;
  const float* lh = a.lse2 + (int64_t)head * a.T_q;
  const float* dh = a.neg_d + (int64_t)head * a.T_q;
  const int wave_qmin = wk0 >= k1 ? 0x7fffffff : a.causal ? wk0 - delta - BQ + 1 : -0x7fffffff;

  // DMA: blocks w + 8j of each chunk's Q / dO tiles (kinds wave-uniform)
  int off[NBW], row_of[NBW];
#pragma unroll
  for (int j = 0; j < NBW; ++j) {
    const int b = w + 2 * NPF * j;
    const int k = S::kind(b);
    const int t = (k == 1 ? b - S::RB : k == 0 ? b : 0) * 64 + lane;
    const int ts = t % SUB, r = ts / 4;
    row_of[j] = r;
    off[j] = 2 * (r * hstride + (t / SUB) * 32 + blk_chunk(r, ts % 4) * 8);  // bytes
  }
  auto issue = [&](int c) {
    const int qc = qc_last - c * BQ;
    u32x4* stg = smem + (c % NSTF) * STAGE;
    const bool tail = qc + BQ > a.T_q;
    auto copy = [&](int j, int o) {
      const int b = w + 2 * NPF * j;
      const int k = S::kind(b);
      dma16s((k == 1 ? oh : qh) + (int64_t)qc * hstride, o, k == 2 ? smem + S::JUNK : stg + b * 64);
    };
    if (!tail) {
#pragma unroll
      for (int j = 0; j < NBW; ++j) copy(j, off[j]);
    } else {  // rows past T_q are clamped to the last row
#pragma unroll
      for (int j = 0; j < NBW; ++j)
        copy(j, off[j] + 2 * (min(qc + row_of[j], Tq1) - qc - row_of[j]) * hstride);
    }
    if (w == 0) {  // the chunk's L and -D rows: one copy is enough
      const int rr = min(qc + (lane & (BQ - 1)), Tq1);
      dma4((lane < BQ ? lh : dh) + rr, stg + S::OFF_LD);
    }
  };

  // B operands: K rows (P-wavefront) or V rows (dS-wavefront) of this pair's keys
  u32x4 bf[KS];
  {
    const int64_t koff = ((int64_t)(key_ok ? key : k0) * a.Hkv + kvh) * D + hh * 8;
    const uint16_t* src = PWAVE ? a.k : a.v;
#pragma unroll
    for (int s = 0; s < KS; ++s) bf[s] = *(const u32x4*)(src + koff + s * 16);
  }
  f32x16 acc[DB];
#pragma unroll
  for (int d = 0; d < DB; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[d][r] = 0.f;
  const float c2 = a.scale_log2;
  const int qr = perm32(l32);
  // plain A fragments: Q (S) or dO (dP); transposed ones: dO (dV) or Q (dK)
  const int af0 = (PWAVE ? 0 : S::OFF_O) + qr * 4 + blk_chunk(qr, hh);
  const int af1 = (PWAVE ? 0 : S::OFF_O) + qr * 4 + blk_chunk(qr, 2 + hh);
  const int tr0 = (PWAVE ? S::OFF_O * 8 : 0) + blk_tr_off(lane);
  const int tr1 = (PWAVE ? S::OFF_O * 8 : 0) + blk_tr_off2(lane);
  const int xo = S::OFF_X + pr * 128 + lane;  // this lane's P exchange chunk (+64 second half)

  // chunk c sits in stage (and exchange slot) `st` == c % NSTF
  auto chunk = [&](int c, int st) {
    const int qc = qc_last - c * BQ;
    if (qc < wave_qmin) return;  // no row of the chunk sees this pair's keys
    const u32x4* stg = smem + st * STAGE;
    const uint16_t* stg16 = (const uint16_t*)stg;
    u32x4* xs = smem + st * S::XSLOT + xo;
    // A fragments of S = Q K^T (resp. dP = dO V^T), issued ahead of the
    // MFMAs, which the compiler places among them
    u32x4 afr[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) afr[ks] = stg[(ks >> 1) * SUB + ((ks & 1) ? af1 : af0)];
    // per-row statistic of the lane's 16 C rows: L (P-wavefront) or -D
    const f32x4* vLD = (const f32x4*)(stg + S::OFF_LD) + (PWAVE ? 0 : BQ / 4);
    f32x16 s;
    if constexpr (PWAVE) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[r] = 0.f;
    } else {
      // dP starts from -D of its row, so the MFMAs leave dP - D
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const f32x4 x = vLD[half * 4 + hh * 2], y = vLD[half * 4 + hh * 2 + 1];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          s[half * 8 + i] = x[i];
          s[half * 8 + 4 + i] = y[i];
        }
      }
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) s = mfma32(afr[ks], bf[ks], s);
    // transposed fragments of the dV (resp. dK) product, read while P / dS
    // are formed
    u32x4 tfr[DB * 2];
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const int o = d * SUB * 8 + ks * 16 * 32;
        const u32x2 lo = lds_tr16(stg16 + tr0 + o), hi = lds_tr16(stg16 + tr1 + o);
        tfr[d * 2 + ks] = u32x4{lo[0], lo[1], hi[0], hi[1]};
      }
    u32x4 pb[2];
    if constexpr (PWAVE) {
      // S -> masked -> P; P to the partner (fp16) and into dV (bf16)
      const bool need_mask = (qc < qb) | (qc + BQ > qe) | (wk0 + 32 > k1) |
                             (a.causal & (wk0 + 31 > qc + delta));
      if (need_mask) {
        int lo = qb - qc, hi = qe - qc;
        if (a.causal) lo = max(lo, key - delta - qc);
        if (!key_ok) hi = lo;
        lo -= hh * 8;
        hi -= hh * 8;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int br = (r >> 3) * 16 + (r & 7);
          s[r] = (br >= lo && br < hi) ? s[r] : neg_inf();
        }
      }
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const f32x4 La = vLD[half * 4 + hh * 2], Lb = vLD[half * 4 + hh * 2 + 1];
        const float Lr[8] = {La[0], La[1], La[2], La[3], Lb[0], Lb[1], Lb[2], Lb[3]};
        f32x8 p;
#pragma unroll
        for (int i = 0; i < 8; ++i) p[i] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[half * 8 + i], c2, -Lr[i]));
        pb[half] = __builtin_bit_cast(u32x4, __builtin_convertvector(p, bf16x8));
        xs[half * 64] = __builtin_bit_cast(u32x4, __builtin_convertvector(p, f16x8));
      }
    } else {
      // dP - D (in s) and the partner's P -> dS
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        // P (fp16) times dP - D as one mixed-precision FMA with a zero addend
        // (v_fma_mix_f32 reads the fp16 half directly: no conversion)
        const f16x8 p = __builtin_bit_cast(f16x8, xs[half * 64]);
        f32x8 ds;
#pragma unroll
        for (int i = 0; i < 8; ++i) ds[i] = __builtin_fmaf((float)p[i], s[half * 8 + i], 0.f);
        pb[half] = __builtin_bit_cast(u32x4, __builtin_convertvector(ds, bf16x8));
      }
    }
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int d = 0; d < DB; ++d) acc[d] = mfma32(tfr[d * 2 + ks], pb[ks], acc[d]);
  };

  constexpr int NGS = NSTF / TPBF;  // groups per stage cycle
  for (int t = 0; t < TPBF && t < n_chunks; ++t) issue(t);
  for (int g0 = 0; g0 <= n_groups; g0 += NGS) {
#pragma unroll
    for (int u = 0; u < NGS; ++u) {
      const int g = g0 + u;
      if (g > n_groups) break;
      // group g has landed; every wavefront is done with group g-2 (its
      // stages and exchange slots receive group g+1)
      wait_vmcnt<0>();
      __syncthreads();
#pragma unroll
      for (int t = 0; t < TPBF; ++t)
        if ((g + 1) * TPBF + t < n_chunks) issue((g + 1) * TPBF + t);
      const int gw = PWAVE ? g : g - 1;
      if (gw >= 0 && gw < n_groups) {
#pragma unroll
        for (int t = 0; t < TPBF; ++t)
          if (gw * TPBF + t < n_chunks)
            chunk(gw * TPBF + t, (TPBF * (PWAVE ? u : u + NGS - 1) + t) % NSTF);
      }
    }
  }

  if (!key_ok) return;
  const float sc = PWAVE ? 1.f : a.scale;
#pragma unroll
  for (int d = 0; d < DB; ++d)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int dim = d * 32 + j * 8 + hh * 4;
      const float x0 = acc[d][j * 4] * sc, x1 = acc[d][j * 4 + 1] * sc;
      const float x2 = acc[d][j * 4 + 2] * sc, x3 = acc[d][j * 4 + 3] * sc;
      if (a.direct) {
        const int64_t o = ((int64_t)key * a.Hkv + kvh) * D + dim;
        *(u32x2*)((PWAVE ? a.dv : a.dk) + o) = pack_bf16x4(x0, x1, x2, x3);
      } else {
        const int64_t o = ((int64_t)head * a.T_k + key) * D + dim;
        *(float4*)((PWAVE ? a.part_v : a.part_k) + o) = make_float4(x0, x1, x2, x3);
      }
    }
}

template <int D>
__global__ __launch_bounds__(64 * 2 * NPF, 1) void attn_dkdv_kernel(DkdvArgs a) {
  __shared__ u32x4 smem[DkdvStage<D>::SMEM];
  int32_t it[kItemInts];
  load_item(a.items, blockIdx.x, it);
  if (it[7] == kItemFillKV) {  // KV head no real query head reads: dK = dV = +0
    fill_rows_bf16(a.dk, it[0], it[1], a.Hkv, it[6], D, threadIdx.x, 64 * 2 * NPF);
    fill_rows_bf16(a.dv, it[0], it[1], a.Hkv, it[6], D, threadIdx.x, 64 * 2 * NPF);
    return;
  }
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (w < NPF)
    dkdv_body<D, true>(a, it, smem, w, lane);
  else
    dkdv_body<D, false>(a, it, smem, w, lane);
}

}  // namespace

hipError_t launch_attn_dq(const DqArgs& a, int n_items, int D, hipStream_t st) {
  if (n_items <= 0) return hipSuccess;
  if (D == 128) return sp_launch(kKDq, attn_dq_kernel<128>, dim3(n_items), dim3(NTQ), st, a);
  return sp_launch(kKDq, attn_dq_kernel<64>, dim3(n_items), dim3(NTQ), st, a);
}

hipError_t launch_attn_dkdv(const DkdvArgs& a, int n_items, int D, hipStream_t st) {
  if (n_items <= 0) return hipSuccess;
  const dim3 g(n_items), b(64 * 2 * NPF);
  if (D == 128) return sp_launch(kKDkdv, attn_dkdv_kernel<128>, g, b, st, a);
  return sp_launch(kKDkdv, attn_dkdv_kernel<64>, g, b, st, a);
}

}  // namespace spk
