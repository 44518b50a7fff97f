// Attention forward for one SP rank's real heads on gfx950.
//
// One workgroup = 8 wavefronts = 256 query rows of one head (a work item from
// the host block-skip scheduler); wavefront w owns rows q_begin + 32w ..
// +32.  The key loop walks 64-key tiles of the segment.  K and V tiles are
// copied global -> LDS by DMA into the blocked layout of dev_common.h (no
// padding, no transposed copy: V^T fragments come from transposing LDS
// reads), four tiles resident: while a pair of tiles is consumed the next
// pair lands, and the eight wavefronts meet at a barrier once per pair.  Each
// tile is shared by all eight wavefronts.
//
// Per 64-key tile and wavefront:
//   S^T = K Q^T      (32x32x16 bf16 MFMA; Q^T kept in registers as B operand)
//   online softmax   (fp32; the 32x32 C layout gives each lane one query row,
//                     16 keys per tile half; the row max needs one exchange
//                     with lane l^32)
//   O^T += V^T P^T   (V^T by ds_read_b64_tr_b16 from the V tile; P^T from the
//                     C registers directly: K rows are loaded in perm32 order
//                     so each lane half's C registers are 8 consecutive keys,
//                     i.e. a B operand k-slice)
// The running max is only raised when it grows by more than 2^8 (exact:
// the final normalisation uses the same max).  Masking is evaluated only on
// tiles that straddle a segment edge or the causal diagonal; a wavefront
// skips the arithmetic of tiles that lie wholly past its causal diagonal.
//
// The ring variant (MERGE) folds the chunk's normalised (O_c, LSE_c) into
// float32 accumulators with the log-sum-exp rule in the epilogue.
#include "dev_common.h"
#include "launch.h"

namespace spk {

namespace {

constexpr int NW = kFwdWaves;         // wavefronts per workgroup
constexpr int BM = kFwdBM;            // query rows per workgroup
constexpr int BN = kFwdBN;            // keys per tile
constexpr int NT = 64 * NW;
constexpr int NST = kFwdStages;       // resident tiles
constexpr int TPB = kFwdTilesPerSync; // tiles per barrier
static_assert(BM == 32 * NW && NST % TPB == 0 && NST >= 2 * TPB, "fwd tiling");

// LDS stage of the forward: K and V tiles [BN][D] in the blocked layout
// (D/32 sub-tiles [BN][32]), filled by DMA in 1 KB blocks.
template <int D>
struct FwdStage {
  static constexpr int SUB = BN * 4;           // chunks per sub-tile
  static constexpr int KB = BN * (D / 8) / 64; // 1 KB blocks per tile
  static constexpr int NB = 2 * KB;
  static constexpr int NBW = NB / NW;          // blocks per wavefront
  static_assert(KB % NW == 0, "DMA blocks per wavefront");
  static constexpr int OFF_V = KB * 64, STAGE = NB * 64;  // 16-byte chunks
  static constexpr int SMEM = NST * STAGE;
};

template <int D, bool MERGE>
__global__ __launch_bounds__(NT, 1) void attn_fwd_kernel(FwdArgs a) {
  using S = FwdStage<D>;
  constexpr int KS = D / 16;   // MFMA k-steps over D
  constexpr int DB = D / 32;   // 32-dim blocks of O^T
  constexpr int NBW = S::NBW, NBK = NBW / 2, STAGE = S::STAGE, SUB = S::SUB;

  __shared__ u32x4 smem[S::SMEM];

  const int32_t* it = a.items + (int64_t)blockIdx.x * kItemInts;
  const int q0 = it[0], q1 = it[1], k0 = it[2], k1 = it[3], delta = it[4], head = it[5],
            kvh = it[6];
  const int tid = threadIdx.x;
  if (it[7] == kItemFillQ) {
    // dummy slot: O = +0, LSE = -inf (ring: the accumulators' identity on the
    // first chunk, and +0 in the bf16 copy)
    if constexpr (!MERGE) {
      fill_rows_bf16(a.o, q0, q1, a.H, head, D, tid, NT);
      fill_span_f32(a.lse + (int64_t)head * a.T_q + q0, q1 - q0, neg_inf(), tid, NT);
    } else {
      if (a.init) {
        fill_rows_f32(a.o_acc, q0, q1, a.H, head, D, tid, NT);
        fill_span_f32(a.lse_acc + (int64_t)head * a.T_q + q0, q1 - q0, neg_inf(), tid, NT);
      }
      if (a.o_out) fill_rows_bf16(a.o_out, q0, q1, a.H, head, D, tid, NT);
    }
    return;
  }
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63, hh = lane >> 5, l32 = lane & 31;
  const int row = q0 + w * 32 + l32;
  const bool row_ok = row < q1;
  // last key any row of this wavefront may see (tiles past it are skipped)
  const int wave_rows = min(32, q1 - q0 - w * 32);
  const int wave_kmax = wave_rows <= 0 ? -1
                        : a.causal     ? min(k1, q0 + w * 32 + wave_rows + delta)
                                       : k1;

  // Q^T as B operand: lane holds query row `row`, dims ks*16 + hh*8 + [0..7].
  u32x4 qf[KS];
  {
    const uint16_t* qp = a.q + ((int64_t)(row_ok ? row : q0) * a.H + head) * D + hh * 8;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      qf[s] = *(const u32x4*)(qp + s * 16);
      if (!row_ok) qf[s] = u32x4{0u, 0u, 0u, 0u};
    }
  }

  f32x16 oacc[DB];
#pragma unroll
  for (int d = 0; d < DB; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[d][r] = 0.f;
  float m_run = neg_inf(), l_part = 0.f;
  const float c2 = a.scale_log2;
  // Carried with the running max (they change only when it is raised):
  // msc = m_run * c2 (0 while m_run is -inf), and the score above which the
  // max is raised, m_run + 8 / c2 (-inf while m_run is -inf)
  const float raise_by = 8.f / c2;
  float msc = 0.f, m_thr = neg_inf();

  const int kt_first = k0 & ~7;
  const int n_tiles = (k1 > k0) ? (k1 - kt_first + BN - 1) / BN : 0;

  // Per-lane, tile-independent element offsets of this wavefront's DMA
  // blocks w + NW*j: the first NBK of them in the K tile, the rest in V;
  // both tiles have the same shape and source row stride.
  const int kstride = a.Hkv * D;
  int off[NBK], key_of[NBK];
#pragma unroll
  for (int j = 0; j < NBK; ++j) {
    const int t = (w + NW * j) * 64 + lane;   // chunk slot within the tile
    const int ts = t % S::SUB, r = ts / 4;
    key_of[j] = r;
    off[j] = 2 * (r * kstride + (t / S::SUB) * 32 + blk_chunk(r, ts % 4) * 8);  // bytes
  }
  const uint16_t* kbase = a.k + (int64_t)kvh * D;
  const uint16_t* vbase = a.v + (int64_t)kvh * D;
  auto issue = [&](int n) {
    const int kt = kt_first + n * BN;
    u32x4* stg = smem + (n % NST) * STAGE + w * 64;
    const int64_t rowoff = (int64_t)kt * kstride;
    if (kt + BN <= k1) {
#pragma unroll
      for (int j = 0; j < NBK; ++j) {
        dma16s(kbase + rowoff, off[j], stg + NW * j * 64);
        dma16s(vbase + rowoff, off[j], stg + S::OFF_V + NW * j * 64);
      }
    } else {  // keys past k1 (masked) are clamped to k1-1
#pragma unroll
      for (int j = 0; j < NBK; ++j) {
        const int o = off[j] + 2 * (min(kt + key_of[j], k1 - 1) - kt - key_of[j]) * kstride;
        dma16s(kbase + rowoff, o, stg + NW * j * 64);
        dma16s(vbase + rowoff, o, stg + S::OFF_V + NW * j * 64);
      }
    }
  };
  // Lane-constant LDS offsets of the fragments.  K fragment (g, ks): tile row
  // g*32 + perm32(l32), logical chunk 2ks + hh -> sub-tile ks/2 (immediate)
  // and one of two lane bases (ks even / odd).  V^T fragments: transposing
  // reads at two lane offsets; dim block, k-step and stage are immediates.
  const int kr = perm32(l32);
  const int kf0 = kr * 4 + blk_chunk(kr, hh), kf1 = kr * 4 + blk_chunk(kr, 2 + hh);
  const int vt0 = S::OFF_V * 8 + blk_tr_off(lane), vt1 = S::OFF_V * 8 + blk_tr_off2(lane);

  for (int n = 0; n < NST - TPB && n < n_tiles; ++n) issue(n);

  for (int n0 = 0; n0 < n_tiles; n0 += NST) {
#pragma unroll
    for (int u = 0; u < NST; ++u) {
      const int n = n0 + u;
      if (n >= n_tiles) break;
      if (u % TPB == 0) {
        // tiles n .. n+TPB-1 landed; every wavefront is done with the stages
        // of tiles n-TPB .. n-1, which receive tiles n+NST-TPB ..
        const int issued = min(n_tiles, n + NST - TPB);
        wait_batches<NBW, NST - 2 * TPB>(issued - min(n_tiles, n + TPB));
        __syncthreads();
      }
      // tile n + NST - TPB goes to a stage freed at the last barrier; its
      // copy is issued after this tile's first MFMAs (spreads the DMA burst)
      const bool pf = n + NST - TPB < n_tiles;
      const int kt = kt_first + n * BN;
      if (kt >= wave_kmax) {  // wholly past this wavefront's rows
        if (pf) issue(n + NST - TPB);
        continue;
      }
      const u32x4* stg = smem + u * STAGE;

      // ---- S^T = K Q^T for the two 32-key halves of the tile.  The K
      // fragment reads are issued together ahead of the MFMAs; the compiler
      // places the MFMAs among them (measured faster than holding every
      // MFMA behind the last read).
      u32x4 kfr[2 * KS];
#pragma unroll
      for (int g = 0; g < 2; ++g)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          kfr[g * KS + ks] = stg[(ks >> 1) * SUB + g * 128 + ((ks & 1) ? kf1 : kf0)];
      f32x16 s[2];
#pragma unroll
      for (int g = 0; g < 2; ++g)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[g][r] = 0.f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int g = 0; g < 2; ++g) s[g] = mfma32(kfr[g * KS + ks], qf[ks], s[g]);
      // V^T fragments of this tile, read while the softmax runs
      const uint16_t* stg16 = (const uint16_t*)stg;
      u32x4 vfr[DB * 4];
#pragma unroll
      for (int d = 0; d < DB; ++d)
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          const int o = d * SUB * 8 + ks * 16 * 32;
          const u32x2 lo = lds_tr16(stg16 + vt0 + o), hi = lds_tr16(stg16 + vt1 + o);
          vfr[d * 4 + ks] = u32x4{lo[0], lo[1], hi[0], hi[1]};
        }
      __builtin_amdgcn_sched_barrier(0);
      if (pf) issue(n + NST - TPB);

      // ---- mask (only on edge / diagonal tiles)
      const bool need_mask = (kt < k0) | (kt + BN > k1) | (a.causal & (kt + BN - 1 > q0 + w * 32 + delta));
      if (need_mask) {
#pragma unroll
        for (int g = 0; g < 2; ++g)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            int key = kt + g * 32 + c_row_of(r, hh);
            bool ok = key >= k0 && key < k1 && (!a.causal || key <= row + delta);
            if (!ok) s[g][r] = neg_inf();
          }
      }

      // ---- online softmax (lazy rescale).  Row max of the lane's 32
      // scores (finite or -inf): four chains of three-input maxima, 18 VALU
      // operations (a wavefront's dependent VALU operations issue back to
      // back, so short chains buy nothing)
      float mx4[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        mx4[i] = max3_nonan(s[0][i], s[0][i + 4], s[0][i + 8]);
        mx4[i] = max3_nonan(mx4[i], s[0][i + 12], s[1][i]);
        mx4[i] = max3_nonan(mx4[i], s[1][i + 4], s[1][i + 8]);
        mx4[i] = max3_nonan(mx4[i], s[1][i + 12], s[1][i + 12]);
      }
      const float mx = wave_max_xor32(max3_nonan(max3_nonan(mx4[0], mx4[1], mx4[2]), mx4[3], mx4[3]));
      const bool need = mx > m_thr;  // false while every score is -inf
      if (__ballot(need)) {
        float alpha = need ? exp2f((m_run - mx) * c2) : 1.f;
        if (need) {
          m_run = mx;
          msc = mx * c2;
          m_thr = mx + raise_by;
        }
        l_part *= alpha;
#pragma unroll
        for (int d = 0; d < DB; ++d)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[d][r] *= alpha;
      }
      u32x4 pb[4];
      float ps[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        float p[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          p[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[g][r], c2, -msc));
          ps[r & 3] += p[r];
        }
        pb[2 * g] = pack_bf16x8(p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7]);
        pb[2 * g + 1] = pack_bf16x8(p[8], p[9], p[10], p[11], p[12], p[13], p[14], p[15]);
      }
      l_part += (ps[0] + ps[1]) + (ps[2] + ps[3]);

      // ---- O^T += V^T P^T
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
#pragma unroll
        for (int d = 0; d < DB; ++d) oacc[d] = mfma32(vfr[d * 4 + ks], pb[ks], oacc[d]);
    }
  }

  // ---- epilogue
  const float l_tot = wave_sum_xor32(l_part);
  const bool has = l_tot > 0.f;
  const float inv = has ? 1.f / l_tot : 0.f;
  const float lse_v = has ? (m_run * c2 + __log2f(l_tot)) * kLn2 : neg_inf();
  if (!row_ok) return;
  const int64_t obase = ((int64_t)row * a.H + head) * D + hh * 4;
  if constexpr (!MERGE) {
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        u32x2 v = pack_bf16x4(oacc[d][j * 4] * inv, oacc[d][j * 4 + 1] * inv,
                              oacc[d][j * 4 + 2] * inv, oacc[d][j * 4 + 3] * inv);
        *(u32x2*)(a.o + obase + d * 32 + j * 8) = v;
      }
    if (hh == 0) a.lse[(int64_t)head * a.T_q + row] = lse_v;
  } else {
    // every accumulator value is loaded before the first store (the stores
    // could alias later loads for all the compiler knows, which would
    // serialize one memory round trip per 16 bytes), together with the
    // accumulated LSE
    float4 old[DB * 4];
#pragma unroll
    for (int i = 0; i < DB * 4; ++i)
      old[i] = a.init ? make_float4(0.f, 0.f, 0.f, 0.f)
                      : *(const float4*)(a.o_acc + obase + (i >> 2) * 32 + (i & 3) * 8);
    const int64_t li = (int64_t)head * a.T_q + row;
    const float la = a.init ? neg_inf() : a.lse_acc[li];
    float wa = 0.f, wb = 0.f, L = neg_inf();
    const float m = fmaxf(la, lse_v);
    if (m != neg_inf()) {
      float ea = __expf(la - m), eb = __expf(lse_v - m);
      float ssum = ea + eb;
      L = m + __logf(ssum);
      wa = ea / ssum;
      wb = eb / ssum * inv;  // folds the chunk's 1/l normalisation
    }
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float4 o = old[d * 4 + j];
        float4 nv = make_float4(wa * o.x + wb * oacc[d][j * 4], wa * o.y + wb * oacc[d][j * 4 + 1],
                                wa * o.z + wb * oacc[d][j * 4 + 2], wa * o.w + wb * oacc[d][j * 4 + 3]);
        *(float4*)(a.o_acc + obase + d * 32 + j * 8) = nv;
        if (a.o_out) *(u32x2*)(a.o_out + obase + d * 32 + j * 8) = pack_bf16x4(nv.x, nv.y, nv.z, nv.w);
      }
    if (hh == 0) a.lse_acc[li] = L;
  }
}

}  // namespace

hipError_t launch_attn_fwd(const FwdArgs& a, int n_items, int D, bool merge, hipStream_t st) {
  if (n_items <= 0) return hipSuccess;
  dim3 grid(n_items), block(NT);
  if (D == 128)
    return merge ? sp_launch(kKFwd, attn_fwd_kernel<128, true>, grid, block, st, a)
                 : sp_launch(kKFwd, attn_fwd_kernel<128, false>, grid, block, st, a);
  return merge ? sp_launch(kKFwd, attn_fwd_kernel<64, true>, grid, block, st, a)
               : sp_launch(kKFwd, attn_fwd_kernel<64, false>, grid, block, st, a);
}

}  // namespace spk
