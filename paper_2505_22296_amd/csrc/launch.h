// Internal interface between the host-side ABI code and the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace spk {

// Kernel identifiers of the opt-in per-thread launch timer (values match the
// SP_KERNEL_* constants of the public header).
enum KernelId {
  kKFwd = 1, kKDq = 2, kKDkdv = 3, kKPack = 4, kKUnpack = 5, kKMerge = 6, kKUnpackAdd = 7,
  kKLogprob = 8, kKLogprobBwd = 9, kKCount = 10
};

struct KernelTimer {
  hipEvent_t start = nullptr, stop = nullptr;
};
// Thread-local timer slot of a kernel id (defined with the C ABI).
KernelTimer& timer_for(int kernel_id);

// Launch `kernel`; when the calling thread armed events for `id`, record them
// on the same stream immediately before and after the launch.  (Plain event
// records: passing events to hipExtLaunchKernelGGL was measured to stall the
// running kernels by ~5 ms per dispatch for ~0.2 s after new events are first
// used that way.)
template <typename F, typename... Args>
inline hipError_t sp_launch(int id, F kernel, dim3 grid, dim3 block, hipStream_t st,
                            Args... args) {
  KernelTimer& t = timer_for(id);
  if (t.start) {
    hipError_t e = hipEventRecord(t.start, st);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(kernel, grid, block, 0, st, args...);
  hipError_t e = hipGetLastError();
  if (e == hipSuccess && t.stop) e = hipEventRecord(t.stop, st);
  return e;
}

// Maximum head-map entries a pack/unpack carries by value in its arguments.
static constexpr int kMaxMap = 512;
// Maximum local KV heads for the GQA dK/dV reduction.
static constexpr int kMaxKv = 64;

struct PackArgs {
  int sp, T, Hs, Hd, nch;  // nch = 16-byte chunks per head row (D / 8)
  int map[kMaxMap];        // pack: slot -> source head; unpack: dest head -> j*Hs + h
};

// Summing unpack: destination head g sums source slots slot[start[g]] ..
// slot[start[g+1]-1] (each j*Hs + h, ascending).  int16 keeps the arguments
// small (slots < kMaxMap, heads <= kMaxAddDst).
static constexpr int kMaxAddDst = 256;
struct PackAddArgs {
  int sp, T, Hs, Hd, nch;
  int16_t start[kMaxAddDst + 1];
  int16_t slot[kMaxMap];
};

// Loss path: vocabulary size V (multiple of 8), the sequences' token
// ranges [cu[s], cu[s+1]) (host copy by value) and the ignored label.
static constexpr int kMaxLossSeqs = 256;
struct LossArgs {
  int T, V, ignore_index, n_seqs;
  int cu[kMaxLossSeqs + 1];
};
struct LossReduceArgs {
  int sp, n, kind;  // kind 0 = SFT, 1 = DPO
  float coef;       // SFT: loss scale; DPO: beta
};

struct ReduceArgs {
  int T, Hkv, D;
  int head_lo[kMaxKv], head_hi[kMaxKv];  // query heads [lo, hi) feeding each KV head
};

// Work item of the attention kernels: 8 int32.
//   fwd / dq:  {q_begin, q_end, k_begin, k_end, delta, head, kv_head, 0}
//   dk/dv:     {k_begin, k_end, q_begin, q_end, delta, head, kv_head, 1}
//   zero fill of a dummy query slot (fwd / dq): {r_begin, r_end, 0, 0, 0, slot, 0, 2}
//   zero fill of a KV head no real query head reads (dk/dv):
//              {k_begin, k_end, 0, 0, 0, 0, kv_head, 3}
// Causal visibility of key j from row i is j <= i + delta.
static constexpr int kItemInts = 8;
static constexpr int kItemFillQ = 2, kItemFillKV = 3;
static constexpr int kFillRows = 8192;  // rows (keys) per zero-fill item

struct FwdArgs {
  const uint16_t* q;   // [T_q, H, D]
  const uint16_t* k;   // [T_k, Hkv, D]
  const uint16_t* v;   // [T_k, Hkv, D]
  uint16_t* o;         // [T_q, H, D] (plain forward)
  float* lse;          // [H, T_q]
  float* o_acc;        // ring: [T_q, H, D] float32 in/out
  float* lse_acc;      // ring: [H, T_q] in/out
  uint16_t* o_out;     // ring: optional bf16 copy of the merged O
  const int32_t* items;
  int T_q, T_k, H, Hkv;
  float scale_log2;    // softmax_scale * log2(e)
  int causal, init;
};

struct DqArgs {
  const uint16_t* q;     // [T_q, H, D]
  const uint16_t* k;     // [T_k, Hkv, D]
  const uint16_t* v;     // [T_k, Hkv, D]
  const uint16_t* dout;  // [T_q, H, D]
  const float* lse;      // [H, T_q]
  const float* neg_d;    // -D = -(dO . O) per row: [n_real, T_q]
  uint16_t* dq;          // bf16 [T_q, H, D] or null
  float* dq_acc;         // float32 [T_q, H, D] or null: with dq, read only
                         // (dq = bf16(dq_acc + dQ)); without, dq_acc += dQ
  int dq_init;           // dq_acc taken as zero (not read)
  const int32_t* items;
  int T_q, T_k, H, Hkv;
  float scale_log2, scale;
  int causal;
};

struct DkdvArgs {
  const uint16_t* q;     // [T_q, H, D]
  const uint16_t* dout;  // [T_q, H, D]
  const float* lse2;     // [n_real, T_q]: LSE * log2(e), +inf for rows without keys
  const float* neg_d;    // -D = -(dO . O) per row: [n_real, T_q]
  const uint16_t* k;     // [T_k, Hkv, D]
  const uint16_t* v;     // [T_k, Hkv, D]
  uint16_t* dk;          // bf16 [T_k, Hkv, D] (direct mode)
  uint16_t* dv;
  float* part_k;         // float32 [n_real, T_k, D] (GQA partial mode)
  float* part_v;
  const int32_t* items;
  int T_q, T_k, H, Hkv;
  float scale_log2, scale;
  int causal, direct;
};

hipError_t launch_pack(const void* src, void* dst, const PackArgs& a, hipStream_t st);
hipError_t launch_unpack(const void* src, void* dst, const PackArgs& a, hipStream_t st);
hipError_t launch_unpack_add(const void* src, void* dst, const PackAddArgs& a, hipStream_t st);
hipError_t launch_token_logprob(const LossArgs& a, const void* logits, const int32_t* labels,
                                float* logp, float* lse, float* seq_sum, hipStream_t st);
hipError_t launch_token_logprob_bwd(const LossArgs& a, const void* logits, const int32_t* labels,
                                    const float* lse, const float* grad_seq, void* dlogits,
                                    hipStream_t st);
hipError_t launch_loss_reduce(const LossReduceArgs& a, const float* ps, const float* refs,
                              float* loss, float* grad, hipStream_t st);
hipError_t launch_merge(float* o_acc, float* lse_acc, const void* o_part, bool part_bf16,
                        const float* lse_part, int T, int H, int D, void* o_out, hipStream_t st);
hipError_t launch_zero_heads_bf16(void* x, int T, int H, int D, int h0, int h1, hipStream_t st);
hipError_t launch_zero_heads_f32(float* x, int T, int H, int D, int h0, int h1, hipStream_t st);
hipError_t launch_fill_f32(float* x, int64_t n, float v, hipStream_t st);
hipError_t launch_f32_to_bf16(const float* s, void* d, int64_t n, hipStream_t st);
hipError_t launch_rowdot(const void* o, const void* dout, const float* lse, float* neg_d,
                         float* lse2, int T, int H, int nh, int D, hipStream_t st);
hipError_t launch_reduce_kv(const float* part_k, const float* part_v, void* dk, void* dv,
                            const ReduceArgs& a, hipStream_t st);

hipError_t launch_attn_fwd(const FwdArgs& a, int n_items, int D, bool merge, hipStream_t st);
hipError_t launch_attn_dq(const DqArgs& a, int n_items, int D, hipStream_t st);
hipError_t launch_attn_dkdv(const DkdvArgs& a, int n_items, int D, hipStream_t st);

// Tile sizes the host scheduler must use (rows per fwd/dq item, keys per
// dk/dv item) and the kernels' LDS pipelines.
static constexpr int kFwdWaves = 8;                 // wavefronts per forward workgroup
static constexpr int kFwdBM = 32 * kFwdWaves;
static constexpr int kFwdBN = 64;
static constexpr int kFwdStages = 4;                // K/V tiles resident in LDS
static constexpr int kFwdTilesPerSync = 2;          // tiles between workgroup barriers
static constexpr int kDqWaves = 8;                  // wavefronts per dQ workgroup
static constexpr int kDqBM = 32 * kDqWaves;
static constexpr int kDqBN = 32;
static constexpr int kDqStages = 4;
static constexpr int kDqTilesPerSync = 2;
static constexpr int kDkdvWaves = 8;                // wavefronts per dK/dV workgroup (4 pairs)
static constexpr int kDkdvBN = 16 * kDkdvWaves;     // keys per dK/dV item
static constexpr int kDkdvBQ = 32;                  // query rows per chunk

}  // namespace spk
