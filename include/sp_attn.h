/*
 * sp_attn.h -- C ABI of the per-rank sequence-parallel attention library
 * (MI355X / gfx950).
 *
 * The library computes one sequence-parallel (SP) rank's share of a causal,
 * packed-varlen attention layer, forward and backward, for the two SP modes
 * of arXiv 2505.22296:
 *
 *   - Dummy-Head Ulysses (Section 4, Listing 1).  Query heads are padded at
 *     the END of the head axis with zero "dummy" heads up to a multiple of
 *     the SP size; after the all-to-all a rank holds the full sequence over
 *     H_loc = hs_new / sp head slots.  Dummy slots are never computed: their
 *     outputs and gradients are written as +0.0 (LSE -inf).
 *   - Ring-Attention (Section 2.1, Table 1).  A rank's Q chunk is run against
 *     successive KV chunks and partial results are combined through
 *     log-sum-exp.
 *
 * Conventions shared by every entry point
 *   Memory      All tensor pointers are DEVICE pointers owned by the caller;
 *               the library allocates no device memory.  Scratch space is a
 *               caller-provided workspace of the size sp_attn_workspace_size
 *               reports (256-byte aligned).  Arrays documented as HOST are
 *               read during the call only.
 *   Layout      Activations are contiguous [T, H, D] (token-major, D
 *               innermost), bf16 stored as uint16 bit patterns, 16-byte
 *               aligned.  LSE arrays are float32 [H, T] (head-major), natural
 *               logarithm.
 *   Streams     `stream` is a hipStream_t (NULL = the default stream).  Calls
 *               enqueue work and return; results are ready when the stream
 *               reaches them.  Host arrays may be freed on return.
 *   Errors      Every call returns sp_status.  Arguments are validated before
 *               anything is enqueued; on error nothing is launched and no
 *               output is touched.  SP_ERR_HIP reports a failed launch or copy.
 *               No C++ exception crosses this interface.
 *   Threading   The library holds no state (apart from the opt-in per-thread
 *               kernel timer of sp_profile_events); calls are reentrant.  Calls
 *               that share a workspace must be ordered on one stream.
 *   Graphs      The attention entry points (sp_attn_fwd, sp_ring_step,
 *               sp_attn_bwd) copy their host-built work lists into the
 *               workspace on every call; a HIP graph would replay that copy
 *               from freed host memory, so on a stream that is being
 *               captured they return SP_ERR_UNSUPPORTED (after argument and
 *               workspace validation) and enqueue nothing.  Calls with no
 *               query rows, which at most zero-fill outputs, are unaffected.
 *               Every other entry point passes its host arrays by value in
 *               the kernel arguments and may be recorded into a graph.
 *
 * Numerics: bf16 operands, float32 accumulation, float32 softmax statistics,
 * outputs rounded to bf16 with round-to-nearest-even.
 */
#ifndef SP_ATTN_H
#define SP_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum sp_status {
  SP_OK = 0,
  SP_ERR_INVALID_ARG = 1, /* inconsistent shapes, heads, segments, positions, pointers */
  SP_ERR_UNSUPPORTED = 2, /* valid but not supported (head_dim not 64/128, a limit, a capturing stream) */
  SP_ERR_WORKSPACE = 3,   /* workspace missing, misaligned or too small */
  SP_ERR_HIP = 4          /* a HIP launch or copy failed */
} sp_status;

/* Operation selector for sp_attn_workspace_size / sp_attn_schedule. */
enum { SP_OP_FWD = 0, SP_OP_BWD = 1, SP_OP_RING_STEP = 2 };

/*
 * One rank's attention problem.
 *
 * Heads.  Global query heads 0..num_padded_heads-1 exist after dummy-head
 * padding (Listing 1: hs_new = hs + (sp - hs % sp) % sp); heads >= hs =
 * num_real_heads are dummies.  This rank holds the H_loc consecutive slots
 * starting at global head head_offset (Ulysses: rank * H_loc; ring: 0).
 * Real query head g reads KV head g / gqa_group; the rank holds the Hkv_loc
 * consecutive KV heads starting at kv_head_offset.  Requirements:
 * num_padded_heads % H_loc == 0, head_offset % H_loc == 0,
 * num_padded_heads - num_real_heads < num_padded_heads / H_loc (fewer dummies
 * than ranks), num_real_heads % gqa_group == 0, and every real local head's KV
 * head lies in the local KV range.
 *
 * Segments (neat packing, Section 3.2).  num_seqs segments; query rows
 * [cu_seqlens_q[s], cu_seqlens_q[s+1]) attend to keys
 * [cu_seqlens_k[s], cu_seqlens_k[s+1]) only.  Rows/keys past the last
 * segment are padding: they attend to nothing (O = 0, LSE = -inf) and are
 * attended by nothing.  cu arrays start at 0, are non-decreasing, and end at
 * or below T.
 *
 * Positions (Section 5.2: explicit global position IDs).  When causal, key j
 * is visible to row i iff position_ids_k[j] <= position_ids_q[i] (diagonal
 * included).  Inside each segment positions must be a +1 ramp; only each
 * segment's first position matters, so ring chunks express their global
 * offsets here (Q chunk r at r*C.., KV chunk c at c*C..).  NULL means
 * positions 0,1,.. restarting at every segment.  Every call checks the ramps
 * (O(T) host work, SP_ERR_INVALID_ARG on a break) unless the environment
 * holds SPATTN_VALIDATE=0 when the library first validates a descriptor;
 * then only each segment's first position is read, and a broken ramp gives
 * a wrong mask, never an out-of-bounds access.
 *
 * Limits.  T_q, T_k < 2^30 and, per segment, |(first key position - first
 * key index) - (first query position - first query index)| <= 2^30
 * (SP_ERR_INVALID_ARG beyond); Hkv_loc <= 64 and H_loc <= 4096
 * (SP_ERR_UNSUPPORTED beyond).
 */
/*
 * SP_DESC_SINGLE_SEQUENCE: the num_seqs segments on each side are PIECES of
 * one sequence rather than separate sequences -- e.g. the zigzag split of
 * Ring-Attention (Section 3.2), where a rank holds chunks r and 2*sp-1-r of
 * the sequence and each ring step brings two KV chunks.  Every query row may
 * see every key; with causal = 1, key j is visible from row i iff
 * position_ids_k[j] <= position_ids_q[i].  Both position arrays are then
 * required, and over the rows [0, cu_seqlens_q[num_seqs]) (keys
 * [0, cu_seqlens_k[num_seqs])) they must increase strictly -- pieces in
 * ascending position order, each a +1 ramp.  Rows / keys past the last
 * piece are padding as usual.
 */
#define SP_DESC_SINGLE_SEQUENCE 1
/*
 * SP_DESC_ROWSTATS_READY (sp_attn_bwd only; ignored elsewhere): the per-row
 * statistics of the backward -- D_i = dO_i . O_i and LSE_i log2(e) of every
 * real query head -- are already in the workspace, left there by an earlier
 * sp_attn_bwd on the same workspace for the same query rows (same q, o, lse
 * and dout, same T_q, H_loc, head_offset and num_real_heads), ordered before
 * this call on the stream; this call does not recompute them.  They sit at
 * the start of the workspace whatever the keys, so a Ring-Attention
 * backward (Section 2.1) forms them once: the first KV chunk's call without
 * the flag, the other chunks' calls with it.  The library cannot check the
 * premise: stale statistics give wrong gradients (never an out-of-bounds
 * access).
 */
#define SP_DESC_ROWSTATS_READY 4
/*
 * SP_DESC_DQ_ACC_INIT (sp_attn_bwd when dq_acc is given; ignored otherwise):
 * the call starts the dQ accumulator instead of adding to it -- dq_acc is not
 * read, and is written with this call's dQ (with dq given too, dq = bf16(dQ)
 * and dq_acc is not touched at all), so it needs no clearing before the
 * first KV chunk of a ring backward.  Dummy slots of dq_acc stay untouched
 * either way.
 */
#define SP_DESC_DQ_ACC_INIT 8

typedef struct sp_attn_desc {
  int32_t T_q;              /* query tokens at this rank (rows of q, o, dq)         */
  int32_t T_k;              /* key tokens (rows of k, v, dk, dv)                     */
  int32_t head_dim;         /* D: 64 or 128                                          */
  int32_t H_loc;            /* query-head slots at this rank, real and dummy        */
  int32_t head_offset;      /* global index of local query slot 0                    */
  int32_t num_real_heads;   /* hs                                                    */
  int32_t num_padded_heads; /* hs_new                                                */
  int32_t gqa_group;        /* real query heads per KV head (1 = MHA)                */
  int32_t Hkv_loc;          /* KV heads at this rank                                 */
  int32_t kv_head_offset;   /* global index of local KV head 0                       */
  int32_t num_seqs;         /* segments (>= 0)                                       */
  int32_t causal;           /* 1 = causal by position inside a segment, 0 = full     */
  float softmax_scale;      /* multiplies q.k (callers pass 1/sqrt(D))               */
  int32_t flags;            /* 0 or an OR of the SP_DESC_* flags above               */
  const int32_t* cu_seqlens_q;   /* HOST, num_seqs + 1                               */
  const int32_t* cu_seqlens_k;   /* HOST, num_seqs + 1                               */
  const int32_t* position_ids_q; /* HOST, T_q, or NULL                               */
  const int32_t* position_ids_k; /* HOST, T_k, or NULL                               */
} sp_attn_desc;

/* Human-readable name of a status code (static storage). */
const char* sp_status_string(sp_status s);

/* Library version as major*10000 + minor*100 + patch. */
int32_t sp_version(void);

/*
 * Dummy-head padding + Ulysses send-side pack (Section 4.1, Listing 1, and
 * the [L/sp, hs, d] -> [L, hs/sp, d] all-to-all layout of Section 4):
 *
 *   dst[j, t, h, :] = src[t, head_map[j*H_dst_loc + h], :]   (map entry >= 0)
 *   dst[j, t, h, :] = 0                                       (map entry == -1)
 *
 * src: [T_loc, H_src, D] bf16; dst: [sp, T_loc, H_dst_loc, D] bf16, where
 * chunk j is what goes to rank j.  head_map: HOST, sp*H_dst_loc entries in
 * [-1, H_src); a source head may appear several times (GQA K/V replicated to
 * two ranks).  For Ulysses Q (and MHA K/V) the map is
 * j*H_loc + h if < hs else -1, which is Listing 1's pad followed by the even
 * head split.  Bit copy: the output is exact.  D must be a multiple of 8.
 * T_loc == 0 is a no-op.
 */
sp_status sp_ulysses_pack(const void* src, int32_t T_loc, int32_t H_src, int32_t head_dim,
                          int32_t sp, int32_t H_dst_loc, const int32_t* head_map, void* dst,
                          void* stream);

/*
 * Ulysses receive-side unpack + unpad (Listing 1 unpad_heads, after the
 * reverse all-to-all):
 *
 *   dst[t, head_map[j*H_src_loc + h], :] = src[j, t, h, :]   (map entry >= 0)
 *
 * src: [sp, T_loc, H_src_loc, D] bf16; dst: [T_loc, H_dst, D] bf16.
 * Entries equal to -1 (dummy slots) are dropped.  Every destination head
 * 0..H_dst-1 must be named exactly once (otherwise SP_ERR_INVALID_ARG).
 * Bit copy.
 */
sp_status sp_ulysses_unpack(const void* src, int32_t T_loc, int32_t H_src_loc, int32_t head_dim,
                            int32_t sp, const int32_t* head_map, int32_t H_dst, void* dst,
                            void* stream);

/*
 * Summing unpack of GQA K/V gradients after the reverse all-to-all (the
 * backward of the K/V pack, Section 4.1 / Listing 1 with GQA: the pack sends
 * one KV head to every rank whose real query heads read it, so the gradients
 * those ranks return for it are added):
 *
 *   dst[t, g, :] = sum over slots s = j*H_src_loc + h with head_map[s] == g,
 *                  in ascending s (source rank j, then slot h), of src[j, t, h, :]
 *
 * src: [sp, T_loc, H_src_loc, D] bf16 (the receive buffer: chunk j came from
 * rank j); dst: [T_loc, H_dst, D] bf16; head_map: HOST, the same map the
 * forward pack used (-1 slots are dropped).  Each sum is formed in float32,
 * one slot at a time in that order, and rounded once to bf16 (nearest-even),
 * so the result is deterministic bit for bit.  A head named by no slot is
 * written as +0.  Limits: sp*H_src_loc <= 512, H_dst <= 256
 * (SP_ERR_UNSUPPORTED); map entries outside [-1, H_dst) are
 * SP_ERR_INVALID_ARG.  T_loc == 0 is a no-op.  Reads sp*T_loc*H_src_loc*D*2
 * bytes and writes T_loc*H_dst*D*2.
 */
sp_status sp_ulysses_unpack_add(const void* src, int32_t T_loc, int32_t H_src_loc,
                                int32_t head_dim, int32_t sp, const int32_t* head_map,
                                int32_t H_dst, void* dst, void* stream);

/* Workspace bytes needed by `op` (SP_OP_FWD, SP_OP_BWD, SP_OP_RING_STEP) for
 * this problem.  Validates the descriptor. */
sp_status sp_attn_workspace_size(const sp_attn_desc* desc, int32_t op, size_t* bytes);

/*
 * Attention forward over the rank's real heads (the FlashAttention-style
 * fused kernel: bf16 MFMA for QK^T and PV, fp32 online softmax, causal and
 * varlen block skipping; dummy slots are not computed).
 *
 * q: [T_q, H_loc, D]; k, v: [T_k, Hkv_loc, D]   (bf16, inputs, not modified)
 * o: [T_q, H_loc, D] bf16 output; lse: [H_loc, T_q] float32 output.
 * Real head rows: O = softmax(scale q k^T + mask) v, LSE = log-sum-exp of the
 * masked scaled scores.  Rows without visible keys and all dummy slots:
 * O = +0.0, LSE = -inf.  Empty inputs: pointers are only required for
 * tensors with elements; T_q == 0 is a no-op, T_k == 0 gives every row
 * O = +0.0 and LSE = -inf (the same holds for sp_ring_step, and sp_attn_bwd
 * then writes dQ = +0.0; with T_q == 0 it writes dK = dV = +0.0).
 */
sp_status sp_attn_fwd(const sp_attn_desc* desc, const void* q, const void* k, const void* v,
                      void* o, float* lse, void* workspace, size_t workspace_bytes,
                      void* stream);

/*
 * Allocation-free forward, for callers that cannot allocate device memory or
 * pass a workspace (tight serving loops, harnesses that forbid hipMalloc):
 * the same operation, kernels and outputs as sp_attn_fwd (bit for bit), with
 * the work list kept in a library-owned device array of
 * SP_STATIC_SCRATCH_BYTES instead of a caller workspace.  Every GPU the
 * library runs on holds its own copy of that array until the process ends;
 * its address is looked up once per device on the first call there.  The
 * call allocates no device memory (and calls no allocating HIP or library
 * routine); its host-side scheduling uses ordinary host heap memory.
 *
 * Limit: the work list (SP_SCHED_ITEM_INTS int32 per item, as reported by
 * sp_attn_schedule for SP_OP_FWD) must fit in SP_STATIC_SCRATCH_BYTES, i.e.
 * at most 32768 items -- about 8.4M query rows x real heads; larger
 * problems return SP_ERR_UNSUPPORTED before anything is enqueued.
 * `stream` must belong to the current device (else SP_ERR_INVALID_ARG).
 * Every call on one GPU shares that GPU's array and overwrites the part it
 * uses (nothing in it needs to start at zero): calls that overlap on one GPU
 * -- on different streams without ordering between them, or from several
 * host threads -- race on it.  Order them on one stream or synchronize.
 * Like sp_attn_fwd it refuses a capturing stream (SP_ERR_UNSUPPORTED).
 */
#define SP_STATIC_SCRATCH_BYTES (1u << 20)
sp_status sp_attn_fwd_static(const sp_attn_desc* desc, const void* q, const void* k,
                             const void* v, void* o, float* lse, void* stream);

/*
 * Attention backward (gradients of sum(dO * O)), with P recomputed from LSE:
 * dV = P^T dO, dP = dO V^T, dS = P (dP - rowsum(dO o O)), dQ = scale dS K,
 * dK = scale dS^T Q.  dK/dV of a KV head sum over its real query heads.
 *
 * o, lse: the forward's outputs (for ring: the FINAL merged O and LSE).
 * dout: [T_q, H_loc, D] bf16.
 * dq: bf16 [T_q, H_loc, D], written; or NULL.
 * dq_acc: float32 [T_q, H_loc, D], dQ is ADDED to it (ring: accumulate over
 *         KV chunks, Section 2.1); or NULL.  At least one of dq / dq_acc must
 *         be non-NULL:
 *           dq only:         dq = bf16(dQ);
 *           dq_acc only:     dq_acc += dQ (with SP_DESC_DQ_ACC_INIT in the
 *                            flags: dq_acc = dQ, nothing read -- the first KV
 *                            chunk of a ring backward);
 *           both:            dq = bf16(dq_acc + dQ) (bf16(dQ) under
 *                            SP_DESC_DQ_ACC_INIT), dq_acc not written -- the
 *                            last KV chunk: the accumulator's final sum goes
 *                            straight to bf16, with no separate cast.
 * dk, dv: bf16 [T_k, Hkv_loc, D], written.
 * Dummy slots: dq = +0.0 (dq_acc untouched); KV heads read by no real query
 * head get dk = dv = +0.0.  Deterministic: no atomics.
 */
sp_status sp_attn_bwd(const sp_attn_desc* desc, const void* q, const void* k, const void* v,
                      const void* o, const float* lse, const void* dout, void* dq,
                      float* dq_acc, void* dk, void* dv, void* workspace,
                      size_t workspace_bytes, void* stream);

/*
 * One Ring-Attention step (Section 2.1): attention of the rank's Q chunk
 * against one KV chunk, merged into running float32 accumulators:
 *   (O, L) <- (O, L) (+) (O_c, L_c),  L = logaddexp(L, L_c),
 *   O = e^(L_old - L) O + e^(L_c - L) O_c.
 * desc positions carry the chunk offsets.  init = 1 on the first chunk:
 * the accumulators are overwritten with this chunk's partial (rows that see
 * no key: O = 0, L = -inf).  init = 0: rows that see no key of this chunk are
 * left untouched (the merge identity).
 * o_acc: float32 [T_q, H_loc, D] in/out; lse_acc: float32 [H_loc, T_q] in/out.
 * o_out: optional bf16 [T_q, H_loc, D]; when non-NULL the merged O is also
 * written there rounded to bf16 (use on the last chunk).  Dummy slots: with
 * init the accumulators get (0, -inf); o_out gets +0.0.
 */
sp_status sp_ring_step(const sp_attn_desc* desc, const void* q, const void* k_chunk,
                       const void* v_chunk, float* o_acc, float* lse_acc, int32_t init,
                       void* o_out, void* workspace, size_t workspace_bytes, void* stream);

/*
 * Standalone log-sum-exp merge of two partial attention results over disjoint
 * key sets (the ring combine, Section 2.1), in float32:
 *   L = logaddexp(L_acc, L_part); O_acc = e^(L_acc-L) O_acc + e^(L_part-L) O_part;
 *   both -inf gives (0, -inf).
 * o_acc: float32 [T, H, D] in/out; lse_acc: float32 [H, T] in/out.
 * o_part: [T, H, D], bf16 when o_part_is_bf16 else float32; lse_part: [H, T].
 * o_out_bf16: optional bf16 [T, H, D] copy of the merged O (RNE), or NULL.
 * D must be a multiple of 8.
 */
sp_status sp_lse_merge(float* o_acc, float* lse_acc, const void* o_part, int32_t o_part_is_bf16,
                       const float* lse_part, int32_t T, int32_t H, int32_t head_dim,
                       void* o_out_bf16, void* stream);

/* dst[i] = bf16_rne(src[i]) for i < n (e.g. a ring dQ accumulator). */
sp_status sp_f32_to_bf16(const float* src, void* dst, int64_t n, void* stream);

/*
 * Introspection of the block-skip scheduler (host only, no GPU work): the
 * work items `op` would launch, SP_SCHED_ITEM_INTS int32 each, in launch
 * order, which is laid out per XCD (workgroup i of a launch runs on XCD
 * i % 8, counting the fill items below; an XCD feeds its four shader
 * engines in turn, in order): every XCD's share (positions x, x + 8, ...)
 * is longest first.  Row items (SP_OP_FWD / SP_OP_RING_STEP) are dealt to
 * the XCDs in groups of four consecutive items of the longest-first order,
 * eight groups a round, the rounds alternately forwards and backwards over
 * the XCDs (the rest item by item); dK/dV items one by one in list order.
 * Within each cost the items an XCD gets are a contiguous share of that
 * cost's items taken head by head, so each XCD's L2 serves a few
 * neighbouring heads.
 *   SP_OP_FWD / SP_OP_RING_STEP (init=1): {q_begin, q_end, k_begin, k_end,
 *       delta, head, kv_head, 0} -- query rows [q_begin, q_end) of local
 *       head `head` against keys [k_begin, k_end); causal visibility is
 *       key <= row + delta.  Row tiles hold 256 rows; under a causal mask
 *       they end at the segment's end, so a partial tile is the segment's
 *       first (its rows see the fewest keys).
 *   SP_OP_BWD, dK/dV items: {k_begin, k_end, q_begin, q_end, delta, head,
 *       kv_head, 1}.
 * Writes at most `capacity` items to `items` (may be NULL) and the total
 * count to *n_items.  Not listed: the zero fills of dummy query slots (and,
 * for one query head per KV head, of KV heads no real query head reads),
 * which the entry points put at the front of the same launch as fill items
 * of up to 8192 rows (keys) of one head, so a rank with dummy slots
 * launches no extra kernel.
 */
#define SP_SCHED_ITEM_INTS 8
sp_status sp_attn_schedule(const sp_attn_desc* desc, int32_t op, int32_t* items, int32_t capacity,
                           int32_t* n_items);

/*
 * SP-aware loss (Section 3.3, Correct Loss Calculation; Section 5.1 and
 * Listing 2).  Each rank holds a slice of the sequence, so it forms the
 * label log-probabilities of its own tokens only; the SFT loss (Eq. 1) is
 * the sum over all tokens, and DPO (Eq. 2, read with the log on both
 * ratios) needs the four sequence log-probabilities summed over the ranks
 * before the sigmoid.  The sums cross ranks through an all-reduce that
 * carries gradients (its backward all-reduces the upstream gradient).
 *
 * sp_token_logprob: for token t with label y = labels[t] (DEVICE int32 [T])
 * inside a sequence and y in [0, V), y != ignore_index:
 *   lse[t]  = log sum_v exp(logits[t, v])            (float32, natural log)
 *   logp[t] = logits[t, y] - lse[t]                   (0 for other tokens)
 *   seq_sum[s] = sum of logp over [cu[s], cu[s+1])   (fixed order: deterministic)
 * logits: DEVICE bf16 [T, V] row-major, 16-byte aligned, V a multiple of 8.
 * cu_seqlens: HOST, num_seqs + 1 non-decreasing entries, cu[0] >= 0,
 * cu[num_seqs] <= T; tokens outside every sequence get logp = 0.  lse is
 * written for every token (the backward reads it).  Limits: num_seqs <= 256
 * (SP_ERR_UNSUPPORTED).  Reads T*V*2 bytes once.
 */
enum { SP_LOSS_SFT = 0, SP_LOSS_DPO = 1 };
sp_status sp_token_logprob(const void* logits, const int32_t* labels, int32_t T, int32_t V,
                           int32_t ignore_index, const int32_t* cu_seqlens, int32_t num_seqs,
                           float* logp, float* lse, float* seq_sum, void* stream);

/*
 * Backward of sum_s grad_seq[s] * seq_sum[s] to the logits (DEVICE bf16
 * [T, V] out): for a token t of sequence s with a counted label y,
 *   dlogits[t, v] = g * (1[v == y] - exp(logits[t, v] - lse[t])),  g = grad_seq[s]
 * rounded to bf16 (nearest-even); every other row is written as zeros.
 * grad_seq: DEVICE float32 [num_seqs] (from sp_loss_reduce); lse from the
 * forward.  Same shape rules as sp_token_logprob.  Reads T*V*2 bytes, writes
 * T*V*2 bytes.
 */
sp_status sp_token_logprob_bwd(const void* logits, const int32_t* labels, const float* lse,
                               int32_t T, int32_t V, int32_t ignore_index,
                               const int32_t* cu_seqlens, int32_t num_seqs,
                               const float* grad_seq, void* dlogits, void* stream);

/*
 * Loss over the ranks' partial sums and every rank's upstream gradient.
 * partial_sums: DEVICE float32 [sp, num_seqs], row r = rank r's seq_sum
 * (on one GPU all rows are available; across GPUs, the rows an all-gather
 * delivers).  Totals are summed over ranks in ascending order.
 *   SP_LOSS_SFT: loss = -coef * sum over sequences of the totals
 *                (coef = 1 for Eq. 1, 1 / #tokens for a mean).
 *   SP_LOSS_DPO: sequences are pairs (2p chosen, 2p+1 rejected);
 *                z_p = coef * ((pi_w - ref_w) - (pi_l - ref_l)) with coef = beta
 *                and ref totals from ref_partial_sums (DEVICE [sp, num_seqs],
 *                the reference model's seq_sum, no gradient);
 *                loss = mean over pairs of -log sigmoid(z_p).
 * grad: DEVICE float32 [sp, num_seqs], rank r's upstream gradient for its
 * own seq_sum: sp times d loss / d total, the gradient a gradient-carrying
 * all-reduce returns to every rank (each rank computes the same loss, and
 * the backward of the all-reduce sums their upstream gradients).  Averaging
 * parameter gradients over the sp ranks then gives the gradient without SP
 * (Listing 2: 8 and 12 average to the local 10; a plain all-reduce gives 4
 * and 6).  loss: DEVICE float32 [1].  Errors: SP_ERR_INVALID_ARG for sp < 1,
 * num_seqs < 1, an odd DPO count, missing pointers, non-finite coef;
 * SP_ERR_UNSUPPORTED for num_seqs > 256.
 */
sp_status sp_loss_reduce(const float* partial_sums, const float* ref_partial_sums, int32_t sp,
                         int32_t num_seqs, int32_t kind, float coef, float* loss, float* grad,
                         void* stream);

/*
 * Opt-in kernel timer (measurement support, per calling thread).  After
 * sp_profile_events(id, start, stop) with hipEvent_t handles created by the
 * caller, every launch of kernel `id` made by THIS thread records `start` on
 * the stream of the call immediately before the kernel is launched and `stop`
 * immediately after it (hipEventRecord).  If a call launches that kernel more
 * than once, the events describe the last launch.  Pass NULL events to disarm.  This is the
 * only state the library keeps (thread-local, no allocation).
 */
enum {
  SP_KERNEL_ATTN_FWD = 1, /* forward / ring-step attention kernel        */
  SP_KERNEL_ATTN_DQ = 2,  /* backward dQ kernel (S, dP, dQ)              */
  SP_KERNEL_ATTN_DKDV = 3,/* backward dK/dV kernel (S, P, dV, dP, dS, dK) */
  SP_KERNEL_PACK = 4,     /* Ulysses pack                                */
  SP_KERNEL_UNPACK = 5,   /* Ulysses unpack                              */
  SP_KERNEL_LSE_MERGE = 6,/* standalone LSE merge                        */
  SP_KERNEL_UNPACK_ADD = 7,/* summing unpack of GQA K/V gradients        */
  SP_KERNEL_TOKEN_LOGPROB = 8,     /* token log-probabilities (forward)  */
  SP_KERNEL_TOKEN_LOGPROB_BWD = 9  /* their backward to the logits       */
};
sp_status sp_profile_events(int32_t kernel_id, void* start_event, void* stop_event);

#ifdef __cplusplus
}
#endif

#endif /* SP_ATTN_H */
