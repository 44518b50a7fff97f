// Host side of the SP attention library: argument validation, the block-skip
// scheduler, workspace layout and the C ABI declared in include/sp_attn.h.
//
// The scheduler replaces full masks (the paper notes the varlen path's
// overhead, Section 6.3): from cu_seqlens and the segments' position bases it
// lists one work item per (real head, segment, row tile) -- or per (real
// head, segment, key tile) for dK/dV -- carrying the tile's visible key (row)
// range and the causal offset delta (key j visible from row i iff
// j <= i + delta).  Dummy head slots (Section 4.1) never enter the list.
// Items are ordered longest first on every XCD, laid out for the order in
// which the hardware hands workgroups to XCDs and shader engines (see
// sort_items), so that its dispatch fills the 256 CUs the way
// longest-processing-time scheduling would.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <vector>

#include "../../include/sp_attn.h"
#include "launch.h"

namespace {

using spk::kItemInts;

constexpr int64_t kMaxTokens = int64_t(1) << 30;

struct Seg {
  int qa, qb, ka, kb, delta;
};

struct Problem {
  int D = 0;
  int n_real = 0;  // real local query heads: slots [0, n_real)
  // Row-side and key-side runs: rows [qa, qb) x keys [ka, kb) with key j
  // visible from row i iff j <= i + delta (causal).  For separate sequences
  // both lists are the segments; for one sequence in pieces they are the
  // maximal row (key) ranges over which the visible key (row) range grows
  // by 0 or 1 per row (key).
  std::vector<Seg> segs, segs_k;
  int q_pad = 0, k_pad = 0;  // first padding row / key
  std::vector<int> kv_of;    // per real local head
  std::vector<int> kv_lo, kv_hi;  // per local KV head: real heads [lo, hi) reading it
  bool direct = true;        // every KV head read by at most one real local head
};


// One sequence in pieces (SP_DESC_SINGLE_SEQUENCE): rows [0, Qn) and keys
// [0, Kn) have strictly increasing positions, so the keys visible from row i
// are a prefix [0, n(i)) and the rows that see key j a suffix [m(j), Qn).
// n and m are split into maximal runs of constant step 0 or 1; each run is a
// Seg whose linear rule j <= i + delta reproduces the prefix / suffix.
sp_status single_sequence_runs(const sp_attn_desc* d, Problem& p) {
  const int n = d->num_seqs;
  if (n < 1 || !d->position_ids_q || !d->position_ids_k) return SP_ERR_INVALID_ARG;
  const int Qn = d->cu_seqlens_q[n], Kn = d->cu_seqlens_k[n];
  const int32_t* pq = d->position_ids_q;
  const int32_t* pk = d->position_ids_k;
  for (int i = 1; i < Qn; ++i)
    if (pq[i] <= pq[i - 1]) return SP_ERR_INVALID_ARG;
  for (int j = 1; j < Kn; ++j)
    if (pk[j] <= pk[j - 1]) return SP_ERR_INVALID_ARG;
  std::vector<int> cnt(Qn), first(Kn);
  for (int i = 0, j = 0; i < Qn; ++i) {  // n(i) = #keys with pos_k <= pos_q[i]
    if (d->causal)
      while (j < Kn && pk[j] <= pq[i]) ++j;
    cnt[i] = d->causal ? j : Kn;
  }
  for (int j = 0, i = 0; j < Kn; ++j) {  // m(j) = first row with pos_q >= pos_k[j]
    if (d->causal)
      while (i < Qn && pq[i] < pk[j]) ++i;
    first[j] = d->causal ? i : 0;
  }
  p.segs.clear();
  for (int i0 = 0; i0 < Qn;) {
    const int step = (i0 + 1 < Qn) ? cnt[i0 + 1] - cnt[i0] : 0;
    int i1 = i0 + 1;
    if (step == 0 || step == 1)
      while (i1 < Qn && cnt[i1] - cnt[i1 - 1] == step) ++i1;
    // step 1: keys [0, cnt[i]) = j <= i + cnt[i0] - 1 - i0; step 0 (or a
    // single row): keys [0, cnt[i0]), every one of them visible
    const int delta = (i1 - i0 > 1 && step == 1) ? cnt[i0] - 1 - i0 : cnt[i0];
    p.segs.push_back(Seg{i0, i1, 0, cnt[i1 - 1], delta});
    i0 = i1;
  }
  p.segs_k.clear();
  for (int j0 = 0; j0 < Kn;) {
    const int step = (j0 + 1 < Kn) ? first[j0 + 1] - first[j0] : 0;
    int j1 = j0 + 1;
    if (step == 0 || step == 1)
      while (j1 < Kn && first[j1] - first[j1 - 1] == step) ++j1;
    // step 1: rows [first[j], Qn) = j <= i + j0 - first[j0]; step 0 (or a
    // single key): rows [first[j0], Qn), visible from every key of the run
    const int delta = (j1 - j0 > 1 && step == 1) ? j0 - first[j0] : (j1 - 1) - first[j0];
    p.segs_k.push_back(Seg{first[j0], Qn, j0, j1, delta});
    j0 = j1;
  }
  return SP_OK;
}

// The O(T) checks that every segment's positions form a +1 ramp run unless
// the environment sets SPATTN_VALIDATE=0 (read once per process); without
// them only each segment's first position is read, and a malformed ramp
// gives a wrong mask, never an out-of-bounds access.
bool ramp_checks() {
  static const bool on = [] {
    const char* e = std::getenv("SPATTN_VALIDATE");
    return !(e && e[0] == '0' && e[1] == '\0');
  }();
  return on;
}

sp_status validate(const sp_attn_desc* d, Problem& p) {
  if (!d) return SP_ERR_INVALID_ARG;
  if (d->flags & ~(SP_DESC_SINGLE_SEQUENCE | SP_DESC_ROWSTATS_READY | SP_DESC_DQ_ACC_INIT))
    return SP_ERR_INVALID_ARG;
  const bool single = (d->flags & SP_DESC_SINGLE_SEQUENCE) != 0;
  if (d->T_q < 0 || d->T_k < 0 || d->T_q >= kMaxTokens || d->T_k >= kMaxTokens)
    return SP_ERR_INVALID_ARG;
  if (d->head_dim != 64 && d->head_dim != 128) return SP_ERR_UNSUPPORTED;
  if (d->H_loc < 1 || d->Hkv_loc < 1 || d->num_padded_heads < 1 || d->num_real_heads < 1 ||
      d->gqa_group < 1 || d->head_offset < 0 || d->kv_head_offset < 0 || d->num_seqs < 0)
    return SP_ERR_INVALID_ARG;
  if (d->Hkv_loc > spk::kMaxKv || d->H_loc > 4096) return SP_ERR_UNSUPPORTED;
  if (d->num_real_heads > d->num_padded_heads) return SP_ERR_INVALID_ARG;
  if (d->num_padded_heads % d->H_loc != 0 || d->head_offset % d->H_loc != 0 ||
      d->head_offset + d->H_loc > d->num_padded_heads)
    return SP_ERR_INVALID_ARG;
  const int sp = d->num_padded_heads / d->H_loc;
  if (d->num_padded_heads - d->num_real_heads >= sp) return SP_ERR_INVALID_ARG;
  if (d->num_real_heads % d->gqa_group != 0) return SP_ERR_INVALID_ARG;
  if (!(d->softmax_scale > 0.f) || !std::isfinite(d->softmax_scale)) return SP_ERR_INVALID_ARG;
  if (d->causal != 0 && d->causal != 1) return SP_ERR_INVALID_ARG;

  p.D = d->head_dim;
  p.n_real = std::max(0, std::min(d->H_loc, d->num_real_heads - d->head_offset));
  p.kv_of.resize(p.n_real);
  p.kv_lo.assign(d->Hkv_loc, 0);
  p.kv_hi.assign(d->Hkv_loc, 0);
  std::vector<int> cnt(d->Hkv_loc, 0);
  for (int y = 0; y < p.n_real; ++y) {
    int kv = (d->head_offset + y) / d->gqa_group - d->kv_head_offset;
    if (kv < 0 || kv >= d->Hkv_loc) return SP_ERR_INVALID_ARG;
    if (y > 0 && kv < p.kv_of[y - 1]) return SP_ERR_INVALID_ARG;  // monotone by construction
    p.kv_of[y] = kv;
    if (cnt[kv] == 0) p.kv_lo[kv] = y;
    p.kv_hi[kv] = y + 1;
    ++cnt[kv];
  }
  p.direct = true;
  for (int c : cnt)
    if (c > 1) p.direct = false;

  // segments
  const int n = d->num_seqs;
  p.segs.clear();
  p.q_pad = 0;
  p.k_pad = 0;
  if (n > 0) {
    if (!d->cu_seqlens_q || !d->cu_seqlens_k) return SP_ERR_INVALID_ARG;
    const int32_t* cq = d->cu_seqlens_q;
    const int32_t* ck = d->cu_seqlens_k;
    if (cq[0] != 0 || ck[0] != 0) return SP_ERR_INVALID_ARG;
    for (int s = 0; s < n; ++s)
      if (cq[s + 1] < cq[s] || ck[s + 1] < ck[s]) return SP_ERR_INVALID_ARG;
    if (cq[n] > d->T_q || ck[n] > d->T_k) return SP_ERR_INVALID_ARG;
    p.q_pad = cq[n];
    p.k_pad = ck[n];
    for (int s = 0; s < n; ++s) {
      Seg g{cq[s], cq[s + 1], ck[s], ck[s + 1], 0};
      int64_t pq = g.qa, pk = g.ka;  // default: positions restart at 0 per segment
      if (d->position_ids_q && g.qb > g.qa) {
        const int32_t* pos = d->position_ids_q;
        if (ramp_checks())
          for (int i = g.qa + 1; i < g.qb; ++i)
            if ((int64_t)pos[i] != (int64_t)pos[i - 1] + 1) return SP_ERR_INVALID_ARG;
        pq = (int64_t)g.qa - pos[g.qa];
      }
      if (d->position_ids_k && g.kb > g.ka) {
        const int32_t* pos = d->position_ids_k;
        if (ramp_checks())
          for (int i = g.ka + 1; i < g.kb; ++i)
            if ((int64_t)pos[i] != (int64_t)pos[i - 1] + 1) return SP_ERR_INVALID_ARG;
        pk = (int64_t)g.ka - pos[g.ka];
      }
      // key j visible from row i iff pos_k[j] <= pos_q[i]
      //   <=> j - pk <= i - pq  <=>  j <= i + (pk - pq)
      int64_t delta = pk - pq;
      if (delta > (int64_t(1) << 30) || delta < -(int64_t(1) << 30)) return SP_ERR_INVALID_ARG;
      g.delta = (int)delta;
      p.segs.push_back(g);
    }
  }
  p.segs_k = p.segs;
  if (single) return single_sequence_runs(d, p);
  return SP_OK;
}

struct Item {
  int v[kItemInts];
  int64_t cost;
};

// Launch order.  MI355X hands workgroup i of a launch to XCD i % 8, and an
// XCD hands its own workgroups, in order, to its four shader engines in
// turn, each to a free CU there; a workgroup whose shader engine has no free
// CU holds up the XCD's later ones even when other engines have free CUs.
// So the list is built per XCD:
//  (1) items sorted longest first (enumerated head by head; the sort keeps
//      that order among equal costs);
//  (2) with `grouped` (row items: forward, dQ), dealt to the XCDs in groups
//      of four consecutive items -- equal or near-equal costs, which the
//      XCD then runs one per shader engine, so its engines free CUs in
//      step -- eight groups a round, the rounds alternately forwards and
//      backwards over the XCDs so that no XCD always takes the round's
//      longest group; what is left after the last full round, and every
//      dK/dV item list (measured better that way), goes item by item in
//      list order;
//  (3) within each cost, the items an XCD was dealt are replaced by a
//      contiguous share of that cost's items, taken head by head, so each
//      XCD's L2 serves a few neighbouring heads (the costs per XCD stay);
//  (4) XCD x's items, longest first, fill the list positions that land on
//      XCD x.
// `n_front` items (zero fills) precede these in the launch and shift the
// position -> XCD map.
constexpr int kXcds = 8, kEngines = 4;

void sort_items(std::vector<Item>& items, std::vector<int32_t>& out, size_t n_front,
                bool grouped) {
  std::stable_sort(items.begin(), items.end(),
                   [](const Item& a, const Item& b) { return a.cost > b.cost; });
  const size_t N = items.size();
  auto xcd_of = [&](size_t p) { return (int)((n_front + p) % kXcds); };
  // (2) owner[i] = XCD of sorted item i
  std::vector<int> owner(N);
  constexpr size_t kRound = (size_t)kXcds * kEngines;
  const size_t full = grouped ? N / kRound * kRound : 0;
  for (size_t i = 0; i < full; ++i) {
    const size_t k = i % kRound / kEngines;      // group within the round
    const bool back = (i / kRound) & 1;
    owner[i] = xcd_of(back ? kXcds - 1 - k : k);
  }
  for (size_t i = full; i < N; ++i) owner[i] = xcd_of(i);
  // (3) contiguous per-XCD shares within each cost
  for (size_t s = 0; s < N;) {
    size_t e = s + 1;
    while (e < N && items[e].cost == items[s].cost) ++e;
    size_t n_x[kXcds] = {};
    for (size_t i = s; i < e; ++i) ++n_x[owner[i]];
    size_t i = s;
    for (int x = 0; x < kXcds; ++x)
      for (size_t j = 0; j < n_x[x]; ++j) owner[i++] = x;
    s = e;
  }
  // (4) per-XCD queues (longest first, as sorted) into their positions
  std::vector<std::vector<const Item*>> q(kXcds);
  for (size_t i = 0; i < N; ++i) q[owner[i]].push_back(&items[i]);
  size_t next[kXcds] = {};
  out.resize(N * kItemInts);
  for (size_t p = 0; p < N; ++p) {
    const int x = xcd_of(p);
    std::memcpy(&out[p * kItemInts], q[x][next[x]++]->v, sizeof(int) * kItemInts);
  }
}

// Row-tile items (forward, ring step, dQ).
void schedule_rows(const sp_attn_desc* d, const Problem& p, int BM, int BN, bool include_empty,
                   std::vector<int32_t>& out, size_t n_front) {
  std::vector<Item> items;
  for (int y = 0; y < p.n_real; ++y) {
    for (const Seg& g : p.segs) {
      // Causal row tiles end at the segment's end, so a partial tile is the
      // segment's first: its rows see the fewest keys.  (Aligned to the
      // start, the partial tile would be the last -- the segment's longest
      // item -- with most of its wavefronts idle.)
      const int len = g.qb - g.qa;
      const int first = d->causal && len % BM ? len % BM : BM;
      for (int a = g.qa, b = g.qa + std::min(first, len); a < g.qb;
           a = b, b = std::min(b + BM, g.qb)) {
        int k1 = g.kb;
        if (d->causal) k1 = (int)std::min<int64_t>(g.kb, (int64_t)b + g.delta);
        const int k0 = g.ka;
        const bool empty = k1 <= k0;
        if (empty && !include_empty) continue;
        Item it{{a, b, k0, empty ? k0 : k1, g.delta, y, p.kv_of[y], 0}, 0};
        it.cost = empty ? 0 : (int64_t)((k1 - (k0 & ~7)) + BN - 1) / BN;
        items.push_back(it);
      }
    }
    if (include_empty)
      for (int a = p.q_pad; a < d->T_q; a += BM)
        items.push_back(Item{{a, std::min(a + BM, d->T_q), 0, 0, 0, y, p.kv_of[y], 0}, 0});
  }
  sort_items(items, out, n_front, true);
}

// Key-tile items (dK / dV).  Every key of every real head gets exactly one item.
void schedule_keys(const sp_attn_desc* d, const Problem& p, int BNK, int BQ,
                   std::vector<int32_t>& out, size_t n_front) {
  std::vector<Item> items;
  for (int y = 0; y < p.n_real; ++y) {
    for (const Seg& g : p.segs_k) {
      for (int a = g.ka; a < g.kb; a += BNK) {
        const int b = std::min(a + BNK, g.kb);
        int q0 = g.qa;
        if (d->causal) q0 = (int)std::max<int64_t>(g.qa, (int64_t)a - g.delta);
        const bool empty = q0 >= g.qb;
        Item it{{a, b, empty ? g.qb : q0, g.qb, g.delta, y, p.kv_of[y], 1}, 0};
        it.cost = empty ? 0 : (int64_t)((g.qb - (q0 & ~7)) + BQ - 1) / BQ;
        items.push_back(it);
      }
    }
    for (int a = p.k_pad; a < d->T_k; a += BNK)
      items.push_back(Item{{a, std::min(a + BNK, d->T_k), 0, 0, 0, y, p.kv_of[y], 1}, 0});
  }
  sort_items(items, out, n_front, false);
}

// Zero fills as work items of the same launch (no extra kernels): dummy
// query slots (O = +0 and LSE = -inf, in the ring variant the accumulators'
// identity; dQ = +0) and, in the direct dK/dV mode, KV heads no real query
// head reads (dK = dV = +0).  One item covers kFillRows rows of one head;
// the items go to the FRONT of the list, so they finish in microseconds on
// a few CUs while the longest items start.
std::vector<int32_t> row_fills(const sp_attn_desc* d, const Problem& p) {
  std::vector<int32_t> out;
  for (int y = p.n_real; y < d->H_loc; ++y)
    for (int a = 0; a < d->T_q; a += spk::kFillRows) {
      const int32_t it[kItemInts] = {a, std::min(a + spk::kFillRows, d->T_q), 0, 0, 0, y, 0,
                                     spk::kItemFillQ};
      out.insert(out.end(), it, it + kItemInts);
    }
  return out;
}
bool kv_unread(const Problem& p, int kv) { return p.n_real == 0 || p.kv_hi[kv] == p.kv_lo[kv]; }
std::vector<int32_t> key_fills(const sp_attn_desc* d, const Problem& p) {
  std::vector<int32_t> out;
  if (!p.direct && p.n_real > 0) return out;  // the GQA reduction writes every KV head
  for (int kv = 0; kv < d->Hkv_loc; ++kv) {
    if (!kv_unread(p, kv)) continue;
    for (int a = 0; a < d->T_k; a += spk::kFillRows) {
      const int32_t it[kItemInts] = {a, std::min(a + spk::kFillRows, d->T_k), 0, 0, 0, 0, kv,
                                     spk::kItemFillKV};
      out.insert(out.end(), it, it + kItemInts);
    }
  }
  return out;
}
void prepend(std::vector<int32_t> fills, std::vector<int32_t>& items) {
  if (!fills.empty()) items.insert(items.begin(), fills.begin(), fills.end());
}
int n_unread_kv(const sp_attn_desc* d, const Problem& p) {
  if (!p.direct && p.n_real > 0) return 0;
  int n = 0;
  for (int kv = 0; kv < d->Hkv_loc; ++kv) n += kv_unread(p, kv);
  return n;
}

// Workspace layout.
struct Layout {
  size_t items_dq = 0, items_kv = 0, neg_d = 0, lse2 = 0, part_k = 0, part_v = 0, total = 0;
};

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

Layout layout_for(const sp_attn_desc* d, const Problem& p, int op, size_t n_items_a,
                  size_t n_items_b) {
  Layout L;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align256(off + bytes);
    return o;
  };
  const size_t D = p.D;
  if (op == SP_OP_FWD || op == SP_OP_RING_STEP) {
    L.items_dq = take(n_items_a * kItemInts * 4);
  } else {
    // the row statistics first: their offsets depend on T_q and the real
    // heads only, so calls over other KV chunks can reuse them
    // (SP_DESC_ROWSTATS_READY)
    L.neg_d = take((size_t)std::max(p.n_real, 1) * d->T_q * 4);
    L.lse2 = take((size_t)std::max(p.n_real, 1) * d->T_q * 4);
    L.items_dq = take(n_items_a * kItemInts * 4);
    L.items_kv = take(n_items_b * kItemInts * 4);
    if (!p.direct) {
      L.part_k = take((size_t)p.n_real * d->T_k * D * 4);
      L.part_v = take((size_t)p.n_real * d->T_k * D * 4);
    }
  }
  L.total = std::max<size_t>(off, 256);
  return L;
}

// Item counts of schedule_rows with empty items included (the worst case
// the workspace is sized for) and of schedule_keys, without building them.
// (With the zero-fill items appended at launch.)
size_t row_item_count(const sp_attn_desc* d, const Problem& p, int BM) {
  size_t per_head = 0;
  for (const Seg& g : p.segs) per_head += (size_t)((g.qb - g.qa) + BM - 1) / BM;
  per_head += (size_t)((d->T_q - p.q_pad) + BM - 1) / BM;
  const size_t fills =
      (size_t)(d->H_loc - p.n_real) * (size_t)((d->T_q + spk::kFillRows - 1) / spk::kFillRows);
  return per_head * (size_t)p.n_real + fills;
}
size_t key_item_count(const sp_attn_desc* d, const Problem& p, int BNK) {
  size_t per_head = 0;
  for (const Seg& g : p.segs_k) per_head += (size_t)((g.kb - g.ka) + BNK - 1) / BNK;
  per_head += (size_t)((d->T_k - p.k_pad) + BNK - 1) / BNK;
  const size_t fills =
      (size_t)n_unread_kv(d, p) * (size_t)((d->T_k + spk::kFillRows - 1) / spk::kFillRows);
  return per_head * (size_t)p.n_real + fills;
}

// Worst-case item counts (with empty items) for sizing.
void item_counts(const sp_attn_desc* d, const Problem& p, int op, size_t& a, size_t& b) {
  if (op == SP_OP_BWD) {
    a = row_item_count(d, p, spk::kDqBM);
    b = key_item_count(d, p, spk::kDkdvBN);
  } else {
    a = row_item_count(d, p, spk::kFwdBM);
    b = 0;
  }
}

inline bool aligned16(const void* ptr) { return ((uintptr_t)ptr & 15u) == 0; }

#define SP_HIP(call)                          \
  do {                                        \
    if ((call) != hipSuccess) return SP_ERR_HIP; \
  } while (0)

sp_status upload(void* dst, const std::vector<int32_t>& v, hipStream_t st) {
  if (v.empty()) return SP_OK;
  SP_HIP(hipMemcpyAsync(dst, v.data(), v.size() * sizeof(int32_t), hipMemcpyHostToDevice, st));
  return SP_OK;
}

// The attention entry points upload host-built work lists on every call,
// which a captured graph would replay from freed host memory: they refuse a
// stream that is being captured.
sp_status refuse_capture(hipStream_t st) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(st, &cs) != hipSuccess) return SP_ERR_HIP;
  return cs == hipStreamCaptureStatusNone ? SP_OK : SP_ERR_UNSUPPORTED;
}

sp_status check_ws(const Layout& L, void* ws, size_t ws_bytes) {
  if (!ws || ws_bytes < L.total || ((uintptr_t)ws & 255u) != 0) return SP_ERR_WORKSPACE;
  return SP_OK;
}

char* at(void* ws, size_t off) { return (char*)ws + off; }

}  // namespace

namespace spk {
KernelTimer& timer_for(int kernel_id) {
  static thread_local KernelTimer slots[kKCount];
  return slots[(kernel_id > 0 && kernel_id < kKCount) ? kernel_id : 0];
}
}  // namespace spk

extern "C" {

sp_status sp_profile_events(int32_t kernel_id, void* start_event, void* stop_event) {
  if (kernel_id < 1 || kernel_id >= spk::kKCount) return SP_ERR_INVALID_ARG;
  spk::KernelTimer& t = spk::timer_for(kernel_id);
  t.start = (hipEvent_t)start_event;
  t.stop = (hipEvent_t)stop_event;
  return SP_OK;
}

const char* sp_status_string(sp_status s) {
  switch (s) {
    case SP_OK: return "ok";
    case SP_ERR_INVALID_ARG: return "invalid argument";
    case SP_ERR_UNSUPPORTED: return "unsupported configuration";
    case SP_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case SP_ERR_HIP: return "HIP launch or copy failed";
  }
  return "unknown status";
}

int32_t sp_version(void) { return 100; }

sp_status sp_ulysses_pack(const void* src, int32_t T_loc, int32_t H_src, int32_t head_dim,
                          int32_t sp, int32_t H_dst_loc, const int32_t* head_map, void* dst,
                          void* stream) {
  if (T_loc < 0 || H_src < 1 || head_dim < 8 || head_dim % 8 != 0 || sp < 1 || H_dst_loc < 1 ||
      !head_map)
    return SP_ERR_INVALID_ARG;
  if ((int64_t)sp * H_dst_loc > spk::kMaxMap) return SP_ERR_UNSUPPORTED;
  spk::PackArgs a;
  a.sp = sp; a.T = T_loc; a.Hs = H_src; a.Hd = H_dst_loc; a.nch = head_dim / 8;
  for (int i = 0; i < sp * H_dst_loc; ++i) {
    if (head_map[i] < -1 || head_map[i] >= H_src) return SP_ERR_INVALID_ARG;
    a.map[i] = head_map[i];
  }
  if (T_loc == 0) return SP_OK;
  if (!src || !dst || !aligned16(src) || !aligned16(dst)) return SP_ERR_INVALID_ARG;
  SP_HIP(spk::launch_pack(src, dst, a, (hipStream_t)stream));
  return SP_OK;
}

sp_status sp_ulysses_unpack(const void* src, int32_t T_loc, int32_t H_src_loc, int32_t head_dim,
                            int32_t sp, const int32_t* head_map, int32_t H_dst, void* dst,
                            void* stream) {
  if (T_loc < 0 || H_src_loc < 1 || head_dim < 8 || head_dim % 8 != 0 || sp < 1 || H_dst < 1 ||
      !head_map)
    return SP_ERR_INVALID_ARG;
  if ((int64_t)sp * H_src_loc > spk::kMaxMap || H_dst > spk::kMaxMap) return SP_ERR_UNSUPPORTED;
  spk::PackArgs a;
  a.sp = sp; a.T = T_loc; a.Hs = H_src_loc; a.Hd = H_dst; a.nch = head_dim / 8;
  std::vector<int> seen(H_dst, 0);
  for (int i = 0; i < sp * H_src_loc; ++i) {
    int g = head_map[i];
    if (g < -1 || g >= H_dst) return SP_ERR_INVALID_ARG;
    if (g >= 0) {
      if (seen[g]++) return SP_ERR_INVALID_ARG;
      a.map[g] = i;  // inverse map: dest head -> j*H_src_loc + h
    }
  }
  for (int g = 0; g < H_dst; ++g)
    if (seen[g] != 1) return SP_ERR_INVALID_ARG;
  if (T_loc == 0) return SP_OK;
  if (!src || !dst || !aligned16(src) || !aligned16(dst)) return SP_ERR_INVALID_ARG;
  SP_HIP(spk::launch_unpack(src, dst, a, (hipStream_t)stream));
  return SP_OK;
}

sp_status sp_ulysses_unpack_add(const void* src, int32_t T_loc, int32_t H_src_loc,
                                int32_t head_dim, int32_t sp, const int32_t* head_map,
                                int32_t H_dst, void* dst, void* stream) {
  if (T_loc < 0 || H_src_loc < 1 || head_dim < 8 || head_dim % 8 != 0 || sp < 1 || H_dst < 1 ||
      !head_map)
    return SP_ERR_INVALID_ARG;
  if ((int64_t)sp * H_src_loc > spk::kMaxMap || H_dst > spk::kMaxAddDst) return SP_ERR_UNSUPPORTED;
  spk::PackAddArgs a;
  a.sp = sp; a.T = T_loc; a.Hs = H_src_loc; a.Hd = H_dst; a.nch = head_dim / 8;
  // counting sort of the slots by destination head keeps each head's slots
  // in ascending order
  std::vector<int> cnt(H_dst + 1, 0);
  const int n_slots = sp * H_src_loc;
  for (int i = 0; i < n_slots; ++i) {
    const int g = head_map[i];
    if (g < -1 || g >= H_dst) return SP_ERR_INVALID_ARG;
    if (g >= 0) ++cnt[g + 1];
  }
  for (int g = 0; g < H_dst; ++g) cnt[g + 1] += cnt[g];
  for (int g = 0; g <= H_dst; ++g) a.start[g] = (int16_t)cnt[g];
  std::vector<int> fill(cnt.begin(), cnt.end() - 1);
  for (int i = 0; i < n_slots; ++i)
    if (head_map[i] >= 0) a.slot[fill[head_map[i]]++] = (int16_t)i;
  if (T_loc == 0) return SP_OK;
  if (!src || !dst || !aligned16(src) || !aligned16(dst)) return SP_ERR_INVALID_ARG;
  SP_HIP(spk::launch_unpack_add(src, dst, a, (hipStream_t)stream));
  return SP_OK;
}

namespace {
// Shared validation of the loss calls: vocabulary, sequences (host copy),
// alignment.  Fills the kernel arguments.
sp_status loss_args(int32_t T, int32_t V, int32_t ignore_index, const int32_t* cu,
                    int32_t num_seqs, spk::LossArgs& a) {
  if (T < 0 || V < 8 || V % 8 != 0 || num_seqs < 0) return SP_ERR_INVALID_ARG;
  if (num_seqs > spk::kMaxLossSeqs) return SP_ERR_UNSUPPORTED;
  if (num_seqs > 0 && !cu) return SP_ERR_INVALID_ARG;
  a.T = T; a.V = V; a.ignore_index = ignore_index; a.n_seqs = num_seqs;
  a.cu[0] = num_seqs > 0 ? cu[0] : 0;
  if (a.cu[0] < 0) return SP_ERR_INVALID_ARG;
  for (int s = 0; s < num_seqs; ++s) {
    if (cu[s + 1] < cu[s]) return SP_ERR_INVALID_ARG;
    a.cu[s + 1] = cu[s + 1];
  }
  if (a.cu[num_seqs] > T) return SP_ERR_INVALID_ARG;
  return SP_OK;
}
}  // namespace

sp_status sp_token_logprob(const void* logits, const int32_t* labels, int32_t T, int32_t V,
                           int32_t ignore_index, const int32_t* cu_seqlens, int32_t num_seqs,
                           float* logp, float* lse, float* seq_sum, void* stream) {
  spk::LossArgs a;
  sp_status st = loss_args(T, V, ignore_index, cu_seqlens, num_seqs, a);
  if (st != SP_OK) return st;
  if (T > 0 && (!logits || !labels || !logp || !lse || !aligned16(logits)))
    return SP_ERR_INVALID_ARG;
  if (num_seqs > 0 && !seq_sum) return SP_ERR_INVALID_ARG;
  SP_HIP(spk::launch_token_logprob(a, logits, labels, logp, lse, seq_sum, (hipStream_t)stream));
  return SP_OK;
}

sp_status sp_token_logprob_bwd(const void* logits, const int32_t* labels, const float* lse,
                               int32_t T, int32_t V, int32_t ignore_index,
                               const int32_t* cu_seqlens, int32_t num_seqs,
                               const float* grad_seq, void* dlogits, void* stream) {
  spk::LossArgs a;
  sp_status st = loss_args(T, V, ignore_index, cu_seqlens, num_seqs, a);
  if (st != SP_OK) return st;
  if (T == 0) return SP_OK;
  if (!logits || !labels || !lse || !dlogits || !aligned16(logits) || !aligned16(dlogits) ||
      (num_seqs > 0 && !grad_seq))
    return SP_ERR_INVALID_ARG;
  SP_HIP(spk::launch_token_logprob_bwd(a, logits, labels, lse, grad_seq, dlogits,
                                       (hipStream_t)stream));
  return SP_OK;
}

sp_status sp_loss_reduce(const float* partial_sums, const float* ref_partial_sums, int32_t sp,
                         int32_t num_seqs, int32_t kind, float coef, float* loss, float* grad,
                         void* stream) {
  if (sp < 1 || num_seqs < 1 || (kind != SP_LOSS_SFT && kind != SP_LOSS_DPO) || !partial_sums ||
      !loss || !grad || !std::isfinite(coef))
    return SP_ERR_INVALID_ARG;
  if (kind == SP_LOSS_DPO && (num_seqs % 2 != 0 || !ref_partial_sums)) return SP_ERR_INVALID_ARG;
  if (num_seqs > 256 || sp > 4096) return SP_ERR_UNSUPPORTED;
  spk::LossReduceArgs a;
  a.sp = sp; a.n = num_seqs; a.kind = kind; a.coef = coef;
  SP_HIP(spk::launch_loss_reduce(a, partial_sums, ref_partial_sums, loss, grad,
                                 (hipStream_t)stream));
  return SP_OK;
}

sp_status sp_attn_workspace_size(const sp_attn_desc* desc, int32_t op, size_t* bytes) {
  if (!bytes) return SP_ERR_INVALID_ARG;
  if (op != SP_OP_FWD && op != SP_OP_BWD && op != SP_OP_RING_STEP) return SP_ERR_INVALID_ARG;
  Problem p;
  sp_status s = validate(desc, p);
  if (s != SP_OK) return s;
  size_t a = 0, b = 0;
  item_counts(desc, p, op, a, b);
  *bytes = layout_for(desc, p, op, a, b).total;
  return SP_OK;
}

sp_status sp_attn_schedule(const sp_attn_desc* desc, int32_t op, int32_t* items, int32_t capacity,
                           int32_t* n_items) {
  if (!n_items || capacity < 0) return SP_ERR_INVALID_ARG;
  Problem p;
  sp_status s = validate(desc, p);
  if (s != SP_OK) return s;
  std::vector<int32_t> v;
  // in launch order: the fill items that precede the listed ones there
  // shift the workgroup -> XCD map
  if (op == SP_OP_FWD || op == SP_OP_RING_STEP)
    schedule_rows(desc, p, spk::kFwdBM, spk::kFwdBN, true, v,
                  row_fills(desc, p).size() / kItemInts);
  else if (op == SP_OP_BWD)
    schedule_keys(desc, p, spk::kDkdvBN, spk::kDkdvBQ, v, key_fills(desc, p).size() / kItemInts);
  else
    return SP_ERR_INVALID_ARG;
  const int32_t n = (int32_t)(v.size() / kItemInts);
  *n_items = n;
  if (items) std::memcpy(items, v.data(), sizeof(int32_t) * kItemInts * std::min(n, capacity));
  return SP_OK;
}

}  // extern "C"

namespace {

// ---- Scratch of the allocation-free forward (sp_attn_fwd_static).  A
// file-scope device array: every GPU the library runs on holds its own copy
// at its own address until the process ends.  In host code `scratch` is a
// host-side stand-in, never a device address: the device copy's address is
// looked up once per device with hipGetSymbolAddress (that device current)
// and only that pointer is handed to kernels and copies.
__device__ __align__(256) unsigned char scratch[SP_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
std::atomic<void*> g_scratch_ptr[kMaxDevices];

// Device address of the current device's scratch (looked up on first use).
sp_status static_scratch(void** out) {
  int dev = -1;
  SP_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return SP_ERR_UNSUPPORTED;
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (!p) {
      if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return SP_ERR_HIP;
      g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return SP_OK;
}

// The stream must belong to the current device (the scratch looked up is
// that device's).
sp_status stream_on_current_device(hipStream_t st) {
  if (!st) return SP_OK;
  int cur = -1, sdev = -1;
  SP_HIP(hipGetDevice(&cur));
  SP_HIP(hipStreamGetDevice(st, &sdev));
  return sdev == cur ? SP_OK : SP_ERR_INVALID_ARG;
}

}  // namespace

extern "C" {

// Forward / ring step.  `static_ws`: the work list goes to the current
// device's static scratch instead of the caller's workspace (sp_attn_fwd_static).
static sp_status fwd_common(const sp_attn_desc* d, const void* q, const void* k, const void* v,
                            void* o, float* lse, float* o_acc, float* lse_acc, int init,
                            void* o_out, void* ws, size_t ws_bytes, void* stream, bool ring,
                            bool static_ws = false) {
  Problem p;
  sp_status s = validate(d, p);
  if (s != SP_OK) return s;
  // pointers are required for tensors that have elements: no query rows is a
  // no-op; no keys leaves every row with O = 0 and LSE = -inf
  if (d->T_q > 0 && !q) return SP_ERR_INVALID_ARG;
  if (d->T_k > 0 && (!k || !v)) return SP_ERR_INVALID_ARG;
  if (d->T_q > 0 && (ring ? (!o_acc || !lse_acc) : (!o || !lse))) return SP_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || (o && !aligned16(o)) ||
      (o_acc && !aligned16(o_acc)) || (o_out && !aligned16(o_out)))
    return SP_ERR_INVALID_ARG;
  if (init != 0 && init != 1) return SP_ERR_INVALID_ARG;
  if (d->T_q == 0) return SP_OK;
  const bool include_empty = !ring || init || o_out;
  std::vector<int32_t> items;
  const std::vector<int32_t> fills = include_empty ? row_fills(d, p) : std::vector<int32_t>();
  schedule_rows(d, p, spk::kFwdBM, spk::kFwdBN, include_empty, items, fills.size() / kItemInts);
  prepend(fills, items);
  const int n_items = (int)(items.size() / kItemInts);
  hipStream_t st = (hipStream_t)stream;
  void* items_dev = nullptr;
  if (static_ws) {
    if (items.size() * sizeof(int32_t) > SP_STATIC_SCRATCH_BYTES) return SP_ERR_UNSUPPORTED;
    if ((s = refuse_capture(st)) != SP_OK) return s;
    if ((s = stream_on_current_device(st)) != SP_OK) return s;
    if ((s = static_scratch(&items_dev)) != SP_OK) return s;
  } else {
    Layout L = layout_for(d, p, ring ? SP_OP_RING_STEP : SP_OP_FWD,
                          row_item_count(d, p, spk::kFwdBM), 0);
    if ((s = check_ws(L, ws, ws_bytes)) != SP_OK) return s;
    if ((s = refuse_capture(st)) != SP_OK) return s;
    items_dev = at(ws, L.items_dq);
  }
  if (n_items > 0) {
    if ((s = upload(items_dev, items, st)) != SP_OK) return s;
    spk::FwdArgs a{};
    a.q = (const uint16_t*)q;
    a.k = (const uint16_t*)k;
    a.v = (const uint16_t*)v;
    a.o = (uint16_t*)o;
    a.lse = lse;
    a.o_acc = o_acc;
    a.lse_acc = lse_acc;
    a.o_out = (uint16_t*)o_out;
    a.items = (const int32_t*)items_dev;
    a.T_q = d->T_q; a.T_k = d->T_k; a.H = d->H_loc; a.Hkv = d->Hkv_loc;
    a.scale_log2 = d->softmax_scale * 1.4426950408889634f;
    a.causal = d->causal;
    a.init = init;
    SP_HIP(spk::launch_attn_fwd(a, n_items, p.D, ring, st));
  }
  return SP_OK;
}

sp_status sp_attn_fwd(const sp_attn_desc* desc, const void* q, const void* k, const void* v,
                      void* o, float* lse, void* workspace, size_t workspace_bytes,
                      void* stream) {
  return fwd_common(desc, q, k, v, o, lse, nullptr, nullptr, 1, nullptr, workspace,
                    workspace_bytes, stream, false);
}

sp_status sp_attn_fwd_static(const sp_attn_desc* desc, const void* q, const void* k,
                             const void* v, void* o, float* lse, void* stream) {
  return fwd_common(desc, q, k, v, o, lse, nullptr, nullptr, 1, nullptr, nullptr, 0, stream,
                    false, true);
}

sp_status sp_ring_step(const sp_attn_desc* desc, const void* q, const void* k_chunk,
                       const void* v_chunk, float* o_acc, float* lse_acc, int32_t init,
                       void* o_out, void* workspace, size_t workspace_bytes, void* stream) {
  return fwd_common(desc, q, k_chunk, v_chunk, nullptr, nullptr, o_acc, lse_acc, init, o_out,
                    workspace, workspace_bytes, stream, true);
}

sp_status sp_attn_bwd(const sp_attn_desc* d, const void* q, const void* k, const void* v,
                      const void* o, const float* lse, const void* dout, void* dq,
                      float* dq_acc, void* dk, void* dv, void* ws, size_t ws_bytes,
                      void* stream) {
  Problem p;
  sp_status s = validate(d, p);
  if (s != SP_OK) return s;
  // pointers are required for tensors that have elements
  if (d->T_q > 0 && (!q || !o || !lse || !dout || (!dq && !dq_acc))) return SP_ERR_INVALID_ARG;
  if (d->T_k > 0 && (!k || !v || !dk || !dv)) return SP_ERR_INVALID_ARG;
  for (const void* ptr : {q, k, v, o, dout, (const void*)dk, (const void*)dv})
    if (!aligned16(ptr)) return SP_ERR_INVALID_ARG;
  if ((dq && !aligned16(dq)) || (dq_acc && !aligned16(dq_acc))) return SP_ERR_INVALID_ARG;
  if (d->T_q == 0) {  // no rows: the keys receive no gradient
    SP_HIP(spk::launch_zero_heads_bf16(dk, d->T_k, d->Hkv_loc, p.D, 0, d->Hkv_loc,
                                       (hipStream_t)stream));
    SP_HIP(spk::launch_zero_heads_bf16(dv, d->T_k, d->Hkv_loc, p.D, 0, d->Hkv_loc,
                                       (hipStream_t)stream));
    return SP_OK;
  }
  std::vector<int32_t> it_dq, it_kv;
  // a dq_acc's dummy slots stay untouched
  const std::vector<int32_t> fq = dq ? row_fills(d, p) : std::vector<int32_t>();
  const std::vector<int32_t> fkv = key_fills(d, p);
  schedule_rows(d, p, spk::kDqBM, spk::kDqBN, true, it_dq, fq.size() / kItemInts);
  prepend(fq, it_dq);
  schedule_keys(d, p, spk::kDkdvBN, spk::kDkdvBQ, it_kv, fkv.size() / kItemInts);
  prepend(fkv, it_kv);
  const size_t na = it_dq.size() / kItemInts, nb = it_kv.size() / kItemInts;
  Layout L = layout_for(d, p, SP_OP_BWD, na, nb);
  if ((s = check_ws(L, ws, ws_bytes)) != SP_OK) return s;
  hipStream_t st = (hipStream_t)stream;
  if ((s = refuse_capture(st)) != SP_OK) return s;
  const int D = p.D;
  {
    // both work lists in one copy (they are adjacent in the workspace): every
    // host-to-device copy sits between two kernels on the stream
    {
      const size_t gap = (L.items_kv - L.items_dq) / sizeof(int32_t);
      std::vector<int32_t> both(gap + it_kv.size(), 0);
      std::copy(it_dq.begin(), it_dq.end(), both.begin());
      std::copy(it_kv.begin(), it_kv.end(), both.begin() + gap);
      if ((s = upload(at(ws, L.items_dq), both, st)) != SP_OK) return s;
    }
    float* neg_d = (float*)at(ws, L.neg_d);
    float* lse2 = (float*)at(ws, L.lse2);
    if (p.n_real > 0 && !(d->flags & SP_DESC_ROWSTATS_READY))
      SP_HIP(spk::launch_rowdot(o, dout, lse, neg_d, lse2, d->T_q, d->H_loc, p.n_real, D, st));
    const float sl2 = d->softmax_scale * 1.4426950408889634f;
    spk::DqArgs a{};
    a.q = (const uint16_t*)q; a.k = (const uint16_t*)k; a.v = (const uint16_t*)v;
    a.dout = (const uint16_t*)dout;
    a.lse = lse; a.neg_d = neg_d; a.dq = (uint16_t*)dq; a.dq_acc = dq_acc;
    a.dq_init = dq_acc && (d->flags & SP_DESC_DQ_ACC_INIT) ? 1 : 0;
    a.items = (const int32_t*)at(ws, L.items_dq);
    a.T_q = d->T_q; a.T_k = d->T_k; a.H = d->H_loc; a.Hkv = d->Hkv_loc;
    a.scale_log2 = sl2; a.scale = d->softmax_scale; a.causal = d->causal;
    SP_HIP(spk::launch_attn_dq(a, (int)na, D, st));

    spk::DkdvArgs b{};
    b.q = (const uint16_t*)q;
    b.dout = (const uint16_t*)dout;
    b.lse2 = lse2; b.neg_d = neg_d; b.k = (const uint16_t*)k; b.v = (const uint16_t*)v;
    b.dk = (uint16_t*)dk; b.dv = (uint16_t*)dv;
    b.part_k = p.direct ? nullptr : (float*)at(ws, L.part_k);
    b.part_v = p.direct ? nullptr : (float*)at(ws, L.part_v);
    b.items = (const int32_t*)at(ws, L.items_kv);
    b.T_q = d->T_q; b.T_k = d->T_k; b.H = d->H_loc; b.Hkv = d->Hkv_loc;
    b.scale_log2 = sl2; b.scale = d->softmax_scale; b.causal = d->causal; b.direct = p.direct;
    SP_HIP(spk::launch_attn_dkdv(b, (int)nb, D, st));
    if (!p.direct && p.n_real > 0) {
      spk::ReduceArgs r{};
      r.T = d->T_k; r.Hkv = d->Hkv_loc; r.D = D;
      for (int kv = 0; kv < d->Hkv_loc; ++kv) {
        r.head_lo[kv] = p.kv_lo[kv];
        r.head_hi[kv] = p.kv_hi[kv];
      }
      SP_HIP(spk::launch_reduce_kv(b.part_k, b.part_v, dk, dv, r, st));
    }
  }
  return SP_OK;
}

sp_status sp_lse_merge(float* o_acc, float* lse_acc, const void* o_part, int32_t o_part_is_bf16,
                       const float* lse_part, int32_t T, int32_t H, int32_t head_dim,
                       void* o_out_bf16, void* stream) {
  if (T < 0 || H < 1 || head_dim < 8 || head_dim > 512 || (head_dim & (head_dim - 1)) != 0)
    return SP_ERR_INVALID_ARG;
  if (o_part_is_bf16 != 0 && o_part_is_bf16 != 1) return SP_ERR_INVALID_ARG;
  if (T == 0) return SP_OK;
  if (!o_acc || !lse_acc || !o_part || !lse_part) return SP_ERR_INVALID_ARG;
  if (!aligned16(o_acc) || !aligned16(o_part) || (o_out_bf16 && !aligned16(o_out_bf16)))
    return SP_ERR_INVALID_ARG;
  SP_HIP(spk::launch_merge(o_acc, lse_acc, o_part, o_part_is_bf16 != 0, lse_part, T, H, head_dim,
                           o_out_bf16, (hipStream_t)stream));
  return SP_OK;
}

sp_status sp_f32_to_bf16(const float* src, void* dst, int64_t n, void* stream) {
  if (n < 0) return SP_ERR_INVALID_ARG;
  if (n == 0) return SP_OK;
  if (!src || !dst || !aligned16(src) || !aligned16(dst)) return SP_ERR_INVALID_ARG;
  SP_HIP(spk::launch_f32_to_bf16(src, dst, n, (hipStream_t)stream));
  return SP_OK;
}

}  // extern "C"
