// SP-aware loss path on gfx950 (Sections 3.3 and 5.1): per-token label
// log-probabilities over one rank's token slice, their per-sequence sums,
// the SFT / DPO loss over the ranks' all-reduced sums with the upstream
// gradient a gradient-carrying all-reduce gives every rank, and the backward
// to the logits.  The logits passes are HBM-bound: each reads the [T, V]
// bf16 rows once with 16-byte loads (the backward also writes them once).
#include <math.h>

#include "dev_common.h"
#include "launch.h"

namespace spk {

namespace {

constexpr int kLB = 256;  // threads per row (four wavefronts)

SP_DEV void decode8(const u32x4& v, float* x) {
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    x[2 * k] = __uint_as_float(v[k] << 16);
    x[2 * k + 1] = __uint_as_float(v[k] & 0xffff0000u);
  }
}

// Combine two (max, sum of exp(x - max)) states, log2 domain for the sum.
SP_DEV void lse_combine(float& m, float& s, float m2, float s2) {
  const float mn = fmaxf(m, m2);
  if (mn == neg_inf()) return;
  s = s * __builtin_amdgcn_exp2f((m - mn) * kLog2e) + s2 * __builtin_amdgcn_exp2f((m2 - mn) * kLog2e);
  m = mn;
}

SP_DEV int seq_of(const LossArgs& a, int t) {
  // sequence s with cu[s] <= t < cu[s+1], or -1
  if (t < a.cu[0] || t >= a.cu[a.n_seqs]) return -1;
  int lo = 0, hi = a.n_seqs;  // cu[lo] <= t < cu[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (a.cu[mid] <= t) lo = mid; else hi = mid;
  }
  return lo;
}

// One workgroup per token row: online max / sum over the vocabulary, then
// lse and the label's log-probability.
__global__ __launch_bounds__(kLB) void token_logprob_kernel(LossArgs a, const u32x4* __restrict__ logits,
                                                            const int32_t* __restrict__ labels,
                                                            float* __restrict__ logp,
                                                            float* __restrict__ lse) {
  const int t = blockIdx.x;
  const int nch = a.V / 8;
  const u32x4* row = logits + (int64_t)t * nch;
  float m = neg_inf(), s = 0.f;
  int c = threadIdx.x;
  for (; c + 3 * kLB < nch; c += 4 * kLB) {  // four loads in flight
    u32x4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = ld_stream(&row[c + u * kLB]);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      float x[8];
      decode8(v[u], x);
      const float cm = fmaxf(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])),
                             fmaxf(fmaxf(x[4], x[5]), fmaxf(x[6], x[7])));
      const float mn = fmaxf(m, cm);
      const float b = mn * kLog2e;
      float acc = (m == neg_inf()) ? 0.f : s * __builtin_amdgcn_exp2f(m * kLog2e - b);
#pragma unroll
      for (int k = 0; k < 8; ++k) acc += __builtin_amdgcn_exp2f(__builtin_fmaf(x[k], kLog2e, -b));
      s = acc;
      m = mn;
    }
  }
  for (; c < nch; c += kLB) {
    float x[8];
    decode8(row[c], x);
    float cm = x[0];
#pragma unroll
    for (int k = 1; k < 8; ++k) cm = fmaxf(cm, x[k]);
    const float mn = fmaxf(m, cm);
    const float b = mn * kLog2e;
    float acc = (m == neg_inf()) ? 0.f : s * __builtin_amdgcn_exp2f(m * kLog2e - b);
#pragma unroll
    for (int k = 0; k < 8; ++k) acc += __builtin_amdgcn_exp2f(__builtin_fmaf(x[k], kLog2e, -b));
    s = acc;
    m = mn;
  }
  // wavefront reduction, then across the four wavefronts
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) lse_combine(m, s, __shfl_xor(m, off), __shfl_xor(s, off));
  __shared__ float sm[4], ss[4];
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    sm[w] = m;
    ss[w] = s;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float M = sm[0], S = ss[0];
    for (int i = 1; i < 4; ++i) lse_combine(M, S, sm[i], ss[i]);
    const float L = M + __log2f(S) * kLn2;
    lse[t] = L;
    const int lab = labels[t];
    float lp = 0.f;
    if (lab != a.ignore_index && lab >= 0 && lab < a.V && seq_of(a, t) >= 0) {
      const uint16_t* r16 = (const uint16_t*)row;
      lp = bf16_to_f32(r16[lab]) - L;
    }
    logp[t] = lp;
  }
}

// One workgroup per sequence: fixed-order sum of its tokens' log-probs.
__global__ __launch_bounds__(kLB) void seq_sum_kernel(LossArgs a, const float* __restrict__ logp,
                                                      float* __restrict__ seq_sum) {
  const int s = blockIdx.x;
  float acc = 0.f;
  for (int t = a.cu[s] + threadIdx.x; t < a.cu[s + 1]; t += kLB) acc += logp[t];
  __shared__ float red[kLB];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int h = kLB / 2; h >= 1; h >>= 1) {
    if (threadIdx.x < h) red[threadIdx.x] += red[threadIdx.x + h];
    __syncthreads();
  }
  if (threadIdx.x == 0) seq_sum[s] = red[0];
}

// dlogits[t, v] = g * (1[v == label] - exp(x - lse)), g = grad_seq[seq(t)].
__global__ __launch_bounds__(kLB) void token_logprob_bwd_kernel(LossArgs a, const u32x4* __restrict__ logits,
                                                                const int32_t* __restrict__ labels,
                                                                const float* __restrict__ lse,
                                                                const float* __restrict__ grad_seq,
                                                                u32x4* __restrict__ dlogits) {
  const int t = blockIdx.x;
  const int nch = a.V / 8;
  const int64_t base = (int64_t)t * nch;
  const int lab = labels[t];
  const int sq = seq_of(a, t);
  const bool live = sq >= 0 && lab != a.ignore_index && lab >= 0 && lab < a.V;
  if (!live) {
    for (int c = threadIdx.x; c < nch; c += kLB) dlogits[base + c] = u32x4{0u, 0u, 0u, 0u};
    return;
  }
  const float g = grad_seq[sq];
  const float b = lse[t] * kLog2e;
  const float ng = -g;
  for (int c = threadIdx.x; c < nch; c += kLB) {
    float x[8];
    decode8(ld_stream(&logits[base + c]), x);
    float d[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      d[k] = ng * __builtin_amdgcn_exp2f(__builtin_fmaf(x[k], kLog2e, -b));
      if (c * 8 + k == lab) d[k] += g;
    }
    st_stream(pack_bf16x8(d[0], d[1], d[2], d[3], d[4], d[5], d[6], d[7]), &dlogits[base + c]);
  }
}

// Loss over the ranks' partial sums [sp, n] and every rank's upstream
// gradient.  The all-reduce is a sum over ranks in ascending order; its
// gradient-carrying backward gives each rank sp times the local upstream.
__global__ __launch_bounds__(kLB) void loss_reduce_kernel(LossReduceArgs a, const float* __restrict__ ps,
                                                          const float* __restrict__ refs,
                                                          float* __restrict__ loss,
                                                          float* __restrict__ grad) {
  __shared__ float term[kLB];
  const int i = threadIdx.x;
  const int n = a.n;
  auto total = [&](const float* x, int j) {
    float acc = 0.f;
    for (int r = 0; r < a.sp; ++r) acc += x[r * n + j];
    return acc;
  };
  float local = 0.f, tm = 0.f;
  if (a.kind == 0) {  // SFT: loss = -coef * sum
    if (i < n) {
      local = -a.coef;
      tm = -a.coef * total(ps, i);
    }
  } else {  // DPO over pairs (2p chosen, 2p+1 rejected)
    const int P = n / 2;
    if (i < n) {
      const int p = i >> 1;
      const float pw = total(ps, 2 * p), pl = total(ps, 2 * p + 1);
      const float rw = total(refs, 2 * p), rl = total(refs, 2 * p + 1);
      const float z = a.coef * ((pw - rw) - (pl - rl));
      const float sig_neg = 1.f / (1.f + __expf(z));  // sigmoid(-z)
      local = ((i & 1) ? a.coef : -a.coef) * sig_neg / (float)P;
      if ((i & 1) == 0) tm = (fmaxf(-z, 0.f) + log1pf(__expf(-fabsf(z)))) / (float)P;
    }
  }
  if (i < n)
    for (int r = 0; r < a.sp; ++r) grad[r * n + i] = (float)a.sp * local;
  term[i] = tm;
  __syncthreads();
  if (i == 0) {
    float acc = 0.f;
    for (int j = 0; j < n; ++j) acc += term[j];
    loss[0] = acc;
  }
}

}  // namespace

hipError_t launch_token_logprob(const LossArgs& a, const void* logits, const int32_t* labels,
                                float* logp, float* lse, float* seq_sum, hipStream_t st) {
  if (a.T > 0) {
    hipError_t e = sp_launch(kKLogprob, token_logprob_kernel, dim3(a.T), dim3(kLB), st, a,
                             (const u32x4*)logits, labels, logp, lse);
    if (e != hipSuccess) return e;
  }
  if (a.n_seqs > 0 && seq_sum)
    return sp_launch(0, seq_sum_kernel, dim3(a.n_seqs), dim3(kLB), st, a, (const float*)logp,
                     seq_sum);
  return hipSuccess;
}

hipError_t launch_token_logprob_bwd(const LossArgs& a, const void* logits, const int32_t* labels,
                                    const float* lse, const float* grad_seq, void* dlogits,
                                    hipStream_t st) {
  if (a.T <= 0) return hipSuccess;
  return sp_launch(kKLogprobBwd, token_logprob_bwd_kernel, dim3(a.T), dim3(kLB), st, a,
                   (const u32x4*)logits, labels, lse, grad_seq, (u32x4*)dlogits);
}

hipError_t launch_loss_reduce(const LossReduceArgs& a, const float* ps, const float* refs,
                              float* loss, float* grad, hipStream_t st) {
  return sp_launch(0, loss_reduce_kernel, dim3(1), dim3(kLB), st, a, ps, refs, loss, grad);
}

}  // namespace spk
