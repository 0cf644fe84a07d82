// Full-sequence beam search with max-symbols 1: the comparison search of Table 5
// ("beam search"), whose state space is the whole label sequence (footnote to
// Sec. 2.2) rather than the (context, graph state) tuples of the FSA-based search.
//
// A hypothesis is a distinct blank-free label sequence y with a score.  On frame t each
// hypothesis expands to blank (y kept) and to every label c (y + c), weighted by
// log P(label | last two labels of y, t) with no blank factor; equal sequences merge by
// max or by log-add (the two merge operations of Table 3); the N best candidates by
// (score desc, first candidate index asc) are kept, in that order, where candidate
// (i, c) has index i * V + c (blank c = 0).  Two candidates can only be equal as the
// blank of a hypothesis y_i and label last(y_i) of the hypothesis y_j = y_i minus its
// last label, so sequences are carried as 64-bit hashes (of y and of y without its last
// label) plus their length; equal hashes are taken as equal sequences.
//
// Frame schedule, two launches per frame: the joiner GEMM over the rows of every
// stream's distinct hypothesis contexts, then k_hyp_step (one workgroup per stream:
// merge, top-N selection, and the next frame's joiner rows).
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstdint>

#include "internal.h"

namespace tbs {
namespace {

constexpr int kHT = 256;
constexpr int kHypCache = 16;  // candidates per thread scored once into registers
constexpr unsigned long long kHashInit = 0x9e3779b97f4a7c15ull;  // hash of the empty sequence
constexpr unsigned long long kHashMul = 0x100000001b3ull;       // odd multiplier

__device__ __forceinline__ unsigned long long hash_push(unsigned long long h, int c) {
  return h * kHashMul + (unsigned long long)(unsigned)c;
}

__device__ __forceinline__ double neg_inf_d() { return -__builtin_inf(); }

// Joiner rows of frame t for stream b from the hypotheses in buffer buf: the distinct
// contexts, ascending, go to rows b * N + r (rowctx, hrow), and each row's input
// h = tanh(enc[b][t] + ReLU(P0[a] + P1[c])) for context (a, c), fp32 or bf16 (RNE).
// Every thread of the workgroup calls it.
__device__ void hyp_rows(const ModelDev& m, const HypDev& d, int b, int t, int buf, int* s_c,
                         int* s_rc, int* s_nd) {
  const int tid = threadIdx.x, N = d.N;
  const size_t o = (size_t)b * N;
  const int nh = d.nh[buf][b];
  if (tid < N) s_c[tid] = tid < nh ? d.ctx[buf][o + tid] : -1;
  __syncthreads();
  if (tid < N) {
    const int c = s_c[tid];
    int rank = 0, first = 1, nd = 0;
    for (int j = 0; j < nh; ++j) {
      const int cj = s_c[j];
      bool fj = true;  // j is the first hypothesis with context cj
      for (int i = 0; i < j; ++i) fj = fj && s_c[i] != cj;
      if (fj) {
        ++nd;
        if (cj < c) ++rank;
      }
      if (j < tid && cj == c) first = 0;
    }
    if (tid < nh) {
      d.hrow[o + tid] = rank;
      if (first) {
        d.rowctx[o + rank] = c;
        s_rc[rank] = c;
      }
    }
    if (tid >= nd) d.rowctx[o + tid] = -1;
    if (tid == 0) *s_nd = nd;
  }
  __syncthreads();
  const int nd = *s_nd, C = m.C, Kpad = m.Kpad, V = m.V;
  const float* e = d.enc + ((size_t)b * d.T + t) * C;
  for (int i = tid; i < nd * Kpad; i += blockDim.x) {
    const int r = i / Kpad, k = i - r * Kpad;
    const int c = s_rc[r], a = c / V, cc = c - a * V;
    const float x = k < C ? tanh_fast(e[k] + fmaxf(m.P0[(size_t)a * Kpad + k] +
                                                   m.P1[(size_t)cc * Kpad + k], 0.f))
                          : 0.f;
    const size_t q = (o + r) * Kpad + k;
    if (m.bf16)
      reinterpret_cast<uint16_t*>(d.h)[q] = f32_to_bf16_rne(x);
    else
      reinterpret_cast<float*>(d.h)[q] = x;
  }
}

// The empty hypothesis of every stream and its joiner row for frame 0.
__global__ __launch_bounds__(256) void k_hyp_init(ModelDev m, HypDev d) {
  __shared__ int s_c[kMaxHyps], s_rc[kMaxHyps], s_nd;
  const int b = blockIdx.x;
  const size_t o = (size_t)b * d.N;
  if (threadIdx.x == 0) {
    d.nh[0][b] = 1;
    d.hash[0][o] = kHashInit;
    d.phash[0][o] = 0;
    d.n[0][o] = 0;
    d.ctx[0][o] = 0;
    d.score[0][o] = 0.0;
  }
  __syncthreads();
  if (d.len[b] > 0) hyp_rows(m, d, b, 0, 0, s_c, s_rc, &s_nd);
}

// (score, first, slot) ordered by score desc, then first asc.
struct Cand {
  double score;
  int first;
  int slot;
};

__device__ __forceinline__ bool cand_before(const Cand& x, const Cand& y) {
  if (x.score != y.score) return x.score > y.score;
  return x.first < y.first;
}

__global__ __launch_bounds__(kHT) void k_hyp_step(ModelDev m, HypDev d, int t,
                                                  const float* __restrict__ logits,
                                                  const float2* __restrict__ stats, int* trace) {
  __shared__ double s_lse[kMaxHyps], s_sc[kMaxHyps], s_gs[kMaxHyps];
  __shared__ int s_gfirst[kMaxHyps], s_rpar[kMaxHyps], s_rlab[kMaxHyps], s_mj[kMaxHyps];
  __shared__ int s_last[kMaxHyps], s_row[kMaxHyps], s_n[kMaxHyps];
  __shared__ unsigned long long s_h[kMaxHyps];
  __shared__ Cand s_w[kHT / 64];
  __shared__ Cand s_win[kMaxHyps];
  __shared__ int s_hc[kMaxHyps], s_hrc[kMaxHyps], s_hnd;
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (t >= d.len[b]) return;
  const int N = d.N, V = m.V, Vpad = m.Vpad, nvt = m.Vpad / kJoinerBN;
  const int cur = t & 1, nx = cur ^ 1;
  const size_t o = (size_t)b * N;
  const int nh = d.nh[cur][b];
  // normaliser of each hypothesis's joiner row
  if (tid < nh) {
    const int row = d.hrow[o + tid];
    const float2* st = stats + (o + row) * nvt;
    float M = -INFINITY;
    for (int i = 0; i < nvt; ++i) M = fmaxf(M, st[i].x);
    float S = 0.f;
    for (int i = 0; i < nvt; ++i) S += st[i].y == 0.f ? 0.f : st[i].y * expf(st[i].x - M);
    s_lse[tid] = (double)M + log((double)S);
    s_sc[tid] = d.score[cur][o + tid];
    s_row[tid] = row;
    const int nn = d.n[cur][o + tid];
    s_last[tid] = nn > 0 ? d.ctx[cur][o + tid] % V : -1;
    s_n[tid] = nn;
    s_h[tid] = d.hash[cur][o + tid];
  }
  __syncthreads();
  auto logp = [&](int i, int c) {
    const float z = logits[(o + s_row[i]) * Vpad + c];
    return (double)(float)((double)z - s_lse[i]);
  };
  // blank of y_i merges with label last(y_i) of y_j when y_j is y_i minus that label
  if (tid < nh) {
    const int i = tid;
    const double a = s_sc[i] + logp(i, 0);
    double gs = a;
    int gfirst = i * V, rpar = i, rlab = 0, mj = -1;
    const int ni = s_n[i];
    if (ni > 0) {
      const unsigned long long ph = d.phash[cur][o + i];
      for (int j = 0; j < nh; ++j)
        if (s_h[j] == ph && s_n[j] == ni - 1) mj = j;
    }
    if (mj >= 0) {
      const int c = s_last[i];
      const double bs = s_sc[mj] + logp(mj, c);
      const double hi = fmax(a, bs), lo = fmin(a, bs);
      gs = d.merge_logadd ? hi + log1p(exp(lo - hi)) : hi;
      const int jidx = mj * V + c;
      if (jidx < gfirst) gfirst = jidx;
      if (bs > a || (bs == a && jidx < i * V)) {
        rpar = mj;
        rlab = c;
      }
    }
    s_gs[i] = gs;
    s_gfirst[i] = gfirst;
    s_rpar[i] = rpar;
    s_rlab[i] = rlab;
    s_mj[i] = mj;
  }
  __syncthreads();
  // top-N: rounds of a workgroup argmax over the candidates not taken yet.  Up to
  // kHypCache candidates per thread are scored once into registers (all their logit
  // loads in flight together); larger sets are rescored every round.
  const int total = nh * V;
  auto score_of = [&](int idx, Cand& x) {
    const int i = idx / V, c = idx - i * V;
    if (c == 0) {
      x = Cand{s_gs[i], s_gfirst[i], idx};
      return true;
    }
    bool merged = false;  // label c of y_i is the blank group of some y_k
    for (int k = 0; k < nh; ++k) merged = merged || (s_mj[k] == i && s_last[k] == c);
    if (merged) return false;
    x = Cand{s_sc[i] + logp(i, c), idx, idx};
    return true;
  };
  const bool cached = total <= kHypCache * kHT;
  double cs[kHypCache];
  int cf[kHypCache];
  if (cached) {
#pragma unroll
    for (int q = 0; q < kHypCache; ++q) {
      const int idx = tid + q * kHT;
      Cand x{neg_inf_d(), 0x7fffffff, idx};
      if (idx >= total || !score_of(idx, x)) x.score = neg_inf_d();
      cs[q] = x.score;
      cf[q] = x.first;
    }
  }
  int kept = 0;
  for (int r = 0; r < N; ++r) {
    Cand best{neg_inf_d(), 0x7fffffff, -1};
    if (cached) {
#pragma unroll
      for (int q = 0; q < kHypCache; ++q) {
        const Cand x{cs[q], cf[q], tid + q * kHT};
        if (x.score != neg_inf_d() && (best.slot < 0 || cand_before(x, best))) best = x;
      }
    } else {
      for (int idx = tid; idx < total; idx += kHT) {
        bool taken = false;
        for (int q = 0; q < r; ++q) taken = taken || s_win[q].slot == idx;
        Cand x;
        if (taken || !score_of(idx, x)) continue;
        if (x.score != neg_inf_d() && (best.slot < 0 || cand_before(x, best))) best = x;
      }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      Cand y;
      y.score = __shfl_xor(best.score, off, 64);
      y.first = __shfl_xor(best.first, off, 64);
      y.slot = __shfl_xor(best.slot, off, 64);
      if (y.slot >= 0 && (best.slot < 0 || cand_before(y, best))) best = y;
    }
    if (lane == 0) s_w[wave] = best;
    __syncthreads();
    if (tid == 0) {
      Cand w = s_w[0];
      for (int q = 1; q < kHT / 64; ++q)
        if (s_w[q].slot >= 0 && (w.slot < 0 || cand_before(s_w[q], w))) w = s_w[q];
      s_win[r] = w;
    }
    __syncthreads();
    const int ws = s_win[r].slot;
    if (ws < 0) break;  // uniform: no candidate left
    kept = r + 1;
    if (cached && ws % kHT == tid) {
#pragma unroll
      for (int q = 0; q < kHypCache; ++q)
        if (tid + q * kHT == ws) cs[q] = neg_inf_d();  // taken
    }
  }
  // the kept hypotheses, in rank order, and their back-pointers
  if (tid < kept) {
    const int k = tid, slot = s_win[k].slot;
    const int i = slot / V, c = slot - i * V;
    const size_t q = o + k, p = o + i;
    int par, lab;
    if (c == 0) {
      d.hash[nx][q] = d.hash[cur][p];
      d.phash[nx][q] = d.phash[cur][p];
      d.n[nx][q] = d.n[cur][p];
      d.ctx[nx][q] = d.ctx[cur][p];
      par = s_rpar[i];
      lab = s_rlab[i];
    } else {
      d.hash[nx][q] = hash_push(d.hash[cur][p], c);
      d.phash[nx][q] = d.hash[cur][p];
      d.n[nx][q] = d.n[cur][p] + 1;
      d.ctx[nx][q] = (d.ctx[cur][p] % V) * V + c;
      par = i;
      lab = c;
    }
    d.score[nx][q] = s_win[k].score;
    d.hist[((size_t)t * d.B + b) * N + k] = par << 16 | lab;
    if (trace) {
      int* tr = trace + (((size_t)(t + 1) * d.B + b) * N + k) * 2;
      tr[0] = par;
      tr[1] = lab;
    }
  }
  if (tid == 0) d.nh[nx][b] = kept;
  if (t + 1 < d.len[b]) {  // uniform: the next frame's joiner rows
    __syncthreads();  // the kept hypotheses (and their count) are written
    __threadfence_block();
    hyp_rows(m, d, b, t + 1, nx, s_hc, s_hrc, &s_hnd);
  }
}

// Result: the first hypothesis after the stream's last frame, traced back.
__global__ __launch_bounds__(64) void k_hyp_final(HypDev d, int* out_tokens, int* out_ntok,
                                                  double* out_scores) {
  __shared__ int s_n;
  const int b = blockIdx.x, lane = threadIdx.x, T = d.T, N = d.N;
  const int len = d.len[b];
  if (lane == 0) {
    const int buf = len & 1;
    out_scores[b] = d.score[buf][(size_t)b * N];
    // count the labels, then write them from the end
    int k = 0, n = 0;
    for (int f = len - 1; f >= 0; --f) {
      const int v = d.hist[((size_t)f * d.B + b) * N + k];
      if ((v & 0xffff) > 0) ++n;
      k = v >> 16;
    }
    k = 0;
    int w = n;
    for (int f = len - 1; f >= 0; --f) {
      const int v = d.hist[((size_t)f * d.B + b) * N + k];
      if ((v & 0xffff) > 0) out_tokens[(size_t)b * T + --w] = v & 0xffff;
      k = v >> 16;
    }
    out_ntok[b] = n;
    s_n = n;
  }
  __syncthreads();
  for (int f = s_n + lane; f < T; f += 64) out_tokens[(size_t)b * T + f] = -1;
}

}  // namespace

hipError_t launch_hyp_init(const ModelDev& m, const HypDev& d, hipStream_t st) {
  hipLaunchKernelGGL(k_hyp_init, dim3(d.B), dim3(256), 0, st, m, d);
  return hipGetLastError();
}

hipError_t launch_hyp_step(const ModelDev& m, const HypDev& d, int t, const float* logits,
                           const float2* stats, int* trace, hipStream_t st) {
  hipEvent_t ea, eb;
  if (take_launch_events(&ea, &eb))  // per-kernel profiling: events in the dispatch packet
    hipExtLaunchKernelGGL(k_hyp_step, dim3(d.B), dim3(kHT), 0, st, ea, eb, 0u, m, d, t, logits,
                          stats, trace);
  else
    hipLaunchKernelGGL(k_hyp_step, dim3(d.B), dim3(kHT), 0, st, m, d, t, logits, stats, trace);
  return hipGetLastError();
}

hipError_t launch_hyp_final(const HypDev& d, int* out_tokens, int* out_ntok, double* out_scores,
                            hipStream_t st) {
  hipLaunchKernelGGL(k_hyp_final, dim3(d.B), dim3(64), 0, st, d, out_tokens, out_ntok,
                     out_scores);
  return hipGetLastError();
}

}  // namespace tbs
