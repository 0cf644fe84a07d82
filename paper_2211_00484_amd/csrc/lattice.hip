// Lattice output of the search and the n-best label-sequence search (Sec. 2.5 of
// "Fast and parallel decoding for transducer"): the search's output is an FSA whose
// states are the tuples that survived each frame; the label sequence with the highest
// probability is found by sampling paths from it, removing blanks, keeping the distinct
// sequences, and scoring each by its total probability in the lattice (the "LogAdd"
// merge of Tables 3 and 6).
//
// Lattice arcs of frame f: every expansion (blank, or a graph arc) from a survivor of
// frame f whose (state, context) survived frame f+1, whichever candidate won the
// max-merge; ordered by (destination, source, arc position) with blank first.  The
// arcs are built from the survivor trace, so the search kernels are unchanged: for a
// destination with context (x, c) and state s', its sources are the survivors whose
// context ends in x, through their arcs with label c into s' (and blank from the
// survivor with the same context and state).
//
// Kernels (one workgroup per (stream, frame) unless noted):
//   k_lat_frame<false>  count the arcs of each frame, list each frame's joiner contexts
//   k_lat_scan          exclusive scan of the counts (one workgroup)
//   k_lat_frame<true>   write the arcs and the per-destination offsets
//   joiner GEMM over the dense (stream, frame, context) rows, then k_lat_weights
//   k_lat_forward       forward log scores, final weights, totals (one workgroup per stream)
//   k_lat_sample        one thread per sampled path: backward sampling by inversion
//   k_lat_unique        distinct blank-free sequences in order of first occurrence
//   k_lat_seqscore      one workgroup per distinct sequence: composition with the lattice
//   k_lat_best          the best distinct sequence per stream
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "internal.h"

namespace tbs {
namespace {

constexpr int kLT = 256;  // threads per workgroup

__device__ __forceinline__ double neg_inf() { return -__builtin_inf(); }

// Exclusive prefix sum over a 256-thread workgroup; *total receives the sum.
__device__ int block_exclusive_scan(int v, int* s_w, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) s_w[wave] = x;
  __syncthreads();
  int base = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kLT / 64; ++w) {
    if (w < wave) base += s_w[w];
    tot += s_w[w];
  }
  __syncthreads();
  *total = tot;
  return base + x - v;
}

// Arcs from node (ci, si) of frame f into node (cj, sj) of frame f+1, in arc-position
// order with blank first; emit(label, graph arc or -1) for each.  Returns the count.
template <class F>
__device__ int pair_arcs(const GraphDev& g, int V, int ci, int si, int cj, int sj, F emit) {
  int n = 0;
  if (ci == cj && si == sj) {
    emit(0, -1);
    ++n;
  }
  const int x = cj / V, c = cj - x * V;
  if (c >= 1 && ci - (ci / V) * V == x) {
    if (g.trivial) {
      // one state; the arc at position c - 1 carries label c back to it
      if (sj == 0) {
        emit(c, c - 1);
        ++n;
      }
    } else {
      const int k1 = g.rp[si + 1];
      for (int k = g.rp[si]; k < k1; ++k)
        if (g.label[k] == c && g.dest[k] == sj) {
          emit(c, k);
          ++n;
        }
    }
  }
  return n;
}

struct FrameNodes {
  int c0[kMaxStates], s0[kMaxStates], c1[kMaxStates], s1[kMaxStates];
  int row[kMaxStates];  // joiner row (context rank) of each frame-f node
  int w[kLT / 64];
  int n0, n1;
};

// Loads the nodes of frames f and f+1 of stream b and ranks the frame-f contexts.
__device__ void load_frame_nodes(const LatticeDev& L, int b, int f, FrameNodes& s) {
  const int tid = threadIdx.x, Ns = L.Ns;
  const int* p0 = L.nodes + ((size_t)f * L.B + b) * Ns * 4;
  const int* p1 = L.nodes + ((size_t)(f + 1) * L.B + b) * Ns * 4;
  int c0 = -1, c1 = -1;
  if (tid < Ns) {
    c0 = p0[4 * tid];
    c1 = p1[4 * tid];
    s.c0[tid] = c0;
    s.s0[tid] = p0[4 * tid + 1];
    s.c1[tid] = c1;
    s.s1[tid] = p1[4 * tid + 1];
  }
  const int n0 = __syncthreads_count(c0 >= 0);
  const int n1 = __syncthreads_count(c1 >= 0);
  // survivors are stored from slot 0 in (ctx, state) order: rank the distinct contexts
  const int flag = tid < n0 && (tid == 0 || s.c0[tid - 1] != c0);
  int tot;
  const int pre = block_exclusive_scan(flag, s.w, &tot);
  if (tid < n0) s.row[tid] = pre + flag - 1;
  if (tid == 0) {
    s.n0 = n0;
    s.n1 = n1;
  }
  __syncthreads();
}

template <bool FILL>
__global__ __launch_bounds__(kLT) void k_lat_frame(LatticeDev L, GraphDev g0) {
  __shared__ FrameNodes s;
  __shared__ int s_red[kLT / 64];
  const int f = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const size_t fi = (size_t)b * L.T + f;
  if (f >= L.len[b]) {
    if (!FILL) {
      if (tid == 0) L.cnt[fi] = 0;
      for (int r = tid; r < L.Nc; r += kLT) L.rowctx[fi * L.Nc + r] = -1;
    }
    return;
  }
  const GraphDev g = L.graphs ? L.graphs[b] : g0;
  load_frame_nodes(L, b, f, s);
  const int n0 = s.n0, n1 = s.n1, V = L.V;
  if (!FILL) {
    // the frame's joiner rows: its distinct contexts in ascending order
    for (int r = tid; r < L.Nc; r += kLT) L.rowctx[fi * L.Nc + r] = -1;
    __syncthreads();
    // (the search keeps at most Nc contexts per stream)
    if (tid < n0 && (tid == 0 || s.c0[tid - 1] != s.c0[tid]) && s.row[tid] < L.Nc)
      L.rowctx[fi * L.Nc + s.row[tid]] = s.c0[tid];
  }
  const int P = n0 * n1;
  int acc = 0, base = 0;
  const long long o0 = FILL ? L.off[fi] : 0;
  int* dptr = L.dptr + fi * (L.Ns + 1);
  for (int q0 = 0; q0 < P; q0 += kLT) {
    const int q = q0 + tid;
    int j = 0, i = 0, c = 0;
    if (q < P) {
      j = q / n0;
      i = q - j * n0;
      c = pair_arcs(g, V, s.c0[i], s.s0[i], s.c1[j], s.s1[j], [](int, int) {});
    }
    if (!FILL) {
      acc += c;
    } else {
      int tot;
      const int pre = block_exclusive_scan(c, s_red, &tot);
      if (q < P) {
        if (i == 0) dptr[j] = base + pre;
        long long o = o0 + base + pre;
        int4* arcs = L.arcs;
        const int ii = i, jj = j;
        pair_arcs(g, V, s.c0[i], s.s0[i], s.c1[j], s.s1[j], [&](int lab, int k) {
          arcs[o] = make_int4(ii, jj, lab, k);
          ++o;
        });
      }
      base += tot;
    }
  }
  if (!FILL) {
    int tot;
    (void)block_exclusive_scan(acc, s_red, &tot);
    if (tid == 0) L.cnt[fi] = tot;
  } else {
    for (int j = n1 + tid; j <= L.Ns; j += kLT) dptr[j] = base;  // empty slots: no arcs
  }
}

// Exclusive scan of the B*T frame counts into 64-bit offsets (one workgroup).
__global__ __launch_bounds__(kLT) void k_lat_scan(const int* __restrict__ cnt,
                                                  long long* __restrict__ off, long long N) {
  __shared__ long long s_w[kLT / 64];
  __shared__ long long s_base;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0) s_base = 0;
  __syncthreads();
  for (long long i0 = 0; i0 < N; i0 += kLT) {
    const long long i = i0 + tid;
    const long long v = i < N ? cnt[i] : 0;
    long long x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const long long y = __shfl_up(x, o, 64);
      if (lane >= o) x += y;
    }
    if (lane == 63) s_w[wave] = x;
    __syncthreads();
    long long pre = s_base, tot = 0;
#pragma unroll
    for (int w = 0; w < kLT / 64; ++w) {
      if (w < wave) pre += s_w[w];
      tot += s_w[w];
    }
    if (i < N) off[i] = pre + x - v;
    __syncthreads();
    if (tid == 0) s_base += tot;
    __syncthreads();
  }
  if (tid == 0) off[N] = s_base;
}

// Arc weights of streams [b0, b0 + gridDim.y): q + log P(label | context, frame), the
// log-softmax taken from the joiner logits and per-tile (max, sum exp) statistics of
// the dense rows ((b - b0) * T + f) * Nc + r.
__global__ __launch_bounds__(kLT) void k_lat_weights(LatticeDev L, GraphDev g0,
                                                     const float* __restrict__ logits,
                                                     const float2* __restrict__ stats, int nvt,
                                                     int Vpad, int b0) {
  __shared__ FrameNodes s;
  __shared__ double s_lse[kMaxStates];
  const int f = blockIdx.x, b = b0 + blockIdx.y, tid = threadIdx.x;
  if (f >= L.len[b]) return;
  const GraphDev g = L.graphs ? L.graphs[b] : g0;
  load_frame_nodes(L, b, f, s);
  const size_t fi = (size_t)b * L.T + f;
  const size_t rbase = ((size_t)blockIdx.y * L.T + f) * L.Nc;
  if (tid < L.Nc) {
    const float2* st = stats + (rbase + tid) * nvt;
    float M = -INFINITY;
    for (int i = 0; i < nvt; ++i) M = fmaxf(M, st[i].x);
    float S = 0.f;
    for (int i = 0; i < nvt; ++i) S += st[i].y == 0.f ? 0.f : st[i].y * expf(st[i].x - M);
    s_lse[tid] = (double)M + log((double)S);
  }
  __syncthreads();
  const long long a0 = L.off[fi], a1 = L.off[fi + 1];
  for (long long a = a0 + tid; a < a1; a += kLT) {
    const int4 x = L.arcs[a];
    const int r = s.row[x.x];
    if (r >= L.Nc) continue;  // not reached: the search keeps at most Nc contexts
    const float z = logits[(rbase + r) * Vpad + x.z];
    const float lp = (float)((double)z - s_lse[r]);
    L.w[a] = x.w >= 0 ? g.q[x.w] + lp : lp;
  }
}

// Log of the sum of exp(alpha[src] + w) over the arcs [a0, a1).
__device__ double arcs_logsum(const LatticeDev& L, const double* alpha_f, long long a0,
                              long long a1) {
  double m = neg_inf();
  for (long long a = a0; a < a1; ++a) m = fmax(m, alpha_f[L.arcs[a].x] + (double)L.w[a]);
  if (m == neg_inf()) return m;
  double sum = 0.0;
  for (long long a = a0; a < a1; ++a) sum += exp(alpha_f[L.arcs[a].x] + (double)L.w[a] - m);
  return m + log(sum);
}

// Forward scores, final weights and totals; one workgroup per stream.
__global__ __launch_bounds__(kLT) void k_lat_forward(LatticeDev L, GraphDev g0) {
  const int b = blockIdx.x, tid = threadIdx.x, Ns = L.Ns, T = L.T;
  const int len = L.len[b];
  const GraphDev g = L.graphs ? L.graphs[b] : g0;
  double* al = L.alpha + (size_t)b * (T + 1) * Ns;
  if (tid < Ns) al[tid] = tid == 0 ? 0.0 : neg_inf();
  if (tid == 0) L.nn[(size_t)b * (T + 1)] = 1;
  __syncthreads();
  for (int f = 0; f < len; ++f) {
    const size_t fi = (size_t)b * T + f;
    const int* p1 = L.nodes + ((size_t)(f + 1) * L.B + b) * Ns * 4;
    const bool here = tid < Ns && p1[4 * tid] >= 0;
    const int n1 = __syncthreads_count(here);
    if (tid == 0) L.nn[(size_t)b * (T + 1) + f + 1] = n1;
    if (tid < Ns) {
      double v = neg_inf();
      if (here) {
        const int* dp = L.dptr + fi * (Ns + 1);
        const long long o = L.off[fi];
        v = arcs_logsum(L, al + (size_t)f * Ns, o + dp[tid], o + dp[tid + 1]);
      }
      al[(size_t)(f + 1) * Ns + tid] = v;
    }
    __syncthreads();
  }
  // final weights: the graph's, or 0 for every node if none of them is final
  const int* pl = L.nodes + ((size_t)len * L.B + b) * Ns * 4;
  const bool node = tid < Ns && pl[4 * tid] >= 0;
  const double fin = node ? (g.fin ? (double)g.fin[pl[4 * tid + 1]] : 0.0) : neg_inf();
  const int nfinal = __syncthreads_count(node && fin != neg_inf());
  if (tid < Ns) L.fw[(size_t)b * Ns + tid] = node ? (nfinal > 0 ? fin : 0.0) : neg_inf();
  __syncthreads();
  if (tid == 0) {
    const double* fw = L.fw + (size_t)b * Ns;
    const double* a = al + (size_t)len * Ns;
    double m = neg_inf();
    for (int j = 0; j < Ns; ++j) m = fmax(m, a[j] + fw[j]);
    double sum = 0.0;
    if (m != neg_inf())
      for (int j = 0; j < Ns; ++j) sum += a[j] + fw[j] == neg_inf() ? 0.0 : exp(a[j] + fw[j] - m);
    L.total[b] = m == neg_inf() ? m : m + log(sum);
    L.status[b] = nfinal > 0 ? 0 : 1;
  }
}

// Inversion pick among K items of log weight v(k): the first item whose running sum of
// exp(v - max) exceeds u times the full sum; if rounding leaves none, the last item
// with a nonzero share.
template <class F>
__device__ int pick_by_inversion(int K, double u, F v) {
  double m = neg_inf();
  for (int k = 0; k < K; ++k) m = fmax(m, v(k));
  double sum = 0.0;
  for (int k = 0; k < K; ++k) {
    const double x = v(k);
    sum += x == neg_inf() ? 0.0 : exp(x - m);
  }
  const double target = u * sum;
  double cum = 0.0;
  int last = -1;
  for (int k = 0; k < K; ++k) {
    const double x = v(k);
    if (x == neg_inf()) continue;
    cum += exp(x - m);
    last = k;
    if (cum > target) return k;
  }
  return last;
}

// One thread per (stream, path): the final node, then backwards the arc into the path's
// node of each frame, picked by inversion with the path's uniforms.
__global__ __launch_bounds__(64) void k_lat_sample(LatticeDev L, NBestDev N) {
  const int b = blockIdx.y, p = blockIdx.x * 64 + threadIdx.x;
  if (p >= N.n) return;
  const int Ns = L.Ns, T = L.T, len = L.len[b];
  const size_t pi = (size_t)b * N.n + p;
  const double* up = N.u + pi * (T + 1);
  int* pp = N.paths ? N.paths + pi * (T + 1) : nullptr;
  const double* al = L.alpha + (size_t)b * (T + 1) * Ns;
  const double* fw = L.fw + (size_t)b * Ns;
  const int nl = L.nn[(size_t)b * (T + 1) + len];
  int node = pick_by_inversion(nl, up[len],
                               [&](int j) { return al[(size_t)len * Ns + j] + fw[j]; });
  if (pp) {
    pp[len] = node;
    for (int f = len + 1; f <= T; ++f) pp[f] = -1;
  }
  int* seq = N.seq + pi * T;
  int nt = 0;
  for (int f = len - 1; f >= 0 && node >= 0; --f) {
    const size_t fi = (size_t)b * T + f;
    const int* dp = L.dptr + fi * (Ns + 1);
    const long long a0 = L.off[fi] + dp[node];
    const int K = dp[node + 1] - dp[node];
    const double* af = al + (size_t)f * Ns;
    const int k = pick_by_inversion(K, up[f], [&](int kk) {
      return af[L.arcs[a0 + kk].x] + (double)L.w[a0 + kk];
    });
    if (k < 0) break;  // no arc with a nonzero share (not reached: every node has one)
    const int4 x = L.arcs[a0 + k];
    if (pp) pp[f] = dp[node] + k;
    if (x.z > 0) seq[T - 1 - nt++] = x.z;  // labels arrive last first
    node = x.x;
  }
  // move the sequence to the front in forward order and hash it (FNV-1a, 64-bit)
  unsigned long long h = 1469598103934665603ull;
  for (int k = 0; k < nt; ++k) {
    const int y = seq[T - nt + k];
    seq[k] = y;
    h = (h ^ (unsigned)y) * 1099511628211ull;
  }
  N.ntok[pi] = nt;
  N.hash[pi] = h ^ (unsigned long long)nt;
}

// Distinct sequences of each stream, in order of first occurrence.
__global__ __launch_bounds__(kLT) void k_lat_unique(LatticeDev L, NBestDev N) {
  __shared__ int s_w[kLT / 64];
  const int b = blockIdx.x, tid = threadIdx.x, n = N.n, T = L.T;
  const size_t b0 = (size_t)b * n;
  int base = 0;
  for (int p0 = 0; p0 < n; p0 += kLT) {
    const int p = p0 + tid;
    int is_first = 0;
    if (p < n) {
      is_first = 1;
      const unsigned long long h = N.hash[b0 + p];
      const int nt = N.ntok[b0 + p];
      const int* sp = N.seq + (b0 + p) * T;
      for (int q = 0; q < p && is_first; ++q) {
        if (N.hash[b0 + q] != h || N.ntok[b0 + q] != nt) continue;
        const int* sq = N.seq + (b0 + q) * T;
        int k = 0;
        while (k < nt && sq[k] == sp[k]) ++k;
        if (k == nt) is_first = 0;
      }
    }
    int tot;
    const int pre = block_exclusive_scan(is_first, s_w, &tot);
    if (is_first) N.first[b0 + base + pre] = p;
    base += tot;
  }
  if (tid == 0) N.nuniq[b] = base;
}

// Total probability of each distinct sequence y: the lattice composed with the linear
// acceptor of y (blanks as epsilon), summed over paths.  State (node, k): k labels of y
// consumed; at frame f only k in [max(0, |y| - (len - f)), min(f, |y|)] can reach the
// end, and the DP keeps that band.  One workgroup per (stream, sequence), grid-strided.
__global__ __launch_bounds__(kLT) void k_lat_seqscore(LatticeDev L, NBestDev N) {
  extern __shared__ double dyn[];
  const int tid = threadIdx.x, Ns = L.Ns, T = L.T, n = N.n;
  const int W = N.dp_stride;  // band width capacity
  double* A0 = N.dp ? N.dp + (size_t)blockIdx.x * 2 * Ns * W : dyn;
  double* A1 = A0 + (size_t)Ns * W;
  for (long long item = blockIdx.x; item < (long long)L.B * n; item += gridDim.x) {
    const int b = (int)(item / n), u = (int)(item - (long long)b * n);
    if (u >= N.nuniq[b]) continue;  // uniform over the workgroup
    const int len = L.len[b];
    const size_t pi = (size_t)b * n + N.first[(size_t)b * n + u];
    const int Ly = N.ntok[pi];
    const int* y = N.seq + pi * T;
    double* cur = A0;
    double* nxt = A1;
    // frame 0: the initial node with nothing consumed (band [lo, hi] = [max(0, Ly - len), 0])
    int lo = Ly - len > 0 ? Ly - len : 0, hi = 0;
    if (tid == 0) cur[0] = lo == 0 ? 0.0 : neg_inf();
    __syncthreads();
    for (int f = 0; f < len; ++f) {
      const int lo1 = Ly - (len - f - 1) > 0 ? Ly - (len - f - 1) : 0;
      const int hi1 = f + 1 < Ly ? f + 1 : Ly;
      const int w1 = hi1 - lo1 + 1;
      const size_t fi = (size_t)b * T + f;
      const int* dp = L.dptr + fi * (Ns + 1);
      const long long o = L.off[fi];
      const int n1 = L.nn[(size_t)b * (T + 1) + f + 1];
      for (int q = tid; q < n1 * w1; q += kLT) {
        const int j = q / w1, k = lo1 + (q - j * w1);
        const long long a0 = o + dp[j], a1 = o + dp[j + 1];
        double m = neg_inf();
        for (int pass = 0; pass < 2; ++pass) {
          double sum = 0.0;
          for (long long a = a0; a < a1; ++a) {
            const int4 x = L.arcs[a];
            const int kk = x.z == 0 ? k : (k >= 1 && y[k - 1] == x.z ? k - 1 : -1);
            if (kk < lo || kk > hi) continue;
            const double v = cur[(size_t)x.x * W + (kk - lo)] + (double)L.w[a];
            if (pass == 0)
              m = fmax(m, v);
            else if (v != neg_inf())
              sum += exp(v - m);
          }
          if (pass == 0 && m == neg_inf()) break;
          if (pass == 1) m = m + log(sum);
        }
        nxt[(size_t)j * W + (k - lo1)] = m;
      }
      __syncthreads();
      double* t = cur;
      cur = nxt;
      nxt = t;
      lo = lo1;
      hi = hi1;
    }
    if (tid == 0) {
      // band at the last frame is [Ly, Ly]
      const double* fw = L.fw + (size_t)b * Ns;
      const int nl = L.nn[(size_t)b * (T + 1) + len];
      double m = neg_inf();
      for (int j = 0; j < nl; ++j) m = fmax(m, cur[(size_t)j * W] + fw[j]);
      double sum = 0.0;
      if (m != neg_inf())
        for (int j = 0; j < nl; ++j) {
          const double v = cur[(size_t)j * W] + fw[j];
          if (v != neg_inf()) sum += exp(v - m);
        }
      N.score[(size_t)b * n + u] = m == neg_inf() ? m : m + log(sum);
    }
    __syncthreads();
  }
}

// Best distinct sequence of each stream (first on ties) and the optional outputs.
__global__ __launch_bounds__(kLT) void k_lat_best(LatticeDev L, NBestDev N, int* out_tokens,
                                                  int* out_ntok, double* out_scores,
                                                  int* out_nuniq, double* out_uscores,
                                                  int* out_ufirst) {
  __shared__ int s_best;
  const int b = blockIdx.x, tid = threadIdx.x, n = N.n, T = L.T;
  const int nu = N.nuniq[b];
  const size_t b0 = (size_t)b * n;
  if (tid == 0) {
    int best = 0;
    for (int u = 1; u < nu; ++u)
      if (N.score[b0 + u] > N.score[b0 + best]) best = u;
    s_best = best;
    out_scores[b] = N.score[b0 + best];
    out_ntok[b] = N.ntok[b0 + N.first[b0 + best]];
    if (out_nuniq) out_nuniq[b] = nu;
  }
  __syncthreads();
  const size_t pi = b0 + N.first[b0 + s_best];
  const int nt = N.ntok[pi];
  for (int k = tid; k < T; k += kLT) out_tokens[(size_t)b * T + k] = k < nt ? N.seq[pi * T + k] : -1;
  for (int u = tid; u < n; u += kLT) {
    if (out_uscores) out_uscores[b0 + u] = u < nu ? N.score[b0 + u] : neg_inf();
    if (out_ufirst) out_ufirst[b0 + u] = u < nu ? N.first[b0 + u] : -1;
  }
}

}  // namespace

hipError_t launch_lattice_count(const LatticeDev& L, const GraphDev& g, hipStream_t st) {
  if (L.B == 0 || L.T == 0) return hipSuccess;
  hipLaunchKernelGGL(k_lat_frame<false>, dim3(L.T, L.B), dim3(kLT), 0, st, L, g);
  return hipGetLastError();
}

hipError_t launch_lattice_scan(const LatticeDev& L, hipStream_t st) {
  hipLaunchKernelGGL(k_lat_scan, dim3(1), dim3(kLT), 0, st, L.cnt, L.off,
                     (long long)L.B * L.T);
  return hipGetLastError();
}

hipError_t launch_lattice_fill(const LatticeDev& L, const GraphDev& g, hipStream_t st) {
  if (L.B == 0 || L.T == 0) return hipSuccess;
  hipLaunchKernelGGL(k_lat_frame<true>, dim3(L.T, L.B), dim3(kLT), 0, st, L, g);
  return hipGetLastError();
}

hipError_t launch_lattice_weights(const ModelDev& m, const LatticeDev& L, const GraphDev& g,
                                  const float* enc, int b0, int b1, void* h, float* logits,
                                  float2* stats, int ncu, hipStream_t st) {
  if (b1 <= b0 || L.T == 0) return hipSuccess;
  const long long row0 = (long long)b0 * L.T * L.Nc;
  const int R = (b1 - b0) * L.T * L.Nc;
  hipError_t e =
      launch_joiner_dense(m, enc, L.rowctx, row0, L.Nc, R, h, logits, stats, ncu, st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_lat_weights, dim3(L.T, b1 - b0), dim3(kLT), 0, st, L, g, logits, stats,
                     m.Vpad / kJoinerBN, m.Vpad, b0);
  return hipGetLastError();
}

hipError_t launch_lattice_forward(const LatticeDev& L, const GraphDev& g, hipStream_t st) {
  if (L.B == 0) return hipSuccess;
  hipLaunchKernelGGL(k_lat_forward, dim3(L.B), dim3(kLT), 0, st, L, g);
  return hipGetLastError();
}

hipError_t launch_nbest(const LatticeDev& L, const NBestDev& N, int* out_tokens, int* out_ntok,
                        double* out_scores, int* out_nuniq, double* out_uscores,
                        int* out_ufirst, int dp_grid, size_t dp_lds, hipStream_t st) {
  if (L.B == 0) return hipSuccess;
  hipLaunchKernelGGL(k_lat_sample, dim3((N.n + 63) / 64, L.B), dim3(64), 0, st, L, N);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_lat_unique, dim3(L.B), dim3(kLT), 0, st, L, N);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (dp_lds > 0) {
    e = hipFuncSetAttribute((const void*)k_lat_seqscore,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)dp_lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_lat_seqscore, dim3(dp_grid), dim3(kLT), dp_lds, st, L, N);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(k_lat_best, dim3(L.B), dim3(kLT), 0, st, L, N, out_tokens, out_ntok,
                     out_scores, out_nuniq, out_uscores, out_ufirst);
  return hipGetLastError();
}

}  // namespace tbs
