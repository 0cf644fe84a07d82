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
// The last three walk the frames from LDS stages of consecutive frames (stage_frames).
//   k_lat_sample        one thread per sampled path: backward sampling by inversion
//                       (one workgroup per stream)
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

// Workgroup barrier that orders LDS accesses only: global stores issued before it may
// still be in flight (they are read by later kernels only).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

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
      if (tid == 0 && f == 0) L.nn[(size_t)b * (L.T + 1)] = 1;  // the initial node
      for (int r = tid; r < L.Nc; r += kLT) L.rowctx[fi * L.Nc + r] = -1;
    }
    return;
  }
  const GraphDev g = L.graphs ? L.graphs[b] : g0;
  load_frame_nodes(L, b, f, s);
  const int n0 = s.n0, n1 = s.n1, V = L.V;
  if (!FILL) {
    if (tid == 0) {
      L.nn[(size_t)b * (L.T + 1) + f + 1] = n1;
      if (f == 0) L.nn[(size_t)b * (L.T + 1)] = n0;
    }
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

// ---------------------------------------------------------------------------
// Frame-chunk staging.  The kernels that walk a stream's frames in order (forward
// scores, path sampling, sequence scoring) first copy the arcs (source, label,
// weight), per-destination offsets, node counts and, if asked, forward scores of a run
// of consecutive frames into LDS with coalesced loads, then walk those frames from LDS:
// the walk's dependent loads hit LDS instead of global memory.  A single frame larger
// than the stage is read from global memory.

constexpr int kStageF = kLT;  // frames per stage at most (one candidate per thread)

template <int ACAP, int DCAP, int XCAP>
struct Stage {
  int src[ACAP];
  int lab[ACAP];
  float w[ACAP];
  int dp[DCAP];                     // [frames][Ns+1]
  double pc[XCAP > 0 ? ACAP : 1];   // arc shares (XCAP > 0)
  int fo[kStageF + 1];              // first arc of each frame, relative to a0
  int nn1[kStageF];                 // nodes of frame f+1
  long long a0;
  int lo, hi, staged;
};

struct FrameView {
  const int* dp;   // [Ns+1] offsets of each destination's arcs within the frame
  const int* src;  // arc k: src[k * stride], lab[k * stride]
  const int* lab;
  int stride;
  const float* w;
  const double* pc;  // arc shares of the destination's score (XCAP > 0 only)
  int n1;            // nodes of frame f+1
};

// Stages frames [lo, hi) of stream b: forward from f (lo = f, hi <= fend), or backward
// (hi = f, lo >= fend).  Every thread must call it; it begins and ends with a barrier.
template <int ACAP, int DCAP, int XCAP>
__device__ void stage_frames(const LatticeDev& L, Stage<ACAP, DCAP, XCAP>& s, int b, int f,
                             bool backward, int fend) {
  const int tid = threadIdx.x, Ns = L.Ns, T = L.T;
  const long long* off = L.off + (size_t)b * T;
  __syncthreads();  // the previous stage is no longer read
  // thread t tries t + 1 frames; the valid counts form a prefix 1..m
  const int nf = tid + 1;
  bool ok = backward ? f - nf >= fend : f + nf <= fend;
  if (ok) {
    const int lo = backward ? f - nf : f, hi = lo + nf;
    ok = off[hi] - off[lo] <= ACAP && nf * (Ns + 1) <= DCAP;
  }
  const int m = __syncthreads_count(ok);
  const int nfr = m > 0 ? m : 1;
  const int lo = backward ? f - nfr : f, hi = lo + nfr;
  if (tid == 0) {
    s.lo = lo;
    s.hi = hi;
    s.staged = m > 0;
    s.a0 = off[lo];
  }
  if (m > 0) {
    const long long a0 = off[lo];
    const int na = (int)(off[hi] - a0);
    for (int i = tid; i < na; i += kLT) {
      const int4 x = L.arcs[a0 + i];
      s.src[i] = x.x;
      s.lab[i] = x.z;
      s.w[i] = L.w[a0 + i];
      if (XCAP > 0) s.pc[i] = L.pc[a0 + i];
    }
    const int* dsrc = L.dptr + ((size_t)b * T + lo) * (Ns + 1);
    for (int i = tid; i < nfr * (Ns + 1); i += kLT) s.dp[i] = dsrc[i];
    for (int i = tid; i <= nfr; i += kLT) s.fo[i] = (int)(off[lo + i] - a0);
    for (int i = tid; i < nfr; i += kLT) s.nn1[i] = L.nn[(size_t)b * (T + 1) + lo + i + 1];
  }
  __syncthreads();
}

template <int ACAP, int DCAP, int XCAP>
__device__ FrameView frame_view(const LatticeDev& L, const Stage<ACAP, DCAP, XCAP>& s, int b,
                                int f) {
  const int Ns = L.Ns, T = L.T;
  FrameView v;
  if (s.staged) {
    const int i = f - s.lo, a = s.fo[i];
    v.dp = s.dp + i * (Ns + 1);
    v.src = s.src + a;
    v.lab = s.lab + a;
    v.stride = 1;
    v.w = s.w + a;
    v.pc = XCAP > 0 ? s.pc + a : nullptr;
    v.n1 = s.nn1[i];
  } else {
    const size_t fi = (size_t)b * T + f;
    const long long a = L.off[fi];
    v.dp = L.dptr + fi * (Ns + 1);
    v.src = reinterpret_cast<const int*>(L.arcs + a);
    v.lab = v.src + 2;
    v.stride = 4;
    v.w = L.w + a;
    v.pc = L.pc + a;
    v.n1 = L.nn[(size_t)b * (T + 1) + f + 1];
  }
  return v;
}

// Forward scores, final weights and totals; one workgroup per stream.
__global__ __launch_bounds__(kLT) void k_lat_forward(LatticeDev L, GraphDev g0) {
  __shared__ Stage<1024, 1024, 0> s;
  __shared__ double s_al[2][kMaxStates];
  const int b = blockIdx.x, tid = threadIdx.x, Ns = L.Ns, T = L.T;
  const int len = L.len[b];
  const GraphDev g = L.graphs ? L.graphs[b] : g0;
  double* al = L.alpha + (size_t)b * (T + 1) * Ns;
  if (tid < Ns) {
    const double v = tid == 0 ? 0.0 : neg_inf();
    s_al[0][tid] = v;
    al[tid] = v;
  }
  int cur = 0;
  for (int f0 = 0; f0 < len; f0 = s.hi) {
    stage_frames(L, s, b, f0, false, len);
    for (int f = s.lo; f < s.hi; ++f) {
      const FrameView v = frame_view(L, s, b, f);
      if (tid < Ns) {
        double x = neg_inf();
        if (tid < v.n1) {
          const int k0 = v.dp[tid], k1 = v.dp[tid + 1];
          // each arc's share of the destination's score (sampling, sequence scores)
          double* pc = L.pc + s.a0 + (s.staged ? s.fo[f - s.lo] : L.off[(size_t)b * T + f] - s.a0);
          if (k1 - k0 <= 8) {
            // few arcs: their terms stay in registers, one exp each
            double e[8];
#pragma unroll
            for (int i = 0; i < 8; ++i)
              e[i] = k0 + i < k1 ? s_al[cur][v.src[(k0 + i) * v.stride]] + (double)v.w[k0 + i]
                                 : neg_inf();
#pragma unroll
            for (int i = 0; i < 8; ++i) x = fmax(x, e[i]);
            if (x != neg_inf()) {
              // the terms relative to the largest, in fp32 (relative error ~1e-7 per
              // frame); the scores accumulate in fp64
              float ef[8], sum = 0.f;
#pragma unroll
              for (int i = 0; i < 8; ++i) {
                ef[i] = e[i] == neg_inf() ? 0.f : __expf((float)(e[i] - x));
                sum += ef[i];
              }
              x += (double)__logf(sum);
              const float inv = 1.f / sum;
#pragma unroll
              for (int i = 0; i < 8; ++i)
                if (k0 + i < k1) pc[k0 + i] = (double)(ef[i] * inv);
            }
          } else {
            for (int k = k0; k < k1; ++k)
              x = fmax(x, s_al[cur][v.src[k * v.stride]] + (double)v.w[k]);
            if (x != neg_inf()) {
              double sum = 0.0;
              for (int k = k0; k < k1; ++k)
                sum += exp(s_al[cur][v.src[k * v.stride]] + (double)v.w[k] - x);
              x += log(sum);
              for (int k = k0; k < k1; ++k)
                pc[k] = exp(s_al[cur][v.src[k * v.stride]] + (double)v.w[k] - x);
            }
          }
        }
        s_al[cur ^ 1][tid] = x;
        al[(size_t)(f + 1) * Ns + tid] = x;
      }
      lds_barrier();  // the next frame reads s_al only
      cur ^= 1;
    }
  }
  // frames after the stream's end hold no nodes
  for (size_t i = (size_t)(len + 1) * Ns + tid; i < (size_t)(T + 1) * Ns; i += kLT) al[i] = neg_inf();
  // final weights: the graph's, or 0 for every node if none of them is final
  const int nl = L.nn[(size_t)b * (T + 1) + len];
  const int* pl = L.nodes + ((size_t)len * L.B + b) * Ns * 4;
  const bool node = tid < nl;
  const double fin = node ? (g.fin ? (double)g.fin[pl[4 * tid + 1]] : 0.0) : neg_inf();
  const int nfinal = __syncthreads_count(node && fin != neg_inf());
  if (tid < Ns) L.fw[(size_t)b * Ns + tid] = node ? (nfinal > 0 ? fin : 0.0) : neg_inf();
  __syncthreads();
  if (tid == 0) {
    const double* fw = L.fw + (size_t)b * Ns;
    double m = neg_inf();
    for (int j = 0; j < nl; ++j) m = fmax(m, s_al[cur][j] + fw[j]);
    double sum = 0.0;
    if (m != neg_inf())
      for (int j = 0; j < nl; ++j) {
        const double x = s_al[cur][j] + fw[j];
        if (x != neg_inf()) sum += exp(x - m);
      }
    L.total[b] = m == neg_inf() ? m : m + log(sum);
    L.status[b] = nfinal > 0 ? 0 : 1;
  }
}

// Inversion pick among K items with nonnegative shares p(k): the first item whose
// running sum exceeds u times the full sum; if rounding leaves none, the last item
// with a nonzero share.
template <class F>
__device__ int pick_by_share(int K, double u, F p) {
  double sum = 0.0;
  for (int k = 0; k < K; ++k) sum += p(k);
  const double target = u * sum;
  double cum = 0.0;
  int last = -1;
  for (int k = 0; k < K; ++k) {
    const double x = p(k);
    if (x == 0.0) continue;
    cum += x;
    last = k;
    if (cum > target) return k;
  }
  return last;
}

// The same with log weights v(k): shares exp(v - max v).
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

// One thread per path, kLT paths per workgroup (grid: path groups x streams): the final
// node, then backwards the arc into the path's node of each frame, picked by inversion
// with the path's uniforms (arc shares from the forward pass); the paths of a
// workgroup walk the staged frames together.
__global__ __launch_bounds__(kLT) void k_lat_sample(LatticeDev L, NBestDev N) {
  __shared__ Stage<2048, 1024, 1> s;
  const int b = blockIdx.y, tid = threadIdx.x;
  const int Ns = L.Ns, T = L.T, len = L.len[b], n = N.n;
  const double* al = L.alpha + (size_t)b * (T + 1) * Ns;
  const double* fw = L.fw + (size_t)b * Ns;
  const int nl = L.nn[(size_t)b * (T + 1) + len];
  {
    const int p = blockIdx.x * kLT + tid;
    const bool act = p < n;
    const size_t pi = (size_t)b * n + (act ? p : 0);
    const double* up = N.u + pi * (T + 1);
    int* pp = act && N.paths ? N.paths + pi * (T + 1) : nullptr;
    int* seq = N.seq + pi * T;
    int node = -1, nt = 0;
    if (act) {
      node = pick_by_inversion(nl, up[len],
                               [&](int j) { return al[(size_t)len * Ns + j] + fw[j]; });
      if (pp) {
        pp[len] = node;
        for (int f = len + 1; f <= T; ++f) pp[f] = -1;
      }
    }
    // the uniforms of the next four frames are loaded ahead of their use
    double q0 = 0.0, q1 = 0.0, q2 = 0.0, q3 = 0.0;
    if (act) {
      if (len - 1 >= 0) q0 = up[len - 1];
      if (len - 2 >= 0) q1 = up[len - 2];
      if (len - 3 >= 0) q2 = up[len - 3];
      if (len - 4 >= 0) q3 = up[len - 4];
    }
    for (int f1 = len; f1 > 0; f1 = s.lo) {
      stage_frames(L, s, b, f1, true, 0);
      for (int f = s.hi - 1; f >= s.lo; --f) {
        const double uf = q0;
        q0 = q1;
        q1 = q2;
        q2 = q3;
        q3 = act && f - 4 >= 0 ? up[f - 4] : 0.0;
        if (!act || node < 0) continue;
        const FrameView v = frame_view(L, s, b, f);
        const int a0 = v.dp[node], K = v.dp[node + 1] - a0;
        const int k = pick_by_share(K, uf, [&](int kk) { return v.pc[a0 + kk]; });
        if (k < 0) {  // no arc with a nonzero share (not reached: every node has one)
          node = -1;
          continue;
        }
        if (pp) pp[f] = a0 + k;
        const int lab = v.lab[(a0 + k) * v.stride];
        if (lab > 0) seq[T - 1 - nt++] = lab;  // labels arrive last first
        node = v.src[(a0 + k) * v.stride];
      }
    }
    if (act) {
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
  }
}

// Distinct sequences of each stream, in order of first occurrence.
constexpr int kUniqStage = 2048;

__global__ __launch_bounds__(kLT) void k_lat_unique(LatticeDev L, NBestDev N) {
  __shared__ int s_w[kLT / 64];
  __shared__ unsigned long long s_h[kUniqStage];
  __shared__ int s_n[kUniqStage];
  const int b = blockIdx.x, tid = threadIdx.x, n = N.n, T = L.T;
  const size_t b0 = (size_t)b * n;
  const bool staged = n <= kUniqStage;
  if (staged)
    for (int p = tid; p < n; p += kLT) {
      s_h[p] = N.hash[b0 + p];
      s_n[p] = N.ntok[b0 + p];
    }
  __syncthreads();
  const unsigned long long* hh = staged ? s_h : N.hash + b0;
  const int* nn = staged ? s_n : N.ntok + b0;
  int base = 0;
  for (int p0 = 0; p0 < n; p0 += kLT) {
    const int p = p0 + tid;
    int is_first = 0;
    if (p < n) {
      is_first = 1;
      const unsigned long long h = hh[p];
      const int nt = nn[p];
      const int* sp = N.seq + (b0 + p) * T;
      for (int q = 0; q < p && is_first; ++q) {
        if (hh[q] != h || nn[q] != nt) continue;
        const int* sq = N.seq + (b0 + q) * T;
        // compare 16 labels per step (independent loads in flight together)
        bool eq = true;
        int k = 0;
        for (; eq && k + 16 <= nt; k += 16) {
          int x[16], y[16];
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            x[i] = sq[k + i];
            y[i] = sp[k + i];
          }
#pragma unroll
          for (int i = 0; i < 16; ++i) eq = eq && x[i] == y[i];
        }
        for (; eq && k < nt; ++k) eq = sq[k] == sp[k];
        if (eq) is_first = 0;
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
// end, and the DP keeps that band.  The DP runs on ratios to the forward scores,
// R_f(j, k) = A_f(j, k) / exp(alpha_f(j)) in [0, 1], so that one frame is
// R_{f+1}(j, k) = sum over arcs a into j of R_f(src, k') * share(a), with the arc
// shares of the forward pass (no exp or log per arc); each frame is rescaled by its
// largest ratio, whose log is accumulated.  One wave per sequence; the four waves of a
// workgroup take four sequences of one stream and walk its staged frames together
// (grid: sequence groups x streams, grid-strided over the groups).
constexpr int kYStage = 512;
constexpr int kSeqWaves = kLT / 64;

__device__ __forceinline__ double wave_max_f64(double x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fmax(x, __shfl_xor(x, o, 64));
  return x;
}

// DP buffers: per wave kSeqLds doubles of LDS (small enough for three workgroups per
// compute unit), used when the sequence's band fits
// (2 * Ns * band width); otherwise the wave's slice of the global scratch.
constexpr int kSeqLds = 768;

__global__ __launch_bounds__(kLT) void k_lat_seqscore(LatticeDev L, NBestDev N) {
  __shared__ Stage<512, 512, 1> s;
  __shared__ int s_y[kSeqWaves][kYStage];
  __shared__ double s_dp[kSeqWaves][kSeqLds];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int Ns = L.Ns, T = L.T, n = N.n, b = blockIdx.y;
  const size_t blk = (size_t)blockIdx.y * gridDim.x + blockIdx.x;
  double* gdp = N.dp ? N.dp + (blk * kSeqWaves + wv) * 2 * (size_t)Ns * N.dp_stride : nullptr;
  const int len = L.len[b], nu = N.nuniq[b];
  const double* fw = L.fw + (size_t)b * Ns;
  const double* al_len = L.alpha + ((size_t)b * (T + 1) + len) * Ns;
  const int nl = L.nn[(size_t)b * (T + 1) + len];
  // the stream's largest node count sizes the DP buffers (usually far below Ns)
  int nmax = 1;
  for (int f = lane; f <= len; f += 64) nmax = max(nmax, L.nn[(size_t)b * (T + 1) + f]);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) nmax = max(nmax, __shfl_xor(nmax, o, 64));
  for (int u0 = blockIdx.x * kSeqWaves; u0 < nu; u0 += gridDim.x * kSeqWaves) {
    const int u = u0 + wv;
    const bool act = u < nu;
    int Ly = 0;
    const int* y = s_y[wv];
    // band width of this sequence: min(|y|, len - |y|) + 1
    int W = 1;
    bool in_lds = true;
    double* A0 = s_dp[wv];
    if (act) {
      const size_t pi = (size_t)b * n + N.first[(size_t)b * n + u];
      Ly = N.ntok[pi];
      const int* yg = N.seq + pi * T;
      if (Ly <= kYStage)
        for (int k = lane; k < Ly; k += 64) s_y[wv][k] = yg[k];
      else
        y = yg;
      W = (Ly < len - Ly ? Ly : len - Ly) + 1;
      in_lds = 2 * nmax * W <= kSeqLds;
      if (!in_lds) A0 = gdp;  // the host allots it whenever a band may not fit
      if (lane == 0) A0[0] = 1.0;  // frame 0: the initial node, nothing consumed
    }
    double* cur = A0;
    double* nxt = A0 + (size_t)nmax * W;
    double logscale = 0.0;
    int lo = 0, hi = 0;
    for (int f0 = 0; f0 < len; f0 = s.hi) {
      stage_frames(L, s, b, f0, false, len);  // also orders the writes above
      for (int f = s.lo; f < s.hi; ++f) {
        if (act) {
          const int lo1 = Ly - (len - f - 1) > 0 ? Ly - (len - f - 1) : 0;
          const int hi1 = f + 1 < Ly ? f + 1 : Ly;
          const int w1 = hi1 - lo1 + 1;
          const FrameView v = frame_view(L, s, b, f);
          double mx = 0.0;
          for (int q = lane; q < v.n1 * w1; q += 64) {
            const int j = q / w1, k = lo1 + (q - j * w1);
            const int a0 = v.dp[j], a1 = v.dp[j + 1];
            const int yk = k >= 1 ? y[k - 1] : -1;
            double r = 0.0;
            if (a1 - a0 <= 8) {
              // few arcs: all their loads in flight together
              int sr[8], lb[8];
              double pcv[8];
#pragma unroll
              for (int i = 0; i < 8; ++i) {
                const bool in = a0 + i < a1;
                sr[i] = in ? v.src[(a0 + i) * v.stride] : 0;
                lb[i] = in ? v.lab[(a0 + i) * v.stride] : -2;
                pcv[i] = in ? v.pc[a0 + i] : 0.0;
              }
#pragma unroll
              for (int i = 0; i < 8; ++i) {
                const int kk = lb[i] == 0 ? k : (lb[i] == yk ? k - 1 : -1);
                if (kk >= lo && kk <= hi) r += cur[(size_t)sr[i] * W + (kk - lo)] * pcv[i];
              }
            } else {
              for (int a = a0; a < a1; ++a) {
                const int lab = v.lab[a * v.stride];
                const int kk = lab == 0 ? k : (lab == yk ? k - 1 : -1);
                if (kk < lo || kk > hi) continue;
                r += cur[(size_t)v.src[a * v.stride] * W + (kk - lo)] * v.pc[a];
              }
            }
            nxt[(size_t)j * W + (k - lo1)] = r;
            mx = fmax(mx, r);
          }
          // every 8 frames, rescale by the largest ratio (no underflow on long streams)
          if ((f & 7) == 7) {
            mx = wave_max_f64(mx);
            if (mx > 0.0) {
              const double inv = 1.0 / mx;
              for (int q = lane; q < v.n1 * w1; q += 64) {
                const int j = q / w1, k = lo1 + (q - j * w1);
                nxt[(size_t)j * W + (k - lo1)] *= inv;
              }
              logscale += log(mx);
            }
          }
          lo = lo1;
          hi = hi1;
          double* t = cur;
          cur = nxt;
          nxt = t;
        }
        // the wave's next frame reads what its lanes wrote for this one: a wave's
        // memory operations are performed in order, so a wavefront-scope fence
        // (ordering only) suffices, for LDS and global buffers alike
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        __builtin_amdgcn_wave_barrier();
      }
    }
    if (act && lane == 0) {
      // band at the last frame is [Ly, Ly]: log sum_j R(j, Ly) exp(alpha(j) + final(j))
      double m = neg_inf();
      for (int j = 0; j < nl; ++j)
        if (cur[(size_t)j * W] > 0.0) m = fmax(m, log(cur[(size_t)j * W]) + al_len[j] + fw[j]);
      double sum = 0.0;
      if (m != neg_inf())
        for (int j = 0; j < nl; ++j)
          if (cur[(size_t)j * W] > 0.0) {
            const double x = log(cur[(size_t)j * W]) + al_len[j] + fw[j];
            if (x != neg_inf()) sum += exp(x - m);
          }
      N.score[(size_t)b * n + u] = m == neg_inf() ? m : m + log(sum) + logscale;
    }
    __syncthreads();  // s_y and the DP buffers are reused by the next group
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
      launch_joiner_dense(m, enc, m.C, L.rowctx, row0, L.Nc, R, h, logits, stats, ncu, st);
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
  hipLaunchKernelGGL(k_lat_sample, dim3((N.n + kLT - 1) / kLT, L.B), dim3(kLT), 0, st, L, N);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_lat_unique, dim3(L.B), dim3(kLT), 0, st, L, N);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  (void)dp_lds;
  hipLaunchKernelGGL(k_lat_seqscore, dim3(dp_grid, L.B), dim3(kLT), 0, st, L, N);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(k_lat_best, dim3(L.B), dim3(kLT), 0, st, L, N, out_tokens, out_ntok,
                     out_scores, out_nuniq, out_uscores, out_ufirst);
  return hipGetLastError();
}

}  // namespace tbs
