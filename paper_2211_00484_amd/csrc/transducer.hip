// Forward recursions of the transducer losses over the (frame t, labels emitted u) grid
// (Sec. 3): the standard recursion, eq. (1); the modified transducer, eq. (2), where
// emitting a label also moves to the next frame; and the constrained transducer, eq. (3),
// where a label is followed by the blank of the new context on the same frame.  Inputs
// are the log-probabilities the joiner gives at each cell: blank [B][T][U+1] and label
// [B][T][U] (the label u+1 of the utterance, after u labels).
//
// One wave per utterance; lane l owns the K consecutive cells u in [l*K, l*K + K) of a
// row (U + 1 <= 64 K), with the row in registers and the next row's log-probabilities
// loaded while the current one is combined.
//  - eq. (2), (3): row t depends on row t-1 only; the cell left of a lane's first comes
//    from the previous lane (one shuffle per row).
//  - eq. (1): row t also depends on its own left neighbour.  With A(u) = alpha(t-1, u) +
//    blank(t-1, u) and S(u) = sum_{j<u} label(t, j), alpha(t, u) = S(u) + log sum_{k<=u}
//    exp(A(k) - S(k)): an exclusive prefix sum and an inclusive prefix log-sum-exp over
//    the row, each a lane-serial scan plus a wave scan of the lane totals.
// Scores are fp64.
#include <hip/hip_runtime.h>

#include <cmath>

#include "internal.h"

namespace tbs {
namespace {

__device__ __forceinline__ double ninf() { return -__builtin_inf(); }

__device__ __forceinline__ double log_add2(double a, double b) {
  const double hi = fmax(a, b), lo = fmin(a, b);
  return hi == ninf() ? hi : hi + log1p(exp(lo - hi));
}

template <int K, int KIND>
__global__ __launch_bounds__(256) void k_transducer(const float* __restrict__ blank,
                                                    const float* __restrict__ label,
                                                    const int* __restrict__ lengths, int B,
                                                    int T, int U, double* __restrict__ total,
                                                    float* __restrict__ alpha,
                                                    int* __restrict__ status) {
  const int lane = threadIdx.x & 63;
  const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (b >= B) return;  // whole wave
  const int Tb = lengths[2 * b], Ub = lengths[2 * b + 1];
  const bool bad = Tb < 1 || Tb > T || Ub < 0 || Ub > U;
  if (bad) {
    if (lane == 0) {
      total[b] = __builtin_nan("");
      if (status) status[b] = 1;
    }
    return;
  }
  const int U1 = U + 1;
  const float* bl = blank + (size_t)b * T * U1;
  const float* lb = label + (size_t)b * T * U;
  float* al = alpha ? alpha + (size_t)b * (T + 1) * U1 : nullptr;
  const int u0 = lane * K;
  double a[K];
#pragma unroll
  for (int k = 0; k < K; ++k) a[k] = u0 + k == 0 ? 0.0 : ninf();
  // log-probabilities of one row for this lane's cells: blank(r, u), label(r, u - 1)
  // (eq. 2, 3) or label(r, u) (eq. 1); 0 outside the utterance (never used)
  auto load_row = [&](int r, float* xb, float* xl) {
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const int u = u0 + k;
      xb[k] = r >= 0 && r < Tb && u <= Ub ? bl[(size_t)r * U1 + u] : 0.f;
      const int ul = KIND == 0 ? u : u - 1;
      xl[k] = r >= 0 && r < Tb && ul >= 0 && ul < Ub ? lb[(size_t)r * U + ul] : 0.f;
    }
  };
  auto store_row = [&](int t) {
    if (!al) return;
#pragma unroll
    for (int k = 0; k < K; ++k)
      if (u0 + k < U1) al[(size_t)t * U1 + u0 + k] = u0 + k <= Ub ? (float)a[k] : -INFINITY;
  };
  float nb[K], nl[K];
  double res;
  if (KIND != 0) {
    store_row(0);
    load_row(0, nb, nl);
    for (int t = 1; t <= Tb; ++t) {
      float cb[K], cl[K];
#pragma unroll
      for (int k = 0; k < K; ++k) {
        cb[k] = nb[k];
        cl[k] = nl[k];
      }
      load_row(t, nb, nl);  // next row, in flight while this one is combined
      double left = __shfl_up(a[K - 1], 1, 64);
      if (lane == 0) left = ninf();
      double na[K];
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const int u = u0 + k;
        double v = ninf();
        if (u <= Ub) {
          v = a[k] + (double)cb[k];
          if (u > 0) {
            double w = (k == 0 ? left : a[k - 1]) + (double)cl[k];
            if (KIND == 2) w += (double)cb[k];
            v = log_add2(v, w);
          }
        }
        na[k] = v;
      }
#pragma unroll
      for (int k = 0; k < K; ++k) a[k] = na[k];
      store_row(t);
    }
    // alpha(Tb, Ub)
    double mine = ninf();
#pragma unroll
    for (int k = 0; k < K; ++k)
      if (u0 + k == Ub) mine = a[k];
    res = __shfl(mine, Ub / K, 64);
  } else {
    float pb[K], pl[K];  // blank of the previous row
#pragma unroll
    for (int k = 0; k < K; ++k) pb[k] = 0.f;
    load_row(0, nb, nl);
    for (int t = 0; t < Tb; ++t) {
      float cl[K];
#pragma unroll
      for (int k = 0; k < K; ++k) {
        pl[k] = pb[k];  // blank(t - 1, u), loaded with row t - 1
        pb[k] = nb[k];  // blank(t, u)
        cl[k] = nl[k];  // label(t, u)
      }
      load_row(t + 1, nb, nl);
      // A(u) and the label weights of this row
      double A[K], y[K];
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const int u = u0 + k;
        A[k] = t == 0 ? (u == 0 ? 0.0 : ninf()) : (u <= Ub ? a[k] + (double)pl[k] : ninf());
        y[k] = u < Ub ? (double)cl[k] : 0.0;
      }
      // exclusive prefix sum S(u) of y over the row
      double S[K], run = 0.0;
#pragma unroll
      for (int k = 0; k < K; ++k) {
        S[k] = run;
        run += y[k];
      }
      double x = run;  // wave inclusive scan of the lane totals
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const double z = __shfl_up(x, o, 64);
        if (lane >= o) x += z;
      }
      const double off = x - run;  // the lanes to the left
#pragma unroll
      for (int k = 0; k < K; ++k) S[k] += off;
      // inclusive prefix log-sum-exp of A(k) - S(k)
      double L[K], acc = ninf();
#pragma unroll
      for (int k = 0; k < K; ++k) {
        acc = log_add2(acc, A[k] - S[k]);
        L[k] = acc;
      }
      double g = acc;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const double z = __shfl_up(g, o, 64);
        if (lane >= o) g = log_add2(g, z);
      }
      double gl = __shfl_up(g, 1, 64);  // exclusive: the lanes to the left
      if (lane == 0) gl = ninf();
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const int u = u0 + k;
        a[k] = u <= Ub ? S[k] + log_add2(gl, L[k]) : ninf();
      }
      store_row(t);
    }
    // alpha(Tb - 1, Ub) + blank(Tb - 1, Ub)
    double mine = ninf();
#pragma unroll
    for (int k = 0; k < K; ++k)
      if (u0 + k == Ub) mine = a[k] + (double)pb[k];
    res = __shfl(mine, Ub / K, 64);
  }
  if (lane == 0) {
    total[b] = res;
    if (status) status[b] = 0;
  }
}

template <int KIND>
hipError_t launch_kind(int K, const float* blank, const float* label, const int* lengths, int B,
                       int T, int U, double* total, float* alpha, int* status, hipStream_t st) {
  const dim3 grid((B + 3) / 4), block(256);
  switch (K) {
    case 1: hipLaunchKernelGGL((k_transducer<1, KIND>), grid, block, 0, st, blank, label, lengths, B, T, U, total, alpha, status); break;
    case 2: hipLaunchKernelGGL((k_transducer<2, KIND>), grid, block, 0, st, blank, label, lengths, B, T, U, total, alpha, status); break;
    case 4: hipLaunchKernelGGL((k_transducer<4, KIND>), grid, block, 0, st, blank, label, lengths, B, T, U, total, alpha, status); break;
    case 8: hipLaunchKernelGGL((k_transducer<8, KIND>), grid, block, 0, st, blank, label, lengths, B, T, U, total, alpha, status); break;
    default: hipLaunchKernelGGL((k_transducer<16, KIND>), grid, block, 0, st, blank, label, lengths, B, T, U, total, alpha, status); break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_transducer_forward(int kind, const float* blank, const float* label,
                                     const int* lengths, int B, int T, int U, double* total,
                                     float* alpha, int* status, hipStream_t st) {
  if (B == 0) return hipSuccess;
  int K = 1;
  while (64 * K < U + 1) K *= 2;
  if (K > kTransducerMaxK) return hipErrorInvalidValue;
  if (kind == 0) return launch_kind<0>(K, blank, label, lengths, B, T, U, total, alpha, status, st);
  if (kind == 1) return launch_kind<1>(K, blank, label, lengths, B, T, U, total, alpha, status, st);
  return launch_kind<2>(K, blank, label, lengths, B, T, U, total, alpha, status, st);
}

}  // namespace tbs
