// gfx950 kernels for batched FSA-based one-symbol-per-frame transducer beam
// search (Kang et al., arXiv 2211.00484, Sec. 2.2-2.5 and Algorithm 1).
//
// Per frame t (the loop body of Algorithm 1):
//   k_joiner  joiner GEMM on MFMA over the rows h = tanh(enc_t + dec(ctx)) of
//             every active (stream, context): logits plus per-tile (max, sum
//             exp) partials of the log-softmax; for the trivial graph the
//             epilogue keeps only each row's best labels per tile.
//   k_search  one workgroup per stream: log-softmax normaliser, ExpandArcs
//             over the CSR graph without pruning, max-merge of equal (state,
//             context) keys, beam + max-states selection, max-contexts
//             selection, canonical (context, state) order, renormalisation,
//             back-pointers; then GetContexts + decoder + IndexSelect + tanh
//             for frame t+1, so the next joiner reads ready rows.
// k_init seeds the initial tuple and its joiner row; k_final picks the best
// final tuple and traces the back-pointers.
#include "internal.h"

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstddef>
#include <cstdint>
#include <type_traits>

namespace tbs {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));

constexpr unsigned long long kEmpty = ~0ull;

// ---------------------------------------------------------------------------
// small helpers


// Order-preserving map float -> uint32 (larger float -> larger code).
__device__ __forceinline__ uint32_t f2ord(float f) {
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float ord2f(uint32_t o) {
  uint32_t u = (o & 0x80000000u) ? (o & 0x7fffffffu) : ~o;
  return __uint_as_float(u);
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

// Cross-lane reductions on DPP row rotations (16-lane rows) and readlane, which
// stay in the VALU instead of taking an LDS round trip per step.
template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xf, 0xf, false);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(dpp_i<CTRL>(__float_as_int(v)));
}
template <int CTRL>
__device__ __forceinline__ unsigned long long dpp_u64(unsigned long long v) {
  const int lo = dpp_i<CTRL>((int)(unsigned)v), hi = dpp_i<CTRL>((int)(unsigned)(v >> 32));
  return ((unsigned long long)(unsigned)hi << 32) | (unsigned)lo;
}
constexpr int kRor8 = 0x128, kRor4 = 0x124, kRor2 = 0x122, kRor1 = 0x121;

// reductions over the 16 lanes of a DPP row; every lane of the row gets the result
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp_f<kRor8>(v));
  v = fmaxf(v, dpp_f<kRor4>(v));
  v = fmaxf(v, dpp_f<kRor2>(v));
  return fmaxf(v, dpp_f<kRor1>(v));
}
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_f<kRor8>(v);
  v += dpp_f<kRor4>(v);
  v += dpp_f<kRor2>(v);
  return v + dpp_f<kRor1>(v);
}
// v of lane (this lane xor M), M a power of two up to 32, in the cheapest form for M:
// DPP within 16-lane rows (1, 2: quad permutations; 4: half-row mirror then quad
// reversal; 8: row mirror then half-row mirror), a swizzle across the halves of 32
// lanes (16), and a permute through LDS only across the wave's halves (32).
__device__ __forceinline__ int xor_lane(int v, int M) {
  switch (M) {
    case 1: return __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xf, 0xf, false);
    case 2: return __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xf, 0xf, false);
    case 4:
      return __builtin_amdgcn_update_dpp(0, __builtin_amdgcn_update_dpp(0, v, 0x141, 0xf, 0xf, false),
                                         0x1B, 0xf, 0xf, false);
    case 8:
      return __builtin_amdgcn_update_dpp(0, __builtin_amdgcn_update_dpp(0, v, 0x140, 0xf, 0xf, false),
                                         0x141, 0xf, 0xf, false);
    case 16: return __builtin_amdgcn_ds_swizzle(v, 0x401F);  // and 31, or 0, xor 16
    default: return __shfl_xor(v, M, 64);
  }
}
__device__ __forceinline__ unsigned long long umax64(unsigned long long a, unsigned long long b) {
  return a > b ? a : b;
}
__device__ __forceinline__ unsigned long long row16_max_u64(unsigned long long v) {
  v = umax64(v, dpp_u64<kRor8>(v));
  v = umax64(v, dpp_u64<kRor4>(v));
  v = umax64(v, dpp_u64<kRor2>(v));
  return umax64(v, dpp_u64<kRor1>(v));
}
__device__ __forceinline__ float rdlane_f(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
// whole-wave reductions (all 64 lanes active); uniform result.  After the row
// reductions, two DPP row broadcasts fold the rows into the last one (lane 15 into
// rows 1 and 3, then lane 31 into rows 2 and 3; rows outside the mask keep their
// value, or add 0) and one readlane of lane 63 returns ((r3 + r2) + (r1 + r0)).
__device__ __forceinline__ float wave_max_f(float v) {
  v = row16_max(v);
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), 0x142, 0xa, 0xf, false)));
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), 0x143, 0xc, 0xf, false)));
  return rdlane_f(v, 63);
}
__device__ __forceinline__ float wave_sum_f(float v) {
  v = row16_sum(v);
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x142, 0xa, 0xf, false));
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x143, 0xc, 0xf, false));
  return rdlane_f(v, 63);
}
__device__ __forceinline__ unsigned long long umin64(unsigned long long a, unsigned long long b) {
  return a < b ? a : b;
}
__device__ __forceinline__ unsigned long long wave_min_u64(unsigned long long v) {
  v = umin64(v, dpp_u64<kRor8>(v));
  v = umin64(v, dpp_u64<kRor4>(v));
  v = umin64(v, dpp_u64<kRor2>(v));
  v = umin64(v, dpp_u64<kRor1>(v));
  unsigned long long r = ~0ull;
#pragma unroll
  for (int l = 0; l < 64; l += 16) {
    const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)v, l);
    const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(v >> 32), l);
    r = umin64(r, ((unsigned long long)hi << 32) | lo);
  }
  return r;
}
// (row maxima, then the row broadcasts of lane 15 into rows 1 and 3 and of lane 31
// into rows 2 and 3, so that lane 63 holds the wave maximum: one readlane)
__device__ __forceinline__ unsigned wave_max_u32(unsigned v) {
  v = max(v, (unsigned)dpp_i<kRor8>((int)v));
  v = max(v, (unsigned)dpp_i<kRor4>((int)v));
  v = max(v, (unsigned)dpp_i<kRor2>((int)v));
  v = max(v, (unsigned)dpp_i<kRor1>((int)v));
  v = max(v, (unsigned)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x142, 0xa, 0xf, false));  // row_bcast:15
  v = max(v, (unsigned)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x143, 0xc, 0xf, false));  // row_bcast:31
  return (unsigned)__builtin_amdgcn_readlane((int)v, 63);
}
__device__ __forceinline__ unsigned wave_min_u32(unsigned v) {
  v = min(v, (unsigned)dpp_i<kRor8>((int)v));
  v = min(v, (unsigned)dpp_i<kRor4>((int)v));
  v = min(v, (unsigned)dpp_i<kRor2>((int)v));
  v = min(v, (unsigned)dpp_i<kRor1>((int)v));
  return min(min((unsigned)__builtin_amdgcn_readlane((int)v, 0), (unsigned)__builtin_amdgcn_readlane((int)v, 16)),
             min((unsigned)__builtin_amdgcn_readlane((int)v, 32), (unsigned)__builtin_amdgcn_readlane((int)v, 48)));
}
__device__ __forceinline__ unsigned long long wave_max_u64(unsigned long long v) {
  v = row16_max_u64(v);
  unsigned long long r = 0;
#pragma unroll
  for (int l = 0; l < 64; l += 16) {
    const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)v, l);
    const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(v >> 32), l);
    r = umax64(r, ((unsigned long long)hi << 32) | lo);
  }
  return r;
}

// Inclusive prefix sum over the wave's 64 lanes on DPP: shifts by 1, 2, 4 and 8 within
// each row of 16 (lanes before the shift's source add 0), then the row broadcasts of
// lane 15 (into rows 1 and 3) and lane 31 (into rows 2 and 3); no LDS round trip.
__device__ __forceinline__ unsigned wave_incl_scan_u32(unsigned v) {
  v += (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xf, 0xf, true);  // row_shr:1
  v += (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xf, 0xf, true);  // row_shr:2
  v += (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xf, 0xf, true);  // row_shr:4
  v += (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xf, 0xf, true);  // row_shr:8
  v += (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xa, 0xf, false);  // row_bcast:15
  v += (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return v;
}

// log-sum-exp of one joiner row from its per-tile (max, sum exp) partials.  The
// logarithm is taken in double: the device logf is biased low by a fraction of
// an ulp, which would otherwise accumulate over the frames of a stream.
__device__ __forceinline__ double lse_of(float M, float S) { return (double)M + log((double)S); }

// log-probability of one logit, rounded once to fp32
__device__ __forceinline__ float logp_of(float z, double lse) { return (float)((double)z - lse); }

// ---------------------------------------------------------------------------
// model setup: P0 = tap0 * E, P1 = tap1 * E (padded to Kpad), W packed to
// [Vpad][Kpad] in fp32 or bf16, bias copied (zeros if absent).  Wi holds W once
// more, interleaved as [Kpad / KQ][Vpad][KQ] (KQ = 16 bytes of elements: 4 fp32
// or 8 bf16), so that 64 lanes loading 16 bytes each for 64 consecutive
// vocabulary columns read one contiguous kilobyte (per-stream kernel).

__global__ void k_model_setup(const float* __restrict__ E, const float* __restrict__ conv,
                              const float* __restrict__ W, const float* __restrict__ b_out, int V,
                              int C, int Kpad, int Vpad, int bf16, float* __restrict__ P0,
                              float* __restrict__ P1, float* __restrict__ Wf,
                              uint16_t* __restrict__ Wb, void* __restrict__ Wi,
                              float* __restrict__ bias) {
  const long long n = (long long)Vpad * Kpad;
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n;
       i += (long long)gridDim.x * blockDim.x) {
    const int v = (int)(i / Kpad), k = (int)(i - (long long)v * Kpad);
    const bool in = v < V && k < C;
    const float e = in ? E[(size_t)v * C + k] : 0.f;
    const float w = in ? W[(size_t)v * C + k] : 0.f;
    if (v < V) {
      P0[i] = in ? conv[2 * k + 0] * e : 0.f;
      P1[i] = in ? conv[2 * k + 1] * e : 0.f;
    }
    if (bf16) {
      const uint16_t wb = f32_to_bf16_rne(w);
      Wb[i] = wb;
      reinterpret_cast<uint16_t*>(Wi)[((size_t)(k >> 3) * Vpad + v) * 8 + (k & 7)] = wb;
    } else {
      Wf[i] = w;
      reinterpret_cast<float*>(Wi)[((size_t)(k >> 2) * Vpad + v) * 4 + (k & 3)] = w;
    }
    if (k == 0 && v < V) bias[v] = b_out ? b_out[v] : 0.f;
  }
}

__global__ void k_fill_i32(int* p, long long n, int v) {
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n;
       i += (long long)gridDim.x * blockDim.x)
    p[i] = v;
}

// out[b] = in[b] clamped to [0, T] (stream lengths handed over in device memory).
__global__ void k_clamp_lengths(const int* __restrict__ in, int* __restrict__ out, int B, int T) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < B) out[b] = min(max(in[b], 0), T);
}

// ---------------------------------------------------------------------------
// tanh_fast (internal.h) has absolute error ~2e-7, which moves a joiner logit by at
// most ~C * max|W| * 2e-7.

// Joiner input rows (Algorithm 1: decoder, IndexSelect of the encoder frame):
// h[k] = tanh(enc[k] + ReLU(P0[a][k] + P1[b][k])) for k < C, 0 for C <= k < Kpad,
// stored as fp32 or bf16 (RNE) at hbase + r * hstride elements (global memory or
// LDS).  Row r reads P0/P1 at rowoff[r] = (a * Kpad, b * Kpad) and the encoder
// row enc_rows + r * enc_stride (enc_stride = 0: one shared frame).
// Thread tid owns columns tid, tid + NT, ... of every row (Kpad is a multiple of
// 512); a batch's loads are all issued before any tanh.
template <int NT, int U = 16>  // U: (row, column) elements per thread per batch
__device__ void write_h_rows(const ModelDev& m, const float* __restrict__ enc_rows,
                             long long enc_stride, const int2* rowoff, int nrows,
                             void* __restrict__ hbase, int hstride, int tid) {
  const int C = m.C, Kpad = m.Kpad;
  const float* __restrict__ P0 = m.P0;
  const float* __restrict__ P1 = m.P1;
  const int cols = Kpad / NT;  // columns per thread per row
  int r = 0, j = 0;            // (row, column slot) of the next element
  while (r < nrows) {
    float e[U], p0[U], p1[U];
    int ro[U], ko[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      ro[u] = r;
      ko[u] = tid + j * NT;
      if (++j == cols) {
        j = 0;
        ++r;
      }
    }
    // the elements' table rows (LDS reads issued together), then every load; past
    // the last row or column an element loads a valid one and drops it, so that no
    // branch separates the loads (all of them in flight at once)
    int2 off[U];
#pragma unroll
    for (int u = 0; u < U; ++u) off[u] = rowoff[min(ro[u], nrows - 1)];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int rc = min(ro[u], nrows - 1), kc = min(ko[u], C - 1);
      e[u] = enc_rows[(size_t)rc * enc_stride + kc];
      p0[u] = P0[(size_t)off[u].x + kc];
      p1[u] = P1[(size_t)off[u].y + kc];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (ro[u] >= nrows) continue;
      const int k = ko[u];
      const float h = k < C ? tanh_fast(e[u] + fmaxf(p0[u] + p1[u], 0.f)) : 0.f;
      const size_t o = (size_t)ro[u] * hstride + k;
      if (m.bf16)
        reinterpret_cast<uint16_t*>(hbase)[o] = f32_to_bf16_rne(h);
      else
        reinterpret_cast<float*>(hbase)[o] = h;
    }
  }
}

// The same rows for C a multiple of 4, four adjacent columns per item: item i of the
// nrows x Kpad / 4 (row, column quad) items is thread i mod NT's; a batch of U items per
// thread issues U 16-byte loads of P0 and of P1 (all in flight at once), then U 16-byte
// (fp32) or 8-byte (bf16) stores.  enc is one frame shared by every row.
template <int NT, int U>
__device__ void write_h_rows_quads(const ModelDev& m, const float* __restrict__ enc,
                                   const int2* rowoff, int nrows, void* __restrict__ hbase,
                                   int hstride, int tid) {
  const int C = m.C, qpr = m.Kpad / 4;  // column quads per row
  // (32-bit byte offsets from the uniform table bases: P0 and P1 stay below 4 GiB)
  const char* P0b = reinterpret_cast<const char*>(m.P0);
  const char* P1b = reinterpret_cast<const char*>(m.P1);
  const int total = nrows * qpr;
  for (int i0 = 0; i0 < total; i0 += U * NT) {
    int ro[U], ko[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int it = min(i0 + tid + u * NT, total - 1);  // past the end: a valid item, dropped
      ro[u] = it / qpr;
      ko[u] = 4 * (it - ro[u] * qpr);
    }
    // the items' table rows (LDS reads together), then every load
    int2 off[U];
#pragma unroll
    for (int u = 0; u < U; ++u) off[u] = rowoff[ro[u]];
    float4 p0[U], p1[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const unsigned kc = (unsigned)min(ko[u], C - 4);
      p0[u] = *reinterpret_cast<const float4*>(P0b + ((unsigned)off[u].x + kc) * 4u);
      p1[u] = *reinterpret_cast<const float4*>(P1b + ((unsigned)off[u].y + kc) * 4u);
    }
    // every value first, then the stores (fully unrolled: a rolled loop would load
    // every item again, one round trip each, and stores between the uses would make
    // each use wait for all of them)
    float4 h[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = ko[u];
      const float4 e = *reinterpret_cast<const float4*>(enc + k);
      h[u] = k < C ? make_float4(tanh_fast(e.x + fmaxf(p0[u].x + p1[u].x, 0.f)),
                                 tanh_fast(e.y + fmaxf(p0[u].y + p1[u].y, 0.f)),
                                 tanh_fast(e.z + fmaxf(p0[u].z + p1[u].z, 0.f)),
                                 tanh_fast(e.w + fmaxf(p0[u].w + p1[u].w, 0.f)))
                   : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    if (m.bf16) {
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (i0 + tid + u * NT < total)
          *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(hbase) + (size_t)ro[u] * hstride + ko[u]) =
              make_uint2((unsigned)f32_to_bf16_rne(h[u].x) | ((unsigned)f32_to_bf16_rne(h[u].y) << 16),
                         (unsigned)f32_to_bf16_rne(h[u].z) | ((unsigned)f32_to_bf16_rne(h[u].w) << 16));
    } else {
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (i0 + tid + u * NT < total)
          *reinterpret_cast<float4*>(reinterpret_cast<float*>(hbase) + (size_t)ro[u] * hstride + ko[u]) = h[u];
    }
  }
}

// The same rows for an even C, two adjacent columns per item: thread tid owns the
// column pairs (2 tid, 2 tid + 1), (2 tid + 2 NT, ...), ... of every row, so a batch
// of U items issues U 8-byte loads of P0 and of P1 (all in flight at once) and U
// 8-byte (fp32) or 4-byte (bf16) stores.  enc is one frame shared by every row.
template <int NT, int U = 16>
__device__ void write_h_rows_pairs(const ModelDev& m, const float* __restrict__ enc,
                                   const int2* rowoff, int nrows, void* __restrict__ hbase,
                                   int hstride, int tid) {
  const int C = m.C, Kpad = m.Kpad;
  // (32-bit byte offsets from the uniform table bases: P0 and P1 stay below 4 GiB)
  const char* P0b = reinterpret_cast<const char*>(m.P0);
  const char* P1b = reinterpret_cast<const char*>(m.P1);
  const int cols = Kpad / (2 * NT);  // column pairs per thread per row
  int r = 0, j = 0;                  // (row, pair slot) of the next item
  while (r < nrows) {
    float2 p0[U], p1[U];
    int ro[U], ko[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      ro[u] = r;
      ko[u] = 2 * (tid + j * NT);
      if (++j == cols) {
        j = 0;
        ++r;
      }
    }
    // the items' table rows (LDS reads issued together), then every load; past the
    // last row or column an item loads a valid pair and drops it (no branch
    // separates the loads)
    int2 off[U];
#pragma unroll
    for (int u = 0; u < U; ++u) off[u] = rowoff[min(ro[u], nrows - 1)];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const unsigned kc = (unsigned)min(ko[u], C - 2);
      p0[u] = *reinterpret_cast<const float2*>(P0b + ((unsigned)off[u].x + kc) * 4u);
      p1[u] = *reinterpret_cast<const float2*>(P1b + ((unsigned)off[u].y + kc) * 4u);
    }
    // (one fully unrolled loop per store type: a rolled loop would load every item
    // again, one round trip each, instead of indexing the registers above)
    auto hpair = [&](int u) {
      const int k = ko[u];
      float2 h = make_float2(0.f, 0.f);
      if (k < C) {
        h.x = tanh_fast(enc[k] + fmaxf(p0[u].x + p1[u].x, 0.f));
        h.y = tanh_fast(enc[k + 1] + fmaxf(p0[u].y + p1[u].y, 0.f));
      }
      return h;
    };
    if (m.bf16) {
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (ro[u] < nrows) {
          const float2 h = hpair(u);
          *reinterpret_cast<unsigned*>(reinterpret_cast<uint16_t*>(hbase) + (size_t)ro[u] * hstride + ko[u]) =
              (unsigned)f32_to_bf16_rne(h.x) | ((unsigned)f32_to_bf16_rne(h.y) << 16);
        }
    } else {
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (ro[u] < nrows)
          *reinterpret_cast<float2*>(reinterpret_cast<float*>(hbase) + (size_t)ro[u] * hstride + ko[u]) = hpair(u);
    }
  }
}

// h rows for explicit (encoder row, context) pairs: one workgroup per row.
__global__ __launch_bounds__(256) void k_h_rows(ModelDev m, const float* __restrict__ enc_rows,
                                                const int* __restrict__ ctx, void* __restrict__ h) {
  __shared__ int2 off;
  const int r = blockIdx.x;
  if (threadIdx.x == 0) {
    const int c = ctx[r], a = c / m.V;
    off = make_int2(a * m.Kpad, (c - a * m.V) * m.Kpad);
  }
  __syncthreads();
  const size_t esz = m.bf16 ? 2 : 4;
  write_h_rows<256>(m, enc_rows + (size_t)r * m.C, 0, &off, 1,
                    reinterpret_cast<char*>(h) + (size_t)r * m.Kpad * esz, m.Kpad, threadIdx.x);
}

// Rows of a dense (encoder row, context) table: batch row r is table row row0 + r,
// with context ctx[row0 + r] (-1: an empty slot, written as zeros) and encoder row
// enc + ((row0 + r) / per_enc) * enc_stride.
__global__ __launch_bounds__(256) void k_h_rows_dense(ModelDev m, const float* __restrict__ enc,
                                                      const int* __restrict__ ctx, long long row0,
                                                      int per_enc, long long enc_stride,
                                                      void* __restrict__ h) {
  __shared__ int2 off;
  const long long g = row0 + blockIdx.x;
  const int c = ctx[g];
  const size_t esz = m.bf16 ? 2 : 4;
  char* hrow = reinterpret_cast<char*>(h) + (size_t)blockIdx.x * m.Kpad * esz;
  if (c < 0) {
    for (int k = threadIdx.x; k < m.Kpad; k += blockDim.x) {
      if (m.bf16)
        reinterpret_cast<uint16_t*>(hrow)[k] = 0;
      else
        reinterpret_cast<float*>(hrow)[k] = 0.f;
    }
    return;
  }
  if (threadIdx.x == 0) {
    const int a = c / m.V;
    off = make_int2(a * m.Kpad, (c - a * m.V) * m.Kpad);
  }
  __syncthreads();
  write_h_rows<256>(m, enc + (size_t)(g / per_enc) * enc_stride, 0, &off, 1, hrow, m.Kpad,
                    threadIdx.x);
}

// ---------------------------------------------------------------------------
// joiner

struct JoinArgs {
  const void* h;            // [R][Kpad]
  float* logits;            // [R][Vpad] or null
  float2* stats;            // [R][nvt]
  float* tk_z;              // [R][nvt][KT] (TOPK)
  int* tk_c;
  float* z0;                // [R] (TOPK)
  int KT;
  int R, n_rt, n_ct;        // rows; row and column tiles (128 x 128)
  int nvt;                  // 64-column vocabulary tiles (stats and label lists)
  int rows_mode;            // 1: every row < R is active
  const int* len;
  const int* nctx;
  int t, Nc;
};

__device__ __forceinline__ bool joiner_row_active(const JoinArgs& a, int r) {
  if (r >= a.R) return false;
  if (a.rows_mode) return true;
  const int b = r / a.Nc, j = r - b * a.Nc;
  return a.t < a.len[b] && j < a.nctx[b];
}

// Small joiner tile, for batches too small to give every compute unit a 128 x 128
// tile: (16 * MB rows) x 64 vocabulary columns; wave w owns columns 16w..16w+15
// and keeps its W fragment (16 columns x up to 512 of K) in registers while it
// sweeps the tile's row blocks, whose h rows are staged once in LDS.
struct JoinShared {
  int act[64];
  float m[4][64], s[4][64];
};

// One joiner tile (16 * MB rows x 64 vocabulary columns) of frame a.t.  Uniform
// across the workgroup; a tile without active rows computes nothing.
template <bool BF16, int MB, bool TOPK>
__device__ __forceinline__ void joiner_tile_small(const ModelDev& m, const JoinArgs& a, int ct, int rt,
                                            unsigned char* smem, JoinShared& js) {
  int* s_act = js.act;
  float(*s_m)[64] = js.m;
  float(*s_s)[64] = js.s;
  constexpr int BM = 16 * MB;
  constexpr int ESZ = BF16 ? 2 : 4;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r0 = rt * BM, n0 = ct * kJoinerBN;
  const int Kpad = m.Kpad, V = m.V, nvt = a.n_ct;
  const int lr = lane & 15, lg = lane >> 4;
  const int col = n0 + 16 * wave + lr;
  const bool cvalid = col < V;

  if (tid < BM) s_act[tid] = joiner_row_active(a, r0 + tid);
  // W fragment of the first K chunk (registers) and the bias: issued before the
  // h staging so that all of the tile's loads are in flight together
  // (Kpad is a multiple of 512: one chunk of W per lane is 32 float4 or 16 uint4).
  // W is read from its interleaved copy (16-byte k slices, columns consecutive),
  // where the 16 lanes of a k slice read 256 contiguous bytes.
  float4 wf[BF16 ? 1 : 32];
  uint4 wb[BF16 ? 16 : 1];
  const uint4* __restrict__ wi = reinterpret_cast<const uint4*>(m.Wi);
  const size_t Vp = (size_t)m.Vpad;
  auto load_w = [&](int kc) {
    if (BF16) {
      const size_t q0 = (size_t)(kc / 8 + 2 * lg);
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        wb[2 * s] = wi[(q0 + 8 * s) * Vp + col];
        wb[2 * s + 1] = wi[(q0 + 8 * s + 1) * Vp + col];
      }
    } else {
      const size_t q0 = (size_t)(kc / 4 + lg);
#pragma unroll
      for (int s = 0; s < 32; ++s) {
        const uint4 v = wi[(q0 + 4 * s) * Vp + col];
        wf[s] = make_float4(__uint_as_float(v.x), __uint_as_float(v.y), __uint_as_float(v.z),
                            __uint_as_float(v.w));
      }
    }
  };
  load_w(0);
  const float bias = cvalid ? m.bias[col] : 0.f;
  __syncthreads();
  int any = 0;
#pragma unroll
  for (int i = 0; i < BM; ++i) any |= s_act[i];
  if (!any) return;  // uniform across the workgroup: nothing to compute in this tile

  // stage the tile's h rows in LDS (16-byte chunks, all loads in flight together)
  const int ldk = Kpad + (BF16 ? 8 : 4);             // row stride in elements (16-byte pad)
  const int cpr = Kpad * ESZ / 16;                   // 16-byte chunks per row
  const int nchunk = BM * cpr;
  const char* hsrc = reinterpret_cast<const char*>(a.h) + (size_t)r0 * Kpad * ESZ;
  for (int base = tid; base < nchunk; base += 256 * 16) {
    uint4 v[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int c = base + u * 256;
      v[u] = make_uint4(0, 0, 0, 0);
      if (c < nchunk && s_act[c / cpr]) v[u] = reinterpret_cast<const uint4*>(hsrc)[c];
    }
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int c = base + u * 256;
      if (c < nchunk) {
        const int r = c / cpr, cc = c - r * cpr;
        *reinterpret_cast<uint4*>(smem + (size_t)r * ldk * ESZ + (size_t)cc * 16) = v[u];
      }
    }
  }

  // Four accumulator chains per row block, and consecutive MFMAs rotate over
  // (row block, chain), so no MFMA waits for the one before it.
  f32x4 acc[MB][4];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[mb][c] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int kc = 0; kc < Kpad; kc += 512) {
    if (kc > 0) load_w(kc);  // later K chunks (C > 512)
    __syncthreads();
    if (BF16) {
      const uint16_t* hb = reinterpret_cast<const uint16_t*>(smem) + (size_t)lr * ldk + kc + 16 * lg;
#pragma unroll
      for (int s = 0; s < 8; ++s) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const uint16_t* hr = hb + (size_t)mb * 16 * ldk + s * 64;
          const uint4 a0 = *reinterpret_cast<const uint4*>(hr);
          const uint4 a1 = *reinterpret_cast<const uint4*>(hr + 8);
          f32x4& c0 = acc[mb][(2 * s) & 3];
          f32x4& c1 = acc[mb][(2 * s + 1) & 3];
          c0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a0), as_bf16x8(wb[2 * s]), c0, 0, 0,
                                                       0);
          c1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a1), as_bf16x8(wb[2 * s + 1]), c1,
                                                       0, 0, 0);
        }
      }
    } else {
      const float* hs = reinterpret_cast<const float*>(smem) + (size_t)lr * ldk + kc + 4 * lg;
#pragma unroll
      for (int s = 0; s < 32; ++s) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const float4 av = *reinterpret_cast<const float4*>(hs + (size_t)mb * 16 * ldk + s * 16);
          acc[mb][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(av.x, wf[s].x, acc[mb][0], 0, 0, 0);
          acc[mb][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(av.y, wf[s].y, acc[mb][1], 0, 0, 0);
          acc[mb][2] = __builtin_amdgcn_mfma_f32_16x16x4f32(av.z, wf[s].z, acc[mb][2], 0, 0, 0);
          acc[mb][3] = __builtin_amdgcn_mfma_f32_16x16x4f32(av.w, wf[s].w, acc[mb][3], 0, 0, 0);
        }
      }
    }
  }

  // epilogue.  First everything that needs the workgroup barrier (per-row max
  // and sum exp over the tile, combined across the 4 waves in LDS); the global
  // stores come after it, so the barrier never waits on them.
  float zr[MB][4];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = mb * 16 + 4 * lg + i;  // the 16 lanes of a DPP row share this row
      const float zs = (acc[mb][0][i] + acc[mb][1][i]) + (acc[mb][2][i] + acc[mb][3][i]);
      const float z = cvalid ? zs + bias : -INFINITY;
      zr[mb][i] = z;
      const float mx = row16_max(z);
      const float e = row16_sum(cvalid ? expf(z - mx) : 0.f);
      if (lr == 0) {
        s_m[wave][row] = mx;
        s_s[wave][row] = e;
      }
    }
  }
  __syncthreads();
  if (tid < BM && s_act[tid]) {
    float M = s_m[0][tid];
    for (int w = 1; w < 4; ++w) M = fmaxf(M, s_m[w][tid]);
    float S = 0.f;
    for (int w = 0; w < 4; ++w) S += s_s[w][tid] == 0.f ? 0.f : s_s[w][tid] * expf(s_m[w][tid] - M);
    a.stats[(size_t)(r0 + tid) * nvt + ct] = make_float2(M, S);
  }
  // logits (general graphs) or each row's best KT labels per 16-column sub-tile
  // (trivial graph), found with DPP row reductions
  const int nsub = nvt * (kJoinerBN / 16);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = mb * 16 + 4 * lg + i;
      const float z = zr[mb][i];
      const bool act = s_act[row];
      if (!TOPK) {
        if (act && cvalid) a.logits[(size_t)(r0 + row) * (nvt * kJoinerBN) + col] = z;
      } else {
        unsigned long long key = (cvalid && col >= 1)
                                     ? ((unsigned long long)f2ord(z) << 32) | (0xffffffffu - (unsigned)col)
                                     : 0ull;
        const size_t ob = ((size_t)(r0 + row) * nsub + ct * (kJoinerBN / 16) + wave) * a.KT;
        for (int q = 0; q < a.KT; ++q) {
          const unsigned long long best = row16_max_u64(key);
          if (act && best != 0ull && key == best) {
            a.tk_z[ob + q] = z;
            a.tk_c[ob + q] = col;
          }
          if (act && best == 0ull && lr == 0) {
            a.tk_z[ob + q] = -INFINITY;
            a.tk_c[ob + q] = -1;
          }
          if (key == best) key = 0ull;
        }
        if (act && ct == 0 && wave == 0 && lr == 0) a.z0[r0 + row] = z;
      }
    }
  }
}

template <bool BF16, int MB, bool TOPK>
__global__ __launch_bounds__(256) void k_joiner_small(ModelDev m, JoinArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ JoinShared js;
  // Workgroup i runs on XCD i mod 8.  XCD x owns the column tiles x, x + 8, ...
  // and walks row tiles in order, its column tiles fastest: its W columns stay
  // in its L2 while each h row tile is read once per XCD.
  const int bid = blockIdx.x, xcd = bid & 7, slot = bid >> 3;
  const int ncx = (a.n_ct + 7) >> 3;
  const int rt = slot / ncx, ct = xcd + 8 * (slot - rt * ncx);
  if (ct >= a.n_ct) return;
  joiner_tile_small<BF16, MB, TOPK>(m, a, ct, rt, smem, js);
}

constexpr float kLog2e = 1.44269504088896341f;

// Joiner GEMM tile: BM = 32 MBW rows x BN = 64 WN vocabulary columns, 2 x WN waves,
// each wave 16 MBW rows x 64 columns (MBW x 4 MFMA blocks of 16 x 16):
//  - 128 x 128 (MBW = 4, WN = 2; four waves), for batches with at least four such
//    tiles per compute unit;
//  - 64 x 128 (MBW = 2, WN = 2; four waves, three workgroups per compute unit), for
//    batches with one to four 128 x 128 tiles per compute unit, which it splits into
//    finer, more evenly spread parts;
//  - 256 x 256 (MBW = 8, WN = 4; eight waves), for bf16 batches with several such
//    tiles per compute unit: half the operand bytes per product of the 128 tile, and
//    a quarter fewer LDS fragment reads per MFMA.
// Both operands go through LDS in K slices of 128 bytes per row (64 bf16 or 32 fp32
// values), two buffers deep, one barrier per slice.  The 128 and 64 tiles keep slices
// s + 1 and s + 2 in flight to registers during the MFMAs of slice s; the 256 tile,
// whose slices hold twice the MFMAs, keeps slice s + 1.  A wave's 64 columns are one
// vocabulary tile, so its epilogue produces that tile's (max, sum exp) per row and
// either the logits or each row's best labels per 16-column sub-tile.
constexpr int kJBM = 128, kJBN = 128;          // the 128 tile: rows, columns
constexpr int kJSlice = 128;                   // bytes of K per row and slice
constexpr int kJRow = kJSlice;                 // LDS row stride (16-byte chunks swizzled per row)
constexpr int kJStage = (kJBM + kJBN) * kJRow; // bytes per buffer: A rows, then B rows
constexpr size_t kJLds = 2 * (size_t)kJStage;  // 65,536 bytes
constexpr int kJHalfBM = 64;                   // the 64 x 128 tile
constexpr size_t kJHalfLds = 2 * (size_t)(kJHalfBM + kJBN) * kJRow;  // 49,152 bytes
constexpr int kJWideBM = 256, kJWideBN = 256;  // the 256 tile
constexpr size_t kJWideLds = 2 * (size_t)(kJWideBM + kJWideBN) * kJRow;  // 131,072 bytes
// LDS chunk swizzle: chunk k of a row with index r mod 16 = l sits at slot k ^ jswz(l).
// A fragment read (16 rows of a block, one chunk each) then touches 16 distinct 4-bank
// groups whether the LDS serves 8 lanes from 32 banks or 16 lanes from 64 banks per
// cycle, and so does a slice write (8 lanes per row, two rows per 16 lanes).
__device__ __forceinline__ int jswz(int l) { return (l & 7) ^ ((l >> 3) & 1); }

template <bool BF16, bool TOPK, int WN, int MBW>
__global__ __launch_bounds__(128 * WN) void k_joiner(ModelDev m, JoinArgs a) {
  constexpr int NT = 128 * WN, BM = 32 * MBW, BN = 64 * WN;
  constexpr int STAGE = (BM + BN) * kJRow;
  constexpr bool DEEP = MBW <= 4;  // two slices in flight (else one)
  constexpr int UA = BM * 8 / NT, UB = BN * 8 / NT;  // 16-byte chunks per thread and slice
  static_assert(UA * NT == BM * 8 && UB * NT == BN * 8 && UA <= UB, "slice loads");
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ int s_act[BM];
  const int bid = blockIdx.x, xcd = bid & 7, slot = bid >> 3;
  int rt, ct;
  if (WN == 2) {
    // Workgroup i runs on XCD i mod 8.  XCD x owns the column tiles x, x + 8, ...
    // and walks row tiles in order, its column tiles fastest: its W columns stay
    // in its L2 while each h row tile is read once per XCD.
    const int ncx = (a.n_ct + 7) >> 3;
    rt = slot / ncx;
    ct = xcd + 8 * (slot - rt * ncx);
    if (ct >= a.n_ct) return;
  } else {
    // Tiles in row-major order, tile q on XCD q mod 8: with a column-tile count that
    // is not a multiple of 8, each XCD still gets an equal share, and sees only the
    // column tiles congruent to its index modulo gcd(n_ct, 8).
    const int q = xcd + 8 * slot;
    rt = q / a.n_ct;
    ct = q - rt * a.n_ct;
    if (rt >= a.n_rt) return;
  }
  constexpr int ESZ = BF16 ? 2 : 4;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave / WN, wc = wave % WN;
  const int lr = lane & 15, lg = lane >> 4;
  const int r0 = rt * BM, c0 = ct * BN;
  const int Kpad = m.Kpad, V = m.V, Vpad = m.Vpad, nvt = a.nvt;
  const int vt = WN * ct + wc;  // this wave's vocabulary tile
  const int act = tid < BM ? (int)joiner_row_active(a, r0 + tid) : 0;
  if (tid < BM) s_act[tid] = act;
  if (!__syncthreads_or(act)) return;  // uniform: no active row in this tile
  // the epilogue's bias values, requested now so that their round trip is hidden
  // behind the main loop (clamped: past the vocabulary they are never used)
  float bias_r[4];
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) bias_r[nb] = m.bias[min(64 * vt + 16 * nb + lr, V - 1)];

  // slice loads: UA (h) and UB (W) chunks of 16 bytes per thread (BM and BN rows x 8 chunks)
  const char* hsrc = reinterpret_cast<const char*>(a.h);
  const char* wsrc = BF16 ? reinterpret_cast<const char*>(m.Wb) : reinterpret_cast<const char*>(m.Wf);
  const size_t rowb = (size_t)Kpad * ESZ;
  const unsigned rowb32 = (unsigned)rowb;  // h and W each stay below 4 GiB (checked at launch)
  // slices in flight: register sets 0 and 1 (set 1 only with DEEP)
  uint4 ra0[UA], rb0[UB], ra1[UA], rb1[UB];
  auto gload = [&](int s, int set) {
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const int c = tid + NT * u, row = c >> 3, part = c & 7;
      const size_t off = (size_t)s * kJSlice + part * 16;
      // Rows past the batch or the padded vocabulary read the last valid row: their
      // products land only in rows and columns the epilogue never writes.  (No
      // branches around the loads, so their waits stay exact.)
      // (32-bit offsets from the uniform bases: one register per load address)
      const int hr = min(r0 + row, a.R - 1), wr_ = min(c0 + row, Vpad - 1);
      const uint4 vb = *reinterpret_cast<const uint4*>(wsrc + ((unsigned)wr_ * rowb32 + (unsigned)off));
      if (set == 0)
        rb0[u] = vb;
      else
        rb1[u] = vb;
      if (u < UA) {
        const uint4 va = *reinterpret_cast<const uint4*>(hsrc + ((unsigned)hr * rowb32 + (unsigned)off));
        if (set == 0)
          ra0[u < UA ? u : 0] = va;
        else
          ra1[u < UA ? u : 0] = va;
      }
    }
  };
  auto lstore = [&](int buf, int set) {
    unsigned char* base = smem + (size_t)buf * STAGE;
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const int c = tid + NT * u, row = c >> 3, part = c & 7;
      const int slot = (part ^ jswz(row & 15)) * 16;
      if (u < UA)
        *reinterpret_cast<uint4*>(base + (size_t)row * kJRow + slot) =
            set == 0 ? ra0[u < UA ? u : 0] : ra1[u < UA ? u : 0];
      *reinterpret_cast<uint4*>(base + (size_t)(BM + row) * kJRow + slot) = set == 0 ? rb0[u] : rb1[u];
    }
  };
  f32x4 acc[MBW][4];
#pragma unroll
  for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  // one slice of MFMAs from LDS buffer buf; fragments: lane (lr, lg) reads 16 bytes
  // of row lr of a block at byte 64 j + 16 lg of the slice (bf16: k-step j of 32;
  // fp32: group j of 16, the four values feeding four k-steps)
  auto compute = [&](int buf) {
    const unsigned char* base = smem + (size_t)buf * STAGE;
    const unsigned char* abase = base + (size_t)(16 * MBW * wr + lr) * kJRow;
    const unsigned char* bbase = base + (size_t)(BM + 64 * wc + lr) * kJRow;
    const int cs = (lg ^ jswz(lr)) * 16;  // chunk lg (j = 0) or 4 + lg (j = 1), swizzled
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      uint4 fa[MBW], fb[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) fb[q] = *reinterpret_cast<const uint4*>(bbase + (size_t)16 * q * kJRow + (cs ^ (64 * j)));
      if (BF16) {
        // row blocks in groups of 4: with 8 row blocks, the fragments of the second
        // group are read after the first group's MFMAs (fewer live registers)
        constexpr int GB = MBW < 4 ? MBW : 4;
#pragma unroll
        for (int g = 0; g < MBW; g += GB) {
#pragma unroll
          for (int q = g; q < g + GB; ++q)
            fa[q] = *reinterpret_cast<const uint4*>(abase + (size_t)16 * q * kJRow + (cs ^ (64 * j)));
#pragma unroll
          for (int mb = g; mb < g + GB; ++mb)
#pragma unroll
            for (int nb = 0; nb < 4; ++nb)
              acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(fa[mb]), as_bf16x8(fb[nb]),
                                                                    acc[mb][nb], 0, 0, 0);
          if (MBW > 4) __builtin_amdgcn_sched_barrier(0);
        }
      } else {
#pragma unroll
        for (int q = 0; q < MBW; ++q)
          fa[q] = *reinterpret_cast<const uint4*>(abase + (size_t)16 * q * kJRow + (cs ^ (64 * j)));
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) {
              const float av = __uint_as_float(u == 0 ? fa[mb].x : u == 1 ? fa[mb].y : u == 2 ? fa[mb].z : fa[mb].w);
              const float bv = __uint_as_float(u == 0 ? fb[nb].x : u == 1 ? fb[nb].y : u == 2 ? fb[nb].z : fb[nb].w);
              acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, acc[mb][nb], 0, 0, 0);
            }
      }
    }
  };
  const int nsl = (int)(rowb / kJSlice);  // Kpad is a multiple of 512: 8 (bf16) or 16 (fp32) per 512 (even)
  if constexpr (DEEP) {
    // Slice s + 2 is requested before the MFMAs of slice s, so each fetch has two
    // slices of MFMAs to land; slice s + 1 goes to the other LDS buffer after them.
    // (The scheduling barriers keep each fetch ahead of the MFMAs and LDS writes that
    // follow it, where the compiler would otherwise sink it.)
    gload(0, 0);
    gload(1, 1);
    __builtin_amdgcn_sched_barrier(0);
    lstore(0, 0);
    __syncthreads();
    for (int s = 0; s + 2 < nsl; s += 2) {
      gload(s + 2, 0);
      __builtin_amdgcn_sched_barrier(0);
      compute(0);
      lstore(1, 1);
      __syncthreads();
      gload(s + 3, 1);
      __builtin_amdgcn_sched_barrier(0);
      compute(1);
      lstore(0, 0);
      __syncthreads();
    }
    compute(0);  // the last two slices
    lstore(1, 1);
    __syncthreads();
    compute(1);
  } else {
    gload(0, 0);
    lstore(0, 0);
    __syncthreads();
    for (int s = 0; s < nsl; s += 2) {
      if (s + 1 < nsl) gload(s + 1, 0);
      __builtin_amdgcn_sched_barrier(0);
      compute(0);
      if (s + 1 < nsl) lstore(1, 0);
      __syncthreads();
      if (s + 2 < nsl) gload(s + 2, 0);
      __builtin_amdgcn_sched_barrier(0);
      compute(1);
      if (s + 2 < nsl) lstore(0, 0);
      __syncthreads();
    }
  }

  // epilogue of this wave's vocabulary tile (none beyond the padded vocabulary)
  if (vt >= nvt) return;
  const int nsub = nvt * (kJoinerBN / 16);
  // FULL: every column of the tile is a label (all but the last tile), so no
  // per-column validity selects
  auto epilogue = [&](auto full_tag) {
    constexpr bool FULL = decltype(full_tag)::value;
    float bias[4];
    bool cvalid[4];
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
      const int col = 64 * vt + 16 * nb + lr;
      cvalid[nb] = FULL || col < V;
      bias[nb] = cvalid[nb] ? bias_r[nb] : 0.f;
    }
#pragma unroll
    for (int mb = 0; mb < MBW; ++mb) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = 16 * MBW * wr + 16 * mb + 4 * lg + i;  // the 16 lanes of a DPP row share it
        const bool ract = s_act[row];
        float z[4];
        float mx = -INFINITY;
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) {
          z[nb] = cvalid[nb] ? acc[mb][nb][i] + bias[nb] : -INFINITY;
          mx = fmaxf(mx, z[nb]);
        }
        const float M = row16_max(mx);
        // sum of e^(z - M) on the base-2 exponential: (z - M) log2(e) <= 0, and its
        // rounding moves a term by a few ulp at most
        float e = 0.f;
#pragma unroll
        for (int nb = 0; nb < 4; ++nb)
          e += cvalid[nb] ? __builtin_amdgcn_exp2f((z[nb] - M) * kLog2e) : 0.f;
        const float S = row16_sum(e);
        if (ract && lr == 0) a.stats[(size_t)(r0 + row) * nvt + vt] = make_float2(M, S);
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) {
          const int col = 64 * vt + 16 * nb + lr;
          if (!TOPK) {
            if (ract && cvalid[nb]) a.logits[(size_t)(r0 + row) * (nvt * kJoinerBN) + col] = z[nb];
          } else {
            // each row's best KT labels of this 16-column sub-tile (DPP row reductions)
            unsigned long long key = (cvalid[nb] && col >= 1)
                                         ? ((unsigned long long)f2ord(z[nb]) << 32) | (0xffffffffu - (unsigned)col)
                                         : 0ull;
            const size_t ob = ((size_t)(r0 + row) * nsub + vt * (kJoinerBN / 16) + nb) * a.KT;
            for (int q = 0; q < a.KT; ++q) {
              const unsigned long long best = row16_max_u64(key);
              if (ract && best != 0ull && key == best) {
                a.tk_z[ob + q] = z[nb];
                a.tk_c[ob + q] = col;
              }
              if (ract && best == 0ull && lr == 0) {
                a.tk_z[ob + q] = -INFINITY;
                a.tk_c[ob + q] = -1;
              }
              if (key == best) key = 0ull;
            }
          }
        }
        if (TOPK && ract && vt == 0 && lr == 0) a.z0[r0 + row] = z[0];
      }
    }
  };
  if (64 * vt + 64 <= V)
    epilogue(std::true_type{});
  else
    epilogue(std::false_type{});
}

__global__ void k_logp_rows(const float* __restrict__ logits, const float2* __restrict__ stats,
                            int nvt, int V, int Vpad, float* __restrict__ out) {
  const int r = blockIdx.x;
  __shared__ double s_lse;
  if (threadIdx.x == 0) {
    const float2* st = stats + (size_t)r * nvt;
    float M = -INFINITY;
    for (int i = 0; i < nvt; ++i) M = fmaxf(M, st[i].x);
    float S = 0.f;
    for (int i = 0; i < nvt; ++i) S += st[i].y == 0.f ? 0.f : st[i].y * expf(st[i].x - M);
    s_lse = lse_of(M, S);
  }
  __syncthreads();
  const double l = s_lse;
  for (int v = threadIdx.x; v < V; v += blockDim.x)
    out[(size_t)r * V + v] = logp_of(logits[(size_t)r * Vpad + v], l);
}

// ---------------------------------------------------------------------------
// search

// initial tuple ((blank, blank), start) and its joiner row for frame 0
__global__ __launch_bounds__(256) void k_init(ModelDev m, DecodeDev d, GraphDev g,
                                              int* __restrict__ trace) {
  const int b = blockIdx.x, tid = threadIdx.x;
  if (d.graphs) g = d.graphs[b];  // per-stream graphs
  if (tid == 0) {
    d.nsurv[b] = 1;
    d.surv_ctx[(size_t)b * d.Ns] = 0;
    d.surv_state[(size_t)b * d.Ns] = g.start;
    d.surv_score[(size_t)b * d.Ns] = 0.f;
    d.surv_row[(size_t)b * d.Ns] = 0;
    d.surv_rp[(size_t)b * d.Ns] = make_int2(g.rp[g.start], g.rp[g.start + 1]);
    d.nctx[b] = 1;
    d.ctx_list[(size_t)b * d.Nc] = 0;
    d.offset[b] = 0.0;
    if (trace) {
      int* p = trace + (size_t)b * d.Ns * 4;
      p[0] = 0;
      p[1] = g.start;
      p[2] = -1;
      p[3] = -1;
    }
  }
  if (d.len[b] > 0) {
    const int2 zero_off = make_int2(0, 0);  // context (blank, blank)
    const size_t esz = m.bf16 ? 2 : 4;
    write_h_rows<256>(m, d.enc + (size_t)b * d.T * m.C, 0, &zero_off, 1,
                      reinterpret_cast<char*>(d.h) + (size_t)b * d.Nc * m.Kpad * esz, m.Kpad, tid);
  }
}

// Start of a decode chunk (streaming decode): for each stream that advances in this
// chunk, the joiner rows of its current contexts from the chunk's first encoder
// frame (frame schedule: rows_needed), and for a stream still at its absolute frame
// 0 the trace row of its initial tuple.
__global__ __launch_bounds__(256) void k_resume(ModelDev m, DecodeDev d, GraphDev g,
                                                int* __restrict__ trace, int rows_needed) {
  __shared__ int2 s_off[kMaxStates];
  __shared__ int s_nc, s_ns;
  const int b = blockIdx.x, tid = threadIdx.x;
  if (d.len[b] == 0) return;
  if (d.graphs) g = d.graphs[b];  // per-stream graphs
  if (tid == 0) {
    s_nc = d.nctx[b];
    s_ns = d.nsurv[b];
    if (trace && d.base[b] == 0) {
      int* p = trace + (size_t)b * d.Ns * 4;
      p[0] = d.surv_ctx[(size_t)b * d.Ns];
      p[1] = d.surv_state[(size_t)b * d.Ns];
      p[2] = -1;
      p[3] = -1;
    }
  }
  __syncthreads();
  // the arc ranges of the survivors' states, from the graph this chunk decodes with
  for (int i = tid; i < s_ns; i += blockDim.x) {
    const size_t o = (size_t)b * d.Ns + i;
    const int st = d.surv_state[o];
    d.surv_rp[o] = make_int2(g.rp[st], g.rp[st + 1]);
  }
  if (!rows_needed) return;
  const int nc = s_nc;
  for (int j = tid; j < nc; j += blockDim.x) {
    const int c = d.ctx_list[(size_t)b * d.Nc + j], a = c / m.V;
    s_off[j] = make_int2(a * m.Kpad, (c - a * m.V) * m.Kpad);
  }
  __syncthreads();
  const size_t esz = m.bf16 ? 2 : 4;
  write_h_rows<256>(m, d.enc + (size_t)b * d.T * m.C, 0, s_off, nc,
                    reinterpret_cast<char*>(d.h) + (size_t)b * d.Nc * m.Kpad * esz, m.Kpad, tid);
}

struct SearchSmem {
  unsigned long long hk[kHashSlots];  // hash keys; also stages softmax partials
  unsigned long long hv[kHashSlots];
  unsigned long long uk[kChunk + kMaxStates];  // merged entries / small-path candidates
  unsigned long long uv[kChunk + kMaxStates];
  unsigned long long lk[kMaxStates];  // running best list
  unsigned long long lv[kMaxStates];
  int s_ctx[kMaxStates], s_bprev[kMaxStates], s_state[kMaxStates], s_row[kMaxStates];
  int s_base[kMaxStates], s_off[kMaxStates + 1];
  float s_score[kMaxStates];
  double s_lse[kMaxStates];
  uint4 fent[kMaxStates];    // final stage: (ctx, state, score bits, context-score bits)
  int fflg[kMaxStates];      // bit 0 in beam, bit 1 first tuple of its context, bit 2 kept
  float wmax[4];
  int n_ctx_list[kMaxStates];
  int2 n_rowoff[kMaxStates];  // (a * Kpad, b * Kpad) of each next-frame context (a, b)
  float rk_z[kMaxTopK * kMaxTopK];  // trivial graph: each row's best labels over all tiles
  int rk_c[kMaxTopK * kMaxTopK];
  float s_z0[kMaxTopK];
  alignas(16) unsigned hist[256];  // radix counts; direct path: packed scores
  int wsum[4];
  int misc[8];
  int g_src[4];              // grouped fast path: decoder-row source of each new context row
  int ns, nc, nU, nL, n_gt, n_eq, nK, nC;
  float best;
  double off_d;              // the stream's fp64 score offset (kept here between frames)
  // encoder frame t+1 of this stream (next frame's joiner rows).  Last member: the
  // frame search kernel allocates only its first Kpad entries, which keeps two of its
  // workgroups within one CU's LDS
  alignas(16) float enc_next[kMaxDim];
};

// Copies n dwords from global memory into LDS on the global-load-to-LDS path: no
// registers held, 64 dwords per wave and instruction, all in flight together.  The
// caller waits for the vector memory counter before the barrier that publishes them.
typedef __attribute__((address_space(1))) void global_void;
typedef __attribute__((address_space(3))) void lds_void;
__device__ __forceinline__ void lds_stage_dwords(void* dst, const void* src, int n, int tid) {
  const int lane = tid & 63, wave = tid >> 6;
  const unsigned* gs = reinterpret_cast<const unsigned*>(src);
  unsigned* ld = reinterpret_cast<unsigned*>(dst);
  for (int base = 64 * wave; base < n; base += kSearchThreads)  // wave-uniform LDS base
    if (base + lane < n)
      __builtin_amdgcn_global_load_lds((global_void*)(gs + base + lane), (lds_void*)(ld + base), 4, 0, 0);
}
// s_waitcnt vmcnt(0) (expcnt and lgkmcnt left free)
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

__device__ __forceinline__ uint32_t hash_slot(unsigned long long key) {
  return (uint32_t)((key * 0x9E3779B97F4A7C15ull) >> (64 - kHashBits));
}

__device__ __forceinline__ void hash_insert(SearchSmem& s, unsigned long long key,
                                            unsigned long long val) {
  uint32_t h = hash_slot(key);
  for (;;) {
    const unsigned long long prev = atomicCAS(&s.hk[h], kEmpty, key);
    if (prev == kEmpty || prev == key) {
      atomicMax(&s.hv[h], val);
      return;
    }
    h = (h + 1) & (kHashSlots - 1);
  }
}

// Block-wide: value v* with #(v > v*) < k <= #(v >= v*) over entries i < n for
// which get(i, v) is true.  Requires 1 <= k <= that count.  NBITS in {32, 64}.
template <int NBITS, class Get>
__device__ unsigned long long kth_largest(SearchSmem& s, int n, int k, Get get) {
  unsigned long long prefix = 0, mask = 0;
  for (int shift = NBITS - 8; shift >= 0; shift -= 8) {
    for (int i = threadIdx.x; i < 256; i += blockDim.x) s.hist[i] = 0;
    __syncthreads();
    for (int i = threadIdx.x; i < n; i += blockDim.x) {
      unsigned long long v;
      if (!get(i, v)) continue;
      if ((v & mask) != prefix) continue;
      atomicAdd(&s.hist[(v >> shift) & 255], 1u);
    }
    __syncthreads();
    if (threadIdx.x < 64) {
      const int lane = threadIdx.x;
      unsigned c[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) c[j] = s.hist[255 - 4 * lane - j];
      const unsigned sum = c[0] + c[1] + c[2] + c[3];
      const unsigned incl = wave_incl_scan_u32(sum);
      const unsigned long long bal = __ballot(incl >= (unsigned)k);
      const int first = __ffsll((long long)bal) - 1;
      if (lane == first) {
        unsigned cum = incl - sum;
        int dsel = 255 - 4 * lane - 3;
        unsigned knew = k - cum;
        for (int j = 0; j < 4; ++j) {
          if (cum + c[j] >= (unsigned)k) {
            dsel = 255 - 4 * lane - j;
            knew = k - cum;
            break;
          }
          cum += c[j];
        }
        s.misc[0] = dsel;
        s.misc[1] = (int)knew;
      }
    }
    __syncthreads();
    const int dsel = s.misc[0];
    k = s.misc[1];
    prefix |= (unsigned long long)dsel << shift;
    mask |= 255ull << shift;
    __syncthreads();
  }
  return prefix;
}

// Top `Ns` of the nU > Ns merged entries in uk/uv by (score desc, key asc) into lk/lv,
// by an exact 8-bit radix select of the score code (several passes) and of the key
// among equal scores.
__device__ __attribute__((noinline)) void select_top_radix(SearchSmem& s, int nU, int Ns) {
  const int tid = threadIdx.x;
  const unsigned theta = (unsigned)kth_largest<32>(s, nU, Ns, [&](int i, unsigned long long& v) {
    v = s.uv[i] >> 32;
    return true;
  });
  if (tid == 0) {
    s.n_gt = 0;
    s.n_eq = 0;
    s.nL = 0;
  }
  __syncthreads();
  for (int i = tid; i < nU; i += blockDim.x) {
    const unsigned so = (unsigned)(s.uv[i] >> 32);
    if (so > theta) atomicAdd(&s.n_gt, 1);
    else if (so == theta) atomicAdd(&s.n_eq, 1);
  }
  __syncthreads();
  const int m_need = Ns - s.n_gt;
  unsigned long long keythr = kEmpty;
  if (s.n_eq > m_need) {
    const unsigned long long vk = kth_largest<64>(s, nU, m_need, [&](int i, unsigned long long& v) {
      if ((unsigned)(s.uv[i] >> 32) != theta) return false;
      v = ~s.uk[i];
      return true;
    });
    keythr = ~vk;
  }
  for (int i = tid; i < nU; i += blockDim.x) {
    const unsigned so = (unsigned)(s.uv[i] >> 32);
    if (so > theta || (so == theta && s.uk[i] <= keythr)) {
      const int p = atomicAdd(&s.nL, 1);
      s.lk[p] = s.uk[i];
      s.lv[p] = s.uv[i];
    }
  }
  __syncthreads();
}

// Top `Ns` of the nU merged entries in uk/uv by (score desc, key asc) into lk/lv.  One
// histogram pass over the score codes, binned across their own range (min to max), finds
// the bin holding the Ns-th entry: entries in higher bins are kept, and the bin's own
// entries (listed in hk/hv, free after the merge) are ranked exactly among themselves.
// A bin of more than one entry per thread (a narrow or degenerate range) falls back to
// the radix select.
__device__ __forceinline__ void select_top(SearchSmem& s, int nU, int Ns) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (nU <= Ns) {
    for (int i = tid; i < nU; i += blockDim.x) {
      s.lk[i] = s.uk[i];
      s.lv[i] = s.uv[i];
    }
    if (tid == 0) s.nL = nU;
    __syncthreads();
    return;
  }
  unsigned lo = 0xffffffffu, hi = 0u;
  for (int i = tid; i < nU; i += blockDim.x) {
    const unsigned c = (unsigned)(s.uv[i] >> 32);
    lo = min(lo, c);
    hi = max(hi, c);
  }
  lo = wave_min_u32(lo);
  hi = wave_max_u32(hi);
  if (lane == 0) {
    s.misc[wave] = (int)lo;
    s.misc[4 + wave] = (int)hi;
  }
  for (int i = tid; i < 256; i += blockDim.x) s.hist[i] = 0u;
  if (tid == 0) {
    s.nL = 0;
    s.n_eq = 0;
  }
  __syncthreads();
  lo = min(min((unsigned)s.misc[0], (unsigned)s.misc[1]), min((unsigned)s.misc[2], (unsigned)s.misc[3]));
  hi = max(max((unsigned)s.misc[4], (unsigned)s.misc[5]), max((unsigned)s.misc[6], (unsigned)s.misc[7]));
  const unsigned range = hi - lo;
  const int shift = range < 256u ? 0 : 24 - __clz((int)range);  // (range >> shift) < 256
  auto bin = [&](unsigned c) { return (c - lo) >> shift; };
  for (int i = tid; i < nU; i += blockDim.x) atomicAdd(&s.hist[bin((unsigned)(s.uv[i] >> 32))], 1u);
  __syncthreads();
  if (tid < 64) {
    // the bin holding the Ns-th largest code, scanning from the top bin
    unsigned c[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) c[j] = s.hist[255 - 4 * lane - j];
    const unsigned sum = c[0] + c[1] + c[2] + c[3];
    const unsigned incl = wave_incl_scan_u32(sum);
    const int first = __ffsll((long long)__ballot(incl >= (unsigned)Ns)) - 1;
    if (lane == first) {
      unsigned cum = incl - sum;
      int bsel = 255 - 4 * lane - 3;
      for (int j = 0; j < 4; ++j) {
        if (cum + c[j] >= (unsigned)Ns) {
          bsel = 255 - 4 * lane - j;
          break;
        }
        cum += c[j];
      }
      s.misc[0] = bsel;
      s.misc[1] = Ns - (int)cum;  // entries still needed from that bin (>= 1)
    }
  }
  __syncthreads();
  const unsigned bsel = (unsigned)s.misc[0];
  const int need = s.misc[1], inb = (int)s.hist[bsel];
  if (inb > kSearchThreads) {  // uniform
    select_top_radix(s, nU, Ns);
    return;
  }
  for (int i = tid; i < nU; i += blockDim.x) {
    const unsigned b = bin((unsigned)(s.uv[i] >> 32));
    if (b > bsel) {
      const int p = atomicAdd(&s.nL, 1);
      s.lk[p] = s.uk[i];
      s.lv[p] = s.uv[i];
    } else if (b == bsel) {
      const int q = atomicAdd(&s.n_eq, 1);
      s.hk[q] = s.uk[i];
      s.hv[q] = s.uv[i];
    }
  }
  __syncthreads();
  if (tid < inb) {
    const unsigned long long k = s.hk[tid], v = s.hv[tid];
    const unsigned so = (unsigned)(v >> 32);
    int r = 0;
    for (int j = 0; j < inb; ++j) {
      const unsigned sj = (unsigned)(s.hv[j] >> 32);
      r += (int)((sj > so) | ((sj == so) & (s.hk[j] < k)));
    }
    if (r < need) {
      const int p = atomicAdd(&s.nL, 1);
      s.lk[p] = k;
      s.lv[p] = v;
    }
  }
  __syncthreads();
}

// Candidate c of the flattened list (trivial: survivor-major blank then per-tile
// top labels; general: blanks then arcs).  Returns false if c is an empty slot.
struct CandIdx {
  int i, pos, lab, dest, arc;
  float q, z;
};

// Result of the one-wave selection for one lane (one candidate).
struct WaveSel {
  unsigned ci, st;          // the candidate's key (context, state)
  float sc;                 // its score
  unsigned long long v;     // score << 32 | ~back-pointer
  int keep2, pos;           // kept, and its canonical position (= its context row)
  int src;                  // i * KT + q for label q of survivor i; -(1 + row) for the
                            // blank of a survivor on context row `row`
  float best;               // the frame's best score (uniform)
  int nk;                   // tuples kept (uniform)
};

// Trivial graph, at most 64 candidates (survivor-major: blank, then the row's KT
// best labels): one wave, one candidate per lane.  The key is the context alone
// (one graph state), so after the max-merge every context has one tuple: the
// context score is the tuple's score, the max-contexts rank equals the max-states
// rank among the in-beam tuples, and a tuple is kept iff it represents its key,
// ranks below min(max_states, max_contexts) and lies within the beam of the best.
// The kept tuples are extracted in rank order: each round takes the candidate with
// the largest (score, then smaller key, then smaller back-pointer), which is its
// key's representative and the best remaining one, and retires every candidate
// with that key; the rounds stop at the rank limit, at the beam or when nothing is
// left.  A kept tuple's canonical position is the number of kept keys below its
// own.  Survivors are read at offset sb of the survivor arrays, with the row
// normalisers and each row's best labels (rk_z, rk_c, s_z0).  publish: also write
// n_ctx_list, nK, nC and best.
// KTC > 0: the number of labels per row is the compile-time KTC (KT is ignored), and
// survivor i sits on context row i (every context holds one tuple), so that every LDS
// read of a lane is issued at once.
template <int KTC = 0>
__device__ __forceinline__ WaveSel trivial_select_wave(SearchSmem& s, int ns, int KT_, int V, int Ns,
                                                       int Nc, float beam, unsigned stride_tb,
                                                       int lane, int sb, bool publish) {
  const int KT = KTC > 0 ? KTC : KT_;
  const int P = 1 + KT, n = ns * P;
  unsigned long long myk = kEmpty, myv = 0ull;
  int src = 0;
  if (KTC > 0) {
    if (lane < n) {
      const int i = lane / P, q = lane - i * P - 1;
      const int e = i * KT + max(q, 0);
      const double lse = s.s_lse[i];
      const float sc0 = s.s_score[sb + i];
      const int lab = s.rk_c[e];
      const float zl = s.rk_z[e], z0 = s.s_z0[i];
      const int st = s.s_state[sb + i], ctx = s.s_ctx[sb + i], bp = s.s_bprev[sb + i];
      if (q < 0) {
        const float sc = sc0 + logp_of(z0, lse);
        myk = ((unsigned long long)(unsigned)st << 32) | (unsigned)ctx;
        myv = ((unsigned long long)f2ord(sc) << 32) | (0xffffffffu - (unsigned)i * stride_tb);
        src = -(1 + i);
      } else {
        if (lab >= 0) {
          const float sc = sc0 + logp_of(zl, lse);
          myk = (unsigned)bp * (unsigned)V + (unsigned)lab;
          myv = ((unsigned long long)f2ord(sc) << 32) |
                (0xffffffffu - ((unsigned)i * stride_tb + (unsigned)lab));
        }
        src = e;
      }
    }
  } else if (lane < n) {
    const int i = lane / P, q = lane - i * P - 1;
    const int row = s.s_row[sb + i];
    const double lse = s.s_lse[row];
    if (q < 0) {
      const float sc = s.s_score[sb + i] + logp_of(s.s_z0[row], lse);
      myk = ((unsigned long long)(unsigned)s.s_state[sb + i] << 32) | (unsigned)s.s_ctx[sb + i];
      myv = ((unsigned long long)f2ord(sc) << 32) | (0xffffffffu - (unsigned)i * stride_tb);
      src = -(1 + row);
    } else {
      const int lab = s.rk_c[row * KT + q];
      if (lab >= 0) {
        const float sc = s.s_score[sb + i] + logp_of(s.rk_z[row * KT + q], lse);
        myk = (unsigned)s.s_bprev[sb + i] * (unsigned)V + (unsigned)lab;
        myv = ((unsigned long long)f2ord(sc) << 32) |
              (0xffffffffu - ((unsigned)i * stride_tb + (unsigned)lab));
      }
      src = i * KT + q;
    }
  }
  const unsigned vhi = (unsigned)(myv >> 32), vlo = (unsigned)myv;
  const int K = min(Ns, Nc);
  bool alive = myk != kEmpty;
  int nk = 0, keep2 = 0, pos = 0;
  float bst = -INFINITY;
  for (int r = 0; r < K; ++r) {
    const unsigned mo = wave_max_u32(alive ? vhi : 0u);
    if (mo == 0u) break;  // no candidate left
    const float scr = ord2f(mo);
    if (r == 0) bst = scr;
    else if (!(scr >= bst - beam)) break;  // ranks only fall from here on
    unsigned long long bal = __ballot(alive && vhi == mo);
    if (__popcll(bal) > 1) {  // equal scores: the smaller key, then the smaller back-pointer
      const bool tie = alive && vhi == mo;
      const unsigned long long kmin = wave_min_u64(tie ? myk : ~0ull);
      bal = __ballot(tie && myk == kmin);
      if (__popcll(bal) > 1) {
        const unsigned vmax = wave_max_u32((tie && myk == kmin) ? vlo : 0u);
        bal = __ballot(tie && myk == kmin && vlo == vmax);
      }
    }
    const int wl = __ffsll((long long)bal) - 1;
    const unsigned long long kr =
        ((unsigned long long)(unsigned)__builtin_amdgcn_readlane((int)(myk >> 32), wl) << 32) |
        (unsigned)__builtin_amdgcn_readlane((int)(unsigned)myk, wl);
    // canonical positions: kept keys above the new one move up by one
    const unsigned long long below = __ballot(keep2 && myk < kr);
    if (keep2 && myk > kr) ++pos;
    if (lane == wl) {
      keep2 = 1;
      pos = __popcll(below);
    }
    alive = alive && myk != kr;
    ++nk;
  }
  if (publish) {
    if (keep2) s.n_ctx_list[pos] = (int)(unsigned)myk;
    if (lane == 0) {
      s.nK = nk;
      s.nC = nk;
      s.best = bst;
    }
  }
  WaveSel r;
  r.ci = (unsigned)myk;
  r.st = (unsigned)(myk >> 32);
  r.sc = ord2f(vhi);
  r.v = myv;
  r.keep2 = keep2;
  r.pos = pos;
  r.src = src;
  r.best = bst;
  r.nk = nk;
  return r;
}

// One frame of the search for stream b (t < L), one workgroup.  FUSED (the
// per-stream kernels): the survivors are in LDS and so are the frame's logit rows
// (zl, [row][Vpad], -inf beyond V); the next frame's joiner rows go to LDS (hl,
// row stride hstride) and the survivors stay in LDS; the global survivor arrays
// are written at the stream's last frame only.  prestats: the normalisers
// (s_lse) and, for the trivial graph, the best labels and blank logits are
// already in LDS.  writer: this workgroup writes the stream's history, trace,
// survivors and offset (a stream run redundantly by several workgroups has one
// writer).  enc_ready: the caller has put encoder frame t+1 in enc_next.  dspec
// (trivial graph, max_states = 4, FUSED): LDS decoder rows, [16][Kpad] of the label
// candidates (gathered by waves 1-3 while wave 0 selects) and [2][4][Kpad] of the
// contexts (buffer dcur_buf holds the current ones); the next frame's joiner rows
// are built from them (enc_next must be zero from C to Kpad).  fb: the stream's
// absolute index of frame 0 of this call (history and trace rows; chunked decode).
template <bool TRIV, bool FUSED>
__device__ __forceinline__ void search_frame(const ModelDev& m, const GraphDev& g,
                                             const DecodeDev& d, float beam, int t, int L, int b,
                                             int* __restrict__ trace, SearchSmem& s, void* hl,
                                             int hstride, const float* zl, bool prestats = false,
                                             bool writer = true, bool enc_ready = false,
                                             float* dspec = nullptr, int dcur_buf = 0,
                                             int fb = 0) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int Ns = d.Ns, Nc = d.Nc, V = m.V, nvt = d.nvt;
  const unsigned stride_tb = (unsigned)g.maxdeg + 1u;
  const size_t row0 = (size_t)b * Nc;

  // ---- loads that do not depend on the survivor count ----
  if (!FUSED && tid == 0) {
    s.ns = d.nsurv[b];
    s.nc = d.nctx[b];
    if (writer) s.off_d = d.offset[b];  // read now, updated at the end
  }
  float2* stage = reinterpret_cast<float2*>(s.hk);  // softmax partials, [Nc][nvt]
  const bool staged = Nc * nvt <= kStatStage;
  if (!FUSED && staged) lds_stage_dwords(stage, d.stats + row0 * nvt, 2 * Nc * nvt, tid);
  if (!FUSED)
    for (int i = tid; i < Ns; i += blockDim.x) {
      const size_t o = (size_t)b * Ns + i;
      s.s_ctx[i] = d.surv_ctx[o];
      s.s_state[i] = d.surv_state[o];
      s.s_row[i] = d.surv_row[o];
      s.s_score[i] = d.surv_score[o];
    }
  // general graph: the arc ranges of the survivors' states, stored with them by the
  // previous frame (one survivor per thread; the persistent kernels, whose survivors
  // stay in LDS, read them from the graph below)
  static_assert(kMaxStates <= kSearchThreads, "one survivor per thread");
  int rp_lo = 0, rp_hi = 0;
  if (!TRIV && !FUSED && tid < Ns) {
    const int2 r = d.surv_rp[(size_t)b * Ns + tid];
    rp_lo = r.x;
    rp_hi = r.y;
  }
  if (t + 1 < L && !enc_ready) {
    lds_stage_dwords(s.enc_next, d.enc + ((size_t)b * d.T + t + 1) * m.C, m.C, tid);
  }
  // trivial graph: the joiner's per-tile best labels of this stream's rows
  const int E = TRIV ? nvt * (kJoinerBN / 16) * d.KT : 0;
  float* tz = reinterpret_cast<float*>(s.uk);
  int* tc = reinterpret_cast<int*>(s.uv);
  const bool tstaged = TRIV && Nc * E <= kTopkStage;
  if (TRIV && !FUSED) {
    if (tstaged)
      for (int i = tid; i < Nc * E; i += blockDim.x) {
        tz[i] = d.tk_z[row0 * E + i];
        tc[i] = d.tk_c[row0 * E + i];
      }
    for (int j = tid; j < Nc; j += blockDim.x) s.s_z0[j] = d.z0[row0 + j];
  }
  wait_vmem();  // the staged partials, encoder frame and label lists have landed in LDS
  __syncthreads();
  const int ns = s.ns, nc = s.nc;
  if (!TRIV && FUSED && tid < ns) {  // requested before the normalisers, which overlap them
    const int st = s.s_state[tid];
    rp_lo = g.rp[st];
    rp_hi = g.rp[st + 1];
  }
  // log-softmax normaliser of each context row: 16 threads (one DPP row) per row,
  // 16 rows at a time
  for (int j0 = 0; !FUSED && j0 < nc; j0 += kSearchThreads / 16) {
    const int j = j0 + (tid >> 4), l16 = tid & 15;
    const bool rv = j < nc;
    float M = -INFINITY;
    for (int i = l16; rv && i < nvt; i += 16)
      M = fmaxf(M, staged ? stage[j * nvt + i].x : d.stats[(row0 + j) * nvt + i].x);
    M = row16_max(M);
    float S = 0.f;
    for (int i = l16; rv && i < nvt; i += 16) {
      const float2 p = staged ? stage[j * nvt + i] : d.stats[(row0 + j) * nvt + i];
      S += p.y == 0.f ? 0.f : p.y * expf(p.x - M);
    }
    S = row16_sum(S);
    if (rv && l16 == 0) s.s_lse[j] = lse_of(M, S);
  }
  if (FUSED && !prestats) {
    // straight from the logit rows: normaliser, and for the trivial graph the blank
    // logit and the row's best KT labels (labels are unique within a row, so round q
    // takes the largest key below round q-1's); one wave per row, each lane holding
    // its columns lane, lane + 64, ... in registers (at most kStreamMaxV / 64)
    const int Vpad = m.Vpad, KT = d.KT;
    constexpr int NPL = kStreamMaxV / 64;
    for (int j = wave; j < nc; j += 4) {
      const float* zr = zl + (size_t)j * Vpad;
      float zv[NPL];
#pragma unroll
      for (int i = 0; i < NPL; ++i) {
        const int c = 64 * i + lane;
        const float z = zr[min(c, Vpad - 1)];
        zv[i] = c < Vpad ? z : -INFINITY;
      }
      float M0 = fmaxf(zv[0], zv[1]), M1 = fmaxf(zv[2], zv[3]);
#pragma unroll
      for (int i = 4; i < NPL; i += 2) {
        M0 = fmaxf(M0, zv[i]);
        M1 = fmaxf(M1, zv[i + 1]);
      }
      const float M = wave_max_f(fmaxf(M0, M1));
      float S0 = 0.f, S1 = 0.f;
#pragma unroll
      for (int i = 0; i < NPL; i += 2) {
        S0 += __expf(zv[i] - M);
        S1 += __expf(zv[i + 1] - M);
      }
      const float S = wave_sum_f(S0 + S1);
      if (lane == 0) s.s_lse[j] = lse_of(M, S);
      if (TRIV) {
        // best KT labels by (logit desc, label asc): each lane's best remaining slot
        // (ties to its smaller column), the wave maximum of the order-preserving
        // code, ties across lanes to the smaller column; the winner's slot retires
        unsigned o[NPL];
#pragma unroll
        for (int i = 0; i < NPL; ++i) {
          const int c = 64 * i + lane;
          o[i] = (c >= 1 && c < V) ? f2ord(zv[i]) : 0u;
        }
        for (int q = 0; q < KT; ++q) {
          unsigned lm = 0u;
          int li = 0;
#pragma unroll
          for (int i = 0; i < NPL; ++i)
            if (o[i] > lm) {
              lm = o[i];
              li = i;
            }
          const unsigned mo = wave_max_u32(lm);
          float zq = -INFINITY;
          int cq = -1;
          if (mo != 0u) {
            const unsigned cand = lm == mo ? (unsigned)(64 * li + lane) : 0xffffffffu;
            const unsigned long long bal = __ballot(lm == mo);
            const unsigned cmin = __popcll(bal) == 1
                                      ? (unsigned)__builtin_amdgcn_readlane((int)cand, __ffsll((long long)bal) - 1)
                                      : wave_min_u32(cand);
            zq = ord2f(mo);
            cq = (int)cmin;
#pragma unroll
            for (int i = 0; i < NPL; ++i)
              if (lane == (int)(cmin & 63) && i == (int)(cmin >> 6)) o[i] = 0u;
          }
          if (lane == 0) {
            s.rk_z[j * KT + q] = zq;
            s.rk_c[j * KT + q] = cq;
          }
        }
        if (lane == 0) s.s_z0[j] = zv[0];
      }
    }
  }
  if (TRIV) {
    for (int i = tid; i < ns; i += blockDim.x) {
      s.s_bprev[i] = s.s_ctx[i] % V;
      s.s_base[i] = 0;
    }
    // each row's best KT labels over all tiles (labels are unique within a row, so
    // round q takes the largest key below round q-1's)
    const int KT = d.KT;
    for (int j = wave; !FUSED && j < nc; j += 4) {
      unsigned long long prev = ~0ull;
      for (int q = 0; q < KT; ++q) {
        unsigned long long mine = 0ull;
        for (int e = lane; e < E; e += 64) {
          const int c = tstaged ? tc[j * E + e] : d.tk_c[(row0 + j) * E + e];
          if (c < 0) continue;
          const float z = tstaged ? tz[j * E + e] : d.tk_z[(row0 + j) * E + e];
          const unsigned long long key =
              ((unsigned long long)f2ord(z) << 32) | (0xffffffffu - (unsigned)c);
          if (key < prev && key > mine) mine = key;
        }
        const unsigned long long best = wave_max_u64(mine);
        if (lane == 0) {
          s.rk_z[j * KT + q] = best ? ord2f((unsigned)(best >> 32)) : -INFINITY;
          s.rk_c[j * KT + q] = best ? (int)(0xffffffffu - (unsigned)best) : -1;
        }
        prev = best ? best : 1ull;
      }
    }
  } else if (tid < ns) {
    s.s_bprev[tid] = s.s_ctx[tid] % V;
    s.s_base[tid] = rp_lo;
    s.s_off[tid + 1] = rp_hi - rp_lo;
  }
  if (tid == 0) {
    s.s_off[0] = 0;
    s.nL = 0;
  }
  __syncthreads();

  // What the selection leaves each thread: the kept tuple it places (if any), its
  // canonical position and context row, and the frame's best score.
  float best;
  unsigned my_ci = 0xffffffffu, my_st = 0xffffffffu;
  float my_sc = -INFINITY;
  unsigned long long my_v = 0ull;  // score << 32 | ~back-pointer of the placed tuple
  int my_keep2 = 0, my_pos = 0, my_crow = 0, my_first = 0;

  if (TRIV && ns * (1 + d.KT) <= 64) {
    // trivial graph, at most 64 candidates: one wave (trivial_select_wave)
    if (wave == 0) {
      const WaveSel r = trivial_select_wave(s, ns, d.KT, V, Ns, Nc, beam, stride_tb, lane, 0, true);
      if (dspec && r.keep2) s.g_src[r.pos] = r.src;
      my_keep2 = r.keep2;
      my_pos = r.pos;
      my_crow = r.pos;
      my_first = 1;
      my_ci = r.ci;
      my_st = r.st;
      my_sc = r.sc;
      my_v = r.v;
    } else if (dspec && t + 1 < L) {
      // decoder rows ReLU(P0[a] + P1[b]) of every label candidate (survivor i on context
      // row i, label q): unconditional LDS reads, absent entries mapped into row 0
      const int kq4 = m.Kpad / 4;
      int pa[4], pb[4][4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int a = s.s_bprev[i];
        pa[i] = (i < ns && (unsigned)a < (unsigned)V) ? a : 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int c = s.rk_c[i * 4 + q];
          pb[i][q] = (i < ns && (unsigned)c < (unsigned)V) ? c : 0;
        }
      }
      const float4* __restrict__ P0 = reinterpret_cast<const float4*>(m.P0);
      const float4* __restrict__ P1 = reinterpret_cast<const float4*>(m.P1);
      float4* dc4 = reinterpret_cast<float4*>(dspec);
      for (int kq = tid - 64; kq < kq4; kq += kSearchThreads - 64) {
        float4 p0[4], p1[4][4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          p0[i] = P0[(size_t)pa[i] * kq4 + kq];
#pragma unroll
          for (int q = 0; q < 4; ++q) p1[i][q] = P1[(size_t)pb[i][q] * kq4 + kq];
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            dc4[(4 * i + q) * kq4 + kq] =
                make_float4(fmaxf(p0[i].x + p1[i][q].x, 0.f), fmaxf(p0[i].y + p1[i][q].y, 0.f),
                            fmaxf(p0[i].z + p1[i][q].z, 0.f), fmaxf(p0[i].w + p1[i][q].w, 0.f));
      }
    }
    __syncthreads();
    best = s.best;
  } else {
  // exclusive offsets of each survivor's candidates (block scan over <= 256 entries)
  {
    const int per = TRIV ? d.KT : 0;
    const int v = tid < ns ? (TRIV ? per : s.s_off[tid + 1]) : 0;
    const int incl = (int)wave_incl_scan_u32((unsigned)v);
    if (lane == 63) s.wsum[wave] = incl;
    __syncthreads();
    int woff = 0;
    for (int w = 0; w < wave; ++w) woff += s.wsum[w];
    if (tid < ns) s.s_off[tid + 1] = woff + incl;
    __syncthreads();
  }
  const int N = ns + s.s_off[ns];

  // candidate c -> (survivor, position) and its score/key inputs; loads batched by the caller
  auto locate = [&](int c, int& i, int& pos) {
    if (c < ns) {
      i = c;
      pos = -1;
      return;
    }
    const int k = c - ns;
    int lo = 0, hi = ns - 1;  // largest i with s_off[i] <= k
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (s.s_off[mid] <= k) lo = mid; else hi = mid - 1;
    }
    i = lo;
    pos = k - s.s_off[i];
  };
  const float* zbase = FUSED ? zl : d.logits + row0 * (size_t)m.Vpad;
  // (key, value) of candidate c; key = kEmpty for an empty trivial-graph slot
  auto make_cand = [&](int c) -> ulonglong2 {
    int i, pos;
    locate(c, i, pos);
    const int row = s.s_row[i];
    const double lse = s.s_lse[row];
    float sc;
    unsigned nctx;
    int nst, tbpos;
    if (pos < 0) {
      const float z = TRIV ? s.s_z0[row] : zbase[(size_t)row * m.Vpad];
      sc = s.s_score[i] + logp_of(z, lse);
      nctx = (unsigned)s.s_ctx[i];
      nst = s.s_state[i];
      tbpos = 0;
    } else if (TRIV) {
      const int lab = s.rk_c[row * d.KT + pos];
      if (lab < 0) return make_ulonglong2(kEmpty, 0ull);
      sc = s.s_score[i] + logp_of(s.rk_z[row * d.KT + pos], lse);
      nctx = (unsigned)s.s_bprev[i] * (unsigned)V + (unsigned)lab;
      nst = 0;
      tbpos = lab;  // trivial graph: arc position = label - 1
    } else {
      const int j = s.s_base[i] + pos;
      const int lab = g.label[j];
      const float q = g.q[j];
      nst = g.dest[j];
      sc = (s.s_score[i] + q) + logp_of(zbase[(size_t)row * m.Vpad + lab], lse);
      nctx = (unsigned)s.s_bprev[i] * (unsigned)V + (unsigned)lab;
      tbpos = pos + 1;
    }
    const unsigned tb = (unsigned)i * stride_tb + (unsigned)tbpos;
    return make_ulonglong2(((unsigned long long)(unsigned)nst << 32) | nctx,
                           ((unsigned long long)f2ord(sc) << 32) | (0xffffffffu - tb));
  };

  // Beam pre-filter.  A candidate scoring below (best candidate - beam) can never
  // be kept, and dropping it changes neither the max-merge of the others nor their
  // ranks, so with a finite beam and a candidate set that fits uk/uv, all
  // candidates are made once, their maximum taken, and only those within the beam
  // are listed in hk/hv for merging and ranking (the hash path, when they are
  // still many, skips the others on insertion).
  int Nsel = N;
  bool listed = false;
  unsigned thr_ord = 0u;
  if (N > kDirectCands && beam < INFINITY && N <= kChunk + kMaxStates) {
    float lmax = -INFINITY;
    __syncthreads();  // trivial graph: uk/uv held the staged tile lists until here
    if (TRIV) {
      for (int c = tid; c < N; c += blockDim.x) {
        const ulonglong2 kv = make_cand(c);
        s.uk[c] = kv.x;
        s.uv[c] = kv.y;
        if (kv.x != kEmpty) lmax = fmaxf(lmax, ord2f((unsigned)(kv.y >> 32)));
      }
    } else {
      // make_cand for PF candidates per thread at a time, with each step's loads in
      // flight together: the arcs' (label, score, destination), then the logits they
      // select.  A blank candidate (or one past N) reads arc 0, which every graph
      // buffer holds, and drops it.
      constexpr int PF = 4;
      for (int c0 = tid; c0 < N; c0 += PF * kSearchThreads) {
        int ci[PF], cpos[PF], crow[PF], cj[PF];
#pragma unroll
        for (int u = 0; u < PF; ++u) {
          const int c = c0 + u * kSearchThreads;
          int i = 0, pos = -1;
          if (c < N) locate(c, i, pos);
          ci[u] = i;
          cpos[u] = pos;
          crow[u] = s.s_row[i];
          cj[u] = pos < 0 ? 0 : s.s_base[i] + pos;
        }
        int clab[PF], cdst[PF];
        float cq[PF];
#pragma unroll
        for (int u = 0; u < PF; ++u) {
          clab[u] = g.label[cj[u]];
          cq[u] = g.q[cj[u]];
          cdst[u] = g.dest[cj[u]];
        }
        float cz[PF];
#pragma unroll
        for (int u = 0; u < PF; ++u)
          cz[u] = zbase[(size_t)crow[u] * m.Vpad + (cpos[u] < 0 ? 0 : clab[u])];
#pragma unroll
        for (int u = 0; u < PF; ++u) {
          const int c = c0 + u * kSearchThreads;
          if (c < N) {
            const int i = ci[u], pos = cpos[u];
            const double lse = s.s_lse[crow[u]];
            float sc;
            unsigned nctx;
            int nst, tbpos;
            if (pos < 0) {
              sc = s.s_score[i] + logp_of(cz[u], lse);
              nctx = (unsigned)s.s_ctx[i];
              nst = s.s_state[i];
              tbpos = 0;
            } else {
              sc = (s.s_score[i] + cq[u]) + logp_of(cz[u], lse);
              nctx = (unsigned)s.s_bprev[i] * (unsigned)V + (unsigned)clab[u];
              nst = cdst[u];
              tbpos = pos + 1;
            }
            const unsigned tb = (unsigned)i * stride_tb + (unsigned)tbpos;
            const unsigned long long k = ((unsigned long long)(unsigned)nst << 32) | nctx;
            const unsigned long long v = ((unsigned long long)f2ord(sc) << 32) | (0xffffffffu - tb);
            s.uk[c] = k;
            s.uv[c] = v;
            lmax = fmaxf(lmax, ord2f((unsigned)(v >> 32)));
          }
        }
      }
    }
    lmax = wave_max_f(lmax);
    if (lane == 0) s.wmax[wave] = lmax;
    if (tid == 0) s.nU = 0;
    __syncthreads();
    const float thr0 = fmaxf(fmaxf(s.wmax[0], s.wmax[1]), fmaxf(s.wmax[2], s.wmax[3])) - beam;
    thr_ord = f2ord(thr0);
    for (int c = tid; c < N; c += blockDim.x) {
      const unsigned long long k = s.uk[c], v = s.uv[c];
      if (k != kEmpty && (unsigned)(v >> 32) >= thr_ord) {
        const int p = atomicAdd(&s.nU, 1);
        s.hk[p] = k;
        s.hv[p] = v;
      }
    }
    __syncthreads();
    Nsel = s.nU;
    listed = true;
  }

  if (Nsel <= kDirectCands) {
    // At most DP candidates per thread.  Candidates of one key merge in an LDS hash
    // table (the maximum of their packed values); the candidate holding that maximum
    // represents the key and is listed for the top-Ns selection.
    constexpr int DP = kDirectCands / kSearchThreads;
    constexpr int kDirBits = 10, kDirSlots = 1 << kDirBits;  // load <= 1/2
    static_assert(DP * kSearchThreads == kDirectCands && kDirSlots == 2 * kDirectCands &&
                      kDirSlots <= kHashSlots && kDirectCands <= kChunk + kMaxStates,
                  "direct path");
    const int n = Nsel;
    unsigned long long myk[DP], myv[DP];
#pragma unroll
    for (int u = 0; u < DP; ++u) {
      const int c = tid + u * kSearchThreads;
      myk[u] = kEmpty;
      myv[u] = 0ull;
      if (c < n) {
        if (listed) {
          myk[u] = s.hk[c];
          myv[u] = s.hv[c];
        } else {
          const ulonglong2 kv = make_cand(c);
          myk[u] = kv.x;
          myv[u] = kv.y;
        }
      }
    }
    __syncthreads();  // listed entries read; trivial graph: uk/uv held the staged tile lists until here
    for (int i = tid; i < kDirSlots; i += blockDim.x) {
      s.hk[i] = kEmpty;
      s.hv[i] = 0ull;
    }
    if (tid == 0) s.nU = 0;
    __syncthreads();
    int slot[DP];
#pragma unroll
    for (int u = 0; u < DP; ++u) {
      slot[u] = -1;
      if (myk[u] != kEmpty) {
        uint32_t h = (uint32_t)((myk[u] * 0x9E3779B97F4A7C15ull) >> (64 - kDirBits));
        for (;;) {
          const unsigned long long prev = atomicCAS(&s.hk[h], kEmpty, myk[u]);
          if (prev == kEmpty || prev == myk[u]) break;
          h = (h + 1) & (kDirSlots - 1);
        }
        atomicMax(&s.hv[h], myv[u]);
        slot[u] = (int)h;
      }
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < DP; ++u)
      if (slot[u] >= 0 && s.hv[slot[u]] == myv[u]) {  // values are unique (back-pointers)
        const int p = atomicAdd(&s.nU, 1);
        s.uk[p] = myk[u];
        s.uv[p] = myv[u];
      }
    __syncthreads();
    select_top(s, s.nU, Ns);
  } else {
    // Hash merge.  Listed entries (at most kChunk + kMaxStates) merge in one pass:
    // moved from hk/hv to uk/uv (whose made candidates are no longer needed), then
    // inserted.  Otherwise the candidates are made and merged kChunk at a time, the
    // best Ns so far carried into each pass.
    constexpr int CPT = kChunk / kSearchThreads;
    static_assert(8 * (kChunk + kMaxStates) <= 5 * kHashSlots, "one listed pass");
    const bool one = listed;
    if (one)
      for (int i = tid; i < Nsel; i += blockDim.x) {
        s.uk[i] = s.hk[i];
        s.uv[i] = s.hv[i];
      }
    __syncthreads();
    for (int base = 0; base < (one ? 1 : N); base += kChunk) {
      for (int i = tid; i < kHashSlots; i += blockDim.x) {
        s.hk[i] = kEmpty;
        s.hv[i] = 0ull;
      }
      if (tid == 0) s.nU = 0;
      __syncthreads();
      if (one) {
        for (int i = tid; i < Nsel; i += blockDim.x) hash_insert(s, s.uk[i], s.uv[i]);
      } else {
        const int nL = s.nL;
        for (int i = tid; i < nL; i += blockDim.x) hash_insert(s, s.lk[i], s.lv[i]);
        ulonglong2 kv[CPT];
#pragma unroll
        for (int u = 0; u < CPT; ++u) {
          const int c = base + tid + u * kSearchThreads;
          kv[u] = c < N ? make_cand(c) : make_ulonglong2(kEmpty, 0ull);
        }
#pragma unroll
        for (int u = 0; u < CPT; ++u)
          if (kv[u].x != kEmpty && (unsigned)(kv[u].y >> 32) >= thr_ord) hash_insert(s, kv[u].x, kv[u].y);
      }
      __syncthreads();
      for (int i = tid; i < kHashSlots; i += blockDim.x) {
        if (s.hk[i] != kEmpty) {
          const int u = atomicAdd(&s.nU, 1);
          s.uk[u] = s.hk[i];
          s.uv[u] = s.hv[i];
        }
      }
      __syncthreads();
      select_top(s, s.nU, Ns);
    }
  }

  // ---- beam, then max-contexts, then canonical (ctx, state) order ----
  // All LDS work and barriers precede the global stores, so no barrier waits
  // for stores to complete.
  const int K = s.nL;
  const int Kp = (K + 7) & ~7;
  {
    float bmax = -INFINITY;
    if (tid < K) bmax = ord2f((unsigned)(s.lv[tid] >> 32));
    bmax = wave_max_f(bmax);
    if (lane == 0) s.wmax[wave] = bmax;
  }
  __syncthreads();
  best = fmaxf(fmaxf(s.wmax[0], s.wmax[1]), fmaxf(s.wmax[2], s.wmax[3]));
  const float thr = best - beam;
  int my_keep1 = 0;
  if (tid < K) {
    my_ci = (unsigned)s.lk[tid];
    my_st = (unsigned)(s.lk[tid] >> 32);
    my_sc = ord2f((unsigned)(s.lv[tid] >> 32));
    my_v = s.lv[tid];
    my_keep1 = my_sc >= thr;
  }
  if (tid < Kp) {
    s.fent[tid] = make_uint4(my_ci, my_st, __float_as_uint(my_sc), 0u);
    s.fflg[tid] = my_keep1;
  }
  if (tid == 0) {
    s.nK = 0;
    s.nC = 0;
  }
  __syncthreads();
  if (K <= 16) {
    // One wave, one entry per lane; other lanes' entries are read with readlane
    // (no LDS traffic).  Context score = max over the context's in-beam tuples;
    // its first tuple is the one with the smallest state.
    if (wave == 0) {
      float my_cs = -INFINITY;
      my_first = my_keep1;
      for (int j = 0; j < K; ++j) {
        const unsigned cj = (unsigned)__builtin_amdgcn_readlane((int)my_ci, j);
        const unsigned sj = (unsigned)__builtin_amdgcn_readlane((int)my_st, j);
        const float scj = rdlane_f(my_sc, j);
        const int k1j = __builtin_amdgcn_readlane(my_keep1, j);
        const bool same = k1j && cj == my_ci;
        my_cs = same ? fmaxf(my_cs, scj) : my_cs;
        my_first &= !(same && sj < my_st);
      }
      // max-contexts: rank of the tuple's context among the in-beam contexts
      int rank = 0;
      for (int j = 0; j < K; ++j) {
        const int fj = __builtin_amdgcn_readlane(my_first, j);
        const float csj = rdlane_f(my_cs, j);
        const unsigned cj = (unsigned)__builtin_amdgcn_readlane((int)my_ci, j);
        rank += fj && (csj > my_cs || (csj == my_cs && cj < my_ci));
      }
      my_keep2 = my_keep1 && rank < Nc;
      // canonical position and context row of each kept tuple
      for (int j = 0; j < K; ++j) {
        const int k2j = __builtin_amdgcn_readlane(my_keep2, j);
        const int fj = __builtin_amdgcn_readlane(my_first, j);
        const unsigned cj = (unsigned)__builtin_amdgcn_readlane((int)my_ci, j);
        const unsigned sj = (unsigned)__builtin_amdgcn_readlane((int)my_st, j);
        my_pos += k2j && (cj < my_ci || (cj == my_ci && sj < my_st));
        my_crow += k2j && fj && cj < my_ci;
      }
      const unsigned long long kept = __ballot(my_keep2);
      const unsigned long long firsts = __ballot(my_keep2 && my_first);
      if (my_keep2 && my_first) s.n_ctx_list[my_crow] = (int)my_ci;
      if (lane == 0) {
        s.nK = __popcll(kept);
        s.nC = __popcll(firsts);
      }
    }
  } else if (K <= 64) {
    // One wave.  The entries are sorted by (context, state) with a bitonic network
    // across the lanes (carrying each entry's original lane, whose packed value is
    // fetched once after the sort), so that each context is a run of lanes: its score
    // is the run maximum of the in-beam scores, its first tuple the run's first
    // in-beam lane.  The kept contexts are the run heads at or above the Nc-th largest
    // context score, found bit by bit on ballots (ties: context ascending, the sorted
    // order); canonical positions and context rows are prefix counts of ballots,
    // because the sorted order is the canonical one.
    if (wave == 0) {
      auto xor64 = [](unsigned long long v, int m) {
        const int lo = xor_lane((int)(unsigned)v, m), hi = xor_lane((int)(unsigned)(v >> 32), m);
        return ((unsigned long long)(unsigned)hi << 32) | (unsigned)lo;
      };
      unsigned long long sk = tid < K ? ((unsigned long long)my_ci << 32) | my_st : ~0ull;  // sentinels last
      int ol = lane;  // the entry's original lane
      // (fully unrolled, so that each stage's exchange distance is a constant; keys
      // are unique but for the sentinels, whose order does not matter, so one compare
      // decides the exchange)
      auto stage = [&](int k, int j) {
        const unsigned long long pk = xor64(sk, j);
        const int po = xor_lane(ol, j);
        const bool up = (lane & k) == 0, lower = (lane & j) == 0;
        // (selects rather than a branch: each stage stays a short dependent chain)
        const bool take = (pk < sk) == (lower == up);
        sk = take ? pk : sk;
        ol = take ? po : ol;
      };
#pragma unroll
      for (int k = 2; k <= 32; k <<= 1)
#pragma unroll
        for (int j = k >> 1; j > 0; j >>= 1) stage(k, j);
      // with at most 32 entries the upper half holds sentinels only, and the lower
      // half is sorted: the last merge would exchange nothing
      if (K > 32)
#pragma unroll
        for (int j = 32; j > 0; j >>= 1) stage(64, j);
      const unsigned long long sv =
          ((unsigned long long)(unsigned)__shfl((int)(unsigned)(my_v >> 32), ol) << 32) |
          (unsigned)__shfl((int)(unsigned)my_v, ol);
      const bool valid = sk != ~0ull;
      const unsigned ci = (unsigned)(sk >> 32), stt = (unsigned)sk;
      const float sc = valid ? ord2f((unsigned)(sv >> 32)) : -INFINITY;
      const bool k1 = valid && sc >= thr;
      const unsigned prev = (unsigned)__builtin_amdgcn_update_dpp(0, (int)ci, 0x138, 0xf, 0xf, false);  // wave_shr:1
      const bool head = valid && (lane == 0 || prev != ci);
      const unsigned long long H = __ballot(head), K1 = __ballot(k1);
      const unsigned long long below = lane ? ~0ull >> (64 - lane) : 0ull;  // lanes < this one
      const unsigned long long self = 1ull << lane;
      const int rs = 63 - __clzll((long long)(H & (below | self)));         // run start
      const unsigned long long hnext = H & ~(below | self);
      const int re = hnext ? __ffsll((long long)hnext) - 2 : K - 1;          // run end
      const unsigned long long k1run = K1 & (~0ull << rs);
      const int fl = k1run ? __ffsll((long long)k1run) - 1 : 63;             // run's first in-beam lane
      const bool first = k1 && lane == fl;
      // run maxima by a segmented inclusive scan on DPP: shifts by 1, 2, 4 and 8
      // within each row of 16 (a source outside the row reads -inf), each taken only
      // from a lane of the same run; then the row broadcasts of lane 15 (into rows 1
      // and 3) and lane 31 (into rows 2 and 3), taken when that lane is in the run
      float run = k1 ? sc : -INFINITY;
      {
        const int ninf = __float_as_int(-INFINITY);
        const float u1 = __int_as_float(__builtin_amdgcn_update_dpp(ninf, __float_as_int(run), 0x111, 0xf, 0xf, false));
        if (lane - 1 >= rs) run = fmaxf(run, u1);
        const float u2 = __int_as_float(__builtin_amdgcn_update_dpp(ninf, __float_as_int(run), 0x112, 0xf, 0xf, false));
        if (lane - 2 >= rs) run = fmaxf(run, u2);
        const float u4 = __int_as_float(__builtin_amdgcn_update_dpp(ninf, __float_as_int(run), 0x114, 0xf, 0xf, false));
        if (lane - 4 >= rs) run = fmaxf(run, u4);
        const float u8 = __int_as_float(__builtin_amdgcn_update_dpp(ninf, __float_as_int(run), 0x118, 0xf, 0xf, false));
        if (lane - 8 >= rs) run = fmaxf(run, u8);
        const float b15 = __int_as_float(__builtin_amdgcn_update_dpp(ninf, __float_as_int(run), 0x142, 0xa, 0xf, false));
        if ((lane & 16) && (lane & ~15) - 1 >= rs) run = fmaxf(run, b15);
        const float b31 = __int_as_float(__builtin_amdgcn_update_dpp(ninf, __float_as_int(run), 0x143, 0xc, 0xf, false));
        if (lane >= 32 && 31 >= rs) run = fmaxf(run, b31);
      }
      const float cs = __shfl(run, valid ? re : lane);
      const unsigned co = first ? f2ord(cs) : 0u;  // a head's code is never 0
      int fkeep = first;
      if (__popcll(__ballot(first)) > (unsigned)Nc) {
        // theta: the largest code with at least Nc heads at or above it, i.e. the
        // Nc-th largest head code (> 0).  Other lanes hold code 0, so plain compares
        // count heads only, one ballot per bit.
        unsigned theta = 0u;
        for (int bit = 31; bit >= 0; --bit) {
          const unsigned cand = theta | (1u << bit);
          if (__popcll(__ballot(co >= cand)) >= (unsigned)Nc) theta = cand;
        }
        const int room = Nc - (int)__popcll(__ballot(co > theta));  // >= 1
        const unsigned long long E = __ballot(co == theta);
        fkeep = first && (co > theta || (co == theta && (int)__popcll(E & below) < room));
      }
      const int keep2 = k1 && __shfl(fkeep, fl);
      const unsigned long long K2 = __ballot(keep2), F2 = __ballot(keep2 && first);
      my_pos = __popcll(K2 & below);
      my_crow = __popcll(F2 & (rs ? ~0ull >> (64 - rs) : 0ull));
      my_first = first;
      my_keep2 = keep2;
      my_ci = ci;
      my_st = stt;
      my_sc = sc;
      my_v = sv;
      if (keep2 && first) s.n_ctx_list[my_crow] = (int)ci;
      if (lane == 0) {
        s.nK = __popcll(K2);
        s.nC = __popcll(F2);
      }
    }
  } else {
    // Larger sets: every thread holds one entry and scans the others in LDS.  The
    // loads are unconditional and issued eight at a time (the asm statements pin
    // them before any use) so they pipeline.
    float my_cs = -INFINITY;
    my_first = my_keep1;
    if (tid < K) {
      for (int j0 = 0; j0 < Kp; j0 += 8) {
        uint4 e[8];
        int f[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          e[u] = s.fent[j0 + u];
          f[u] = s.fflg[j0 + u];
        }
        asm volatile("" ::"v"(e[0].x), "v"(e[0].y), "v"(e[0].z), "v"(f[0]), "v"(e[1].x), "v"(e[1].y),
                     "v"(e[1].z), "v"(f[1]), "v"(e[2].x), "v"(e[2].y), "v"(e[2].z), "v"(f[2]),
                     "v"(e[3].x), "v"(e[3].y), "v"(e[3].z), "v"(f[3]));
        asm volatile("" ::"v"(e[4].x), "v"(e[4].y), "v"(e[4].z), "v"(f[4]), "v"(e[5].x), "v"(e[5].y),
                     "v"(e[5].z), "v"(f[5]), "v"(e[6].x), "v"(e[6].y), "v"(e[6].z), "v"(f[6]),
                     "v"(e[7].x), "v"(e[7].y), "v"(e[7].z), "v"(f[7]));
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const bool same = (f[u] & 1) && e[u].x == my_ci;
          my_cs = same ? fmaxf(my_cs, __uint_as_float(e[u].z)) : my_cs;
          my_first &= !(same && e[u].y < my_st);
        }
      }
    }
    __syncthreads();
    if (tid < Kp) {
      s.fent[tid].w = __float_as_uint(my_cs);
      s.fflg[tid] = my_keep1 | (my_first << 1);
    }
    __syncthreads();
    if (my_keep1) {
      int rank = 0;
      for (int j0 = 0; j0 < Kp; j0 += 8) {
        uint4 e[8];
        int f[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          e[u] = s.fent[j0 + u];
          f[u] = s.fflg[j0 + u];
        }
        asm volatile("" ::"v"(e[0].x), "v"(e[0].w), "v"(f[0]), "v"(e[1].x), "v"(e[1].w), "v"(f[1]),
                     "v"(e[2].x), "v"(e[2].w), "v"(f[2]), "v"(e[3].x), "v"(e[3].w), "v"(f[3]));
        asm volatile("" ::"v"(e[4].x), "v"(e[4].w), "v"(f[4]), "v"(e[5].x), "v"(e[5].w), "v"(f[5]),
                     "v"(e[6].x), "v"(e[6].w), "v"(f[6]), "v"(e[7].x), "v"(e[7].w), "v"(f[7]));
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const float csj = __uint_as_float(e[u].w);
          rank += ((f[u] >> 1) & 1) && (csj > my_cs || (csj == my_cs && e[u].x < my_ci));
        }
      }
      my_keep2 = rank < Nc;
    }
    __syncthreads();
    if (tid < Kp) s.fflg[tid] = my_keep1 | (my_first << 1) | (my_keep2 << 2);
    __syncthreads();
    if (my_keep2) {
      for (int j0 = 0; j0 < Kp; j0 += 8) {
        uint4 e[8];
        int f[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          e[u] = s.fent[j0 + u];
          f[u] = s.fflg[j0 + u];
        }
        asm volatile("" ::"v"(e[0].x), "v"(e[0].y), "v"(f[0]), "v"(e[1].x), "v"(e[1].y), "v"(f[1]),
                     "v"(e[2].x), "v"(e[2].y), "v"(f[2]), "v"(e[3].x), "v"(e[3].y), "v"(f[3]));
        asm volatile("" ::"v"(e[4].x), "v"(e[4].y), "v"(f[4]), "v"(e[5].x), "v"(e[5].y), "v"(f[5]),
                     "v"(e[6].x), "v"(e[6].y), "v"(f[6]), "v"(e[7].x), "v"(e[7].y), "v"(f[7]));
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const bool k2 = (f[u] >> 2) & 1;
          my_pos += k2 && (e[u].x < my_ci || (e[u].x == my_ci && e[u].y < my_st));
          my_crow += k2 && ((f[u] >> 1) & 1) && e[u].x < my_ci;
        }
      }
      atomicAdd(&s.nK, 1);
      if (my_first) {
        s.n_ctx_list[my_crow] = (int)my_ci;
        atomicAdd(&s.nC, 1);
      }
    }
  }
  }  // general selection
  __syncthreads();
  const int nC = s.nC;
  if (tid < nC) {
    const int c = s.n_ctx_list[tid], a = c / V;
    s.n_rowoff[tid] = make_int2(a * m.Kpad, (c - a * V) * m.Kpad);
  }
  __syncthreads();
  const bool store_surv = writer && (!FUSED || t + 1 == L);
  // general graph: the kept tuples' arc ranges for the next frame, requested before
  // the next rows so that their round trip overlaps them
  int2 nrp = make_int2(0, 0);
  if (!TRIV && store_surv && my_keep2) nrp = make_int2(g.rp[my_st], g.rp[my_st + 1]);
  // global stores: joiner rows of the next frame, survivors, history, trace
  if (t + 1 < L) {
    if (FUSED && dspec) {
      // h = tanh(enc[t + 1] + decoder row) from the staged rows; the new contexts'
      // decoder rows go to the other context buffer
      const int kq4 = m.Kpad / 4;
      const float4* dc4 = reinterpret_cast<const float4*>(dspec);
      const float4* du4 = reinterpret_cast<const float4*>(dspec + (size_t)(16 + 4 * dcur_buf) * m.Kpad);
      float4* dn4 = reinterpret_cast<float4*>(dspec + (size_t)(16 + 4 * (dcur_buf ^ 1)) * m.Kpad);
      const float4* en4 = reinterpret_cast<const float4*>(s.enc_next);
      for (int e = tid; e < nC * kq4; e += blockDim.x) {
        const int j = e / kq4, kq = e - j * kq4;
        const int src = s.g_src[j];
        const float4 dv = src >= 0 ? dc4[src * kq4 + kq] : du4[(-src - 1) * kq4 + kq];
        const float4 ev = en4[kq];
        const float h0 = tanh_fast(ev.x + dv.x), h1 = tanh_fast(ev.y + dv.y);
        const float h2 = tanh_fast(ev.z + dv.z), h3 = tanh_fast(ev.w + dv.w);
        if (m.bf16) {
          const uint2 hb = make_uint2((unsigned)f32_to_bf16_rne(h0) | ((unsigned)f32_to_bf16_rne(h1) << 16),
                                      (unsigned)f32_to_bf16_rne(h2) | ((unsigned)f32_to_bf16_rne(h3) << 16));
          *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(hl) + (size_t)j * hstride + 4 * kq) = hb;
        } else {
          *reinterpret_cast<float4*>(reinterpret_cast<float*>(hl) + (size_t)j * hstride + 4 * kq) =
              make_float4(h0, h1, h2, h3);
        }
        dn4[e] = dv;
      }
    } else if (FUSED) {
      write_h_rows<kSearchThreads>(m, s.enc_next, 0, s.n_rowoff, nC, hl, hstride, tid);
    } else {
      // (the gathers of up to 16 rows of K = 512 in one batch)
      const size_t esz = m.bf16 ? 2 : 4;
      char* hrows = reinterpret_cast<char*>(d.h) + row0 * m.Kpad * esz;
      // (C a multiple of 4: 16-byte column quads, 4 items per thread and batch for at
      // most 8 rows, else 8; otherwise column pairs, a batch of 8 items when at most 8
      // rows: a row per item at K = 512, so no batch loads rows it drops)
      if ((m.C & 3) == 0 && nC <= 8)
        write_h_rows_quads<kSearchThreads, 4>(m, s.enc_next, s.n_rowoff, nC, hrows, m.Kpad, tid);
      else if ((m.C & 3) == 0)
        write_h_rows_quads<kSearchThreads, 8>(m, s.enc_next, s.n_rowoff, nC, hrows, m.Kpad, tid);
      else if ((m.C & 1) == 0 && nC <= 8)
        write_h_rows_pairs<kSearchThreads, 8>(m, s.enc_next, s.n_rowoff, nC, hrows, m.Kpad, tid);
      else if ((m.C & 1) == 0)
        write_h_rows_pairs<kSearchThreads, 16>(m, s.enc_next, s.n_rowoff, nC, hrows, m.Kpad, tid);
      else
        write_h_rows<kSearchThreads, 32>(m, s.enc_next, 0, s.n_rowoff, nC, hrows, m.Kpad, tid);
    }
  }
  if (my_keep2) {
    const unsigned tb = 0xffffffffu - (unsigned)my_v;
    const int parent = (int)(tb / stride_tb);
    const int apos = (int)(tb - (unsigned)parent * stride_tb) - 1;
    const int arc = apos < 0 ? -1 : s.s_base[parent] + apos;
    // (the arc's label is the newer label of the tuple's context: no load)
    const int label = arc < 0 ? 0 : (int)(my_ci % (unsigned)V);
    const size_t o = (size_t)b * Ns + my_pos;
    if (FUSED) {  // every read of the old survivors precedes the last barrier
      s.s_ctx[my_pos] = (int)my_ci;
      s.s_state[my_pos] = (int)my_st;
      s.s_score[my_pos] = my_sc - best;
      s.s_row[my_pos] = my_crow;
    }
    if (store_surv) {
      d.surv_ctx[o] = (int)my_ci;
      d.surv_state[o] = (int)my_st;
      d.surv_score[o] = my_sc - best;
      d.surv_row[o] = my_crow;
      if (!TRIV) d.surv_rp[o] = nrp;
      if (my_first) d.ctx_list[row0 + my_crow] = (int)my_ci;
    }
    const size_t hbase = ((size_t)(fb + t) * d.B + b) * Ns;
    if (writer) {
      d.hist_pl[hbase + my_pos] = (parent << 16) | label;
      d.hist_arc[hbase + my_pos] = arc;
    }
    if (writer && trace) {
      int* tr = trace + (((size_t)(fb + t + 1) * d.B + b) * Ns + my_pos) * 4;
      tr[0] = (int)my_ci;
      tr[1] = (int)my_st;
      tr[2] = parent;
      tr[3] = label;
    }
  }
  if (tid == 0) {
    if (store_surv) {
      d.nsurv[b] = s.nK;
      d.nctx[b] = nC;
    }
    if (FUSED) {
      s.ns = s.nK;
      s.nc = nC;
    }
    // the offset stays in LDS across the persistent kernels' frames and is stored
    // after the stream's (or chunk's) last one
    if (writer) {
      s.off_d += (double)best;
      if (!FUSED || t + 1 == L) d.offset[b] = s.off_d;
    }
  }
}

template <bool TRIV>
__global__ __launch_bounds__(kSearchThreads) void k_search(ModelDev m, GraphDev g, DecodeDev d,
                                                           float beam, int t,
                                                           int* __restrict__ trace) {
  const int b = blockIdx.x;
  const int L = d.len[b];
  if (t >= L) return;
  extern __shared__ __align__(16) unsigned char smem[];
  SearchSmem& s = *reinterpret_cast<SearchSmem*>(smem);
  const int fb = d.base ? d.base[b] : 0;
  if (d.graphs) g = d.graphs[b];  // per-stream graphs
  search_frame<TRIV, false>(m, g, d, beam, t, L, b, trace, s, nullptr, 0, nullptr, false, true,
                            false, nullptr, 0, fb);
}

// ---------------------------------------------------------------------------
// per-stream kernel: one workgroup owns one stream for all of its frames
// (Algorithm 1's frame loop without a launch or a global round trip per frame).

// Joiner of frame t for this stream's context rows (Algorithm 1: joiner; the
// log-softmax is taken by the search from the rows this writes).  The rows h are
// in LDS at hl (row stride hstride elements, RG groups of 4 rows; rows >= nc hold
// stale or zero values whose outputs are never read); the logits go to LDS at zl
// ([4 RG][Vpad] fp32, -inf beyond V).  Lane l of a wave owns vocabulary column
// 64 cg + l of two 64-column groups at once, cg = wave + 4 (2p) and wave + 4 (2p + 1),
// so that each h value read from LDS feeds both.  W is streamed as 16-byte k
// slices of the interleaved copy (one contiguous kilobyte per wave and load), the
// next chunk always in flight in ping-pong registers.  fp32: VALU FMAs with h
// broadcast from LDS (with 4 to 16 rows, VALU outruns the 4x4 MFMA blocks).
// bf16: v_mfma_f32_4x4x4bf16 computes 16 independent 4x4 blocks, lane l = 4j + c
// supplying row c of A block j and column c of B block j, so A = h[4g + (l & 3)]
// and B = W[64 cg + l] leave z[4g + v][64 cg + l] in accumulator element v.
template <bool BF16, int RG>
__device__ __forceinline__ void stream_joiner(const ModelDev& m, const DecodeDev& d, const void* hl,
                                              int hstride, float* zl) {
  constexpr int KQ = BF16 ? 8 : 4;   // k values per 16-byte slice
  constexpr int CH = 8;              // slices per lane per column group and chunk
  constexpr int NR = 4 * RG;         // rows computed
  constexpr int ESZ = BF16 ? 2 : 4;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int V = m.V, Vpad = m.Vpad, nvt = d.nvt;
  const int nch = m.Kpad / (KQ * CH);                  // chunks per column group
  const int ncgw = (nvt - wave + 3) >> 2;              // column groups of this wave
  const int steps = ((ncgw + 1) >> 1) * nch;           // pairs of groups x chunks
  if (steps == 0) return;
  const uint4* __restrict__ Wi = reinterpret_cast<const uint4*>(m.Wi);
  const char* hrows = reinterpret_cast<const char*>(hl);
  const size_t rstride = (size_t)hstride * ESZ;

  // column groups of pair p; the second may not exist (then it repeats the first
  // and is never written)
  auto pair_cg = [&](int p, int& c0, int& c1) {
    c0 = wave + 8 * p;
    c1 = c0 + 4 < nvt ? c0 + 4 : c0;
  };
  auto load_chunk = [&](int step, uint4 (&w)[2][CH], float (&bias)[2]) {
    const int p = step / nch, ch = step - p * nch;
    int c0, c1;
    pair_cg(p, c0, c1);
    const uint4* s0 = Wi + (size_t)(ch * CH) * Vpad + c0 * 64 + lane;
    const uint4* s1 = Wi + (size_t)(ch * CH) * Vpad + c1 * 64 + lane;
#pragma unroll
    for (int u = 0; u < CH; ++u) {
      w[0][u] = s0[(size_t)u * Vpad];
      w[1][u] = s1[(size_t)u * Vpad];
    }
    bias[0] = m.bias[min(c0 * 64 + lane, V - 1)];
    bias[1] = m.bias[min(c1 * 64 + lane, V - 1)];
  };

  float acc[2][NR];
  f32x4 macc[2][BF16 ? RG : 1][2];
  auto reset = [&]() {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
#pragma unroll
      for (int r = 0; r < NR; ++r) acc[c][r] = 0.f;
#pragma unroll
      for (int g = 0; g < (BF16 ? RG : 1); ++g) {
        macc[c][g][0] = f32x4{0.f, 0.f, 0.f, 0.f};
        macc[c][g][1] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
  };
  auto epilogue = [&](int c, int cg, float bias) {
    const int col = cg * 64 + lane;
    const bool cvalid = col < V;
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      float zs;
      if (BF16) {
        const int g = r >> 2, v = r & 3;
        zs = macc[c][g][0][v] + macc[c][g][1][v];
      } else {
        zs = acc[c][r];
      }
      zl[(size_t)r * Vpad + col] = cvalid ? zs + bias : -INFINITY;
    }
  };
  // step >= steps (the odd tail of the ping-pong) computes on a repeated chunk and
  // writes nothing
  auto compute = [&](int step, const uint4 (&w)[2][CH], const float (&bias)[2]) {
    const int p = step / nch, ch = step - p * nch;
#pragma unroll
    for (int u = 0; u < CH; ++u) {
      const size_t ko = (size_t)(ch * CH + u) * 16;  // byte offset of this k slice in a row
      if (BF16) {
        typedef short s16x4 __attribute__((ext_vector_type(4)));
#pragma unroll
        for (int g = 0; g < RG; ++g) {
          const uint4 a =
              *reinterpret_cast<const uint4*>(hrows + (size_t)(4 * g + (lane & 3)) * rstride + ko);
          const s16x4 alo = __builtin_bit_cast(s16x4, make_uint2(a.x, a.y));
          const s16x4 ahi = __builtin_bit_cast(s16x4, make_uint2(a.z, a.w));
#pragma unroll
          for (int c = 0; c < 2; ++c) {
            macc[c][g][0] = __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(
                alo, __builtin_bit_cast(s16x4, make_uint2(w[c][u].x, w[c][u].y)), macc[c][g][0], 0,
                0, 0);
            macc[c][g][1] = __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(
                ahi, __builtin_bit_cast(s16x4, make_uint2(w[c][u].z, w[c][u].w)), macc[c][g][1], 0,
                0, 0);
          }
        }
      } else {
#pragma unroll
        for (int r = 0; r < NR; ++r) {
          const float4 a = *reinterpret_cast<const float4*>(hrows + (size_t)r * rstride + ko);
#pragma unroll
          for (int c = 0; c < 2; ++c) {
            acc[c][r] = fmaf(a.x, __uint_as_float(w[c][u].x), acc[c][r]);
            acc[c][r] = fmaf(a.y, __uint_as_float(w[c][u].y), acc[c][r]);
            acc[c][r] = fmaf(a.z, __uint_as_float(w[c][u].z), acc[c][r]);
            acc[c][r] = fmaf(a.w, __uint_as_float(w[c][u].w), acc[c][r]);
          }
        }
      }
    }
    if (ch == nch - 1 && step < steps) {
      int c0, c1;
      pair_cg(p, c0, c1);
      epilogue(0, c0, bias[0]);
      if (c1 != c0) epilogue(1, c1, bias[1]);
      reset();
    }
  };

  reset();
  uint4 wa[2][CH], wb[2][CH];
  float ba[2], bb[2];
  // Every load is issued unconditionally (clamped to the last chunk), so the wait
  // before a chunk's first use counts only the loads issued after it.
  load_chunk(0, wa, ba);
  for (int step = 0; step < steps; step += 2) {
    load_chunk(min(step + 1, steps - 1), wb, bb);
    compute(step, wa, ba);
    load_chunk(min(step + 2, steps - 1), wa, ba);
    compute(step + 1, wb, bb);
  }
}

template <bool BF16, bool TRIV, int RG>
__global__ __launch_bounds__(kSearchThreads) void k_stream(ModelDev m, GraphDev g, DecodeDev d,
                                                           float beam, int* __restrict__ trace,
                                                           int hoff, int hstride, int zoff,
                                                           int doff) {
  const int b = blockIdx.x;
  const int L = d.len[b];
  if (L == 0) return;
  extern __shared__ __align__(16) unsigned char smem[];
  SearchSmem& s = *reinterpret_cast<SearchSmem*>(smem);
  void* hl = smem + hoff;
  float* zl = reinterpret_cast<float*>(smem + zoff);
  const int tid = threadIdx.x;
  const int Ns = d.Ns, Nc = d.Nc, V = m.V;
  const int fb = d.base ? d.base[b] : 0;  // absolute index of this call's frame 0
  if (d.graphs) g = d.graphs[b];          // per-stream graphs
  const size_t row0 = (size_t)b * Nc;
  // state after the initial tuple (written by k_init), encoder frame 0, zeroed rows
  if (tid == 0) {
    s.ns = d.nsurv[b];
    s.nc = d.nctx[b];
    s.off_d = d.offset[b];
  }
  for (int i = tid; i < Ns; i += blockDim.x) {
    const size_t o = (size_t)b * Ns + i;
    s.s_ctx[i] = d.surv_ctx[o];
    s.s_state[i] = d.surv_state[o];
    s.s_row[i] = d.surv_row[o];
    s.s_score[i] = d.surv_score[o];
  }
  for (int j = tid; j < Nc; j += blockDim.x) {
    const int c = d.ctx_list[row0 + j], a = c / V;
    s.n_rowoff[j] = make_int2(a * m.Kpad, (c - a * V) * m.Kpad);
  }
  {
    const float* er = d.enc + (size_t)b * d.T * m.C;
    for (int k = tid; k < m.Kpad; k += blockDim.x) s.enc_next[k] = k < m.C ? er[k] : 0.f;
    const int words = RG * 4 * hstride * (m.bf16 ? 2 : 4) / 4;
    for (int i = tid; i < words; i += blockDim.x) reinterpret_cast<int*>(hl)[i] = 0;
  }
  __syncthreads();
  write_h_rows<kSearchThreads>(m, s.enc_next, 0, s.n_rowoff, s.nc, hl, hstride, tid);
  // staged decoder rows (trivial graph, max_states = 4): those of the initial contexts
  float* dspec = (TRIV && doff) ? reinterpret_cast<float*>(smem + doff) : nullptr;
  if (dspec)
    for (int e = tid; e < s.nc * m.Kpad; e += blockDim.x) {
      const int j = e / m.Kpad, k = e - j * m.Kpad;
      const int2 off = s.n_rowoff[j];
      dspec[(size_t)16 * m.Kpad + e] = fmaxf(m.P0[(size_t)off.x + k] + m.P1[(size_t)off.y + k], 0.f);
    }
  __syncthreads();
  int cur = 0;
  constexpr int NEP = kMaxDim / kSearchThreads;
  for (int t = 0; t < L; ++t) {
    // encoder frame t + 1, in flight during the joiner
    float encp[NEP];
    {
      const float* er = d.enc + ((size_t)b * d.T + min(t + 1, L - 1)) * m.C;
#pragma unroll
      for (int u = 0; u < NEP; ++u) {
        const int k = tid + u * kSearchThreads;
        encp[u] = k < m.C ? er[k] : 0.f;
      }
    }
    stream_joiner<BF16, RG>(m, d, hl, hstride, zl);
    if (t + 1 < L) {
#pragma unroll
      for (int u = 0; u < NEP; ++u) {
        const int k = tid + u * kSearchThreads;
        if (k < m.C) s.enc_next[k] = encp[u];
      }
    }
    __syncthreads();
    search_frame<TRIV, true>(m, g, d, beam, t, L, b, trace, s, hl, hstride, zl, false, true, true,
                             dspec, cur, fb);
    __syncthreads();
    cur ^= 1;
  }
}

// ---------------------------------------------------------------------------
// grouped per-stream kernel: G workgroups share one stream (trivial graph, fp32).
// Member g computes the joiner for its NCG 64-column groups starting at cg0 = g NCG,
// and every member runs the same search on the same data, so they stay identical;
// per frame they exchange each row's (max, sum exp), best KT labels and blank logit
// through tagged 64-bit words: relaxed device-scope atomic stores and loads, coherent
// across the compute units and L2 caches of every XCD.

constexpr int kResSlices = kKStep / 16;  // 16-byte k slices per wave of a resident W slice

// Joiner of member columns [64 cg0, 64 (cg0 + NCG)) for all 4 RG rows, split over
// K: wave w accumulates k slices [w Kpad / 16, (w + 1) Kpad / 16) (16-byte fp32
// slices), lane l owning column 64 (cg0 + j) + l, h broadcast from LDS.  RES
// (NCG = 1, Kpad = 512): the lane's 32 slices of W are in registers (wres) for the
// whole decode; otherwise W is streamed from the interleaved copy with the next
// chunk in flight.  Both add the slices in the same order.  The four waves'
// partial sums go to LDS (part, [wave][NCG][4 RG][64]); the caller adds them in
// wave order.
template <int RG, int NCG, bool RES>
__device__ __forceinline__ void group_joiner_f32(const ModelDev& m, const void* hl, int hstride,
                                                 float* part, int cg0,
                                                 const float4 (&wres)[kResSlices]) {
  // v_mfma_f32_4x4x1f32 computes 16 independent 4 x 4 x 1 blocks: lane l = 4 j + c
  // supplies row c of A block j and column c of B block j, and accumulator element
  // v of lane l is (row v, column c) of block j.  With A = h[4 g + (l & 3)][k] and
  // B = W[64 cg + l][k] every block reads the same four rows, so element v of lane l
  // accumulates z[4 g + v][64 cg + l] over this wave's k values: one instruction is
  // 4 rows x 64 columns x 1 k, twice the unpacked fp32 FMA rate of the VALU.
  constexpr int NR = 4 * RG;
  constexpr int CH = 8 / NCG;  // k slices per chunk
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int Vpad = m.Vpad;
  const int qw = m.Kpad / 16;  // k slices per wave (a multiple of 32)
  const int q0 = wave * qw;
  const char* hrows = reinterpret_cast<const char*>(hl) + (size_t)(lane & 3) * hstride * 4;
  const size_t gstride = (size_t)hstride * 16;  // bytes between row groups of 4
  // two accumulator chains (even and odd k of each slice), so that consecutive
  // MFMAs never wait on each other's result
  f32x4 acc[NCG][RG], acc2[NCG][RG];
#pragma unroll
  for (int j = 0; j < NCG; ++j)
#pragma unroll
    for (int g = 0; g < RG; ++g) acc[j][g] = acc2[j][g] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto slice = [&](size_t ko, const float4 (&w)[NCG]) {
#pragma unroll
    for (int g = 0; g < RG; ++g) {
      const float4 a = *reinterpret_cast<const float4*>(hrows + g * gstride + ko);
#pragma unroll
      for (int j = 0; j < NCG; ++j) {
        acc[j][g] = __builtin_amdgcn_mfma_f32_4x4x1f32(a.x, w[j].x, acc[j][g], 0, 0, 0);
        acc2[j][g] = __builtin_amdgcn_mfma_f32_4x4x1f32(a.y, w[j].y, acc2[j][g], 0, 0, 0);
        acc[j][g] = __builtin_amdgcn_mfma_f32_4x4x1f32(a.z, w[j].z, acc[j][g], 0, 0, 0);
        acc2[j][g] = __builtin_amdgcn_mfma_f32_4x4x1f32(a.w, w[j].w, acc2[j][g], 0, 0, 0);
      }
    }
  };
  static_assert(!RES || NCG == 1, "a resident W slice is one column group");
  if constexpr (RES) {
#pragma unroll
    for (int u = 0; u < kResSlices; ++u) {
      const float4 w[1] = {wres[u]};
      slice((size_t)(q0 + u) * 16, w);
    }
  } else {
    const int steps = qw / CH;   // even
    const float4* __restrict__ Wi = reinterpret_cast<const float4*>(m.Wi);
    auto load_chunk = [&](int step, float4 (&w)[CH][NCG]) {
#pragma unroll
      for (int u = 0; u < CH; ++u) {
        const size_t q = (size_t)(q0 + step * CH + u);
#pragma unroll
        for (int j = 0; j < NCG; ++j) w[u][j] = Wi[q * Vpad + (cg0 + j) * 64 + lane];
      }
    };
    auto compute = [&](int step, const float4 (&w)[CH][NCG]) {
#pragma unroll
      for (int u = 0; u < CH; ++u) slice((size_t)(q0 + step * CH + u) * 16, w[u]);
    };
    float4 wa[CH][NCG], wb[CH][NCG];
    load_chunk(0, wa);
    for (int step = 0; step < steps; step += 2) {
      load_chunk(step + 1, wb);
      compute(step, wa);
      load_chunk(min(step + 2, steps - 1), wa);
      compute(step + 1, wb);
    }
  }
#pragma unroll
  for (int j = 0; j < NCG; ++j)
#pragma unroll
    for (int g = 0; g < RG; ++g)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        part[((wave * NCG + j) * NR + 4 * g + v) * 64 + lane] = acc[j][g][v] + acc2[j][g][v];
  __syncthreads();
}

// The member joiner's partial sums (4 waves x 2 column groups x 16 rows x 64 lanes)
// live in hk and hv.
static_assert(offsetof(SearchSmem, hv) == offsetof(SearchSmem, hk) + sizeof(SearchSmem::hk) &&
                  sizeof(SearchSmem::hk) + sizeof(SearchSmem::hv) >= 4 * 2 * 16 * 64 * sizeof(float),
              "member joiner partial sums do not fit hk and hv");

// Exchange slot of (stream b, member g, frame parity): Nc rows of RW words.  A word
// is tag << 48 | payload: the tag (decode epoch << 8 | frame, both mod 256; the
// epoch is never 0, so cleared words never match) tells a word of this decode and
// frame from an older one (the slot of a frame parity is rewritten every other
// frame, and members never drift a frame apart).  Row payloads: the maximum and the
// sum of exp(z - maximum) over the member's columns, the blank logit (member 0),
// then KT candidates label << 32 | logit bits (label 0: none).
struct GroupX {
  unsigned long long* buf;  // device memory (exchange words only)
  int G, xwords;            // members per stream; words per slot
  unsigned epoch;           // decode number (8 bits, never 0)
  unsigned spin_limit;      // polls before a wait is abandoned (recorded in err)
  unsigned* err;            // [1 + B]: timeouts of any stream (checked by every later
                            // wait, which then gives up at once), then per stream
  unsigned* tickets;        // [8][64] (zeroed): per-XCD arrival counters (xlocal)
  int xlocal;               // one workgroup per CU on every CU of 8 XCDs: each stream's
                            // members are placed on one XCD by arrival order there, and
                            // their words pass through that XCD's L2 (stores sc0, loads
                            // sc0 sc1) instead of device-scope atomics
};
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
// Exchange word access of the grouped kernel.  r is a buffer resource over x.buf; the
// L2 path addresses a word by its byte offset there, with cache policy 17 (sc0 sc1) on
// loads and 1 (sc0) on stores.
__device__ __forceinline__ unsigned long long xw_load(const GroupX& x, __amdgpu_buffer_rsrc_t r,
                                                      const unsigned long long* w) {
  if (x.xlocal)
    return __builtin_bit_cast(unsigned long long,
                              __builtin_amdgcn_raw_buffer_load_b64(
                                  r, (unsigned)((const char*)w - (const char*)x.buf), 0, 17));
  return __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void xw_store(const GroupX& x, __amdgpu_buffer_rsrc_t r,
                                         unsigned long long* w, unsigned long long v) {
  if (x.xlocal)
    __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2_t, v), r,
                                          (unsigned)((char*)w - (char*)x.buf), 0, 1);
  else
    __hip_atomic_store(w, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// LDS layout of the grouped kernel beyond SearchSmem.
struct GroupLds {
  int hoff, hstride;        // joiner rows [4 RG][hstride] fp32 (byte offset, row stride)
  int doff;                 // fast path: per-wave decoder rows of the candidates
                            // [4 waves][20][64] float2 (byte offset)
};
constexpr int kFastDecEntries = 20;  // 16 label candidates (i KT + q) + 4 current rows

__device__ __forceinline__ unsigned long long* group_slot(const GroupX& x, int b, int g, int t) {
  return x.buf + ((size_t)(b * x.G + g) * 2 + (t & 1)) * x.xwords;
}

// Grouped per-stream kernel.  Per frame: member joiner (partial sums per wave),
// per-row statistics of the member's columns published as tagged words, the
// members' words of each row polled by the row's wave and combined in member order,
// then the search.
//
// FAST (RG = 1, NCG = 1, resident W, Kpad = 512, at most 4 tuples): every wave runs
// the one-wave selection itself (the results are identical), so that each wave can
// build its own quarter of the next frame's joiner rows, the quarter its joiner
// reads, without a workgroup barrier: the decoder rows ReLU(P0[a] + P1[b]) of every
// candidate context are gathered at the wave's 128 columns (two per lane) into
// registers before the selection, so their latency hides behind it, and the
// decoder rows of the current contexts stay in registers for the blank
// candidates.  The survivors alternate between two LDS buffers (wave 0 writes the
// next frame's while the other waves may still read the current one).
template <int RG, int NCG, bool RES, bool FAST>
__global__ __launch_bounds__(kSearchThreads) void k_stream_group(ModelDev m, GraphDev g, DecodeDev d,
                                                                 float beam, int* __restrict__ trace,
                                                                 GroupLds ly, GroupX x) {
  static_assert(!FAST || (RG == 1 && NCG == 1 && RES), "the fast path is for 4 rows, resident W");
  const int G = x.G;
  extern __shared__ __align__(16) unsigned char smem[];
  SearchSmem& s = *reinterpret_cast<SearchSmem*>(smem);
  int b = blockIdx.x / G, mem = blockIdx.x - b * G;
  if (x.xlocal) {
    // (XCC_ID, the XCD this workgroup runs on; every XCD holds gridDim.x / 8 of them)
    if (threadIdx.x == 0) {
      const unsigned xcc = __builtin_amdgcn_s_getreg((3 << 11) | 20) & 0xfu;
      const unsigned per = gridDim.x / 8;
      const unsigned tk = xcc < 8 ? __hip_atomic_fetch_add(x.tickets + 64 * xcc, 1u, __ATOMIC_RELAXED,
                                                           __HIP_MEMORY_SCOPE_AGENT)
                                  : per;
      s.misc[0] = tk < per ? (int)(xcc * per + tk) : -1;
    }
    __syncthreads();
    const int slot = s.misc[0];
    if (slot < 0) {  // placement not as assumed: the other members' waits time out
      if (threadIdx.x == 0) __hip_atomic_fetch_add(x.err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      return;
    }
    b = slot / G;
    mem = slot - b * G;
  }
  const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
      x.buf, (short)0, (int)(gridDim.x * 2u * (unsigned)x.xwords * 8u), 0x00020000);
  const int L = d.len[b];
  if (L == 0) return;  // every member of the stream returns here
  unsigned char* hl = smem + ly.hoff;
  const int hstride = ly.hstride;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int Ns = d.Ns, Nc = d.Nc, V = m.V, C = m.C, Kpad = m.Kpad;
  const int KT = FAST ? 4 : d.KT;  // the fast path runs max_states = 4 (4 labels per row)
  const int RW = 3 + KT;  // words per row: max, sum exp, blank logit, KT candidates
  const int cg0 = mem * NCG;
  const size_t row0 = (size_t)b * Nc;
  const unsigned stride_tb = (unsigned)g.maxdeg + 1u;
  const bool writer = mem == 0;
  const int fb = d.base ? d.base[b] : 0;  // absolute index of this call's frame 0
  // the member's W slice (RES) and bias, for the whole decode
  float4 wres[kResSlices];
  if (RES) {
    const float4* __restrict__ Wi = reinterpret_cast<const float4*>(m.Wi);
    const int q0 = wave * kResSlices;
#pragma unroll
    for (int u = 0; u < kResSlices; ++u) wres[u] = Wi[(size_t)(q0 + u) * m.Vpad + cg0 * 64 + lane];
  }
  float bias_r[NCG];
#pragma unroll
  for (int jj = 0; jj < NCG; ++jj) bias_r[jj] = m.bias[min((cg0 + jj) * 64 + lane, V - 1)];
  if (tid == 0) {
    s.ns = d.nsurv[b];
    s.nc = d.nctx[b];
    s.off_d = d.offset[b];
  }
  for (int i = tid; i < Ns; i += blockDim.x) {
    const size_t o = (size_t)b * Ns + i;
    s.s_ctx[i] = d.surv_ctx[o];
    s.s_state[i] = d.surv_state[o];
    s.s_row[i] = d.surv_row[o];
    s.s_score[i] = d.surv_score[o];
    s.s_bprev[i] = s.s_ctx[i] % V;
  }
  for (int j = tid; j < Nc; j += blockDim.x) {
    const int c = d.ctx_list[row0 + j], a = c / V;
    s.n_rowoff[j] = make_int2(a * Kpad, (c - a * V) * Kpad);
  }
  {
    const float* er = d.enc + (size_t)b * d.T * C;
    for (int k = tid; k < C; k += blockDim.x) s.enc_next[k] = er[k];
    const int words = RG * 4 * hstride;
    for (int i = tid; i < words; i += blockDim.x) reinterpret_cast<int*>(hl)[i] = 0;
  }
  __syncthreads();
  write_h_rows<kSearchThreads>(m, s.enc_next, 0, s.n_rowoff, s.nc, hl, hstride, tid);
  __syncthreads();
  // FAST: this lane's two columns, the decoder rows of the current contexts there,
  // the survivor buffer and the tuple / context counts of the current frame
  const int k0 = 128 * wave + 2 * lane;
  float2* dstage = reinterpret_cast<float2*>(smem + ly.doff) + (size_t)wave * kFastDecEntries * 64;
  float2 dcur[4];
  int ns_r = s.ns, nc_r = s.nc, sb = 0;
  if (FAST) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      dcur[j] = make_float2(0.f, 0.f);
      if (j < nc_r) {
        const int2 off = s.n_rowoff[j];
        dcur[j].x = fmaxf(m.P0[(size_t)off.x + k0] + m.P1[(size_t)off.y + k0], 0.f);
        dcur[j].y = fmaxf(m.P0[(size_t)off.x + k0 + 1] + m.P1[(size_t)off.y + k0 + 1], 0.f);
      }
    }
  }
  constexpr int NEP = FAST ? 1 : kMaxDim / kSearchThreads;
  for (int t = 0; t < L; ++t) {
    // encoder frame t + 1, in flight during the joiner and the exchange
    float encp[NEP];
    float2 encf = make_float2(0.f, 0.f);
    if (FAST) {
      if (t + 1 < L) {
        const float* er = d.enc + ((size_t)b * d.T + t + 1) * C;
        encf.x = k0 < C ? er[k0] : 0.f;
        encf.y = k0 + 1 < C ? er[k0 + 1] : 0.f;
      }
    } else {
      const float* er = d.enc + ((size_t)b * d.T + min(t + 1, L - 1)) * C;
#pragma unroll
      for (int u = 0; u < NEP; ++u) {
        const int k = tid + u * kSearchThreads;
        encp[u] = k < C ? er[k] : 0.f;
      }
    }
    // the partial sums use the hash table's LDS, idle until the search
    float* part = reinterpret_cast<float*>(s.hk);
    group_joiner_f32<RG, NCG, RES>(m, hl, hstride, part, cg0, wres);
    // FAST: the P0 rows of the survivors' last labels at this lane's columns (read
    // after the joiner's barrier, which orders them after wave 0's survivor writes;
    // the label candidates' decoder rows add P1 rows once the labels are known)
    float2 p0[4];
    if (FAST) {
      const char* P0b = reinterpret_cast<const char*>(m.P0);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int a = s.s_bprev[sb + i];  // (absent survivors: anything, mapped into row 0)
        p0[i] = *reinterpret_cast<const float2*>(
            P0b + (unsigned)(((unsigned)a < (unsigned)V ? a : 0) * kKStep + k0) * 4u);
      }
    }
    const int nc = FAST ? nc_r : s.nc;
    const unsigned long long tg = (unsigned long long)((x.epoch << 8) | ((unsigned)t & 0xffu)) << 48;
    // this member's row statistics over its columns (partial sums added in wave
    // order, bias, -inf beyond V) -> tagged words
    {
      constexpr int NR = 4 * RG, PER = NCG * NR * 64;
      unsigned long long* slot = group_slot(x, b, mem, t);
      for (int j = wave; j < nc; j += 4) {
        float z[NCG];
        float mx = -INFINITY;
#pragma unroll
        for (int jj = 0; jj < NCG; ++jj) {
          const int col = (cg0 + jj) * 64 + lane;
          const int e = (jj * NR + j) * 64 + lane;
          const float zs = ((part[e] + part[PER + e]) + part[2 * PER + e]) + part[3 * PER + e];
          z[jj] = col < V ? zs + bias_r[jj] : -INFINITY;
          mx = fmaxf(mx, z[jj]);
        }
        const float M = wave_max_f(mx);
        float se = 0.f;
#pragma unroll
        for (int jj = 0; jj < NCG; ++jj) se += __expf(z[jj] - M);
        const float S = wave_sum_f(se);
        // the maximum, exp-sum and blank logit go out first: the other members start
        // their normalisers while the candidates are ranked
        unsigned long long* w = slot + (size_t)j * RW;
        if (lane == 0) {
          xw_store(x, xr, w, tg | __float_as_uint(M));
          xw_store(x, xr, w + 1, tg | __float_as_uint(S));
          const float z0 = cg0 == 0 ? z[0] : 0.f;  // lane 0 of the first member holds label 0
          xw_store(x, xr, w + 2, tg | __float_as_uint(z0));
        }
        // best KT labels in 1..V-1 by (logit desc, label asc); lane q keeps the q-th
        float my_z = -INFINITY;
        int my_c = -1;
        if (NCG == 1) {
          // one column per lane: the wave maximum of the order-preserving code, the
          // smallest lane among equal codes (columns rise with the lane)
          const int col = cg0 * 64 + lane;
          unsigned o = (col >= 1 && col < V) ? f2ord(z[0]) : 0u;
          for (int q = 0; q < KT; ++q) {
            const unsigned mo = wave_max_u32(o);
            if (mo == 0u) break;
            const int wl = __ffsll((long long)__ballot(o == mo)) - 1;
            if (lane == q) {
              my_z = ord2f(mo);
              my_c = cg0 * 64 + wl;
            }
            if (lane == wl) o = 0u;
          }
        } else {
          unsigned long long key[NCG];
#pragma unroll
          for (int jj = 0; jj < NCG; ++jj) {
            const int col = (cg0 + jj) * 64 + lane;
            key[jj] = (col >= 1 && col < V)
                          ? ((unsigned long long)f2ord(z[jj]) << 32) | (0xffffffffu - (unsigned)col)
                          : 0ull;
          }
          unsigned long long prev = ~0ull;
          for (int q = 0; q < KT; ++q) {
            unsigned long long mine = 0ull;
#pragma unroll
            for (int jj = 0; jj < NCG; ++jj) mine = (key[jj] < prev && key[jj] > mine) ? key[jj] : mine;
            const unsigned long long best = wave_max_u64(mine);
            if (lane == q && best != 0ull) {
              my_z = ord2f((unsigned)(best >> 32));
              my_c = (int)(0xffffffffu - (unsigned)best);
            }
            prev = best ? best : 1ull;
          }
        }
        if (lane < KT) {
          const unsigned long long c16 = my_c > 0 ? (unsigned long long)my_c << 32 : 0ull;
          xw_store(x, xr, w + 3 + lane, tg | c16 | __float_as_uint(my_z));
        }
      }
    }
    if (!FAST && t + 1 < L) {
#pragma unroll
      for (int u = 0; u < NEP; ++u) {
        const int k = tid + u * kSearchThreads;
        if (k < C) s.enc_next[k] = encp[u];
      }
    }
    // Each wave then takes its rows again: it polls the members' words of the row
    // (bounded) and combines them in member order, identically in every member.  The
    // maxima and exp-sums are waited for first and the normaliser computed while the
    // candidates' words (published later by each member) are still on their way.
    {
      const unsigned tag = (unsigned)(tg >> 48);
      // the payload of word wi of a row once its tag is this frame's; a wait that
      // runs out (or finds another wait already given up) is recorded and yields a
      // neutral payload: -inf with label 0 (none), and a zero exp-sum
      auto settle = [&](const unsigned long long* w, unsigned long long v, int wi) {
        unsigned n = 0;
        while ((unsigned)(v >> 48) != tag) {
          ++n;
          if (n > x.spin_limit ||
              ((n & 255u) == 0 &&
               __hip_atomic_load(x.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u)) {
            __hip_atomic_fetch_add(x.err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_fetch_add(x.err + 1 + b, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            return wi == 1 ? 0ull : 0xff800000ull;
          }
          v = xw_load(x, xr, w);
        }
        return v & 0xffffffffffffull;
      };
      auto wload = [&](const unsigned long long* w) { return xw_load(x, xr, w); };
      const int ne = G * KT;
      for (int j = wave; j < nc; j += 4) {
        // lanes g < G: member g's maximum; G + g: its exp-sum; 2 G: member 0's blank logit
        const bool hasA = lane <= 2 * G;
        const int ga = lane < G ? lane : (lane < 2 * G ? lane - G : 0);
        const int wa = lane < G ? 0 : (lane < 2 * G ? 1 : 2);
        const unsigned long long* pa = group_slot(x, b, ga, t) + (size_t)j * RW + wa;
        // candidate entry e (member e / KT, its (e mod KT)-th): lanes e and e - 64
        const unsigned long long* pb[2];
        unsigned long long vb[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int e = min(lane + 64 * h, ne - 1), g2 = e / KT;
          pb[h] = group_slot(x, b, g2, t) + (size_t)j * RW + 3 + (e - g2 * KT);
        }
        unsigned long long va = hasA ? wload(pa) : 0ull;
#pragma unroll
        for (int h = 0; h < 2; ++h) vb[h] = (lane + 64 * h < ne) ? wload(pb[h]) : 0ull;
        if (hasA) va = settle(pa, va, wa);
        // (the wave reductions combine in a fixed order, the same in every member)
        const unsigned vs = (unsigned)__shfl((int)(unsigned)va, min(lane + G, 63));
        const float Mg = lane < G ? __uint_as_float((unsigned)va) : -INFINITY;
        const float Sg = lane < G ? __uint_as_float(vs) : 0.f;
        const float M = wave_max_f(Mg);
        const float S = wave_sum_f(Sg == 0.f ? 0.f : Sg * __expf(Mg - M));
        const float z0 = __uint_as_float((unsigned)__builtin_amdgcn_readlane((int)(unsigned)va, 2 * G));
        if (lane == 0) {
          s.s_lse[j] = lse_of(M, S);
          s.s_z0[j] = z0;
        }
#pragma unroll
        for (int h = 0; h < 2; ++h)
          if (lane + 64 * h < ne) vb[h] = settle(pb[h], vb[h], 3);
        // best KT labels over the G lists (the members' columns are disjoint, so the
        // labels are distinct)
        if (ne <= 64) {
          // one entry per lane: wave maximum of the code; equal codes (rare) go to the
          // smaller label
          unsigned o = 0u, c = 0xffffffffu;
          if (lane < ne && (vb[0] >> 32) != 0ull) {
            o = f2ord(__uint_as_float((unsigned)vb[0]));
            c = (unsigned)(vb[0] >> 32);
          }
          for (int q = 0; q < KT; ++q) {
            const unsigned mo = wave_max_u32(o);
            float zq = -INFINITY;
            int cq = -1;
            if (mo != 0u) {
              unsigned long long bal = __ballot(o == mo);
              if (__popcll(bal) > 1) {
                const unsigned cm = wave_min_u32(o == mo ? c : 0xffffffffu);
                bal = __ballot(o == mo && c == cm);
              }
              const int wl = __ffsll((long long)bal) - 1;
              zq = ord2f(mo);
              cq = __builtin_amdgcn_readlane((int)c, wl);
              if (lane == wl) o = 0u;
            }
            if (lane == 0) {
              s.rk_z[j * KT + q] = zq;
              s.rk_c[j * KT + q] = cq;
            }
          }
        } else {
          unsigned long long kv[2];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const unsigned c = (unsigned)(vb[h] >> 32);
            kv[h] = (lane + 64 * h < ne && c != 0u)
                        ? ((unsigned long long)f2ord(__uint_as_float((unsigned)vb[h])) << 32) | (0xffffffffu - c)
                        : 0ull;
          }
          unsigned long long prev = ~0ull;
          for (int q = 0; q < KT; ++q) {
            unsigned long long mine = 0ull;
#pragma unroll
            for (int h = 0; h < 2; ++h) mine = (kv[h] < prev && kv[h] > mine) ? kv[h] : mine;
            const unsigned long long best = wave_max_u64(mine);
            if (lane == 0) {
              s.rk_z[j * KT + q] = best ? ord2f((unsigned)(best >> 32)) : -INFINITY;
              s.rk_c[j * KT + q] = best ? (int)(0xffffffffu - (unsigned)best) : -1;
            }
            prev = best ? best : 1ull;
          }
        }
      }
    }
    __syncthreads();
    if (!FAST) {
      search_frame<true, true>(m, g, d, beam, t, L, b, trace, s, hl, hstride, nullptr, true,
                               writer, true, nullptr, 0, fb);
      __syncthreads();
      continue;
    }
    // ---- fast path: no workgroup barrier until the next frame's joiner ----
    // decoder-row inputs of every label candidate (survivor i, label q) at this
    // lane's two columns; every load is issued (clamped), then the selection runs
    // (on this path every context holds one tuple, so survivor i sits on context row
    // i.  The LDS reads are unconditional and issued together; entries of absent
    // survivors or labels may hold anything and are mapped into row 0, never used)
    // (the survivors' P0 rows were requested after the joiner; 32-bit byte offsets
    // from the uniform base: P1 stays below 4 GiB)
    int pb[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int c = s.rk_c[i * 4 + q];
        pb[i][q] = (unsigned)c < (unsigned)V ? c : 0;
      }
    float2 p1[4][4];
    const char* P1b = reinterpret_cast<const char*>(m.P1);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        p1[i][q] = *reinterpret_cast<const float2*>(P1b + (unsigned)(pb[i][q] * kKStep + k0) * 4u);
    const WaveSel sel =
        trivial_select_wave<4>(s, ns_r, 4, V, Ns, Nc, beam, stride_tb, lane, sb, false);
    const int nk = sel.nk;
    const float best = sel.best;
    // decoder rows at this lane's columns of every candidate, staged in the wave's
    // LDS area by source index: label candidate 4 i + q, blank of row r at 16 + r
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        dstage[(4 * i + q) * 64 + lane] =
            make_float2(fmaxf(p0[i].x + p1[i][q].x, 0.f), fmaxf(p0[i].y + p1[i][q].y, 0.f));
#pragma unroll
    for (int r = 0; r < 4; ++r) dstage[(16 + r) * 64 + lane] = dcur[r];
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // each new context row j: its decoder row and its joiner row h = tanh(enc[t + 1] +
    // decoder row) at this lane's columns.  Rows j >= nk are computed from a stale
    // source and never read; columns k >= C come out exactly 0 (all inputs are zero
    // there and tanh(0) = 0); at the stream's last frame the rows are not read.
    int srcj[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const unsigned long long mj = __ballot(sel.keep2 && sel.pos == j);
      const int sj = __builtin_amdgcn_readlane(sel.src, mj ? __ffsll((long long)mj) - 1 : 0);
      srcj[j] = mj ? (sj >= 0 ? sj : 15 - sj) : 16;
    }
    float2 dv[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) dv[j] = dstage[srcj[j] * 64 + lane];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      dcur[j] = dv[j];
      const float2 h = make_float2(tanh_fast(encf.x + dv[j].x), tanh_fast(encf.y + dv[j].y));
      *reinterpret_cast<float2*>(hl + ((size_t)j * hstride + k0) * 4) = h;
    }
    // survivors of the next frame (other buffer), history, trace, outputs
    const int nb = sb ^ 4;
    const bool store_surv = writer && t + 1 == L;
    if (wave == 0 && sel.keep2) {
      const int pos = sel.pos;
      const unsigned tb = 0xffffffffu - (unsigned)sel.v;
      const int parent = (int)(tb / stride_tb);
      const int arc = (int)(tb - (unsigned)parent * stride_tb) - 1;  // label - 1, or -1 (blank)
      const int label = arc + 1;
      s.s_ctx[nb + pos] = (int)sel.ci;
      s.s_state[nb + pos] = (int)sel.st;
      s.s_score[nb + pos] = sel.sc - best;
      s.s_row[nb + pos] = pos;
      s.s_bprev[nb + pos] = (int)(sel.ci % (unsigned)V);
      if (store_surv) {
        const size_t o = (size_t)b * Ns + pos;
        d.surv_ctx[o] = (int)sel.ci;
        d.surv_state[o] = (int)sel.st;
        d.surv_score[o] = sel.sc - best;
        d.surv_row[o] = pos;
        d.ctx_list[row0 + pos] = (int)sel.ci;
      }
      if (writer) {
        const size_t hb = ((size_t)(fb + t) * d.B + b) * Ns + pos;
        d.hist_pl[hb] = (parent << 16) | label;
        d.hist_arc[hb] = arc;
        if (trace) {
          int* tr = trace + (((size_t)(fb + t + 1) * d.B + b) * Ns + pos) * 4;
          tr[0] = (int)sel.ci;
          tr[1] = (int)sel.st;
          tr[2] = parent;
          tr[3] = label;
        }
      }
    }
    if (tid == 0 && writer) {
      if (store_surv) {
        d.nsurv[b] = nk;
        d.nctx[b] = nk;
      }
      s.off_d += (double)best;
      if (t + 1 == L) d.offset[b] = s.off_d;
    }
    sb = nb;
    ns_r = nk;
    nc_r = nk;
    // this wave's joiner reads only the rows it has just written
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
}

// ---------------------------------------------------------------------------
// final selection and traceback

constexpr int kFinalBuf = 4096;

__global__ __launch_bounds__(256) void k_final(GraphDev g, DecodeDev d, int* __restrict__ out_tokens,
                                               int* __restrict__ out_ntok,
                                               double* __restrict__ out_scores,
                                               int* __restrict__ out_status,
                                               int* __restrict__ out_arcs,
                                               const unsigned* __restrict__ xerr) {
  __shared__ int buf_pl[kFinalBuf];
  __shared__ int buf_arc[kFinalBuf];
  __shared__ int s_idx;
  __shared__ int s_wsum[4];
  const int b = blockIdx.x, tid = threadIdx.x;
  const int Ns = d.Ns, T = d.T, len = d.len[b];
  if (d.graphs) g = d.graphs[b];  // per-stream graphs
  if (tid == 0) {
    const int ns = d.nsurv[b];
    int pick = -1, status = 0;
    float pv = -INFINITY;
    for (int pass = 0; pass < 2 && pick < 0; ++pass) {
      for (int i = 0; i < ns; ++i) {
        const int st = d.surv_state[(size_t)b * Ns + i];
        const float f = g.fin ? g.fin[st] : 0.f;
        if (pass == 0 && !(f > -INFINITY)) continue;
        const float v = d.surv_score[(size_t)b * Ns + i] + (pass == 0 ? f : 0.f);
        if (pick < 0 || v > pv) {
          pv = v;
          pick = i;
        }
      }
      status = pass;
    }
    const int st = d.surv_state[(size_t)b * Ns + pick];
    const double f = (status == 0 && g.fin) ? (double)g.fin[st] : 0.0;
    out_scores[b] = (double)d.surv_score[(size_t)b * Ns + pick] + d.offset[b] + f;
    if (xerr && xerr[1 + b]) {  // a grouped stream's exchange wait timed out
      status = 2;
      out_scores[b] = __longlong_as_double(0x7ff8000000000000ll);  // NaN
    }
    if (out_status) out_status[b] = status;
    s_idx = pick;
  }
  __syncthreads();
  // walk back, staging the stream's history rows through LDS
  const int F = kFinalBuf / Ns;
  int* plab = d.path_lab + (size_t)b * T;
  for (int thi = len; thi > 0; thi -= F) {
    const int tlo = max(0, thi - F);
    const int n = (thi - tlo) * Ns;
    for (int i = tid; i < n; i += blockDim.x) {
      const int tt = tlo + i / Ns, p = i - (i / Ns) * Ns;
      const size_t o = ((size_t)tt * d.B + b) * Ns + p;
      buf_pl[i] = d.hist_pl[o];
      if (out_arcs) buf_arc[i] = d.hist_arc[o];
    }
    __syncthreads();
    if (tid == 0) {
      int idx = s_idx;
      for (int tt = thi - 1; tt >= tlo; --tt) {
        const int pl = buf_pl[(tt - tlo) * Ns + idx];
        plab[tt] = pl & 0xffff;
        if (out_arcs) out_arcs[(size_t)b * T + tt] = buf_arc[(tt - tlo) * Ns + idx];
        idx = pl >> 16;
      }
      s_idx = idx;
    }
    __syncthreads();
  }
  // compact non-blank labels in frame order
  int total = 0;
  const int lane = tid & 63, wave = tid >> 6;
  for (int t0 = 0; t0 < len; t0 += 256) {
    const int tt = t0 + tid;
    const int lab = tt < len ? plab[tt] : 0;
    const int flag = lab > 0;
    int incl = flag;
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(incl, o);
      if (lane >= o) incl += y;
    }
    if (lane == 63) s_wsum[wave] = incl;
    __syncthreads();
    int woff = 0;
    for (int w = 0; w < wave; ++w) woff += s_wsum[w];
    const int tile_total = s_wsum[0] + s_wsum[1] + s_wsum[2] + s_wsum[3];
    if (flag) out_tokens[(size_t)b * T + total + woff + incl - 1] = lab;
    total += tile_total;
    __syncthreads();
  }
  for (int i = total + tid; i < T; i += blockDim.x) out_tokens[(size_t)b * T + i] = -1;
  if (out_arcs)
    for (int i = len + tid; i < T; i += blockDim.x) out_arcs[(size_t)b * T + i] = -2;
  if (tid == 0) out_ntok[b] = total;
}

// Timing events for the next launch (per-kernel profiling): when set, the launch
// records them in its own dispatch packet (hipExtLaunchKernel), so the interval
// between them is the kernel's execution and not the enqueue around it.
thread_local hipEvent_t g_ev_start = nullptr, g_ev_stop = nullptr;

template <typename F, typename... Args>
void launch_k(F kernel, dim3 grid, dim3 block, unsigned shmem, hipStream_t st, Args... args) {
  if (g_ev_start) {
    hipExtLaunchKernelGGL(kernel, grid, block, shmem, st, g_ev_start, g_ev_stop, 0u, args...);
    g_ev_start = g_ev_stop = nullptr;
  } else {
    hipLaunchKernelGGL(kernel, grid, block, shmem, st, args...);
  }
}

inline int grid_for(long long n, int threads, int cap = 4096) {
  long long g = (n + threads - 1) / threads;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return (int)g;
}

template <bool BF16, bool TOPK, int WN, int MBW>
hipError_t launch_joiner_t(const ModelDev& m, const JoinArgs& a, const JoinerPlan& p,
                           hipStream_t st) {
  static size_t attr = 0;  // dynamic LDS limit granted so far (kernel default: 64 KiB)
  if (p.lds > 65536 && p.lds > attr) {
    hipError_t e = hipFuncSetAttribute((const void*)k_joiner<BF16, TOPK, WN, MBW>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)p.lds);
    if (e != hipSuccess) return e;
    attr = p.lds;
  }
  launch_k((k_joiner<BF16, TOPK, WN, MBW>), dim3(p.grid), dim3(128 * WN), p.lds, st, m, a);
  return hipGetLastError();
}

template <bool BF16, int MB, bool TOPK>
hipError_t launch_joiner_small_t(const ModelDev& m, const JoinArgs& a, const JoinerPlan& p,
                                 hipStream_t st) {
  static size_t attr = 0;
  if (p.lds > 65536 && p.lds > attr) {
    hipError_t e = hipFuncSetAttribute((const void*)k_joiner_small<BF16, MB, TOPK>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)p.lds);
    if (e != hipSuccess) return e;
    attr = p.lds;
  }
  launch_k((k_joiner_small<BF16, MB, TOPK>), dim3(p.grid), dim3(256), p.lds, st, m, a);
  return hipGetLastError();
}

template <bool BF16, bool TOPK>
hipError_t launch_joiner_small(const ModelDev& m, const JoinArgs& a, const JoinerPlan& p,
                               hipStream_t st) {
  switch (p.MB) {
    case 1: return launch_joiner_small_t<BF16, 1, TOPK>(m, a, p, st);
    case 2: return launch_joiner_small_t<BF16, 2, TOPK>(m, a, p, st);
    default: return launch_joiner_small_t<BF16, 4, TOPK>(m, a, p, st);
  }
}

hipError_t launch_joiner(const ModelDev& m, const JoinArgs& a, const JoinerPlan& p, bool topk,
                         hipStream_t st) {
  if (p.MB == 0) {  // the GEMM tiles address h and W with 32-bit byte offsets
    const unsigned long long rowb = (unsigned long long)m.Kpad * (m.bf16 ? 2 : 4);
    if ((unsigned long long)a.R * rowb >= (1ull << 32) || (unsigned long long)m.Vpad * rowb >= (1ull << 32))
      return hipErrorInvalidValue;
  }
  if (p.MB == 0 && p.shape == 1) {  // bf16 logits only
    if (!m.bf16 || topk) return hipErrorInvalidValue;
    return launch_joiner_t<true, false, 4, 8>(m, a, p, st);
  }
  if (p.MB == 0 && p.shape == 2) {
    if (m.bf16)
      return topk ? launch_joiner_t<true, true, 2, 2>(m, a, p, st)
                  : launch_joiner_t<true, false, 2, 2>(m, a, p, st);
    return topk ? launch_joiner_t<false, true, 2, 2>(m, a, p, st)
                : launch_joiner_t<false, false, 2, 2>(m, a, p, st);
  }
  if (p.MB == 0) {
    if (m.bf16)
      return topk ? launch_joiner_t<true, true, 2, 4>(m, a, p, st)
                  : launch_joiner_t<true, false, 2, 4>(m, a, p, st);
    return topk ? launch_joiner_t<false, true, 2, 4>(m, a, p, st)
                : launch_joiner_t<false, false, 2, 4>(m, a, p, st);
  }
  if (m.bf16)
    return topk ? launch_joiner_small<true, true>(m, a, p, st) : launch_joiner_small<true, false>(m, a, p, st);
  return topk ? launch_joiner_small<false, true>(m, a, p, st) : launch_joiner_small<false, false>(m, a, p, st);
}

}  // namespace

void set_launch_events(hipEvent_t start, hipEvent_t stop) {
  g_ev_start = start;
  g_ev_stop = stop;
}

bool launch_events_pending() { return g_ev_start != nullptr; }

bool take_launch_events(hipEvent_t* start, hipEvent_t* stop) {
  if (!g_ev_start) return false;
  *start = g_ev_start;
  *stop = g_ev_stop;
  g_ev_start = g_ev_stop = nullptr;
  return true;
}

JoinerPlan plan_joiner(int rows, int Vpad, int Kpad, int bf16, int ncu, bool topk) {
  JoinerPlan p;
  p.shape = 0;
  const int esz = bf16 ? 2 : 4;
  const int nvt = Vpad / kJoinerBN;
  // bf16 logits: 256 x 256 GEMM tiles when they give every compute unit several
  if (bf16 && !topk) {
    p.n_rt = (rows + kJWideBM - 1) / kJWideBM;
    p.n_ct = (nvt * kJoinerBN + kJWideBN - 1) / kJWideBN;
    const long long tiles = (long long)p.n_rt * p.n_ct;
    if (tiles >= 4LL * ncu) {
      p.MB = 0;
      p.shape = 1;
      p.grid = (int)(8 * ((tiles + 7) / 8));
      p.lds = kJWideLds;
      return p;
    }
  }
  // 128 x 128 GEMM tiles when they give every compute unit one (MB = 0)
  p.n_rt = (rows + kJBM - 1) / kJBM;
  p.n_ct = (nvt + 1) / 2;
  if ((long long)p.n_rt * p.n_ct >= ncu) {
    p.MB = 0;
    if ((long long)p.n_rt * p.n_ct < 4LL * ncu) {
      // a few 128 x 128 tiles per CU: 64 x 128 tiles (three workgroups per CU), which
      // spread the work over the CUs in finer and more even parts
      p.shape = 2;
      p.n_rt = (rows + kJHalfBM - 1) / kJHalfBM;
      p.lds = kJHalfLds;
    } else {
      p.lds = kJLds;
    }
    p.grid = 8 * ((p.n_ct + 7) / 8) * p.n_rt;
    return p;
  }
  // Otherwise small tiles: the largest row block (4 or 2 MFMA blocks, else 1) whose h
  // tile leaves room for two workgroups per CU and still yields a workgroup per CU.
  int MB = 1;
  for (int cand : {4, 2}) {
    const size_t lds = (size_t)16 * cand * (Kpad + (bf16 ? 8 : 4)) * esz;
    const long long tiles = (long long)((rows + 16 * cand - 1) / (16 * cand)) * nvt;
    if (lds <= 78 * 1024 && tiles >= ncu) {
      MB = cand;
      break;
    }
  }
  p.MB = MB;
  p.n_rt = (rows + 16 * MB - 1) / (16 * MB);
  p.n_ct = nvt;
  p.grid = 8 * ((nvt + 7) / 8) * p.n_rt;
  p.lds = (size_t)16 * MB * (Kpad + (bf16 ? 8 : 4)) * esz;
  return p;
}

hipError_t launch_model_setup(const float* embed, const float* conv, const float* w_out,
                              const float* b_out, int V, int C, int Kpad, int Vpad, int bf16,
                              float* P0, float* P1, float* Wf, uint16_t* Wb, void* Wi,
                              float* bias, hipStream_t st) {
  hipLaunchKernelGGL(k_model_setup, dim3(grid_for((long long)Vpad * Kpad, 256)), dim3(256), 0, st,
                     embed, conv, w_out, b_out, V, C, Kpad, Vpad, bf16, P0, P1, Wf, Wb, Wi, bias);
  return hipGetLastError();
}

hipError_t launch_clamp_lengths(const int* in, int* out, int B, int T, hipStream_t st) {
  if (B <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_clamp_lengths, dim3((B + 255) / 256), dim3(256), 0, st, in, out, B, T);
  return hipGetLastError();
}

hipError_t launch_fill_i32(int* p, long long n, int v, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_fill_i32, dim3(grid_for(n, 256)), dim3(256), 0, st, p, n, v);
  return hipGetLastError();
}

hipError_t launch_resume(const ModelDev& m, const DecodeDev& d, const GraphDev& g, int* trace,
                         int rows_needed, hipStream_t st) {
  hipLaunchKernelGGL(k_resume, dim3(d.B), dim3(256), 0, st, m, d, g, trace, rows_needed);
  return hipGetLastError();
}

hipError_t launch_init(const ModelDev& m, const DecodeDev& d, const GraphDev& g, int* trace,
                       hipStream_t st) {
  hipLaunchKernelGGL(k_init, dim3(d.B), dim3(256), 0, st, m, d, g, trace);
  return hipGetLastError();
}

hipError_t launch_joiner_frame(const ModelDev& m, const DecodeDev& d, const JoinerPlan& p, int t,
                               hipStream_t st) {
  JoinArgs a{};
  a.h = d.h;
  a.logits = d.logits;
  a.stats = d.stats;
  a.tk_z = d.tk_z;
  a.tk_c = d.tk_c;
  a.z0 = d.z0;
  a.KT = d.KT;
  a.R = d.B * d.Nc;
  a.n_rt = p.n_rt;
  a.n_ct = p.n_ct;
  a.nvt = m.Vpad / kJoinerBN;
  a.rows_mode = 0;
  a.len = d.len;
  a.nctx = d.nctx;
  a.t = t;
  a.Nc = d.Nc;
  return launch_joiner(m, a, p, d.KT > 0, st);
}

hipError_t launch_search_frame(const ModelDev& m, const GraphDev& g, const DecodeDev& d,
                               float beam, int t, int* trace, hipStream_t st) {
  // (the attribute admits the whole layout; a launch allocates enc_next up to Kpad)
  const size_t lds = offsetof(SearchSmem, enc_next) + (size_t)m.Kpad * sizeof(float);
  const int lds_max = (int)sizeof(SearchSmem);
  if (d.KT > 0) {
    static bool attr = false;
    if (!attr) {
      hipError_t e = hipFuncSetAttribute((const void*)k_search<true>,
                                         hipFuncAttributeMaxDynamicSharedMemorySize, lds_max);
      if (e != hipSuccess) return e;
      attr = true;
    }
    launch_k(k_search<true>, dim3(d.B), dim3(kSearchThreads), lds, st, m, g, d, beam, t,
                       trace);
  } else {
    static bool attr = false;
    if (!attr) {
      hipError_t e = hipFuncSetAttribute((const void*)k_search<false>,
                                         hipFuncAttributeMaxDynamicSharedMemorySize, lds_max);
      if (e != hipSuccess) return e;
      attr = true;
    }
    launch_k(k_search<false>, dim3(d.B), dim3(kSearchThreads), lds, st, m, g, d, beam, t,
                       trace);
  }
  return hipGetLastError();
}

StreamPlan plan_stream(const ModelDev& m, int Nc, int KT, int trivial) {
  StreamPlan p{};
  const int esz = m.bf16 ? 2 : 4;
  const int nvt = m.Vpad / kJoinerBN;
  p.RG = (Nc + 3) / 4;
  p.hstride = m.Kpad + 16 / esz;
  p.hoff = (int)round_up((int)sizeof(SearchSmem), 16);
  p.zoff = p.hoff + p.RG * 4 * p.hstride * esz;
  p.lds = (size_t)p.zoff + (size_t)p.RG * 4 * m.Vpad * 4;
  p.ok = Nc <= 16 && m.Vpad <= kStreamMaxV && p.lds <= kMaxLds && (!trivial || KT > 0);
  // trivial graph with max_states = 4: staged decoder rows of the candidates and contexts
  p.doff = 0;
  const size_t dbeg = (p.lds + 15) / 16 * 16, dend = dbeg + (size_t)(16 + 8) * m.Kpad * 4;
  if (trivial && KT == 4 && dend <= kMaxLds) {
    p.doff = (int)dbeg;
    p.lds = dend;
  }
  (void)nvt;
  return p;
}

template <bool BF16, bool TRIV, int RG>
hipError_t launch_stream_t(const ModelDev& m, const GraphDev& g, const DecodeDev& d, float beam,
                           int* trace, const StreamPlan& p, hipStream_t st) {
  static size_t attr = 0;
  if (p.lds > attr) {
    hipError_t e = hipFuncSetAttribute((const void*)k_stream<BF16, TRIV, RG>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)p.lds);
    if (e != hipSuccess) return e;
    attr = p.lds;
  }
  launch_k((k_stream<BF16, TRIV, RG>), dim3(d.B), dim3(kSearchThreads), p.lds, st, m, g, d, beam,
           trace, p.hoff, p.hstride, p.zoff, p.doff);
  return hipGetLastError();
}

template <bool BF16, bool TRIV>
hipError_t launch_stream_rg(const ModelDev& m, const GraphDev& g, const DecodeDev& d, float beam,
                            int* trace, const StreamPlan& p, hipStream_t st) {
  switch (p.RG) {
    case 1: return launch_stream_t<BF16, TRIV, 1>(m, g, d, beam, trace, p, st);
    case 2: return launch_stream_t<BF16, TRIV, 2>(m, g, d, beam, trace, p, st);
    case 3: return launch_stream_t<BF16, TRIV, 3>(m, g, d, beam, trace, p, st);
    default: return launch_stream_t<BF16, TRIV, 4>(m, g, d, beam, trace, p, st);
  }
}

hipError_t launch_stream(const ModelDev& m, const GraphDev& g, const DecodeDev& d, float beam,
                         int* trace, const StreamPlan& p, hipStream_t st) {
  if (!p.ok) return hipErrorInvalidValue;
  const bool triv = d.KT > 0;
  if (m.bf16)
    return triv ? launch_stream_rg<true, true>(m, g, d, beam, trace, p, st)
                : launch_stream_rg<true, false>(m, g, d, beam, trace, p, st);
  return triv ? launch_stream_rg<false, true>(m, g, d, beam, trace, p, st)
              : launch_stream_rg<false, false>(m, g, d, beam, trace, p, st);
}

int group_words(int Nc, int KT) { return Nc * (3 + KT); }

template <int RG, int NCG, bool RES, bool FAST>
hipError_t launch_group_t(const ModelDev& m, const GraphDev& g, const DecodeDev& d, float beam,
                          int* trace, const GroupLds& ly, size_t lds, const GroupX& x,
                          hipStream_t st) {
  static size_t attr = 0;
  if (lds > attr) {
    hipError_t e = hipFuncSetAttribute((const void*)k_stream_group<RG, NCG, RES, FAST>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr = lds;
  }
  ModelDev ma = m;
  GraphDev ga = g;
  DecodeDev da = d;
  GroupLds la = ly;
  GroupX xa = x;
  void* args[] = {&ma, &ga, &da, &beam, &trace, &la, &xa};
  return hipLaunchCooperativeKernel((const void*)k_stream_group<RG, NCG, RES, FAST>,
                                    dim3(d.B * x.G), dim3(kSearchThreads), args, (unsigned)lds, st);
}

template <int NCG, bool RES>
hipError_t launch_group_rg(int RG, const ModelDev& m, const GraphDev& g, const DecodeDev& d,
                           float beam, int* trace, const GroupLds& ly, size_t lds, const GroupX& x,
                           hipStream_t st) {
  switch (RG) {
    case 1: return launch_group_t<1, NCG, RES, false>(m, g, d, beam, trace, ly, lds, x, st);
    case 2: return launch_group_t<2, NCG, RES, false>(m, g, d, beam, trace, ly, lds, x, st);
    case 3: return launch_group_t<3, NCG, RES, false>(m, g, d, beam, trace, ly, lds, x, st);
    default: return launch_group_t<4, NCG, RES, false>(m, g, d, beam, trace, ly, lds, x, st);
  }
}

// Compute units of the current device (cached per device).
static int device_cus() {
  static int cus[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  if (cus[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    cus[dev] = n;
  }
  return cus[dev];
}

hipError_t launch_stream_group(const ModelDev& m, const GraphDev& g, const DecodeDev& d, float beam,
                               int* trace, const StreamPlan& p, unsigned long long* xbuf, int G,
                               unsigned epoch, unsigned spin_limit, unsigned* err,
                               hipStream_t st) {
  const int ncg = m.Vpad / kJoinerBN;
  if (!p.ok || m.bf16 || d.KT <= 0 || G < 2 || ncg % G != 0 || ncg / G > 2)
    return hipErrorInvalidValue;
  // one workgroup per CU (the LDS holds one) on all 256 CUs of the 8 XCDs
  const int ncu = device_cus();
  const bool xlocal = ncu == 256 && d.B * G == ncu && (ncu / 8) % G == 0;
  GroupX x{xbuf, G, group_words(d.Nc, d.KT), epoch & 0xffu, spin_limit, err,
           err + 1 + d.B, xlocal ? 1 : 0};
  if (xlocal) {  // the arrival counters start at zero for every launch
    const hipError_t e = launch_fill_i32(reinterpret_cast<int*>(x.tickets), kXTickets, 0, st);
    if (e != hipSuccess) return e;
  }
  // LDS: the search state, the joiner rows and (fast path) the staged decoder rows
  GroupLds ly{p.hoff, p.hstride, p.hoff + p.RG * 4 * p.hstride * 4};
  // one column group per member and K = 512: the member's W slice stays in registers;
  // with at most 4 tuples (4 rows) the per-wave fast path
  const bool res = ncg / G == 1 && m.Kpad == kKStep;
  const bool fast = res && p.RG == 1 && d.Ns == 4 && d.KT == 4;
  const size_t lds = (size_t)ly.doff + (fast ? (size_t)4 * kFastDecEntries * 64 * sizeof(float2) : 0);
  if (lds > kMaxLds) return hipErrorInvalidValue;
  if (ncg / G == 2) return launch_group_rg<2, false>(p.RG, m, g, d, beam, trace, ly, lds, x, st);
  if (fast) return launch_group_t<1, 1, true, true>(m, g, d, beam, trace, ly, lds, x, st);
  return res ? launch_group_rg<1, true>(p.RG, m, g, d, beam, trace, ly, lds, x, st)
             : launch_group_rg<1, false>(p.RG, m, g, d, beam, trace, ly, lds, x, st);
}

hipError_t launch_final(const GraphDev& g, const DecodeDev& d, int* out_tokens, int* out_ntok,
                        double* out_scores, int* out_status, int* out_arcs,
                        const unsigned* exchange_err, hipStream_t st) {
  launch_k(k_final, dim3(d.B), dim3(256), 0, st, g, d, out_tokens, out_ntok, out_scores,
                     out_status, out_arcs, exchange_err);
  return hipGetLastError();
}

hipError_t launch_h_rows_dense(const ModelDev& m, const float* enc, long long enc_stride,
                               const int* ctx, long long row0, int per_enc, int R, void* h,
                               hipStream_t st) {
  if (R <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_h_rows_dense, dim3(R), dim3(256), 0, st, m, enc, ctx, row0, per_enc,
                     enc_stride, h);
  return hipGetLastError();
}

hipError_t launch_joiner_dense(const ModelDev& m, const float* enc, long long enc_stride,
                               const int* ctx, long long row0, int per_enc, int R, void* h,
                               float* logits, float2* stats, int ncu, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  hipError_t e = launch_h_rows_dense(m, enc, enc_stride, ctx, row0, per_enc, R, h, st);
  if (e != hipSuccess) return e;
  return launch_joiner_gemm(m, h, R, logits, stats, ncu, st);
}

hipError_t launch_joiner_gemm(const ModelDev& m, const void* h, int R, float* logits,
                              float2* stats, int ncu, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  const JoinerPlan p = plan_joiner(R, m.Vpad, m.Kpad, m.bf16, ncu);
  JoinArgs a{};
  a.h = h;
  a.logits = logits;
  a.stats = stats;
  a.R = R;
  a.n_rt = p.n_rt;
  a.n_ct = p.n_ct;
  a.nvt = m.Vpad / kJoinerBN;
  a.rows_mode = 1;
  return launch_joiner(m, a, p, false, st);
}

hipError_t launch_joiner_rows(const ModelDev& m, const float* enc_rows, const int* ctx, int R,
                              void* h, float* logits, float2* stats, float* out_logp, int ncu,
                              hipStream_t st) {
  hipLaunchKernelGGL(k_h_rows, dim3(R), dim3(256), 0, st, m, enc_rows, ctx, h);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const JoinerPlan p = plan_joiner(R, m.Vpad, m.Kpad, m.bf16, ncu);
  JoinArgs a{};
  a.h = h;
  a.logits = logits;
  a.stats = stats;
  a.R = R;
  a.n_rt = p.n_rt;
  a.n_ct = p.n_ct;
  a.nvt = m.Vpad / kJoinerBN;
  a.rows_mode = 1;
  e = launch_joiner(m, a, p, false, st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_logp_rows, dim3(R), dim3(256), 0, st, logits, stats, a.nvt, m.V, m.Vpad,
                     out_logp);
  return hipGetLastError();
}

}  // namespace tbs
