// gfx950 kernels for batched FSA-based one-symbol-per-frame transducer beam
// search (Kang et al., arXiv 2211.00484, Sec. 2.2-2.5 and Algorithm 1).
//
// Per frame t (Algorithm 1 loop body):
//   k_joiner  GetContexts rows -> decoder (ReLU of conv-tap-scaled embedding
//             rows) + IndexSelect of enc[b, t] -> tanh -> joiner GEMM on MFMA
//             -> logits and per-tile (max, sum exp) partials of the log-softmax.
//   k_search  one workgroup per stream: log-softmax normaliser, ExpandArcs over
//             the CSR graph without pruning, max-merge of equal (state, context)
//             keys in an LDS hash table, beam + max-states selection by radix
//             select, max-contexts selection, canonical (context, state) order,
//             score renormalisation and the back-pointer history.
// After the last frame, k_final picks the best final tuple and traces back.
#include "internal.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

namespace tbs {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));

constexpr unsigned long long kEmpty = ~0ull;

// ---------------------------------------------------------------------------
// small helpers

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);  // round to nearest, ties to even (finite inputs)
  return (uint16_t)(u >> 16);
}

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

// ---------------------------------------------------------------------------
// model setup: P0 = tap0 * E, P1 = tap1 * E (padded to Kpad), W packed to
// [Vpad][Kpad] in fp32 or bf16, bias copied (zeros if absent).

__global__ void k_model_setup(const float* __restrict__ E, const float* __restrict__ conv,
                              const float* __restrict__ W, const float* __restrict__ b_out, int V,
                              int C, int Kpad, int Vpad, int bf16, float* __restrict__ P0,
                              float* __restrict__ P1, float* __restrict__ Wf,
                              uint16_t* __restrict__ Wb, float* __restrict__ bias) {
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
    if (bf16)
      Wb[i] = f32_to_bf16_rne(w);
    else
      Wf[i] = w;
    if (k == 0 && v < V) bias[v] = b_out ? b_out[v] : 0.f;
  }
}

__global__ void k_fill_i32(int* p, long long n, int v) {
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < n;
       i += (long long)gridDim.x * blockDim.x)
    p[i] = v;
}

// ---------------------------------------------------------------------------
// joiner

struct RowSrc {
  // decode mode: row r = b * Nc + j is context j of stream b at frame t
  const float* enc;
  int T, t, Nc;
  const int* len;
  const int* nctx;
  const int* ctx_list;
  // explicit-rows mode
  const float* enc_rows;
  const int* ctx_rows;
  int R;
  int rows_mode;
};

__device__ __forceinline__ bool row_info(const RowSrc& s, int C, int r, const float*& enc_row,
                                         int& ctx) {
  if (r >= s.R) return false;
  if (s.rows_mode) {
    enc_row = s.enc_rows + (size_t)r * C;
    ctx = s.ctx_rows[r];
    return true;
  }
  const int b = r / s.Nc, j = r - b * s.Nc;
  if (s.t >= s.len[b] || j >= s.nctx[b]) return false;
  enc_row = s.enc + ((size_t)b * s.T + s.t) * C;
  ctx = s.ctx_list[r];
  return true;
}

// One 16-row x 64-column tile per workgroup; wave w owns columns 16w..16w+15.
// The A operand h = tanh(enc + ReLU(P0[a] + P1[b])) is built in LDS (fp32 or
// bf16 RNE); W is streamed from its packed [Vpad][Kpad] copy.
template <bool BF16>
__global__ __launch_bounds__(256) void k_joiner(ModelDev m, RowSrc src, float* __restrict__ logits,
                                                float2* __restrict__ stats, int nvt) {
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ const float* s_enc[kJoinerBM];
  __shared__ int s_a[kJoinerBM], s_b[kJoinerBM], s_act[kJoinerBM];
  __shared__ float s_m[4][kJoinerBM], s_s[4][kJoinerBM];

  const int vt = blockIdx.x, r0 = blockIdx.y * kJoinerBM, n0 = vt * kJoinerBN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int C = m.C, V = m.V, Kpad = m.Kpad;

  if (tid < kJoinerBM) {
    const float* e = nullptr;
    int ctx = 0;
    const bool act = row_info(src, C, r0 + tid, e, ctx);
    s_act[tid] = act;
    s_enc[tid] = e;
    s_a[tid] = act ? ctx / V : 0;
    s_b[tid] = act ? ctx - (ctx / V) * V : 0;
  }
  __syncthreads();
  int any = 0;
#pragma unroll
  for (int i = 0; i < kJoinerBM; ++i) any |= s_act[i];
  if (!any) return;  // uniform across the workgroup

  // prologue: h tile in LDS
  const int ldk = BF16 ? Kpad + 8 : Kpad + 4;  // 16-byte row padding
  float* hs = reinterpret_cast<float*>(smem);
  uint16_t* hb = reinterpret_cast<uint16_t*>(smem);
  for (int r = 0; r < kJoinerBM; ++r) {
    const bool act = s_act[r];
    const float* e = s_enc[r];
    const float* p0 = m.P0 + (size_t)s_a[r] * Kpad;
    const float* p1 = m.P1 + (size_t)s_b[r] * Kpad;
    for (int k = tid; k < Kpad; k += 256) {
      float h = 0.f;
      if (act && k < C) {
        const float d = fmaxf(p0[k] + p1[k], 0.f);
        h = tanhf(e[k] + d);
      }
      if (BF16)
        hb[r * ldk + k] = f32_to_bf16_rne(h);
      else
        hs[r * ldk + k] = h;
    }
  }
  __syncthreads();

  // main loop: 16x16 output block per wave on MFMA
  const int lr = lane & 15, lg = lane >> 4;
  const int col = n0 + 16 * wave + lr;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  if (BF16) {
    const uint16_t* wrow = m.Wb + (size_t)col * Kpad;
    const uint16_t* hrow = hb + lr * ldk;
    for (int k0 = 0; k0 < Kpad; k0 += 64) {
      const int ko = k0 + 16 * lg;
      const uint4 a0 = *reinterpret_cast<const uint4*>(hrow + ko);
      const uint4 a1 = *reinterpret_cast<const uint4*>(hrow + ko + 8);
      const uint4 b0 = *reinterpret_cast<const uint4*>(wrow + ko);
      const uint4 b1 = *reinterpret_cast<const uint4*>(wrow + ko + 8);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a0), as_bf16x8(b0), acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a1), as_bf16x8(b1), acc, 0, 0, 0);
    }
  } else {
    const float* wrow = m.Wf + (size_t)col * Kpad;
    const float* hrow = hs + lr * ldk;
    for (int k0 = 0; k0 < Kpad; k0 += 16) {
      const int ko = k0 + 4 * lg;
      const float4 a = *reinterpret_cast<const float4*>(hrow + ko);
      const float4 w = *reinterpret_cast<const float4*>(wrow + ko);
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, w.x, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, w.y, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, w.z, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, w.w, acc, 0, 0, 0);
    }
  }

  // epilogue: bias, logits store, per-row (max, sum exp) over the tile
  const bool cvalid = col < V;
  const float bias = cvalid ? m.bias[col] : 0.f;
  float z[4], mx[4], sm[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) z[i] = cvalid ? acc[i] + bias : -INFINITY;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float v = z[i];
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) v = fmaxf(v, __shfl_xor(v, o));
    mx[i] = v;
    float e = cvalid ? expf(z[i] - v) : 0.f;
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) e += __shfl_xor(e, o);
    sm[i] = e;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = 4 * lg + i;
    if (s_act[row] && cvalid) logits[(size_t)(r0 + row) * m.Vpad + col] = z[i];
    if (lr == 0) {
      s_m[wave][row] = mx[i];
      s_s[wave][row] = sm[i];
    }
  }
  __syncthreads();
  if (tid < kJoinerBM && s_act[tid]) {
    float M = s_m[0][tid];
    for (int w = 1; w < 4; ++w) M = fmaxf(M, s_m[w][tid]);
    float S = 0.f;
    for (int w = 0; w < 4; ++w) S += s_s[w][tid] == 0.f ? 0.f : s_s[w][tid] * expf(s_m[w][tid] - M);
    stats[(size_t)(r0 + tid) * nvt + vt] = make_float2(M, S);
  }
}

// log-sum-exp of one joiner row from its per-tile (max, sum exp) partials.  The
// logarithm is taken in double: the device logf is biased low by a fraction of
// an ulp, which would otherwise accumulate over the frames of a stream.
__device__ __forceinline__ double row_lse(const float2* st, int nvt) {
  float M = -INFINITY;
  for (int i = 0; i < nvt; ++i) M = fmaxf(M, st[i].x);
  float S = 0.f;
  for (int i = 0; i < nvt; ++i) S += st[i].y == 0.f ? 0.f : st[i].y * expf(st[i].x - M);
  return (double)M + log((double)S);
}

// log-probability of one logit, rounded once to fp32
__device__ __forceinline__ float logp_of(float z, double lse) { return (float)((double)z - lse); }

__global__ void k_logp_rows(const float* __restrict__ logits, const float2* __restrict__ stats,
                            int nvt, int V, int Vpad, float* __restrict__ out) {
  const int r = blockIdx.x;
  __shared__ double s_lse;
  if (threadIdx.x == 0) s_lse = row_lse(stats + (size_t)r * nvt, nvt);
  __syncthreads();
  const double l = s_lse;
  for (int v = threadIdx.x; v < V; v += blockDim.x)
    out[(size_t)r * V + v] = logp_of(logits[(size_t)r * Vpad + v], l);
}

// ---------------------------------------------------------------------------
// search

__global__ void k_init(DecodeDev d, GraphDev g, int* __restrict__ trace) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= d.B) return;
  d.nsurv[b] = 1;
  d.surv_ctx[(size_t)b * d.Ns] = 0;
  d.surv_state[(size_t)b * d.Ns] = g.start;
  d.surv_score[(size_t)b * d.Ns] = 0.f;
  d.surv_row[(size_t)b * d.Ns] = 0;
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

struct SearchSmem {
  unsigned long long hk[kHashSlots];
  unsigned long long hv[kHashSlots];
  unsigned long long uk[kChunk + kMaxStates];
  unsigned long long uv[kChunk + kMaxStates];
  unsigned long long lk[kMaxStates];
  unsigned long long lv[kMaxStates];
  int s_ctx[kMaxStates], s_bprev[kMaxStates], s_state[kMaxStates], s_row[kMaxStates];
  int s_base[kMaxStates], s_off[kMaxStates + 1];
  float s_score[kMaxStates];
  double s_lse[kMaxStates];
  float f_score[kMaxStates], f_cs[kMaxStates];
  int f_keep1[kMaxStates], f_first[kMaxStates], f_keep2[kMaxStates];
  unsigned hist[256];
  int misc[8];
  int nU, nL, n_gt, n_eq;
  float best;
};

__device__ __forceinline__ uint32_t hash_slot(unsigned long long key) {
  return (uint32_t)((key * 0x9E3779B97F4A7C15ull) >> 52) & (kHashSlots - 1);  // 12 bits
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
      unsigned incl = sum;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const unsigned y = __shfl_up(incl, o);
        if (lane >= o) incl += y;
      }
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

__global__ __launch_bounds__(kSearchThreads) void k_search(ModelDev m, GraphDev g, DecodeDev d,
                                                           float beam, int t,
                                                           int* __restrict__ trace) {
  const int b = blockIdx.x;
  if (t >= d.len[b]) return;
  extern __shared__ __align__(16) unsigned char smem[];
  SearchSmem& s = *reinterpret_cast<SearchSmem*>(smem);
  const int tid = threadIdx.x;
  const int Ns = d.Ns, Nc = d.Nc, V = m.V;
  const int ns = d.nsurv[b], nc = d.nctx[b];
  const unsigned stride_tb = (unsigned)g.maxdeg + 1u;

  // survivors of frame t and the log-softmax normaliser of each context row
  for (int i = tid; i < ns; i += blockDim.x) {
    const size_t o = (size_t)b * Ns + i;
    const int ctx = d.surv_ctx[o], st = d.surv_state[o];
    s.s_ctx[i] = ctx;
    s.s_bprev[i] = ctx % V;
    s.s_state[i] = st;
    s.s_row[i] = d.surv_row[o];
    s.s_score[i] = d.surv_score[o];
    s.s_base[i] = g.rp[st];
    s.s_off[i + 1] = g.rp[st + 1] - g.rp[st];
  }
  for (int j = tid; j < nc; j += blockDim.x)
    s.s_lse[j] = row_lse(d.stats + (size_t)(b * Nc + j) * d.nvt, d.nvt);
  if (tid == 0) {
    s.s_off[0] = 0;
    s.nL = 0;
  }
  __syncthreads();
  if (tid == 0)  // inclusive scan of out-degrees (ns <= 256)
    for (int i = 1; i <= ns; ++i) s.s_off[i] += s.s_off[i - 1];
  __syncthreads();
  const int N = ns + s.s_off[ns];
  const float* zbase = d.logits + (size_t)b * Nc * m.Vpad;

  for (int base = 0; base < N; base += kChunk) {
    for (int i = tid; i < kHashSlots; i += blockDim.x) {
      s.hk[i] = kEmpty;
      s.hv[i] = 0ull;
    }
    if (tid == 0) s.nU = 0;
    __syncthreads();
    const int nL = s.nL;
    for (int i = tid; i < nL; i += blockDim.x) hash_insert(s, s.lk[i], s.lv[i]);
    const int end = min(N, base + kChunk);
    for (int c = base + tid; c < end; c += blockDim.x) {
      int i, pos;
      if (c < ns) {
        i = c;
        pos = -1;
      } else {
        const int k = c - ns;
        int lo = 0, hi = ns - 1;  // largest i with s_off[i] <= k
        while (lo < hi) {
          const int mid = (lo + hi + 1) >> 1;
          if (s.s_off[mid] <= k) lo = mid; else hi = mid - 1;
        }
        i = lo;
        pos = k - s.s_off[i];
      }
      const float* z = zbase + (size_t)s.s_row[i] * m.Vpad;
      const double lse = s.s_lse[s.s_row[i]];
      float sc;
      unsigned nctx;
      int nst;
      if (pos < 0) {
        sc = s.s_score[i] + logp_of(z[0], lse);
        nctx = (unsigned)s.s_ctx[i];
        nst = s.s_state[i];
      } else {
        const int j = s.s_base[i] + pos;
        const int lab = g.label[j];
        sc = (s.s_score[i] + g.q[j]) + logp_of(z[lab], lse);
        nctx = (unsigned)s.s_bprev[i] * (unsigned)V + (unsigned)lab;
        nst = g.dest[j];
      }
      const unsigned tb = (unsigned)i * stride_tb + (unsigned)(pos + 1);
      const unsigned long long key = ((unsigned long long)(unsigned)nst << 32) | nctx;
      const unsigned long long val = ((unsigned long long)f2ord(sc) << 32) | (0xffffffffu - tb);
      hash_insert(s, key, val);
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
    const int nU = s.nU;
    if (nU <= Ns) {
      for (int i = tid; i < nU; i += blockDim.x) {
        s.lk[i] = s.uk[i];
        s.lv[i] = s.uv[i];
      }
      if (tid == 0) s.nL = nU;
      __syncthreads();
      continue;
    }
    // beam/max-states order: score desc, then key = (state, ctx) asc
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

  // beam, then max-contexts, then canonical (ctx, state) order
  const int K = s.nL;
  if (tid < 64) {
    float bmax = -INFINITY;
    for (int i = tid; i < K; i += 64) bmax = fmaxf(bmax, ord2f((unsigned)(s.lv[i] >> 32)));
    for (int o = 32; o >= 1; o >>= 1) bmax = fmaxf(bmax, __shfl_xor(bmax, o));
    if (tid == 0) s.best = bmax;
  }
  __syncthreads();
  const float best = s.best;
  const float thr = best - beam;
  for (int i = tid; i < K; i += blockDim.x) {
    const float sc = ord2f((unsigned)(s.lv[i] >> 32));
    s.f_score[i] = sc;
    s.f_keep1[i] = sc >= thr;
  }
  __syncthreads();
  for (int i = tid; i < K; i += blockDim.x) {
    const unsigned ci = (unsigned)s.lk[i], sti = (unsigned)(s.lk[i] >> 32);
    float cs = -INFINITY;
    int first = s.f_keep1[i];
    for (int j = 0; j < K; ++j) {
      if (!s.f_keep1[j] || (unsigned)s.lk[j] != ci) continue;
      cs = fmaxf(cs, s.f_score[j]);
      if ((unsigned)(s.lk[j] >> 32) < sti) first = 0;
    }
    s.f_cs[i] = cs;
    s.f_first[i] = first;
  }
  __syncthreads();
  for (int i = tid; i < K; i += blockDim.x) {
    int keep = 0;
    if (s.f_keep1[i]) {
      const unsigned ci = (unsigned)s.lk[i];
      const float cs = s.f_cs[i];
      int rank = 0;
      for (int j = 0; j < K; ++j) {
        if (!s.f_first[j]) continue;
        const float csj = s.f_cs[j];
        if (csj > cs || (csj == cs && (unsigned)s.lk[j] < ci)) ++rank;
      }
      keep = rank < Nc;
    }
    s.f_keep2[i] = keep;
  }
  __syncthreads();
  const size_t hbase = ((size_t)t * d.B + b) * Ns;
  int* tr = trace ? trace + ((size_t)(t + 1) * d.B + b) * Ns * 4 : nullptr;
  for (int i = tid; i < K; i += blockDim.x) {
    if (!s.f_keep2[i]) continue;
    const unsigned ci = (unsigned)s.lk[i], sti = (unsigned)(s.lk[i] >> 32);
    int pos = 0, crow = 0;
    for (int j = 0; j < K; ++j) {
      if (!s.f_keep2[j]) continue;
      const unsigned cj = (unsigned)s.lk[j], stj = (unsigned)(s.lk[j] >> 32);
      if (cj < ci || (cj == ci && stj < sti)) ++pos;
      if (s.f_first[j] && cj < ci) ++crow;
    }
    const unsigned tb = 0xffffffffu - (unsigned)s.lv[i];
    const int parent = (int)(tb / stride_tb);
    const int apos = (int)(tb - (unsigned)parent * stride_tb) - 1;
    const int arc = apos < 0 ? -1 : s.s_base[parent] + apos;
    const int label = arc < 0 ? 0 : g.label[arc];
    const size_t o = (size_t)b * Ns + pos;
    d.surv_ctx[o] = (int)ci;
    d.surv_state[o] = (int)sti;
    d.surv_score[o] = s.f_score[i] - best;
    d.surv_row[o] = crow;
    if (s.f_first[i]) d.ctx_list[(size_t)b * Nc + crow] = (int)ci;
    d.hist_pl[hbase + pos] = (parent << 16) | label;
    d.hist_arc[hbase + pos] = arc;
    if (tr) {
      tr[4 * pos + 0] = (int)ci;
      tr[4 * pos + 1] = (int)sti;
      tr[4 * pos + 2] = parent;
      tr[4 * pos + 3] = label;
    }
  }
  if (tid == 0) {
    int nk = 0, ncx = 0;
    for (int i = 0; i < K; ++i) {
      nk += s.f_keep2[i];
      ncx += s.f_keep2[i] && s.f_first[i];
    }
    d.nsurv[b] = nk;
    d.nctx[b] = ncx;
    d.offset[b] += (double)best;
  }
}

// ---------------------------------------------------------------------------
// final selection and traceback

constexpr int kFinalBuf = 4096;

__global__ __launch_bounds__(256) void k_final(GraphDev g, DecodeDev d, int* __restrict__ out_tokens,
                                               int* __restrict__ out_ntok,
                                               double* __restrict__ out_scores,
                                               int* __restrict__ out_status,
                                               int* __restrict__ out_arcs) {
  __shared__ int buf_pl[kFinalBuf];
  __shared__ int buf_arc[kFinalBuf];
  __shared__ int s_idx, s_total;
  __shared__ int s_wsum[4];
  const int b = blockIdx.x, tid = threadIdx.x;
  const int Ns = d.Ns, T = d.T, len = d.len[b];
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

inline int grid_for(long long n, int threads, int cap = 4096) {
  long long g = (n + threads - 1) / threads;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return (int)g;
}

template <bool BF16>
hipError_t launch_joiner_impl(const ModelDev& m, const RowSrc& src, float* logits, float2* stats,
                              int R, int nvt, hipStream_t st) {
  const int ldk = BF16 ? m.Kpad + 8 : m.Kpad + 4;
  const size_t lds = (size_t)kJoinerBM * ldk * (BF16 ? 2 : 4);
  dim3 grid(nvt, (R + kJoinerBM - 1) / kJoinerBM);
  hipLaunchKernelGGL(k_joiner<BF16>, grid, dim3(256), lds, st, m, src, logits, stats, nvt);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_model_setup(const float* embed, const float* conv, const float* w_out,
                              const float* b_out, int V, int C, int Kpad, int Vpad, int bf16,
                              float* P0, float* P1, float* Wf, uint16_t* Wb, float* bias,
                              hipStream_t st) {
  hipLaunchKernelGGL(k_model_setup, dim3(grid_for((long long)Vpad * Kpad, 256)), dim3(256), 0, st,
                     embed, conv, w_out, b_out, V, C, Kpad, Vpad, bf16, P0, P1, Wf, Wb, bias);
  return hipGetLastError();
}

hipError_t launch_fill_i32(int* p, long long n, int v, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_fill_i32, dim3(grid_for(n, 256)), dim3(256), 0, st, p, n, v);
  return hipGetLastError();
}

hipError_t launch_init(const DecodeDev& d, const GraphDev& g, int* trace, hipStream_t st) {
  hipLaunchKernelGGL(k_init, dim3((d.B + 255) / 256), dim3(256), 0, st, d, g, trace);
  return hipGetLastError();
}

hipError_t launch_joiner_frame(const ModelDev& m, const DecodeDev& d, const float* enc, int t,
                               hipStream_t st) {
  RowSrc src{};
  src.enc = enc;
  src.T = d.T;
  src.t = t;
  src.Nc = d.Nc;
  src.len = d.len;
  src.nctx = d.nctx;
  src.ctx_list = d.ctx_list;
  src.R = d.B * d.Nc;
  src.rows_mode = 0;
  return m.bf16 ? launch_joiner_impl<true>(m, src, d.logits, d.stats, src.R, d.nvt, st)
                : launch_joiner_impl<false>(m, src, d.logits, d.stats, src.R, d.nvt, st);
}

hipError_t launch_search_frame(const ModelDev& m, const GraphDev& g, const DecodeDev& d,
                               float beam, int t, int* trace, hipStream_t st) {
  static bool attr_set = false;
  const size_t lds = sizeof(SearchSmem);
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)k_search,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL(k_search, dim3(d.B), dim3(kSearchThreads), lds, st, m, g, d, beam, t, trace);
  return hipGetLastError();
}

hipError_t launch_final(const GraphDev& g, const DecodeDev& d, int* out_tokens, int* out_ntok,
                        double* out_scores, int* out_status, int* out_arcs, hipStream_t st) {
  hipLaunchKernelGGL(k_final, dim3(d.B), dim3(256), 0, st, g, d, out_tokens, out_ntok, out_scores,
                     out_status, out_arcs);
  return hipGetLastError();
}

hipError_t launch_joiner_rows(const ModelDev& m, const float* enc_rows, const int* ctx, int R,
                              float* logits, float2* stats, float* out_logp, hipStream_t st) {
  const int nvt = m.Vpad / kJoinerBN;
  RowSrc src{};
  src.enc_rows = enc_rows;
  src.ctx_rows = ctx;
  src.R = R;
  src.rows_mode = 1;
  hipError_t e = m.bf16 ? launch_joiner_impl<true>(m, src, logits, stats, R, nvt, st)
                        : launch_joiner_impl<false>(m, src, logits, stats, R, nvt, st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_logp_rows, dim3(R), dim3(256), 0, st, logits, stats, nvt, m.V, m.Vpad,
                     out_logp);
  return hipGetLastError();
}

}  // namespace tbs
