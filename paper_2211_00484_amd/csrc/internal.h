// Internal declarations shared by the host runtime (api.cpp) and the gfx950
// kernels (kernels.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace tbs {

constexpr int kMaxStates = 256;      // max_states limit (canonical ranking is O(Ns^2) per stream)
constexpr int kMaxDim = 2048;        // joiner dimension limit
constexpr unsigned kDefaultSpinLimit = 1u << 22;  // grouped kernel: polls per exchange wait
constexpr int kXTickets = 8 * 64;   // grouped kernel: per-XCD arrival counters after its [1 + B] timeouts
constexpr int kMaxVocab = 46340;     // contexts a * V + b are int32: V * V < 2^31
constexpr int kJoinerBN = 64;        // joiner vocabulary columns per tile (4 waves x 16)
constexpr int kKStep = 512;          // K padding granule of the packed weights and h rows (one
                                     // register-resident W chunk; keeps the MFMA loop branch-free)
constexpr int kSearchThreads = 256;
constexpr int kChunk = 1024;         // candidates merged per LDS pass (hash path)
constexpr int kHashBits = 11;
constexpr int kHashSlots = 1 << kHashBits;  // LDS open-addressing table (load <= 0.63)
constexpr int kDirectCands = 512;    // candidate sets up to this size (two per thread) merge directly
constexpr int kMaxTopK = 16;         // trivial-graph fast path: max_states limit
constexpr int kStatStage = kHashSlots;  // softmax partials staged in LDS (in hk) per stream (frame kernels)
constexpr int kTopkStage = 2 * (kChunk + kMaxStates);  // trivial-graph label lists staged in LDS (in uk)
constexpr size_t kMaxLds = 160 * 1024;  // LDS per workgroup on gfx950
constexpr int kStreamMaxV = 512;     // per-stream kernel: vocabulary limit (8 logits per lane)
constexpr int kMaxHyps = 16;         // full-sequence beam search: hypotheses per stream
constexpr int kTransducerMaxK = 16;  // transducer recursions: cells per lane (U + 1 <= 1024)

inline int round_up(int x, int m) { return (x + m - 1) / m * m; }

// Round to the nearest bfloat16, ties to even (finite inputs).
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// tanh for the joiner input: (e - 1) / (e + 1), e = exp(2x), with x clamped to [-9, 9]
// (|tanh(9)| rounds to 1 in fp32), the hardware exp and reciprocal.
__device__ __forceinline__ float tanh_fast(float x) {
  const float xc = fminf(fmaxf(x, -9.f), 9.f);
  const float e = __expf(2.f * xc);
  return (e - 1.f) * __builtin_amdgcn_rcpf(e + 1.f);
}

// Device-side model tables (padded: rows to Vpad, columns to Kpad, zeros).
struct ModelDev {
  int V, C, Kpad, Vpad;
  int bf16;
  const float* P0;          // [V][Kpad] conv tap 0 * embedding (older label)
  const float* P1;          // [V][Kpad] conv tap 1 * embedding (newer label)
  const float* Wf;          // [Vpad][Kpad] fp32 joiner weight (fp32 mode)
  const uint16_t* Wb;       // [Vpad][Kpad] bf16 joiner weight (bf16 mode)
  const void* Wi;           // [Kpad/KQ][Vpad][KQ] W interleaved by 16-byte k slices (KQ = 4 fp32
                            // or 8 bf16), read by the per-stream kernel
  const float* bias;        // [V]
};

struct GraphDev {
  int S, start, maxdeg;
  int trivial;              // one state, loops 1..V-1 in label order, q = 0, final 0
  const int* rp;
  const int* dest;
  const int* label;
  const float* q;
  const float* fin;         // [S] or null
};

// Per-decode device state.
struct DecodeDev {
  int B, T, Ns, Nc, nvt;    // nvt = number of joiner vocabulary tiles
  int KT;                   // trivial fast path: candidates kept per (row, tile); 0 = off
  const float* enc;         // [B][T][C]
  const int* len;           // [B]
  const int* base;          // [B] absolute index of frame 0 of this call (chunked decode) or null
  const GraphDev* graphs;   // [B] per-stream decoding graphs, or null (one shared graph)
  int* nsurv;               // [B]
  int* surv_ctx;            // [B][Ns]
  int* surv_state;          // [B][Ns]
  float* surv_score;        // [B][Ns], relative to the stream's best
  int* surv_row;            // [B][Ns], index of the tuple's context in ctx_list
  int2* surv_rp;            // [B][Ns], arc range [lo, hi) of the tuple's state (frame kernels)
  int* nctx;                // [B]
  int* ctx_list;            // [B][Nc], ascending
  double* offset;           // [B]
  void* h;                  // [B*Nc][Kpad] joiner input rows tanh(enc + dec) (fp32 or bf16)
  float* logits;            // [B*Nc][Vpad] (general graphs)
  float2* stats;            // [B*Nc][nvt]: (max, sum exp(z - max)) per vocabulary tile
  float* tk_z;              // [B*Nc][nvt*4][KT] trivial fast path: best logits per 16-column sub-tile
  int* tk_c;                // [B*Nc][nvt*4][KT] and their labels (-1 = none)
  float* z0;                // [B*Nc] blank logit (trivial fast path)
  int* hist_pl;             // [T][B][Ns]: parent << 16 | label
  int* hist_arc;            // [T][B][Ns]: arc id, -1 blank
  int* path_lab;            // [B][T] scratch for the traceback
};

struct JoinerPlan {
  int MB;                   // 0: GEMM tiles (shape); else 16 MB x 64 tiles
  int shape;                // GEMM tiles: 0 = 128 x 128, 1 = 256 x 256 (bf16), 2 = 64 x 128
  int n_rt, n_ct;           // row and column tiles
  int grid;                 // workgroups (XCD-interleaved tile order)
  size_t lds;               // dynamic LDS bytes
};

// topk: the joiner writes each row's best labels (trivial graph) instead of logits
JoinerPlan plan_joiner(int rows, int Vpad, int Kpad, int bf16, int ncu, bool topk = false);

// Events for the next non-cooperative kernel launch of the calling thread, recorded in
// that launch's dispatch packet (per-kernel profiling); pending until a launch takes them.
void set_launch_events(hipEvent_t start, hipEvent_t stop);
bool launch_events_pending();
// Takes the pending events (for a launch made outside kernels.hip); false if none.
bool take_launch_events(hipEvent_t* start, hipEvent_t* stop);

// Per-stream kernel (one workgroup runs every frame of one stream).
struct StreamPlan {
  int ok;                   // the shape fits (contexts, LDS)
  int RG;                   // groups of 4 context rows (1 to 4)
  int hoff, hstride;        // LDS offset of the joiner rows and their stride (elements)
  int zoff;                 // LDS offset of the logit rows [4 RG][Vpad] fp32
  int doff;                 // LDS offset of the staged decoder rows (0: none)
  size_t lds;               // dynamic LDS bytes
};

StreamPlan plan_stream(const ModelDev& m, int Nc, int KT, int trivial);

// Grouped per-stream kernel (trivial graph, fp32): G workgroups per stream, each with
// Vpad / 64 / G (1 or 2) column groups; cooperative launch of B * G workgroups.
// xbuf: device memory of at least B * G * 2 * group_words(Nc, KT) words.
int group_words(int Nc, int KT);
hipError_t launch_stream_group(const ModelDev& m, const GraphDev& g, const DecodeDev& d, float beam,
                               int* trace, const StreamPlan& p, unsigned long long* xbuf, int G,
                               unsigned epoch, unsigned spin_limit, unsigned* err,
                               hipStream_t st);
hipError_t launch_stream(const ModelDev& m, const GraphDev& g, const DecodeDev& d, float beam,
                         int* trace, const StreamPlan& p, hipStream_t st);

hipError_t launch_model_setup(const float* embed, const float* conv, const float* w_out,
                              const float* b_out, int V, int C, int Kpad, int Vpad, int bf16,
                              float* P0, float* P1, float* Wf, uint16_t* Wb, void* Wi,
                              float* bias, hipStream_t st);
hipError_t launch_fill_i32(int* p, long long n, int v, hipStream_t st);
// out[b] = min(max(in[b], 0), T) for b < B (device arrays)
hipError_t launch_clamp_lengths(const int* in, int* out, int B, int T, hipStream_t st);
hipError_t launch_init(const ModelDev& m, const DecodeDev& d, const GraphDev& g, int* trace,
                       hipStream_t st);
hipError_t launch_resume(const ModelDev& m, const DecodeDev& d, const GraphDev& g, int* trace,
                         int rows_needed, hipStream_t st);
hipError_t launch_joiner_frame(const ModelDev& m, const DecodeDev& d, const JoinerPlan& p, int t,
                               hipStream_t st);
hipError_t launch_search_frame(const ModelDev& m, const GraphDev& g, const DecodeDev& d,
                               float beam, int t, int* trace, hipStream_t st);
hipError_t launch_final(const GraphDev& g, const DecodeDev& d, int* out_tokens, int* out_ntok,
                        double* out_scores, int* out_status, int* out_arcs,
                        const unsigned* exchange_err, hipStream_t st);
hipError_t launch_joiner_rows(const ModelDev& m, const float* enc_rows, const int* ctx, int R,
                              void* h, float* logits, float2* stats, float* out_logp, int ncu,
                              hipStream_t st);

// Lattice of a batch (the search's output FSA): nodes are the survivors of each frame
// (the survivor trace, [T+1][B][Ns][4] = (ctx, state, parent, label), -1 padded); the
// arcs of frame f of stream b run from its frame-f survivors into its frame-(f+1)
// survivors, ordered by (destination, source, arc position) with blank first.
struct LatticeDev {
  int B, T, Ns, Nc, V;
  const int* len;           // [B]
  const int* nodes;         // survivor trace
  const GraphDev* graphs;   // [B] per-stream graphs, or null
  int* nn;                  // [B][T+1] nodes per frame (written by the forward pass)
  int* cnt;                 // [B*T] arcs of (b, f)
  long long* off;           // [B*T+1] first arc of (b, f)
  int* dptr;                // [B*T][Ns+1] local offset of each destination's first arc
  int4* arcs;               // [A] (src, dst, label, graph arc or -1)
  float* w;                 // [A] weight: q + log P(label), blank: log P(blank)
  double* pc;               // [A] exp(alpha[src] + w - alpha[dst]): the arc's share of its
                            // destination's forward score (backward sampling)
  int* rowctx;              // [B*T*Nc] context of joiner row (b, f, r), -1 = none
  double* alpha;            // [B][T+1][Ns] forward log scores (-inf for absent nodes)
  double* fw;               // [B][Ns] final weights of the last frame's nodes
  double* total;            // [B]
  int* status;              // [B] 1: no survivor of the last frame is final
};

// n-best scratch of a lattice for n paths.
struct NBestDev {
  int n;
  const double* u;          // [B][n][T+1]
  int* paths;               // [B][n][T+1] or null
  int* seq;                 // [B][n][T] blank-free label sequences
  int* ntok;                // [B][n]
  unsigned long long* hash; // [B][n]
  int* first;               // [B][n] path of each distinct sequence
  int* nuniq;               // [B]
  double* score;            // [B][n] total log probability of each distinct sequence
  double* dp;               // DP scratch in global memory, or null (LDS)
  int dp_stride;            // doubles per DP buffer row: band width cap
};

hipError_t launch_lattice_count(const LatticeDev& L, const GraphDev& g, hipStream_t st);
hipError_t launch_lattice_scan(const LatticeDev& L, hipStream_t st);
hipError_t launch_lattice_fill(const LatticeDev& L, const GraphDev& g, hipStream_t st);
// Joiner rows of streams [b0, b1) (dense (b, f, r) rows, ctx from L.rowctx): h rows,
// logits and per-tile softmax statistics, then the arc weights of those streams.
hipError_t launch_lattice_weights(const ModelDev& m, const LatticeDev& L, const GraphDev& g,
                                  const float* enc, int b0, int b1, void* h, float* logits,
                                  float2* stats, int ncu, hipStream_t st);
hipError_t launch_lattice_forward(const LatticeDev& L, const GraphDev& g, hipStream_t st);
hipError_t launch_nbest(const LatticeDev& L, const NBestDev& N, int* out_tokens, int* out_ntok,
                        double* out_scores, int* out_nuniq, double* out_uscores,
                        int* out_ufirst, int dp_grid, size_t dp_lds, hipStream_t st);

// joiner rows of a dense row table: row r of the batch is table row row0 + r, with
// context ctx[row0 + r] (-1: no row, h = 0) and encoder row
// enc + ((row0 + r) / per_enc) * enc_stride
hipError_t launch_joiner_dense(const ModelDev& m, const float* enc, long long enc_stride,
                               const int* ctx, long long row0, int per_enc, int R, void* h,
                               float* logits, float2* stats, int ncu, hipStream_t st);

// the two halves of launch_joiner_dense: h rows, then the GEMM over R rows of h
hipError_t launch_h_rows_dense(const ModelDev& m, const float* enc, long long enc_stride,
                               const int* ctx, long long row0, int per_enc, int R, void* h,
                               hipStream_t st);
hipError_t launch_joiner_gemm(const ModelDev& m, const void* h, int R, float* logits,
                              float2* stats, int ncu, hipStream_t st);

// Full-sequence beam search (the comparison search of Table 5), frame schedule.
struct HypDev {
  int B, T, N, merge_logadd;
  const int* len;                     // [B]
  const float* enc;                   // [B][T][C] encoder output
  void* h;                            // [B*N][Kpad] joiner rows of the next frame
  unsigned long long* hash[2];        // [B][N] per frame parity: hash of the sequence
  unsigned long long* phash[2];       // hash of the sequence without its last label
  int* n[2];                          // sequence length
  int* ctx[2];                        // last two labels a * V + b
  double* score[2];
  int* nh[2];                         // [B] hypotheses
  int* rowctx;                        // [B*N] joiner row contexts (-1: none)
  int* hrow;                          // [B*N] joiner row of each hypothesis
  int* hist;                          // [T][B][N] parent << 16 | label
};
hipError_t launch_hyp_init(const ModelDev& m, const HypDev& d, hipStream_t st);
hipError_t launch_hyp_step(const ModelDev& m, const HypDev& d, int t, const float* logits,
                           const float2* stats, int* trace, hipStream_t st);
hipError_t launch_hyp_final(const HypDev& d, int* out_tokens, int* out_ntok, double* out_scores,
                            hipStream_t st);

// Transducer forward recursions (kind 0: eq. 1, 1: eq. 2, 2: eq. 3); one wave per
// utterance.  lengths: DEVICE [B][2] (frames, labels).
hipError_t launch_transducer_forward(int kind, const float* blank, const float* label,
                                     const int* lengths, int B, int T, int U, double* total,
                                     float* alpha, int* status, hipStream_t st);

}  // namespace tbs
