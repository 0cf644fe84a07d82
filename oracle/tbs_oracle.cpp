// TEST INFRASTRUCTURE ONLY.  A plain, slow, fp64 CPU oracle for FSA-based
// one-symbol-per-frame transducer beam search (Kang et al., "Fast and parallel
// decoding for transducer": Sec. 2.2 stateless transducer, Sec. 2.3 max-symbols
// decoding with S = 1, Sec. 2.4 FSA-based decoding, Sec. 2.5 beam search with
// its three pruning constraints, Algorithm 1).  Only the test suite, the smoke
// check and the benchmark's CPU-baseline leg may load it; the product path
// never does.  It shares no code, header or table with the HIP library.
//
// Everything is computed in double precision, stream by stream, in the order
// the paper gives: contexts of the current hypotheses, decoder, index-select
// of the encoder frame, joiner, log-softmax, unpruned expansion over the graph
// arcs, merge of equal (graph state, context) tuples by max, the beam and
// max-states pruning in one operation, then max-contexts pruning.  Readings of
// points the paper leaves open are stated where they are used.
//
// Parity pins: the search is checked in the test suite against exhaustive
// enumeration of alignments (tiny T, V, S), a textbook Viterbi recursion over
// the (context, state) product space and per-frame argmax greedy search; the
// joiner against library layers (embedding, depthwise Conv1d, tanh, Linear,
// log_softmax).  The finite-beam / max-states / max-contexts selection rules
// are this implementation's reading of Sec. 2.5 and are pinned only by
// invariants and by the reductions above ("parity unpinned by the paper" for
// the exact tie-breaking rules).

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <limits>
#include <map>
#include <thread>
#include <vector>

namespace {

struct Model {
  int V, C;
  const float* E;     // [V][C] decoder embedding
  const float* conv;  // [C][2] depthwise conv taps, tap 0 = older label
  const float* W;     // [V][C] joiner output weight
  const float* bias;  // [V] or null
  int bf16;           // 1: joiner GEMM operands rounded to bfloat16 (RNE)
};

struct Graph {
  int S, start;
  const int* rp;      // [S+1]
  const int* dest;    // [A]
  const int* label;   // [A]
  const float* q;     // [A] log-domain arc score
  const float* fin;   // [S] or null; -inf = not final
};

struct Params {
  double beam;
  int Ns, Nc;
};

const double kNegInf = -std::numeric_limits<double>::infinity();

// Round a real number to the nearest bfloat16 value (8 significant bits),
// ties to even.  Used only in the bfloat16-operand mode of the joiner.
double round_bf16(double x) {
  if (x == 0.0 || !std::isfinite(x)) return x;
  int e = 0;
  double m = std::frexp(x, &e);           // x = m * 2^e, 0.5 <= |m| < 1
  double r = std::nearbyint(m * 256.0);   // default rounding mode: to nearest, ties to even
  return std::ldexp(r / 256.0, e);
}

// Stateless decoder (Sec. 2.2, Sec. 5.1): embedding of the two most recent
// labels followed by a kernel-2 convolution, read as depthwise with a ReLU
// and no bias; then the joiner tanh(enc + dec) -> Linear(V) -> log-softmax
// over the full vocabulary, blank included (Algorithm 1, decoder and joiner).
void joiner_logp(const Model& m, const float* enc_row, int a, int b, double* logp) {
  const int C = m.C, V = m.V;
  std::vector<double> h(C);
  for (int k = 0; k < C; ++k) {
    double d = (double)m.conv[2 * k + 0] * (double)m.E[(size_t)a * C + k] +
               (double)m.conv[2 * k + 1] * (double)m.E[(size_t)b * C + k];
    if (d < 0.0) d = 0.0;
    double hk = std::tanh((double)enc_row[k] + d);
    h[k] = m.bf16 ? round_bf16(hk) : hk;
  }
  double zmax = kNegInf;
  std::vector<double> z(V);
  for (int v = 0; v < V; ++v) {
    double acc = 0.0;
    const float* wr = m.W + (size_t)v * C;
    for (int k = 0; k < C; ++k) {
      double w = m.bf16 ? round_bf16((double)wr[k]) : (double)wr[k];
      acc += w * h[k];
    }
    if (m.bias) acc += (double)m.bias[v];
    z[v] = acc;
    if (acc > zmax) zmax = acc;
  }
  double s = 0.0;
  for (int v = 0; v < V; ++v) s += std::exp(z[v] - zmax);
  double lse = zmax + std::log(s);
  for (int v = 0; v < V; ++v) logp[v] = z[v] - lse;
}

// One lattice tuple ((a, b), t, s) of Sec. 2.4 with its accumulated score.
struct Tup {
  int64_t ctx;   // a * V + b
  int s;         // graph state
  double score;  // log-domain path score
  int parent;    // index of the predecessor in the previous frame's list
  int label;     // 0 = blank, else the emitted label
  int arc;       // graph arc taken, -1 for blank
};

struct Cand {
  int s;
  int64_t ctx;
  double score;
  int parent;
  int pos;    // arc position within the parent's state, -1 = blank
  int label;
  int arc;
};

// (score desc, then (parent, arc position) asc): the candidate kept when
// several candidates reach the same (state, context).
bool cand_better(const Cand& x, const Cand& y) {
  if (x.score != y.score) return x.score > y.score;
  if (x.parent != y.parent) return x.parent < y.parent;
  return x.pos < y.pos;
}

struct StreamOut {
  std::vector<int> tokens;
  std::vector<int> arcs;     // per frame: arc id, -1 blank
  double score = 0.0;
  int status = 0;
  double margin = std::numeric_limits<double>::infinity();
  double final_margin = std::numeric_limits<double>::infinity();
  std::vector<double> frame_margin;  // per frame: smallest decision margin of that frame
};

// Decodes one stream.  trace (optional) receives, for frame index f in
// [0, len], the surviving tuples (ctx, state, parent, label) in canonical order.
void decode_stream(const Model& m, const Graph& g, const Params& p, const float* enc, int T,
                   int len, StreamOut& out, int* trace, int trace_stride_frame) {
  const int V = m.V, C = m.C;
  std::vector<Tup> H;
  H.push_back(Tup{0, g.start, 0.0, -1, -1, -1});  // ((blank, blank), 0, start), Sec. 2.2 / 2.4
  std::vector<std::vector<Tup>> hist;               // survivors after each frame
  hist.reserve(len);
  auto write_trace = [&](int f, const std::vector<Tup>& L) {
    if (!trace) return;
    int* base = trace + (size_t)f * trace_stride_frame;
    for (int i = 0; i < (int)L.size() && i < p.Ns; ++i) {
      base[4 * i + 0] = (int)L[i].ctx;
      base[4 * i + 1] = L[i].s;
      base[4 * i + 2] = L[i].parent;
      base[4 * i + 3] = L[i].label;
    }
  };
  write_trace(0, H);
  double margin = std::numeric_limits<double>::infinity();
  std::vector<double> logp;
  out.frame_margin.assign(len, std::numeric_limits<double>::infinity());

  for (int t = 0; t < len; ++t) {
    double fmar = std::numeric_limits<double>::infinity();
    // GetContexts: the distinct contexts of the current tuples, ascending.
    std::vector<int64_t> ctxs;
    for (const Tup& x : H) ctxs.push_back(x.ctx);
    std::sort(ctxs.begin(), ctxs.end());
    ctxs.erase(std::unique(ctxs.begin(), ctxs.end()), ctxs.end());
    // Decoder + IndexSelect(enc_t) + joiner + log-softmax, once per context.
    logp.assign(ctxs.size() * (size_t)V, 0.0);
    const float* enc_row = enc + (size_t)t * C;
    for (size_t r = 0; r < ctxs.size(); ++r)
      joiner_logp(m, enc_row, (int)(ctxs[r] / V), (int)(ctxs[r] % V), &logp[r * V]);
    auto row_of = [&](int64_t ctx) {
      return (size_t)(std::lower_bound(ctxs.begin(), ctxs.end(), ctx) - ctxs.begin());
    };

    // ExpandArcs without pruning.  Blank keeps context and state; an arc
    // s -> r with label c and score q moves to ((b, c), t+1, r) with weight
    // q + log P(c | (a, b), t); with S = 1 no blank factor is added.
    std::vector<Cand> cands;
    for (int i = 0; i < (int)H.size(); ++i) {
      const Tup& x = H[i];
      const double* lp = &logp[row_of(x.ctx) * V];
      cands.push_back(Cand{x.s, x.ctx, x.score + lp[0], i, -1, 0, -1});
      const int64_t bprev = x.ctx % V;
      for (int j = g.rp[x.s]; j < g.rp[x.s + 1]; ++j) {
        const int c = g.label[j];
        cands.push_back(Cand{g.dest[j], bprev * V + c, x.score + (double)g.q[j] + lp[c], i,
                             j - g.rp[x.s], c, j});
      }
    }

    // Merge tuples with equal (state, context) by max (Table 3 / Table 6 "Max").
    std::map<std::pair<int, int64_t>, std::vector<const Cand*>> groups;
    for (const Cand& c : cands) groups[{c.s, c.ctx}].push_back(&c);
    struct Entry {
      int s;
      int64_t ctx;
      const Cand* best;
      double runner_up;  // best score among candidates with another (parent, label)
    };
    std::vector<Entry> ents;
    ents.reserve(groups.size());
    for (auto& kv : groups) {
      const Cand* best = kv.second[0];
      for (const Cand* c : kv.second)
        if (cand_better(*c, *best)) best = c;
      double ru = kNegInf;
      for (const Cand* c : kv.second)
        if (!(c->parent == best->parent && c->label == best->label)) ru = std::max(ru, c->score);
      ents.push_back(Entry{kv.first.first, kv.first.second, best, ru});
    }

    // Beam and max-states constraints in one pruning operation: keep a tuple
    // iff its score is within `beam` of the best and it ranks among the first
    // max_states by (score desc, (state, context) asc).
    auto ent_before = [](const Entry& x, const Entry& y) {
      if (x.best->score != y.best->score) return x.best->score > y.best->score;
      if (x.s != y.s) return x.s < y.s;
      return x.ctx < y.ctx;
    };
    std::sort(ents.begin(), ents.end(), ent_before);
    const double best = ents[0].best->score;
    const double thr = best - p.beam;
    size_t n_in_beam = 0;
    while (n_in_beam < ents.size() && ents[n_in_beam].best->score >= thr) ++n_in_beam;
    size_t n1 = std::min(n_in_beam, (size_t)p.Ns);
    if (n_in_beam > (size_t)p.Ns)
      fmar = std::min(fmar, ents[p.Ns - 1].best->score - ents[p.Ns].best->score);
    if (std::isfinite(p.beam)) {
      const size_t lim = std::min(ents.size(), (size_t)p.Ns);
      for (size_t i = 0; i < lim; ++i) fmar = std::min(fmar, std::fabs(ents[i].best->score - thr));
    }
    ents.resize(n1);

    // Max-contexts constraint: a context scores the max over its surviving
    // tuples; keep the max_contexts best by (score desc, context asc) and drop
    // every tuple of the other contexts.
    std::map<int64_t, double> cscore;
    for (const Entry& e : ents) {
      auto it = cscore.find(e.ctx);
      if (it == cscore.end() || e.best->score > it->second) cscore[e.ctx] = e.best->score;
    }
    std::vector<std::pair<double, int64_t>> cl;
    for (auto& kv : cscore) cl.push_back({kv.second, kv.first});
    std::sort(cl.begin(), cl.end(), [](const std::pair<double, int64_t>& x,
                                        const std::pair<double, int64_t>& y) {
      if (x.first != y.first) return x.first > y.first;
      return x.second < y.second;
    });
    if (cl.size() > (size_t)p.Nc) fmar = std::min(fmar, cl[p.Nc - 1].first - cl[p.Nc].first);
    std::vector<int64_t> kept_ctx;
    for (size_t i = 0; i < cl.size() && i < (size_t)p.Nc; ++i) kept_ctx.push_back(cl[i].second);
    std::sort(kept_ctx.begin(), kept_ctx.end());

    // New tuple list in canonical order: (context, state) ascending.
    std::vector<Tup> nH;
    for (const Entry& e : ents) {
      if (!std::binary_search(kept_ctx.begin(), kept_ctx.end(), e.ctx)) continue;
      if (e.runner_up != kNegInf) fmar = std::min(fmar, e.best->score - e.runner_up);
      nH.push_back(Tup{e.ctx, e.s, e.best->score, e.best->parent, e.best->label, e.best->arc});
    }
    std::sort(nH.begin(), nH.end(), [](const Tup& x, const Tup& y) {
      if (x.ctx != y.ctx) return x.ctx < y.ctx;
      return x.s < y.s;
    });
    out.frame_margin[t] = fmar;
    margin = std::min(margin, fmar);
    hist.push_back(nH);
    H.swap(nH);
    write_trace(t + 1, H);
  }

  // Final selection: best score + final weight over final-state tuples (first
  // in canonical order on ties); without any final tuple, the best tuple.
  int pick = -1;
  double pick_v = kNegInf, second = kNegInf;
  for (int pass = 0; pass < 2 && pick < 0; ++pass) {
    for (int i = 0; i < (int)H.size(); ++i) {
      double f = g.fin ? (double)g.fin[H[i].s] : 0.0;
      if (pass == 0 && !std::isfinite(f)) continue;
      double v = H[i].score + (pass == 0 ? f : 0.0);
      if (pick < 0 || v > pick_v) {
        second = pick_v;
        pick_v = v;
        pick = i;
      } else if (v > second) {
        second = v;
      }
    }
    out.status = pass;
  }
  out.final_margin = second != kNegInf ? pick_v - second : std::numeric_limits<double>::infinity();
  margin = std::min(margin, out.final_margin);
  out.score = pick_v;
  out.margin = margin;

  // Trace back through the stored predecessors and drop blanks.
  out.tokens.clear();
  out.arcs.assign(len, -1);
  int idx = pick;
  for (int t = len - 1; t >= 0; --t) {
    const Tup& x = hist[t][idx];
    out.arcs[t] = x.arc;
    if (x.label > 0) out.tokens.push_back(x.label);
    idx = x.parent;
  }
  std::reverse(out.tokens.begin(), out.tokens.end());
}

}  // namespace

extern "C" {

// log-softmax of the joiner for R (encoder row, context) pairs; out [R][V].
int oracle_logp(int C, int V, int R, const float* enc_rows, const int* ctx_a, const int* ctx_b,
                const float* E, const float* conv, const float* W, const float* bias, int bf16,
                double* out) {
  Model m{V, C, E, conv, W, bias, bf16};
  for (int r = 0; r < R; ++r)
    joiner_logp(m, enc_rows + (size_t)r * C, ctx_a[r], ctx_b[r], out + (size_t)r * V);
  return 0;
}

// Full decode.  tokens [B][T] (-1 padded), ntok [B], scores [B] (fp64),
// status [B] (0 = ended in a final state, 1 = no final state survived),
// arcs [B][T] or null (arc id per frame, -1 blank, -2 past the stream's end),
// trace [T+1][B][Ns][4] or null (-1 padded), margins [B] or null (smallest
// decision margin of the stream, +inf if no decision was contested),
// frame_margins [B][T+1] or null (entry t < len: smallest margin of the
// decisions taken on frame t; entry T: margin of the final pick; others +inf).
int oracle_decode(int B, int T, int C, int V, const float* enc, const int* lengths,
                  const float* E, const float* conv, const float* W, const float* bias,
                  int bf16, int S, int start, const int* rp, const int* dest, const int* label,
                  const float* q, const float* fin, double beam, int Ns, int Nc, int nthreads,
                  int* tokens, int* ntok, double* scores, int* status, int* arcs, int* trace,
                  double* margins, double* frame_margins) {
  Model m{V, C, E, conv, W, bias, bf16};
  Graph g{S, start, rp, dest, label, q, fin};
  Params p{beam, Ns, Nc};
  for (size_t i = 0; i < (size_t)B * T; ++i) tokens[i] = -1;
  if (arcs)
    for (size_t i = 0; i < (size_t)B * T; ++i) arcs[i] = -2;
  if (trace)
    for (size_t i = 0; i < (size_t)(T + 1) * B * Ns * 4; ++i) trace[i] = -1;
  std::atomic<int> next{0};
  auto work = [&]() {
    for (;;) {
      int b = next.fetch_add(1);
      if (b >= B) break;
      StreamOut o;
      decode_stream(m, g, p, enc + (size_t)b * T * C, T, lengths[b], o,
                    trace ? trace + (size_t)b * Ns * 4 : nullptr, B * Ns * 4);
      for (size_t k = 0; k < o.tokens.size(); ++k) tokens[(size_t)b * T + k] = o.tokens[k];
      ntok[b] = (int)o.tokens.size();
      scores[b] = o.score;
      status[b] = o.status;
      if (arcs)
        for (int t = 0; t < lengths[b]; ++t) arcs[(size_t)b * T + t] = o.arcs[t];
      if (margins) margins[b] = o.margin;
      if (frame_margins) {
        double* fm = frame_margins + (size_t)b * (T + 1);
        for (int t = 0; t <= T; ++t) fm[t] = std::numeric_limits<double>::infinity();
        for (int t = 0; t < lengths[b]; ++t) fm[t] = o.frame_margin[t];
        fm[T] = o.final_margin;
      }
    }
  };
  int nt = nthreads > 0 ? nthreads : (int)std::thread::hardware_concurrency();
  if (nt < 1) nt = 1;
  if (nt > B) nt = B > 0 ? B : 1;
  std::vector<std::thread> pool;
  for (int i = 1; i < nt; ++i) pool.emplace_back(work);
  work();
  for (auto& th : pool) th.join();
  return 0;
}

// Scores one alignment of one stream: arcs[t] is the graph arc taken at frame
// t (-1 = blank).  Returns 0 and the fp64 path score (final weight included)
// if the alignment is a path of the graph from the start state, -1 otherwise.
int oracle_rescore(int C, int V, int len, const float* enc, const int* arcs, const float* E,
                   const float* conv, const float* W, const float* bias, int bf16, int S,
                   int start, const int* rp, const int* dest, const int* label, const float* q,
                   const float* fin, double* score_out) {
  Model m{V, C, E, conv, W, bias, bf16};
  std::vector<double> lp(V);
  int64_t ctx = 0;
  int s = start;
  double score = 0.0;
  for (int t = 0; t < len; ++t) {
    joiner_logp(m, enc + (size_t)t * C, (int)(ctx / V), (int)(ctx % V), lp.data());
    const int j = arcs[t];
    if (j < 0) {
      score += lp[0];
      continue;
    }
    if (j < rp[s] || j >= rp[s + 1]) return -1;
    score += (double)q[j] + lp[label[j]];
    ctx = (ctx % V) * V + label[j];
    s = dest[j];
  }
  if (fin) {
    if (!std::isfinite((double)fin[s])) {
      *score_out = score;
      return 1;
    }
    score += (double)fin[s];
  }
  *score_out = score;
  return 0;
}

}  // extern "C"
