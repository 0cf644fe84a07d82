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
  std::vector<float> Wr;  // bf16 mode: W rounded to bfloat16 once (each value exact in float)

  Model(int V_, int C_, const float* E_, const float* conv_, const float* W_, const float* bias_,
        int bf16_);
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

Model::Model(int V_, int C_, const float* E_, const float* conv_, const float* W_,
             const float* bias_, int bf16_)
    : V(V_), C(C_), E(E_), conv(conv_), W(W_), bias(bias_), bf16(bf16_) {
  if (bf16) {
    Wr.resize((size_t)V * C);
    for (size_t i = 0; i < Wr.size(); ++i) Wr[i] = (float)round_bf16((double)W[i]);
  }
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
    const float* wr = (m.bf16 ? m.Wr.data() : m.W) + (size_t)v * C;
    for (int k = 0; k < C; ++k) acc += (double)wr[k] * h[k];
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
  double w;   // weight of the expansion: q + log P(label), or log P(blank)
};

// Lattice of one stream (Sec. 2.4 / 2.5: the search's output is an FSA whose
// states are the surviving tuples of each frame).  Arcs of frame f run from a
// survivor of frame f to a survivor of frame f+1: every unpruned expansion
// (blank or graph arc) whose (state, context) survived, whichever candidate won
// the max-merge.  Order within a frame: destination ascending, then source
// ascending, then arc position within the source state (blank first).
struct LatArc {
  int src, dst, label, arc;
  double w;
};

struct Lattice {
  int len = 0;
  std::vector<std::vector<Tup>> nodes;    // nodes[f], f = 0..len, canonical order
  std::vector<std::vector<LatArc>> arcs;  // arcs[f], f = 0..len-1
  std::vector<double> fw;                 // final weight of each node of frame len
  int status = 0;                         // 1: no survivor of frame len is final
};

// (score desc, then (parent, arc position) asc): the candidate kept when
// several candidates reach the same (state, context).
bool cand_better(const Cand& x, const Cand& y) {
  if (x.score != y.score) return x.score > y.score;
  if (x.parent != y.parent) return x.parent < y.parent;
  return x.pos < y.pos;
}

// A merged (state, context) tuple of one frame: the best candidate reaching it
// and the best score among its candidates with another (parent, label).
struct Entry {
  int s;
  int64_t ctx;
  const Cand* best;
  double runner_up;
};

// What one frame of the search decides from a list of tuples.
struct FrameOut {
  std::vector<Cand> cands;   // every unpruned expansion, in (source, arc position) order
  std::map<std::pair<int, int64_t>, std::vector<const Cand*>> groups;  // candidates per (state, ctx)
  std::vector<Entry> ranked; // merged tuples by (score desc, (state, context) asc), unpruned
  std::vector<Tup> next;     // the survivors, canonical order
  double margin = std::numeric_limits<double>::infinity();  // smallest decision margin
  double thr = kNegInf;      // best - beam
  double s_in = kNegInf, s_out = kNegInf;  // scores at ranks Ns-1 and Ns within the beam
  double c_in = kNegInf, c_out = kNegInf;  // context scores at ranks Nc-1 and Nc
  std::map<int64_t, double> cscore;        // context score after beam + max-states
};

// One frame of Algorithm 1 for one stream, from the tuples H (canonical order):
// contexts, decoder, joiner and log-softmax once per context, unpruned expansion,
// merge by max, beam + max-states in one pruning operation, then max-contexts.
void search_frame(const Model& m, const Graph& g, const Params& p, const float* enc_row,
                  const std::vector<Tup>& H, FrameOut& fo) {
  const int V = m.V;
  double fmar = std::numeric_limits<double>::infinity();
  // GetContexts: the distinct contexts of the current tuples, ascending.
  std::vector<int64_t> ctxs;
  for (const Tup& x : H) ctxs.push_back(x.ctx);
  std::sort(ctxs.begin(), ctxs.end());
  ctxs.erase(std::unique(ctxs.begin(), ctxs.end()), ctxs.end());
  // Decoder + IndexSelect(enc_t) + joiner + log-softmax, once per context.
  std::vector<double> logp(ctxs.size() * (size_t)V, 0.0);
  for (size_t r = 0; r < ctxs.size(); ++r)
    joiner_logp(m, enc_row, (int)(ctxs[r] / V), (int)(ctxs[r] % V), &logp[r * V]);
  auto row_of = [&](int64_t ctx) {
    return (size_t)(std::lower_bound(ctxs.begin(), ctxs.end(), ctx) - ctxs.begin());
  };

  // ExpandArcs without pruning.  Blank keeps context and state; an arc
  // s -> r with label c and score q moves to ((b, c), t+1, r) with weight
  // q + log P(c | (a, b), t); with S = 1 no blank factor is added.
  std::vector<Cand>& cands = fo.cands;
  for (int i = 0; i < (int)H.size(); ++i) {
    const Tup& x = H[i];
    const double* lp = &logp[row_of(x.ctx) * V];
    cands.push_back(Cand{x.s, x.ctx, x.score + lp[0], i, -1, 0, -1, lp[0]});
    const int64_t bprev = x.ctx % V;
    for (int j = g.rp[x.s]; j < g.rp[x.s + 1]; ++j) {
      const int c = g.label[j];
      cands.push_back(Cand{g.dest[j], bprev * V + c, x.score + (double)g.q[j] + lp[c], i,
                           j - g.rp[x.s], c, j, (double)g.q[j] + lp[c]});
    }
  }

  // Merge tuples with equal (state, context) by max (Table 3 / Table 6 "Max").
  std::map<std::pair<int, int64_t>, std::vector<const Cand*>>& groups = fo.groups;
  for (const Cand& c : cands) groups[{c.s, c.ctx}].push_back(&c);
  std::vector<Entry>& ents = fo.ranked;
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
  fo.thr = thr;
  size_t n_in_beam = 0;
  while (n_in_beam < ents.size() && ents[n_in_beam].best->score >= thr) ++n_in_beam;
  size_t n1 = std::min(n_in_beam, (size_t)p.Ns);
  if (n_in_beam >= (size_t)p.Ns) fo.s_in = ents[p.Ns - 1].best->score;
  if (n_in_beam > (size_t)p.Ns) {
    fo.s_out = ents[p.Ns].best->score;
    fmar = std::min(fmar, ents[p.Ns - 1].best->score - ents[p.Ns].best->score);
  }
  if (std::isfinite(p.beam)) {
    // the best tuple is never outside its own beam: its distance (the beam) decides nothing
    const size_t lim = std::min(ents.size(), (size_t)p.Ns);
    for (size_t i = 1; i < lim; ++i) fmar = std::min(fmar, std::fabs(ents[i].best->score - thr));
  }

  // Max-contexts constraint: a context scores the max over its surviving
  // tuples; keep the max_contexts best by (score desc, context asc) and drop
  // every tuple of the other contexts.
  std::map<int64_t, double>& cscore = fo.cscore;
  for (size_t i = 0; i < n1; ++i) {
    const Entry& e = ents[i];
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
  if (cl.size() >= (size_t)p.Nc) fo.c_in = cl[p.Nc - 1].first;
  if (cl.size() > (size_t)p.Nc) {
    fo.c_out = cl[p.Nc].first;
    fmar = std::min(fmar, cl[p.Nc - 1].first - cl[p.Nc].first);
  }
  std::vector<int64_t> kept_ctx;
  for (size_t i = 0; i < cl.size() && i < (size_t)p.Nc; ++i) kept_ctx.push_back(cl[i].second);
  std::sort(kept_ctx.begin(), kept_ctx.end());

  // New tuple list in canonical order: (context, state) ascending.
  std::vector<Tup>& nH = fo.next;
  for (size_t i = 0; i < n1; ++i) {
    const Entry& e = ents[i];
    if (!std::binary_search(kept_ctx.begin(), kept_ctx.end(), e.ctx)) continue;
    if (e.runner_up != kNegInf) fmar = std::min(fmar, e.best->score - e.runner_up);
    nH.push_back(Tup{e.ctx, e.s, e.best->score, e.best->parent, e.best->label, e.best->arc});
  }
  std::sort(nH.begin(), nH.end(), [](const Tup& x, const Tup& y) {
    if (x.ctx != y.ctx) return x.ctx < y.ctx;
    return x.s < y.s;
  });
  fo.margin = fmar;
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
                   int len, StreamOut& out, int* trace, int trace_stride_frame,
                   Lattice* lat = nullptr) {
  const int C = m.C;
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
  if (lat) {
    lat->len = len;
    lat->nodes.assign(1, H);
    lat->arcs.clear();
  }
  double margin = std::numeric_limits<double>::infinity();
  out.frame_margin.assign(len, std::numeric_limits<double>::infinity());

  for (int t = 0; t < len; ++t) {
    FrameOut fo;
    search_frame(m, g, p, enc + (size_t)t * C, H, fo);
    out.frame_margin[t] = fo.margin;
    margin = std::min(margin, fo.margin);
    if (lat) {
      // lattice arcs of frame t: the candidates whose (state, context) survived;
      // cands are in (source, arc position) order, blank first
      const std::vector<Tup>& nH = fo.next;
      std::vector<std::vector<LatArc>> into(nH.size());
      for (const Cand& c : fo.cands) {
        auto it = std::lower_bound(nH.begin(), nH.end(), c, [](const Tup& x, const Cand& y) {
          if (x.ctx != y.ctx) return x.ctx < y.ctx;
          return x.s < y.s;
        });
        if (it == nH.end() || it->ctx != c.ctx || it->s != c.s) continue;
        const int j = (int)(it - nH.begin());
        into[j].push_back(LatArc{c.parent, j, c.label, c.arc, c.w});
      }
      std::vector<LatArc> fa;
      for (auto& v : into) fa.insert(fa.end(), v.begin(), v.end());
      lat->arcs.push_back(std::move(fa));
      lat->nodes.push_back(nH);
    }
    hist.push_back(fo.next);
    H = fo.next;
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
  if (lat) {
    // final weights of the lattice: those of the graph, or 0 for every node of
    // the last frame when none of them is final (the same fallback as above)
    lat->fw.assign(H.size(), 0.0);
    lat->status = out.status;
    if (g.fin && out.status == 0)
      for (size_t i = 0; i < H.size(); ++i) lat->fw[i] = (double)g.fin[H[i].s];
  }
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

// log(exp(a) + exp(b)) without overflow.
double log_add(double a, double b) {
  if (a == kNegInf) return b;
  if (b == kNegInf) return a;
  const double hi = std::max(a, b), lo = std::min(a, b);
  return hi + std::log1p(std::exp(lo - hi));
}

// Forward scores of a lattice in the log semiring: alpha[f][j] = log of the sum,
// over lattice paths from the initial node to node j of frame f, of exp(path
// weight); returns the total over complete paths with final weights.
double lattice_forward(const Lattice& L, std::vector<std::vector<double>>& alpha) {
  alpha.assign(L.len + 1, {});
  alpha[0].assign(L.nodes[0].size(), kNegInf);
  alpha[0][0] = 0.0;
  for (int f = 0; f < L.len; ++f) {
    alpha[f + 1].assign(L.nodes[f + 1].size(), kNegInf);
    for (const LatArc& a : L.arcs[f])
      alpha[f + 1][a.dst] = log_add(alpha[f + 1][a.dst], alpha[f][a.src] + a.w);
  }
  double tot = kNegInf;
  for (size_t j = 0; j < L.nodes[L.len].size(); ++j)
    tot = log_add(tot, alpha[L.len][j] + L.fw[j]);
  return tot;
}

// Picks one of K items with probabilities proportional to exp(v[k]) by
// inversion: the first item whose running sum of exp(v - max) exceeds u times
// the full sum (u in [0, 1)).  margin: the distance of u * sum from the nearest
// boundary between two items, as a fraction of the sum (+inf for one item).
int pick_by_inversion(const std::vector<double>& v, double u, double* margin) {
  double mx = kNegInf;
  for (double x : v) mx = std::max(mx, x);
  std::vector<double> cum(v.size());
  double sum = 0.0;
  for (size_t k = 0; k < v.size(); ++k) {
    sum += v[k] == kNegInf ? 0.0 : std::exp(v[k] - mx);
    cum[k] = sum;
  }
  const double target = u * sum;
  int pick = -1;
  for (size_t k = 0; k < v.size(); ++k)
    if (cum[k] > target) {
      pick = (int)k;
      break;
    }
  if (pick < 0)  // rounding: the last item with a nonzero share
    for (size_t k = v.size(); k-- > 0;)
      if (v[k] != kNegInf) {
        pick = (int)k;
        break;
      }
  double m = std::numeric_limits<double>::infinity();
  for (size_t k = 0; k + 1 < v.size(); ++k) m = std::min(m, std::fabs(cum[k] - target) / sum);
  *margin = m;
  return pick;
}

// Total probability (log) of the label sequence y[0..n) in the lattice: the
// lattice composed with the linear acceptor of y, blanks as epsilon, summed over
// every path (Sec. 2.5, label sequence with the highest probability).  Dense
// recursion over (node, labels of y consumed).
double lattice_sequence_score(const Lattice& L, const int* y, int n) {
  std::vector<std::vector<double>> cur(L.nodes[0].size(), std::vector<double>(n + 1, kNegInf));
  cur[0][0] = 0.0;
  for (int f = 0; f < L.len; ++f) {
    std::vector<std::vector<double>> nxt(L.nodes[f + 1].size(),
                                         std::vector<double>(n + 1, kNegInf));
    for (const LatArc& a : L.arcs[f])
      for (int k = 0; k <= n; ++k) {
        if (a.label == 0)
          nxt[a.dst][k] = log_add(nxt[a.dst][k], cur[a.src][k] + a.w);
        else if (k >= 1 && y[k - 1] == a.label)
          nxt[a.dst][k] = log_add(nxt[a.dst][k], cur[a.src][k - 1] + a.w);
      }
    cur.swap(nxt);
  }
  double tot = kNegInf;
  for (size_t j = 0; j < cur.size(); ++j) tot = log_add(tot, cur[j][n] + L.fw[j]);
  return tot;
}

struct Decoded {
  std::vector<Lattice> lat;
};

// Beam search over full label sequences, the comparison search of Table 5 ("beam
// search", max-symbols 1; Sec. 2.2 footnote: the state space is the whole sequence
// y).  A hypothesis is a distinct blank-free sequence with a score.  On each frame
// every hypothesis expands to blank (y kept) and to every label a (y + a), with
// weight log P(label | last two labels of y, t) and no blank factor (as R5); equal
// sequences merge by max or by log-add (Table 3's two merge operations); the N best
// by (score desc, first candidate index asc) are kept, in that order.  A candidate's
// index is hyp_rank * V + label (blank = 0).  The result is the first hypothesis.
struct HypOut {
  std::vector<int> tokens;
  double score = 0.0;
  std::vector<double> frame_margin;  // per frame: smallest gap between neighbouring ranks up
                                     // to the N-best cut, or between the two best members
                                     // of a kept merged sequence
  double final_margin = std::numeric_limits<double>::infinity();
};

void hyp_stream(const Model& m, const float* enc, int len, int N, bool logadd, HypOut& out,
                int* trace, int trace_stride_frame) {
  const int V = m.V, C = m.C;
  struct Hyp {
    std::vector<int> y;
    double score;
  };
  std::vector<Hyp> H{Hyp{{}, 0.0}};
  if (trace) {
    trace[0] = -1;
    trace[1] = -1;
  }
  out.frame_margin.assign(len, std::numeric_limits<double>::infinity());
  std::vector<double> lp(V);
  for (int t = 0; t < len; ++t) {
    struct Group {
      double score;
      int first;             // smallest candidate index of the group
      int rep;               // candidate index of the best member (ties: smaller index)
      double rep_score;
      int parent, label;
      double second;         // best score among the other members (-inf: none)
    };
    std::map<std::vector<int>, Group> groups;
    for (int i = 0; i < (int)H.size(); ++i) {
      const std::vector<int>& y = H[i].y;
      const int a = y.size() >= 2 ? y[y.size() - 2] : 0;
      const int b = y.size() >= 1 ? y[y.size() - 1] : 0;
      joiner_logp(m, enc + (size_t)t * C, a, b, lp.data());
      for (int c = 0; c < V; ++c) {
        std::vector<int> z = y;
        if (c > 0) z.push_back(c);
        const double sc = H[i].score + lp[c];
        const int idx = i * V + c;
        auto it = groups.find(z);
        if (it == groups.end()) {
          groups.emplace(std::move(z), Group{sc, idx, idx, sc, i, c, kNegInf});
          continue;
        }
        Group& g = it->second;
        g.score = logadd ? log_add(g.score, sc) : std::max(g.score, sc);
        if (sc > g.rep_score) {  // candidates arrive in index order: ties keep the first
          g.second = g.rep_score;
          g.rep = idx;
          g.rep_score = sc;
          g.parent = i;
          g.label = c;
        } else {
          g.second = std::max(g.second, sc);
        }
        g.first = std::min(g.first, idx);
      }
    }
    std::vector<std::pair<const std::vector<int>*, const Group*>> order;
    for (auto& kv : groups) order.push_back({&kv.first, &kv.second});
    std::sort(order.begin(), order.end(), [](const auto& x, const auto& y) {
      if (x.second->score != y.second->score) return x.second->score > y.second->score;
      return x.second->first < y.second->first;
    });
    // the kept hypotheses are stored in rank order, so every gap between neighbours up
    // to the cut is a decision
    for (int k = 0; k + 1 < (int)order.size() && k < N; ++k)
      out.frame_margin[t] = std::min(out.frame_margin[t],
                                     order[k].second->score - order[k + 1].second->score);
    std::vector<Hyp> nH;
    for (int k = 0; k < (int)order.size() && k < N; ++k) {
      // the back-pointer of a merged sequence is its best member: a decision too
      const Group& g = *order[k].second;
      if (g.second != kNegInf)
        out.frame_margin[t] = std::min(out.frame_margin[t], g.rep_score - g.second);
      nH.push_back(Hyp{*order[k].first, order[k].second->score});
      if (trace) {
        int* p = trace + (size_t)(t + 1) * trace_stride_frame + 2 * k;
        p[0] = order[k].second->parent;
        p[1] = order[k].second->label;
      }
    }
    H.swap(nH);
  }
  out.tokens = H[0].y;
  out.score = H[0].score;
  if (H.size() > 1) out.final_margin = H[0].score - H[1].score;
}

}  // namespace

extern "C" {

// log-softmax of the joiner for R (encoder row, context) pairs; out [R][V].
int oracle_logp(int C, int V, int R, const float* enc_rows, const int* ctx_a, const int* ctx_b,
                const float* E, const float* conv, const float* W, const float* bias, int bf16,
                double* out) {
  const Model m(V, C, E, conv, W, bias, bf16);
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
  const Model m(V, C, E, conv, W, bias, bf16);
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

// Replays a search trace produced elsewhere, frame by frame: the survivors of
// frame f given in `given` ([T+1][B][Ns][4] (ctx, state, parent, label),
// canonical order, -1 padded, the layout of oracle_decode's trace) are taken
// as the tuples of frame f, each with the fp64 score of its (state, context)
// after the merge of frame f (0 for the initial tuple), and frame f+1 is
// decided again from them (search_frame).  Per stream b and frame f <= len_b,
// with the same layouts:
//   ref [T+1][B][Ns][4]: the survivors decided from the given frame f-1 (f >= 1);
//   ref_score, ref_cscore [T+1][B][Ns]: their scores and context scores;
//   key_score [T+1][B][Ns]: the merged score of each given survivor's
//     (state, context) on its frame, NaN if no candidate reaches it;
//   cand_score [T+1][B][Ns]: the best score among the candidates with the given
//     survivor's (state, context, parent, label), NaN if there is none;
//   margins [B][T+1]: entry f < len_b, the decision margin of frame f;
//   bounds [B][T][5]: per frame, best - beam, the scores at ranks Ns-1 and Ns
//     within the beam and the context scores at ranks Nc-1 and Nc (-inf if absent).
// A stream's replay stops at the first given survivor that is not a candidate.
int oracle_replay(int B, int T, int C, int V, const float* enc, const int* lengths,
                  const float* E, const float* conv, const float* W, const float* bias,
                  int bf16, int S, int start, const int* rp, const int* dest, const int* label,
                  const float* q, const float* fin, double beam, int Ns, int Nc, int nthreads,
                  const int* given, int* ref, double* ref_score, double* ref_cscore,
                  double* key_score, double* cand_score, double* margins, double* bounds) {
  const Model m(V, C, E, conv, W, bias, bf16);
  Graph g{S, start, rp, dest, label, q, fin};
  Params p{beam, Ns, Nc};
  const double nan = std::numeric_limits<double>::quiet_NaN();
  const size_t per_frame = (size_t)B * Ns;
  for (size_t i = 0; i < (size_t)(T + 1) * per_frame * 4; ++i) ref[i] = -1;
  for (size_t i = 0; i < (size_t)(T + 1) * per_frame; ++i)
    ref_score[i] = ref_cscore[i] = key_score[i] = cand_score[i] = nan;
  for (size_t i = 0; i < (size_t)B * (T + 1); ++i) margins[i] = nan;
  for (size_t i = 0; i < (size_t)B * T * 5; ++i) bounds[i] = nan;
  std::atomic<int> next{0};
  auto work = [&]() {
    for (;;) {
      const int b = next.fetch_add(1);
      if (b >= B) break;
      std::vector<Tup> H;
      H.push_back(Tup{0, g.start, 0.0, -1, -1, -1});
      key_score[(size_t)b * Ns] = cand_score[(size_t)b * Ns] = 0.0;
      for (int t = 0; t < lengths[b]; ++t) {
        FrameOut fo;
        search_frame(m, g, p, enc + ((size_t)b * T + t) * C, H, fo);
        margins[(size_t)b * (T + 1) + t] = fo.margin;
        double* bd = bounds + ((size_t)b * T + t) * 5;
        bd[0] = fo.thr;
        bd[1] = fo.s_in;
        bd[2] = fo.s_out;
        bd[3] = fo.c_in;
        bd[4] = fo.c_out;
        const size_t o = (size_t)(t + 1) * per_frame + (size_t)b * Ns;
        for (size_t i = 0; i < fo.next.size() && i < (size_t)Ns; ++i) {
          const Tup& x = fo.next[i];
          int* r = ref + 4 * (o + i);
          r[0] = (int)x.ctx;
          r[1] = x.s;
          r[2] = x.parent;
          r[3] = x.label;
          ref_score[o + i] = x.score;
          ref_cscore[o + i] = fo.cscore.at(x.ctx);
        }
        // the given survivors of frame t+1, scored by the merge of frame t
        std::vector<Tup> nH;
        bool ok = true;
        for (int i = 0; i < Ns; ++i) {
          const int* x = given + 4 * (o + i);
          if (x[0] < 0) break;
          auto it = fo.groups.find({x[1], (int64_t)x[0]});
          if (it == fo.groups.end()) {
            ok = false;
            break;
          }
          double ks = kNegInf, cs = kNegInf;
          for (const Cand* c : it->second) {
            ks = std::max(ks, c->score);
            if (c->parent == x[2] && c->label == x[3]) cs = std::max(cs, c->score);
          }
          key_score[o + i] = ks;
          cand_score[o + i] = cs == kNegInf ? nan : cs;
          nH.push_back(Tup{(int64_t)x[0], x[1], ks, x[2], x[3], -1});
        }
        if (!ok || nH.empty()) break;
        H.swap(nH);
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
  const Model m(V, C, E, conv, W, bias, bf16);
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

// Lattices of a batch (same arguments as oracle_decode): returns a handle for
// the functions below, or null.  frame_margins [B][T+1] or null as in oracle_decode.
void* oracle_lattice(int B, int T, int C, int V, const float* enc, const int* lengths,
                     const float* E, const float* conv, const float* W, const float* bias,
                     int bf16, int S, int start, const int* rp, const int* dest,
                     const int* label, const float* q, const float* fin, double beam, int Ns,
                     int Nc, int nthreads, double* frame_margins) {
  const Model m(V, C, E, conv, W, bias, bf16);
  Graph g{S, start, rp, dest, label, q, fin};
  Params p{beam, Ns, Nc};
  Decoded* D = new Decoded();
  D->lat.resize(B);
  std::atomic<int> next{0};
  auto work = [&]() {
    for (;;) {
      int b = next.fetch_add(1);
      if (b >= B) break;
      StreamOut o;
      decode_stream(m, g, p, enc + (size_t)b * T * C, T, lengths[b], o, nullptr, 0, &D->lat[b]);
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
  return D;
}

void oracle_lattice_free(void* h) { delete static_cast<Decoded*>(h); }

// Sizes of stream b's lattice: *len, nnodes[len+1] (nodes per frame), narcs[len].
int oracle_lattice_sizes(void* h, int b, int* len, int* nnodes, int* narcs) {
  const Lattice& L = static_cast<Decoded*>(h)->lat[b];
  *len = L.len;
  if (nnodes)
    for (int f = 0; f <= L.len; ++f) nnodes[f] = (int)L.nodes[f].size();
  if (narcs)
    for (int f = 0; f < L.len; ++f) narcs[f] = (int)L.arcs[f].size();
  return 0;
}

// Stream b's lattice: nodes [sum nnodes][4] (ctx, state, parent, label), arcs
// [sum narcs][4] (src, dst, label, graph arc), w [sum narcs], fw [nnodes[len]],
// alpha [sum nnodes] (forward scores), *total, *status.
int oracle_lattice_get(void* h, int b, int* nodes, int* arcs, double* w, double* fw,
                       double* alpha, double* total, int* status) {
  const Lattice& L = static_cast<Decoded*>(h)->lat[b];
  size_t n = 0, a = 0;
  for (int f = 0; f <= L.len; ++f)
    for (const Tup& x : L.nodes[f]) {
      nodes[4 * n + 0] = (int)x.ctx;
      nodes[4 * n + 1] = x.s;
      nodes[4 * n + 2] = x.parent;
      nodes[4 * n + 3] = x.label;
      ++n;
    }
  for (int f = 0; f < L.len; ++f)
    for (const LatArc& x : L.arcs[f]) {
      arcs[4 * a + 0] = x.src;
      arcs[4 * a + 1] = x.dst;
      arcs[4 * a + 2] = x.label;
      arcs[4 * a + 3] = x.arc;
      w[a] = x.w;
      ++a;
    }
  for (size_t j = 0; j < L.fw.size(); ++j) fw[j] = L.fw[j];
  std::vector<std::vector<double>> al;
  *total = lattice_forward(L, al);
  size_t k = 0;
  for (auto& v : al)
    for (double x : v) alpha[k++] = x;
  *status = L.status;
  return 0;
}

// n-best label-sequence search on stream b's lattice (Sec. 2.5): sample n paths
// (u [n][len+1]: entry f < len picks the arc into the path's node of frame f+1,
// going backwards from the end; entry len picks the final node first), take the
// distinct blank-free label sequences in order of first occurrence, score each
// by its total probability in the lattice and pick the best (first on ties).
// paths [n][len+1]: local arc index within frame f for f < len, final node at
// len; margins [n][len+1]: the inversion margin of each pick; first [n]: the
// path index of each distinct sequence; uscore [n]: its log probability.
// Returns the number of distinct sequences; *best: index of the best among them.
int oracle_lattice_nbest(void* h, int b, int n, const double* u, int* paths, double* margins,
                         int* first, double* uscore, int* best) {
  const Lattice& L = static_cast<Decoded*>(h)->lat[b];
  std::vector<std::vector<double>> alpha;
  lattice_forward(L, alpha);
  const int len = L.len;
  std::vector<std::vector<int>> seqs(n);
  for (int p = 0; p < n; ++p) {
    const double* up = u + (size_t)p * (len + 1);
    int* pp = paths + (size_t)p * (len + 1);
    double* mp = margins + (size_t)p * (len + 1);
    std::vector<double> v;
    for (size_t j = 0; j < L.nodes[len].size(); ++j) v.push_back(alpha[len][j] + L.fw[j]);
    int node = pick_by_inversion(v, up[len], &mp[len]);
    pp[len] = node;
    std::vector<int> labs;
    for (int f = len - 1; f >= 0; --f) {
      std::vector<int> ids;
      v.clear();
      for (size_t k = 0; k < L.arcs[f].size(); ++k)
        if (L.arcs[f][k].dst == node) {
          ids.push_back((int)k);
          v.push_back(alpha[f][L.arcs[f][k].src] + L.arcs[f][k].w);
        }
      const int k = ids[pick_by_inversion(v, up[f], &mp[f])];
      pp[f] = k;
      if (L.arcs[f][k].label > 0) labs.push_back(L.arcs[f][k].label);
      node = L.arcs[f][k].src;
    }
    std::reverse(labs.begin(), labs.end());
    seqs[p] = labs;
  }
  int nu = 0;
  for (int p = 0; p < n; ++p) {
    bool seen = false;
    for (int k = 0; k < nu && !seen; ++k) seen = seqs[first[k]] == seqs[p];
    if (!seen) first[nu++] = p;
  }
  *best = 0;
  for (int k = 0; k < nu; ++k) {
    const std::vector<int>& y = seqs[first[k]];
    uscore[k] = lattice_sequence_score(L, y.data(), (int)y.size());
    if (uscore[k] > uscore[*best]) *best = k;
  }
  return nu;
}

// Total probability (log) of label sequence y [n] in stream b's lattice.
double oracle_lattice_seqscore(void* h, int b, const int* y, int n) {
  return lattice_sequence_score(static_cast<Decoded*>(h)->lat[b], y, n);
}


// Full-sequence beam search (see hyp_stream) over a batch: tokens [B][T] (-1 padded),
// ntok [B], scores [B]; trace [T+1][B][N][2] or null: per frame the kept hypotheses'
// (parent rank, label), -1 padded; frame_margins [B][T+1] or null (entry T: the gap
// between the best two final hypotheses).
int oracle_hyps(int B, int T, int C, int V, const float* enc, const int* lengths,
                const float* E, const float* conv, const float* W, const float* bias, int bf16,
                int N, int logadd, int nthreads, int* tokens, int* ntok, double* scores,
                int* trace, double* frame_margins) {
  const Model m(V, C, E, conv, W, bias, bf16);
  for (size_t i = 0; i < (size_t)B * T; ++i) tokens[i] = -1;
  if (trace)
    for (size_t i = 0; i < (size_t)(T + 1) * B * N * 2; ++i) trace[i] = -1;
  std::atomic<int> next{0};
  auto work = [&]() {
    for (;;) {
      int b = next.fetch_add(1);
      if (b >= B) break;
      HypOut o;
      hyp_stream(m, enc + (size_t)b * T * C, lengths[b], N, logadd != 0, o,
                 trace ? trace + (size_t)b * N * 2 : nullptr, B * N * 2);
      for (size_t k = 0; k < o.tokens.size(); ++k) tokens[(size_t)b * T + k] = o.tokens[k];
      ntok[b] = (int)o.tokens.size();
      scores[b] = o.score;
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


// Forward recursions of the transducer losses over the (t, u) grid (Sec. 3), on given
// log-probabilities: blank [B][T][U+1] = log P(blank | frame t, u labels emitted),
// label [B][T][U] = log P(label u+1 | frame t, u labels emitted).  kind 0: the standard
// recursion, eq. (1), likelihood alpha(T_b - 1, U_b) + blank(T_b - 1, U_b); kind 1: the
// modified transducer, eq. (2), where a label also moves to the next frame; kind 2: the
// constrained transducer, eq. (3), where a label is followed by the blank of the new
// context on the same frame; both with likelihood alpha(T_b, U_b).  frames [B] and
// labels [B] are each utterance's T_b >= 1 and U_b.  alpha [B][T+1][U+1] (or null)
// receives every cell, -inf where no path reaches; total [B].
int oracle_transducer_forward(int kind, int B, int T, int U, const float* blank,
                              const float* label, const int* frames, const int* labels,
                              double* alpha, double* total) {
  for (int b = 0; b < B; ++b) {
    const int Tb = frames[b], Ub = labels[b];
    const float* bl = blank + (size_t)b * T * (U + 1);
    const float* lb = label + (size_t)b * T * U;
    auto BL = [&](int t, int u) { return (double)bl[(size_t)t * (U + 1) + u]; };
    auto LB = [&](int t, int u) { return (double)lb[(size_t)t * U + u]; };
    std::vector<double> a((size_t)(T + 1) * (U + 1), kNegInf);
    auto A = [&](int t, int u) -> double& { return a[(size_t)t * (U + 1) + u]; };
    A(0, 0) = 0.0;
    if (kind == 0) {
      for (int t = 0; t < Tb; ++t)
        for (int u = 0; u <= Ub; ++u) {
          if (t == 0 && u == 0) continue;
          double v = kNegInf;
          if (t > 0) v = log_add(v, A(t - 1, u) + BL(t - 1, u));
          if (u > 0) v = log_add(v, A(t, u - 1) + LB(t, u - 1));
          A(t, u) = v;
        }
      total[b] = A(Tb - 1, Ub) + BL(Tb - 1, Ub);
    } else {
      for (int t = 1; t <= Tb; ++t)
        for (int u = 0; u <= Ub; ++u) {
          double v = A(t - 1, u) + BL(t - 1, u);
          if (u > 0) {
            double w = A(t - 1, u - 1) + LB(t - 1, u - 1);
            if (kind == 2) w += BL(t - 1, u);
            v = log_add(v, w);
          }
          A(t, u) = v;
        }
      total[b] = A(Tb, Ub);
    }
    if (alpha)
      std::copy(a.begin(), a.end(), alpha + (size_t)b * (T + 1) * (U + 1));
  }
  return 0;
}

}  // extern "C"
