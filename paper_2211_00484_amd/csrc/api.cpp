// Host runtime behind include/tbs.h: argument validation, graph/model handles,
// the cached decode workspace and the frame loop that enqueues the gfx950
// kernels (Algorithm 1 of Kang et al., arXiv 2211.00484).
#include "tbs.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <type_traits>
#include <vector>

#include "internal.h"

using namespace tbs;

// Workspace of tbs_decode_noalloc: one array per device, held until the process ends.
constexpr size_t kScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

thread_local std::string g_last_error;

tbs_status fail(tbs_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

tbs_status hip_fail(hipError_t e, const char* what) {
  return fail(e == hipErrorOutOfMemory ? TBS_ENOMEM : TBS_EDEVICE, "%s: %s", what,
              hipGetErrorString(e));
}

#define HIP_TRY(expr, what)                    \
  do {                                         \
    hipError_t e_ = (expr);                    \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

template <class T>
hipError_t dalloc(T** p, size_t n) {
  *p = nullptr;
  if (n == 0) n = 1;
  return hipMalloc((void**)p, n * sizeof(T));
}

struct Workspace {
  int B = 0, T = 0, Ns = 0, Nc = 0, KT = 0;
  bool has_logits = false;
  int* len = nullptr;
  int* nsurv = nullptr;
  int* surv_ctx = nullptr;
  int* surv_state = nullptr;
  float* surv_score = nullptr;
  int* surv_row = nullptr;
  int2* surv_rp = nullptr;
  int* nctx = nullptr;
  int* ctx_list = nullptr;
  double* offset = nullptr;
  void* h = nullptr;
  float* logits = nullptr;
  float2* stats = nullptr;
  float* tk_z = nullptr;
  int* tk_c = nullptr;
  float* z0 = nullptr;
  int* hist_pl = nullptr;
  int* hist_arc = nullptr;
  int* path_lab = nullptr;
  int* len_host = nullptr;  // pinned staging for lengths (and frame bases), [2B]
  unsigned* xerr = nullptr;  // [1 + B] exchange timeouts of the grouped kernel: any, per stream;
                             // then its [kXTickets] per-XCD arrival counters
  GraphDev* gtab = nullptr;       // [B] per-stream graph table (decodes with one graph per stream)
  GraphDev* gtab_host = nullptr;  // pinned staging for it
  hipEvent_t done = nullptr;
  bool pending = false;

  void release() {
    (void)hipFree(len); (void)hipFree(nsurv); (void)hipFree(surv_ctx); (void)hipFree(surv_state); (void)hipFree(surv_score);
    (void)hipFree(surv_row); (void)hipFree(surv_rp); (void)hipFree(nctx); (void)hipFree(ctx_list); (void)hipFree(offset); (void)hipFree(h);
    (void)hipFree(logits); (void)hipFree(stats); (void)hipFree(tk_z); (void)hipFree(tk_c); (void)hipFree(z0);
    (void)hipFree(hist_pl); (void)hipFree(hist_arc); (void)hipFree(path_lab);
    (void)hipFree(gtab);
    (void)hipFree(xerr);
    if (len_host) (void)hipHostFree(len_host);
    if (gtab_host) (void)hipHostFree(gtab_host);
    if (done) (void)hipEventDestroy(done);
    *this = Workspace();
  }
};

// Workspace of the full-sequence beam search (tbs_hyp_search), cached in the model.
struct HypWork {
  int B = 0, T = 0, N = 0;
  int* len = nullptr;
  unsigned long long* hash[2] = {nullptr, nullptr};
  unsigned long long* phash[2] = {nullptr, nullptr};
  int* n[2] = {nullptr, nullptr};
  int* ctx[2] = {nullptr, nullptr};
  double* score[2] = {nullptr, nullptr};
  int* nh[2] = {nullptr, nullptr};
  int* rowctx = nullptr;
  int* hrow = nullptr;
  int* hist = nullptr;
  void* h = nullptr;
  float* logits = nullptr;
  float2* stats = nullptr;
  hipEvent_t done = nullptr;
  bool pending = false;

  void release() {
    if (done && pending) (void)hipEventSynchronize(done);
    for (int i = 0; i < 2; ++i) {
      (void)hipFree(hash[i]);
      (void)hipFree(phash[i]);
      (void)hipFree(n[i]);
      (void)hipFree(ctx[i]);
      (void)hipFree(score[i]);
      (void)hipFree(nh[i]);
    }
    (void)hipFree(len);
    (void)hipFree(rowctx);
    (void)hipFree(hrow);
    (void)hipFree(hist);
    (void)hipFree(h);
    (void)hipFree(logits);
    (void)hipFree(stats);
    if (done) (void)hipEventDestroy(done);
    *this = HypWork();
  }
};

}  // namespace

void lattice_free(tbs_lattice* L);  // release and delete (defined with tbs_lattice)

struct tbs_graph {
  int S = 0, start = 0, V = 0, A = 0, maxdeg = 0;
  int trivial = 0;  // one state, 0-weight loops 1..V-1 in label order, final weight 0
  int* rp = nullptr;
  int* dest = nullptr;
  int* label = nullptr;
  float* q = nullptr;
  float* fin = nullptr;
};

// Exchange buffers of the grouped per-stream kernel (device memory, accessed with
// device-scope atomics).  A destroyed model returns its buffer to a per-process free
// list for later models, which then skip the allocation and the clear.  Words carry an
// 8-bit decode epoch; when the process-wide epoch wraps, a buffer is cleared before
// its next use.
struct XBuf {
  int dev = -1;
  unsigned long long* p = nullptr;
  size_t words = 0;
  unsigned wrap = 0;  // epoch wrap count at the last clear
};
std::mutex g_xmu;
std::vector<XBuf> g_xfree;
std::atomic<unsigned> g_epoch{0};
std::atomic<unsigned> g_wrap{0};

struct tbs_model {
  int V = 0, C = 0, Kpad = 0, Vpad = 0, bf16 = 0;
  int dev = 0, ncu = 0, coop = 0;   // device, compute units, cooperative launch support
  XBuf xbuf;
  unsigned spin_limit = kDefaultSpinLimit;  // polls before a grouped-kernel wait gives up
  float* P0 = nullptr;
  float* P1 = nullptr;
  float* Wf = nullptr;
  uint16_t* Wb = nullptr;
  void* Wi = nullptr;
  float* bias = nullptr;
  int schedule = TBS_SCHEDULE_AUTO;
  std::mutex mu;
  Workspace ws;
  HypWork hw;
  tbs_lattice* lat_cache = nullptr;  // buffers of the last destroyed lattice, for the next
  // device work of every decode and chunk on this model is serialised on this event
  // (they share the exchange buffer and, for tbs_decode, the workspace)
  hipEvent_t busy = nullptr;
  bool busy_pending = false;
  // per-kernel timing (tbs_model_set_profiling)
  bool prof = false;
  struct Timed {
    int kernel;
    hipEvent_t start, stop;
  };
  std::vector<Timed> prof_pending;
  std::vector<hipEvent_t> prof_pool;
  tbs_kernel_time prof_acc[TBS_KERNEL_COUNT] = {};
  // frame loop of the frame schedule captured in a HIP graph (tbs_model_set_graph_capture):
  // the key is the bytes of every argument of the captured launches; a loop is captured
  // the second time its key is seen and replayed while the key repeats
  bool graphs = true;
  std::vector<unsigned char> fg_key, fg_seen;
  hipGraph_t fg_graph = nullptr;
  hipGraphExec_t fg_exec = nullptr;
  hipStream_t cap_stream = nullptr;  // capture stream (the caller's may be the null stream)
  int fg_captures = 0, fg_replays = 0;
  // scratch for tbs_joiner_logp
  int rows_cap = 0;
  void* rows_h = nullptr;
  float* rows_logits = nullptr;
  float2* rows_stats = nullptr;
};

namespace {

ModelDev model_dev(const tbs_model* m) {
  ModelDev d;
  d.V = m->V;
  d.C = m->C;
  d.Kpad = m->Kpad;
  d.Vpad = m->Vpad;
  d.bf16 = m->bf16;
  d.P0 = m->P0;
  d.P1 = m->P1;
  d.Wf = m->Wf;
  d.Wb = m->Wb;
  d.Wi = m->Wi;
  d.bias = m->bias;
  return d;
}

GraphDev graph_dev(const tbs_graph* g) {
  GraphDev d;
  d.S = g->S;
  d.start = g->start;
  d.maxdeg = g->maxdeg;
  d.trivial = g->trivial;
  d.rp = g->rp;
  d.dest = g->dest;
  d.label = g->label;
  d.q = g->q;
  d.fin = g->fin;
  return d;
}

tbs_status graph_upload(tbs_graph* g, const int32_t* row_ptr, const int32_t* dest,
                        const int32_t* label, const float* score, const float* final_score) {
  const size_t A = (size_t)g->A, S = (size_t)g->S;
  HIP_TRY(dalloc(&g->rp, S + 1), "hipMalloc(graph)");
  HIP_TRY(dalloc(&g->dest, A), "hipMalloc(graph)");
  HIP_TRY(dalloc(&g->label, A), "hipMalloc(graph)");
  HIP_TRY(dalloc(&g->q, A), "hipMalloc(graph)");
  HIP_TRY(hipMemcpy(g->rp, row_ptr, (S + 1) * 4, hipMemcpyHostToDevice), "hipMemcpy(graph)");
  if (A) {
    HIP_TRY(hipMemcpy(g->dest, dest, A * 4, hipMemcpyHostToDevice), "hipMemcpy(graph)");
    HIP_TRY(hipMemcpy(g->label, label, A * 4, hipMemcpyHostToDevice), "hipMemcpy(graph)");
    HIP_TRY(hipMemcpy(g->q, score, A * 4, hipMemcpyHostToDevice), "hipMemcpy(graph)");
  }
  if (final_score) {
    HIP_TRY(dalloc(&g->fin, S), "hipMalloc(graph)");
    HIP_TRY(hipMemcpy(g->fin, final_score, S * 4, hipMemcpyHostToDevice), "hipMemcpy(graph)");
  }
  return TBS_OK;
}

void graph_free(tbs_graph* g) {
  if (!g) return;
  (void)hipFree(g->rp);
  (void)hipFree(g->dest);
  (void)hipFree(g->label);
  (void)hipFree(g->q);
  (void)hipFree(g->fin);
  delete g;
}

hipError_t prof_event(tbs_model* m, hipEvent_t* ev) {
  if (!m->prof_pool.empty()) {
    *ev = m->prof_pool.back();
    m->prof_pool.pop_back();
    return hipSuccess;
  }
  return hipEventCreate(ev);
}

// Launches `fn` on st, timed when profiling is on: a single kernel launch records the
// two events in its own dispatch packet; the cooperative grouped kernel (one launch
// of milliseconds) is bracketed by events recorded on the stream.
template <class F>
hipError_t timed_launch(tbs_model* m, int kernel, hipStream_t st, F fn) {
  if (!m->prof) return fn();
  hipEvent_t a, b;
  hipError_t e = prof_event(m, &a);
  if (e == hipSuccess) e = prof_event(m, &b);
  if (e != hipSuccess) return e;
  if (kernel == TBS_KERNEL_STREAM_GROUP) {
    e = hipEventRecord(a, st);
    if (e == hipSuccess) e = fn();
    if (e == hipSuccess) e = hipEventRecord(b, st);
  } else {
    set_launch_events(a, b);
    e = fn();
    if (launch_events_pending()) {  // not taken by a launch (failed before it)
      set_launch_events(nullptr, nullptr);
      if (e == hipSuccess) e = hipErrorUnknown;
    }
  }
  if (e == hipSuccess) m->prof_pending.push_back({kernel, a, b});
  else {
    m->prof_pool.push_back(a);
    m->prof_pool.push_back(b);
  }
  return e;
}

void prof_drop(tbs_model* m) {
  for (auto& x : m->prof_pending) {
    (void)hipEventSynchronize(x.stop);
    m->prof_pool.push_back(x.start);
    m->prof_pool.push_back(x.stop);
  }
  m->prof_pending.clear();
}

// Allocates w for (B, T, Ns, Nc, KT); w must be empty.  w.len holds 2B entries: the
// frame counts of a call, then (chunked decode) each stream's frame base.
tbs_status alloc_workspace(const tbs_model* m, Workspace& w, int B, int T, int Ns, int Nc, int KT,
                           bool need_logits) {
  const int nvt = m->Vpad / kJoinerBN;
  const size_t BN = (size_t)B * Ns, BC = (size_t)B * Nc;
  const size_t esz = m->bf16 ? 2 : 4;
  HIP_TRY(dalloc(&w.len, 2 * (size_t)B), "hipMalloc(workspace)");
  HIP_TRY(dalloc(&w.nsurv, B), "hipMalloc(workspace)");
  HIP_TRY(dalloc(&w.surv_ctx, BN), "hipMalloc(workspace)");
  HIP_TRY(dalloc(&w.surv_state, BN), "hipMalloc(workspace)");
  HIP_TRY(dalloc(&w.surv_score, BN), "hipMalloc(workspace)");
  HIP_TRY(dalloc(&w.surv_row, BN), "hipMalloc(workspace)");
  HIP_TRY(dalloc(&w.surv_rp, BN), "hipMalloc(workspace)");
  HIP_TRY(dalloc(&w.nctx, B), "hipMalloc(workspace)");
  HIP_TRY(dalloc(&w.ctx_list, BC), "hipMalloc(workspace)");
  HIP_TRY(dalloc(&w.offset, B), "hipMalloc(workspace)");
  HIP_TRY(dalloc((char**)&w.h, BC * m->Kpad * esz), "hipMalloc(workspace)");
  if (need_logits) HIP_TRY(dalloc(&w.logits, BC * m->Vpad), "hipMalloc(workspace)");
  HIP_TRY(dalloc(&w.stats, BC * nvt), "hipMalloc(workspace)");
  if (KT > 0) {
    const size_t nsub = (size_t)nvt * (kJoinerBN / 16);
    HIP_TRY(dalloc(&w.tk_z, BC * nsub * KT), "hipMalloc(workspace)");
    HIP_TRY(dalloc(&w.tk_c, BC * nsub * KT), "hipMalloc(workspace)");
    HIP_TRY(dalloc(&w.z0, BC), "hipMalloc(workspace)");
  }
  HIP_TRY(dalloc(&w.hist_pl, (size_t)T * BN), "hipMalloc(workspace)");
  HIP_TRY(dalloc(&w.hist_arc, (size_t)T * BN), "hipMalloc(workspace)");
  HIP_TRY(dalloc(&w.path_lab, (size_t)B * T), "hipMalloc(workspace)");
  HIP_TRY(dalloc(&w.gtab, B), "hipMalloc(workspace)");
  HIP_TRY(dalloc(&w.xerr, 1 + (size_t)B + kXTickets), "hipMalloc(workspace)");
  HIP_TRY(hipHostMalloc((void**)&w.len_host, (size_t)(B > 0 ? 2 * B : 1) * 4, hipHostMallocDefault),
          "hipHostMalloc(workspace)");
  HIP_TRY(hipHostMalloc((void**)&w.gtab_host, (size_t)(B > 0 ? B : 1) * sizeof(GraphDev),
                        hipHostMallocDefault),
          "hipHostMalloc(workspace)");
  HIP_TRY(hipEventCreateWithFlags(&w.done, hipEventDisableTiming), "hipEventCreate");
  w.B = B;
  w.T = T;
  w.Ns = Ns;
  w.Nc = Nc;
  w.KT = KT;
  w.has_logits = need_logits;
  return TBS_OK;
}

tbs_status ensure_workspace(tbs_model* m, int B, int T, int Ns, int Nc, int KT,
                            bool need_logits) {
  Workspace& w = m->ws;
  if (w.done && w.B >= B && w.T >= T && w.Ns == Ns && w.Nc == Nc && w.KT == KT &&
      (w.has_logits || !need_logits))
    return TBS_OK;
  if (w.done) {
    if (w.pending) (void)hipEventSynchronize(w.done);
    w.release();
  }
  tbs_status st = alloc_workspace(m, w, B, T, Ns, Nc, KT, need_logits);
  if (st != TBS_OK) w.release();
  return st;
}

// The model's exchange buffer with at least `words` words, cleared if the epoch has
// wrapped since its last clear (on st, before the decode that uses it).
hipError_t ensure_xbuf(tbs_model* m, size_t words, hipStream_t st) {
  if (m->xbuf.p && m->xbuf.words < words) {
    std::lock_guard<std::mutex> xl(g_xmu);
    g_xfree.push_back(m->xbuf);
    m->xbuf = XBuf();
  }
  if (!m->xbuf.p) {
    std::lock_guard<std::mutex> xl(g_xmu);
    for (size_t i = 0; i < g_xfree.size(); ++i)
      if (g_xfree[i].dev == m->dev && g_xfree[i].words >= words) {
        m->xbuf = g_xfree[i];
        g_xfree.erase(g_xfree.begin() + (long)i);
        break;
      }
  }
  if (!m->xbuf.p) {
    XBuf x;
    x.dev = m->dev;
    x.words = words;
    hipError_t e = hipMalloc((void**)&x.p, words * 8);
    if (e != hipSuccess) return e;
    x.wrap = ~0u;  // cleared below
    m->xbuf = x;
  }
  const unsigned wrap = g_wrap.load();
  if (m->xbuf.wrap != wrap) {
    hipError_t e = launch_fill_i32((int*)m->xbuf.p, (long long)m->xbuf.words * 2, 0, st);
    if (e != hipSuccess) return e;
    m->xbuf.wrap = wrap;
  }
  return hipSuccess;
}

// Next 8-bit decode epoch of the grouped kernel's exchange tags (never 0, so zeroed
// words never match a tag); a wrap makes every exchange buffer be cleared before its
// next use.
unsigned next_epoch() {
  for (;;) {
    const unsigned e = (g_epoch.fetch_add(1) + 1) & 0xffu;
    if (e != 0) return e;
    g_wrap.fetch_add(1);
  }
}

// Workgroups per stream for the grouped per-stream kernel (1 = not grouped).
int pick_group(const tbs_model* m, const StreamPlan& sp, int B, int KT, int maxlen, int trivial) {
  if (!sp.ok || m->bf16 || !trivial || KT <= 0 || !m->coop || maxlen > 65535) return 1;
  const int ncg = m->Vpad / kJoinerBN;
  for (int G : {8, 4, 2})
    if (ncg % G == 0 && ncg / G <= 2 && (long long)B * G <= m->ncu) return G;
  return 1;
}

// Frame-loop schedule of a decode (tbs_model_set_schedule): persistent per-stream
// kernels or two kernels per frame.
tbs_status choose_schedule(const tbs_model* m, const StreamPlan& splan, int Ns, int Nc,
                           const char* who, bool* per_stream) {
  *per_stream = false;
  if (m->schedule == TBS_SCHEDULE_STREAM || m->schedule == TBS_SCHEDULE_STREAM_SINGLE) {
    if (!splan.ok)
      return fail(TBS_EUNSUPPORTED,
                  "%s: the per-stream schedule does not fit max_contexts %d / "
                  "max_states %d with V %d and dim %d",
                  who, Nc, Ns, m->V, m->C);
    *per_stream = true;
  } else if (m->schedule == TBS_SCHEDULE_AUTO) {
    // One compute unit streams the whole joiner weight every frame: worth it while
    // W stays L2-resident and the fp32 rows (broadcast from LDS to VALU FMAs) are few.
    *per_stream = splan.ok && (size_t)m->Vpad * m->Kpad * (m->bf16 ? 2 : 4) <= (4u << 20) &&
                  (m->bf16 || Nc <= 4);
  }
  return TBS_OK;
}

DecodeDev decode_dev(const tbs_model* m, const Workspace& w, int B, int T, int Ns, int Nc, int KT,
                     const float* enc, const int* len, const int* base, bool per_graph) {
  DecodeDev d;
  d.B = B;
  d.T = T;
  d.Ns = Ns;
  d.Nc = Nc;
  d.nvt = m->Vpad / kJoinerBN;
  d.KT = KT;
  d.enc = enc;
  d.len = len;
  d.base = base;
  d.graphs = per_graph ? w.gtab : nullptr;
  d.nsurv = w.nsurv;
  d.surv_ctx = w.surv_ctx;
  d.surv_state = w.surv_state;
  d.surv_score = w.surv_score;
  d.surv_row = w.surv_row;
  d.surv_rp = w.surv_rp;
  d.nctx = w.nctx;
  d.ctx_list = w.ctx_list;
  d.offset = w.offset;
  d.h = w.h;
  d.logits = w.logits;
  d.stats = w.stats;
  d.tk_z = w.tk_z;
  d.tk_c = w.tk_c;
  d.z0 = w.z0;
  d.hist_pl = w.hist_pl;
  d.hist_arc = w.hist_arc;
  d.path_lab = w.path_lab;
  return d;
}

// Workgroups per stream the decode of d will take (1: not grouped).
int decode_group(const tbs_model* m, const GraphDev& gd, const StreamPlan& splan, bool per_stream,
                 const DecodeDev& d, int maxlen) {
  return (per_stream && m->schedule != TBS_SCHEDULE_STREAM_SINGLE)
             ? pick_group(m, splan, d.B, d.KT, maxlen, gd.trivial)
             : 1;
}

// Enqueues frames 0 .. maxlen-1 of d: the grouped or single-workgroup persistent
// kernel, or the joiner and search kernels per frame.  xerr: the exchange-timeout
// counters ([1 + B]) the grouped kernel adds to.  xbuf: the grouped kernel's exchange
// words (zeroed), or null for the model's own buffer.  timed: per-kernel timing when
// profiling is on.  use_graph: the frame schedule's loop may be captured in a HIP graph
// (the model's capture setting).  *grouped: whether the grouped kernel ran.
tbs_status enqueue_frames(tbs_model* m, const GraphDev& gd, float beam,
                          const StreamPlan& splan, bool per_stream, const DecodeDev& d,
                          int maxlen, int* trace, unsigned* xerr, unsigned long long* xbuf,
                          bool timed, bool use_graph, hipStream_t st, bool* grouped) {
  *grouped = false;
  if (maxlen <= 0) return TBS_OK;
  const ModelDev md = model_dev(m);
  const int G = decode_group(m, gd, splan, per_stream, d, maxlen);
  auto launch = [&](int kernel, auto fn) { return timed ? timed_launch(m, kernel, st, fn) : fn(); };
  if (G > 1) {
    // the epoch first: a wrap it causes must clear the buffer before this decode
    const unsigned epoch = next_epoch();
    if (!xbuf) {
      HIP_TRY(ensure_xbuf(m, (size_t)d.B * G * 2 * group_words(d.Nc, d.KT), st),
              "exchange buffer");
      xbuf = m->xbuf.p;
    }
    hipError_t e = launch(TBS_KERNEL_STREAM_GROUP, [&] {
      return launch_stream_group(md, gd, d, beam, trace, splan, xbuf, G, epoch, m->spin_limit,
                                 xerr, st);
    });
    if (e == hipSuccess) {
      *grouped = true;
    } else if (e == hipErrorCooperativeLaunchTooLarge) {
      (void)hipGetLastError();  // not co-resident here: one workgroup per stream instead
    } else {
      return hip_fail(e, "launch(stream group)");
    }
  }
  if (per_stream && !*grouped)
    HIP_TRY(launch(TBS_KERNEL_STREAM,
                   [&] { return launch_stream(md, gd, d, beam, trace, splan, st); }),
            "launch(stream)");
  if (!per_stream) {
    const JoinerPlan plan = plan_joiner(d.B * d.Nc, m->Vpad, m->Kpad, m->bf16, m->ncu, d.KT > 0);
    auto frames = [&](hipStream_t s2) -> hipError_t {
      for (int t = 0; t < maxlen; ++t) {
        hipError_t e = launch(TBS_KERNEL_JOINER,
                              [&] { return launch_joiner_frame(md, d, plan, t, s2); });
        if (e == hipSuccess)
          e = launch(TBS_KERNEL_SEARCH,
                     [&] { return launch_search_frame(md, gd, d, beam, t, trace, s2); });
        if (e != hipSuccess) return e;
      }
      return hipSuccess;
    };
    if (!use_graph || (timed && m->prof)) {
      HIP_TRY(frames(st), "launch(frame loop)");
      return TBS_OK;
    }
    // the arguments of the loop's launches that can change between decodes on this
    // model, as bytes (GraphDev and DecodeDev hold no padding; the model's tables and
    // the joiner plan follow from the model and d)
    static_assert(sizeof(GraphDev) == 4 * sizeof(int) + 5 * sizeof(void*) &&
                      sizeof(DecodeDev) == 6 * sizeof(int) + 22 * sizeof(void*),
                  "frame-loop key: GraphDev / DecodeDev must have no padding");
    std::vector<unsigned char> key;
    auto put = [&](const void* p, size_t n) {
      const unsigned char* c = static_cast<const unsigned char*>(p);
      key.insert(key.end(), c, c + n);
    };
    put(&gd, sizeof gd);
    put(&d, sizeof d);
    put(&beam, sizeof beam);
    put(&trace, sizeof trace);
    put(&maxlen, sizeof maxlen);
    if (m->fg_exec && key == m->fg_key) {
      HIP_TRY(hipGraphLaunch(m->fg_exec, st), "hipGraphLaunch(frame loop)");
      ++m->fg_replays;
      return TBS_OK;
    }
    if (key != m->fg_seen) {  // first time: launch directly, capture if it repeats
      m->fg_seen = key;
      HIP_TRY(frames(st), "launch(frame loop)");
      return TBS_OK;
    }
    if (!m->cap_stream)
      HIP_TRY(hipStreamCreateWithFlags(&m->cap_stream, hipStreamNonBlocking), "hipStreamCreate");
    HIP_TRY(hipStreamBeginCapture(m->cap_stream, hipStreamCaptureModeThreadLocal),
            "hipStreamBeginCapture");
    hipError_t e = frames(m->cap_stream);
    hipGraph_t g = nullptr;
    const hipError_t e2 = hipStreamEndCapture(m->cap_stream, &g);
    if (e == hipSuccess) e = e2;
    hipGraphExec_t x = nullptr;
    if (e == hipSuccess) e = hipGraphInstantiate(&x, g, nullptr, nullptr, 0);
    if (e != hipSuccess) {
      if (g) (void)hipGraphDestroy(g);
      return hip_fail(e, "capture(frame loop)");
    }
    if (m->fg_exec) (void)hipGraphExecDestroy(m->fg_exec);
    if (m->fg_graph) (void)hipGraphDestroy(m->fg_graph);
    m->fg_exec = x;
    m->fg_graph = g;
    m->fg_key = key;
    ++m->fg_captures;
    HIP_TRY(hipGraphLaunch(m->fg_exec, st), "hipGraphLaunch(frame loop)");
  }
  return TBS_OK;
}

// Checks shared by tbs_decode and tbs_state_create.
tbs_status check_params(const tbs_model* model, const tbs_graph* graph,
                        const tbs_beam_params* params, const char* who) {
  if (!model || !graph || !params) return fail(TBS_EINVAL, "%s: NULL model/graph/params", who);
  if (graph->V != model->V)
    return fail(TBS_EINVAL, "%s: graph vocab_size %d != model vocab_size %d", who, graph->V,
                model->V);
  const float beam = params->beam;
  const int Ns = params->max_states, Nc = params->max_contexts;
  if (std::isnan(beam) || beam < 0.f)
    return fail(TBS_EINVAL, "%s: beam must be >= 0 or INFINITY", who);
  if (Ns < 1 || Nc < 1)
    return fail(TBS_EINVAL, "%s: max_states and max_contexts must be >= 1", who);
  if (Ns > kMaxStates)
    return fail(TBS_ECAPACITY, "%s: max_states %d exceeds the limit %d", who, Ns, kMaxStates);
  if ((long long)Ns * ((long long)graph->maxdeg + 1) >= (1ll << 31))
    return fail(TBS_ECAPACITY, "%s: max_states * (max out-degree + 1) = %lld must be < 2^31", who,
                (long long)Ns * ((long long)graph->maxdeg + 1));
  return TBS_OK;
}

// The graphs of a decode: one shared graph, or one per stream (graphs[B], host array).
// The returned descriptor is the shared graph's, or (per-stream graphs) the first
// graph's with the largest out-degree of all and no trivial-graph fast path; the
// kernels then take each stream's own descriptor from the workspace's graph table.
tbs_status graph_set(const tbs_model* model, const tbs_graph* graph,
                     const tbs_graph* const* graphs, int B, const tbs_beam_params* params,
                     const char* who, GraphDev* out) {
  if (!graphs) {
    tbs_status s = check_params(model, graph, params, who);
    if (s == TBS_OK) *out = graph_dev(graph);
    return s;
  }
  if (B < 1) return fail(TBS_EINVAL, "%s: B must be >= 1", who);
  int maxdeg = 0;
  for (int b = 0; b < B; ++b) {
    if (!graphs[b]) return fail(TBS_EINVAL, "%s: graphs[%d] is NULL", who, b);
    tbs_status s = check_params(model, graphs[b], params, who);
    if (s != TBS_OK) return s;
    if (graphs[b]->maxdeg > maxdeg) maxdeg = graphs[b]->maxdeg;
  }
  *out = graph_dev(graphs[0]);
  out->maxdeg = maxdeg;
  out->trivial = 0;
  return TBS_OK;
}

// Stages the per-stream graph table of w (w's previous device work must be done).
hipError_t upload_graphs(Workspace& w, const tbs_graph* const* graphs, int B, hipStream_t st) {
  for (int b = 0; b < B; ++b) w.gtab_host[b] = graph_dev(graphs[b]);
  return hipMemcpyAsync(w.gtab, w.gtab_host, (size_t)B * sizeof(GraphDev), hipMemcpyHostToDevice,
                        st);
}

// Waits (on st) for the model's previous device work; marks st's work as the latest.
hipError_t model_wait(tbs_model* m, hipStream_t st) {
  return m->busy_pending ? hipStreamWaitEvent(st, m->busy, 0) : hipSuccess;
}
hipError_t model_mark(tbs_model* m, hipStream_t st) {
  hipError_t e = hipEventRecord(m->busy, st);
  if (e == hipSuccess) m->busy_pending = true;
  return e;
}

}  // namespace

struct tbs_state {
  tbs_model* m = nullptr;
  GraphDev gd{};            // the shared graph, or the per-stream graphs' summary
  bool per_graph = false;   // one graph per stream (table in w.gtab)
  float beam = 0.f;
  int Ns = 0, Nc = 0, KT = 0, B = 0, Tcap = 0;
  bool per_stream = false;
  StreamPlan splan{};
  Workspace w;
  std::vector<int> done;     // frames decoded so far per stream
};

extern "C" {

const char* tbs_last_error(void) { return g_last_error.c_str(); }

tbs_status tbs_graph_create(int32_t num_states, int32_t start_state, int32_t vocab_size,
                            const int32_t* row_ptr, const int32_t* dest, const int32_t* label,
                            const float* score, const float* final_score, tbs_graph** out) {
  if (!out) return fail(TBS_EINVAL, "tbs_graph_create: out is NULL");
  *out = nullptr;
  if (num_states < 1) return fail(TBS_EINVAL, "tbs_graph_create: num_states must be >= 1");
  if (start_state < 0 || start_state >= num_states)
    return fail(TBS_EINVAL, "tbs_graph_create: start_state %d outside [0, %d)", start_state,
                num_states);
  if (vocab_size < 2 || vocab_size > kMaxVocab)
    return fail(TBS_EINVAL, "tbs_graph_create: vocab_size %d outside [2, %d]", vocab_size,
                kMaxVocab);
  if (!row_ptr) return fail(TBS_EINVAL, "tbs_graph_create: row_ptr is NULL");
  if (row_ptr[0] != 0) return fail(TBS_EINVAL, "tbs_graph_create: row_ptr[0] must be 0");
  int maxdeg = 0;
  for (int s = 0; s < num_states; ++s) {
    const long long d = (long long)row_ptr[s + 1] - row_ptr[s];
    if (d < 0)
      return fail(TBS_EINVAL, "tbs_graph_create: row_ptr decreases at state %d", s);
    if (d > maxdeg) maxdeg = (int)d;
  }
  const int A = row_ptr[num_states];
  if (A > 0 && (!dest || !label || !score))
    return fail(TBS_EINVAL, "tbs_graph_create: dest/label/score is NULL");
  for (int j = 0; j < A; ++j) {
    if (dest[j] < 0 || dest[j] >= num_states)
      return fail(TBS_EINVAL, "tbs_graph_create: dest[%d] = %d outside [0, %d)", j, dest[j],
                  num_states);
    if (label[j] < 1 || label[j] >= vocab_size)
      return fail(TBS_EINVAL,
                  "tbs_graph_create: label[%d] = %d outside [1, %d] (the graph must be epsilon-free)",
                  j, label[j], vocab_size - 1);
    if (!std::isfinite(score[j]))
      return fail(TBS_EINVAL, "tbs_graph_create: score[%d] is not finite", j);
  }
  if (final_score) {
    for (int s = 0; s < num_states; ++s) {
      const float f = final_score[s];
      if (std::isnan(f) || f == INFINITY)
        return fail(TBS_EINVAL, "tbs_graph_create: final_score[%d] must be finite or -inf", s);
    }
  }
  tbs_graph* g = new tbs_graph();
  g->S = num_states;
  g->start = start_state;
  g->V = vocab_size;
  g->A = A;
  g->maxdeg = maxdeg;
  bool trivial = num_states == 1 && A == vocab_size - 1 &&
                 (!final_score || final_score[0] == 0.f);
  for (int j = 0; trivial && j < A; ++j)
    trivial = label[j] == j + 1 && dest[j] == 0 && score[j] == 0.f;
  g->trivial = trivial;
  tbs_status st = graph_upload(g, row_ptr, dest, label, score, final_score);
  if (st != TBS_OK) {
    graph_free(g);
    return st;
  }
  *out = g;
  return TBS_OK;
}

tbs_status tbs_graph_create_trivial(int32_t vocab_size, tbs_graph** out) {
  if (!out) return fail(TBS_EINVAL, "tbs_graph_create_trivial: out is NULL");
  *out = nullptr;
  if (vocab_size < 2 || vocab_size > kMaxVocab)
    return fail(TBS_EINVAL, "tbs_graph_create_trivial: vocab_size %d outside [2, %d]",
                vocab_size, kMaxVocab);
  const int A = vocab_size - 1;
  std::vector<int32_t> rp = {0, A}, dest(A, 0), label(A);
  std::vector<float> q(A, 0.f);
  for (int j = 0; j < A; ++j) label[j] = j + 1;
  return tbs_graph_create(1, 0, vocab_size, rp.data(), dest.data(), label.data(), q.data(),
                          nullptr, out);
}

void tbs_graph_destroy(tbs_graph* graph) { graph_free(graph); }

tbs_status tbs_model_create(int32_t vocab_size, int32_t dim, int32_t context_size,
                            const float* embed, const float* conv, const float* w_out,
                            const float* b_out, tbs_joiner_dtype dtype, void* hip_stream,
                            tbs_model** out) {
  if (!out) return fail(TBS_EINVAL, "tbs_model_create: out is NULL");
  *out = nullptr;
  if (context_size != 2)
    return fail(TBS_EUNSUPPORTED, "tbs_model_create: context_size %d unsupported (must be 2)",
                context_size);
  if (vocab_size < 2 || vocab_size > kMaxVocab)
    return fail(TBS_EINVAL, "tbs_model_create: vocab_size %d outside [2, %d]", vocab_size,
                kMaxVocab);
  if (dim < 1 || dim > kMaxDim)
    return fail(TBS_EINVAL, "tbs_model_create: dim %d outside [1, %d]", dim, kMaxDim);
  if (!embed || !conv || !w_out)
    return fail(TBS_EINVAL, "tbs_model_create: embed/conv/w_out is NULL");
  if (dtype != TBS_JOINER_FP32 && dtype != TBS_JOINER_BF16)
    return fail(TBS_EINVAL, "tbs_model_create: unknown dtype %d", (int)dtype);
  hipStream_t st = (hipStream_t)hip_stream;
  tbs_model* m = new tbs_model();
  m->V = vocab_size;
  m->C = dim;
  m->Kpad = round_up(dim, kKStep);
  m->Vpad = round_up(vocab_size, kJoinerBN);
  m->bf16 = dtype == TBS_JOINER_BF16;
  const size_t VK = (size_t)m->V * m->Kpad, VpK = (size_t)m->Vpad * m->Kpad;
  hipError_t e = hipGetDevice(&m->dev);
  if (e == hipSuccess)
    e = hipDeviceGetAttribute(&m->ncu, hipDeviceAttributeMultiprocessorCount, m->dev);
  if (e == hipSuccess)
    e = hipDeviceGetAttribute(&m->coop, hipDeviceAttributeCooperativeLaunch, m->dev);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&m->busy, hipEventDisableTiming);
  if (e == hipSuccess) e = dalloc(&m->P0, VK);
  if (e == hipSuccess) e = dalloc(&m->P1, VK);
  if (e == hipSuccess) e = m->bf16 ? dalloc(&m->Wb, VpK) : dalloc(&m->Wf, VpK);
  if (e == hipSuccess) e = dalloc((char**)&m->Wi, VpK * (m->bf16 ? 2 : 4));
  if (e == hipSuccess) e = dalloc(&m->bias, (size_t)m->V);
  if (e == hipSuccess)
    e = launch_model_setup(embed, conv, w_out, b_out, m->V, m->C, m->Kpad, m->Vpad, m->bf16,
                           m->P0, m->P1, m->Wf, m->Wb, m->Wi, m->bias, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) {
    tbs_model_destroy(m);
    return hip_fail(e, "tbs_model_create");
  }
  *out = m;
  return TBS_OK;
}

void tbs_model_destroy(tbs_model* m) {
  if (!m) return;
  {
    std::lock_guard<std::mutex> lk(m->mu);
    if (m->ws.done && m->ws.pending) (void)hipEventSynchronize(m->ws.done);
    m->ws.release();
    m->hw.release();
    if (m->lat_cache) lattice_free(m->lat_cache);
    m->lat_cache = nullptr;
  }
  prof_drop(m);
  for (hipEvent_t e : m->prof_pool) (void)hipEventDestroy(e);
  (void)hipFree(m->P0);
  (void)hipFree(m->P1);
  (void)hipFree(m->Wf);
  (void)hipFree(m->Wb);
  (void)hipFree(m->Wi);
  (void)hipFree(m->bias);
  if (m->busy) {
    if (m->busy_pending) (void)hipEventSynchronize(m->busy);
    (void)hipEventDestroy(m->busy);
  }
  if (m->xbuf.p) {
    std::lock_guard<std::mutex> xl(g_xmu);
    g_xfree.push_back(m->xbuf);
  }
  (void)hipFree(m->rows_h);
  (void)hipFree(m->rows_logits);
  (void)hipFree(m->rows_stats);
  if (m->fg_exec) (void)hipGraphExecDestroy(m->fg_exec);
  if (m->fg_graph) (void)hipGraphDestroy(m->fg_graph);
  if (m->cap_stream) (void)hipStreamDestroy(m->cap_stream);
  delete m;
}

}  // extern "C"

namespace {

// tbs_decode and tbs_decode_graphs: one shared graph, or graphs[B] (one per stream).
tbs_status decode_impl(const tbs_model* model, const tbs_graph* graph,
                       const tbs_graph* const* graphs, const tbs_beam_params* params,
                       const float* encoder_out, const int32_t* lengths, int32_t B, int32_t T,
                       int32_t* out_tokens, int32_t* out_num_tokens, double* out_scores,
                       int32_t* out_status, int32_t* out_arcs, int32_t* trace, void* hip_stream,
                       const char* who) {
  if (B < 0 || T < 0) return fail(TBS_EINVAL, "%s: B and T must be >= 0", who);
  if (B == 0) return graphs ? TBS_OK : check_params(model, graph, params, who);
  GraphDev gd;
  tbs_status s = graph_set(model, graph, graphs, B, params, who, &gd);
  if (s != TBS_OK) return s;
  const float beam = params->beam;
  const int Ns = params->max_states, Nc_req = params->max_contexts;
  if (!lengths) return fail(TBS_EINVAL, "%s: lengths is NULL", who);
  int maxlen = 0;
  for (int b = 0; b < B; ++b) {
    if (lengths[b] < 0 || lengths[b] > T)
      return fail(TBS_EINVAL, "%s: lengths[%d] = %d outside [0, %d]", who, b, lengths[b], T);
    if (lengths[b] > maxlen) maxlen = lengths[b];
  }
  if (maxlen > 0 && !encoder_out) return fail(TBS_EINVAL, "%s: encoder_out is NULL", who);
  if (!out_num_tokens || !out_scores || (T > 0 && !out_tokens))
    return fail(TBS_EINVAL, "%s: NULL output pointer", who);
  // More contexts than tuples can never be active.
  const int Nc = Nc_req < Ns ? Nc_req : Ns;
  // Trivial graph with few tuples: the joiner keeps each row's best labels per
  // vocabulary tile instead of materialising the logits.
  const int KT = (gd.trivial && Ns <= kMaxTopK) ? Ns : 0;

  tbs_model* m = const_cast<tbs_model*>(model);
  std::lock_guard<std::mutex> lk(m->mu);
  hipStream_t st = (hipStream_t)hip_stream;
  const ModelDev md = model_dev(m);
  const StreamPlan splan = plan_stream(md, Nc, KT, gd.trivial);
  bool per_stream = false;
  s = choose_schedule(m, splan, Ns, Nc, who, &per_stream);
  if (s != TBS_OK) return s;
  s = ensure_workspace(m, B, T, Ns, Nc, KT, KT == 0);
  if (s != TBS_OK) return s;
  Workspace& w = m->ws;
  HIP_TRY(model_wait(m, st), "hipStreamWaitEvent");
  if (w.pending) HIP_TRY(hipStreamWaitEvent(st, w.done, 0), "hipStreamWaitEvent");
  // lengths: wait until the previous decode consumed the pinned staging buffers
  if (w.pending) HIP_TRY(hipEventSynchronize(w.done), "hipEventSynchronize");
  std::memcpy(w.len_host, lengths, (size_t)B * 4);
  HIP_TRY(hipMemcpyAsync(w.len, w.len_host, (size_t)B * 4, hipMemcpyHostToDevice, st),
          "hipMemcpyAsync(lengths)");
  if (graphs) HIP_TRY(upload_graphs(w, graphs, B, st), "hipMemcpyAsync(graphs)");

  const DecodeDev d =
      decode_dev(m, w, B, T, Ns, Nc, KT, encoder_out, w.len, nullptr, graphs != nullptr);
  if (trace)
    HIP_TRY(launch_fill_i32(trace, (long long)(T + 1) * B * Ns * 4, -1, st), "fill(trace)");
  HIP_TRY(launch_init(md, d, gd, trace, st), "launch(init)");
  HIP_TRY(launch_fill_i32((int*)w.xerr, 1 + (long long)B + kXTickets, 0, st), "fill(exchange errors)");
  bool grouped = false;
  s = enqueue_frames(m, gd, beam, splan, per_stream, d, maxlen, trace, w.xerr, nullptr, true,
                     m->graphs, st, &grouped);
  if (s != TBS_OK) return s;
  HIP_TRY(timed_launch(m, TBS_KERNEL_FINAL, st,
                       [&] {
                         return launch_final(gd, d, out_tokens, out_num_tokens, out_scores,
                                             out_status, out_arcs, grouped ? w.xerr : nullptr,
                                             st);
                       }),
          "launch(final)");
  HIP_TRY(hipEventRecord(w.done, st), "hipEventRecord");
  w.pending = true;
  HIP_TRY(model_mark(m, st), "hipEventRecord");
  return TBS_OK;
}

// Lays out a decode workspace for (B, T, Ns, Nc, KT) at `base` (an address, or 0 to
// size it only) and returns the bytes it takes: the device arrays tbs_decode allocates
// (no per-stream graph table, no host staging), then `xwords` exchange words.
size_t carve_workspace(const tbs_model* m, uintptr_t base, int B, int T, int Ns, int Nc, int KT,
                       bool need_logits, size_t xwords, Workspace& w,
                       unsigned long long** xbuf) {
  size_t off = 0;
  auto take = [&](auto*& p, size_t n) {
    p = reinterpret_cast<std::remove_reference_t<decltype(p)>>(base + off);
    off += (((n ? n : 1) * sizeof(*p)) + 255) & ~(size_t)255;
  };
  const int nvt = m->Vpad / kJoinerBN;
  const size_t BN = (size_t)B * Ns, BC = (size_t)B * Nc;
  const size_t esz = m->bf16 ? 2 : 4;
  w = Workspace();
  take(w.len, (size_t)B);
  take(w.nsurv, (size_t)B);
  take(w.surv_ctx, BN);
  take(w.surv_state, BN);
  take(w.surv_score, BN);
  take(w.surv_row, BN);
  take(w.surv_rp, BN);
  take(w.nctx, (size_t)B);
  take(w.ctx_list, BC);
  take(w.offset, (size_t)B);
  char* h = nullptr;
  take(h, BC * m->Kpad * esz);
  w.h = h;
  if (need_logits) take(w.logits, BC * m->Vpad);
  take(w.stats, BC * nvt);
  if (KT > 0) {
    const size_t nsub = (size_t)nvt * (kJoinerBN / 16);
    take(w.tk_z, BC * nsub * KT);
    take(w.tk_c, BC * nsub * KT);
    take(w.z0, BC);
  }
  take(w.hist_pl, (size_t)T * BN);
  take(w.hist_arc, (size_t)T * BN);
  take(w.path_lab, (size_t)B * T);
  take(w.xerr, 1 + (size_t)B + kXTickets);
  *xbuf = nullptr;
  if (xwords) take(*xbuf, xwords);
  w.B = B;
  w.T = T;
  w.Ns = Ns;
  w.Nc = Nc;
  w.KT = KT;
  w.has_logits = need_logits;
  return off;
}

tbs_status state_create_impl(const tbs_model* model, const tbs_graph* graph,
                             const tbs_graph* const* graphs, const tbs_beam_params* params,
                             int32_t B, int32_t max_frames, void* hip_stream, tbs_state** out,
                             const char* who) {
  if (!out) return fail(TBS_EINVAL, "%s: out is NULL", who);
  *out = nullptr;
  if (B < 1 || max_frames < 1) return fail(TBS_EINVAL, "%s: B and max_frames must be >= 1", who);
  GraphDev gd;
  tbs_status s = graph_set(model, graph, graphs, B, params, who, &gd);
  if (s != TBS_OK) return s;
  tbs_model* m = const_cast<tbs_model*>(model);
  std::lock_guard<std::mutex> lk(m->mu);
  hipStream_t st = (hipStream_t)hip_stream;
  tbs_state* S = new tbs_state();
  S->m = m;
  S->gd = gd;
  S->per_graph = graphs != nullptr;
  S->beam = params->beam;
  S->Ns = params->max_states;
  S->Nc = params->max_contexts < S->Ns ? params->max_contexts : S->Ns;
  S->KT = (gd.trivial && S->Ns <= kMaxTopK) ? S->Ns : 0;
  S->B = B;
  S->Tcap = max_frames;
  S->done.assign(B, 0);
  const ModelDev md = model_dev(m);
  S->splan = plan_stream(md, S->Nc, S->KT, gd.trivial);
  s = choose_schedule(m, S->splan, S->Ns, S->Nc, who, &S->per_stream);
  if (s == TBS_OK) s = alloc_workspace(m, S->w, B, max_frames, S->Ns, S->Nc, S->KT, S->KT == 0);
  hipError_t e = hipSuccess;
  if (s == TBS_OK) {
    e = launch_fill_i32((int*)S->w.xerr, 1 + (long long)B + kXTickets, 0, st);
    // the initial tuple of every stream (k_init with zero lengths writes no joiner row)
    if (e == hipSuccess) e = launch_fill_i32(S->w.len, 2 * (long long)B, 0, st);
    // the graph table stays for the state's lifetime
    if (e == hipSuccess && graphs) e = upload_graphs(S->w, graphs, B, st);
    if (e == hipSuccess) {
      const DecodeDev d = decode_dev(m, S->w, B, max_frames, S->Ns, S->Nc, S->KT, nullptr,
                                     S->w.len, nullptr, S->per_graph);
      e = launch_init(md, d, gd, nullptr, st);
    }
    if (e == hipSuccess) e = hipEventRecord(S->w.done, st);
    if (e == hipSuccess) S->w.pending = true;
    if (e != hipSuccess) s = hip_fail(e, who);
  }
  if (s != TBS_OK) {
    if (S->w.pending) (void)hipEventSynchronize(S->w.done);
    S->w.release();
    delete S;
    return s;
  }
  *out = S;
  return TBS_OK;
}

}  // namespace

struct tbs_lattice {
  tbs_model* m = nullptr;
  GraphDev gd{};
  int B = 0, T = 0, Ns = 0, Nc = 0;
  long long A = 0;                  // arcs
  // allocated capacity (a destroyed lattice's buffers serve the model's next one)
  int capB = 0, capT = 0, capNs = 0, capNc = 0;
  long long capA = 0;
  size_t cap_rows = 0;
  int* len_host = nullptr;          // pinned staging: lengths [capB]
  GraphDev* gtab_host = nullptr;    // pinned staging: per-stream graphs [capB]
  int* len = nullptr;               // [B]
  int* trace = nullptr;             // [T+1][B][Ns][4] survivors (the lattice nodes)
  int* tokens = nullptr;            // best path of the search (needed by the decode call)
  int* ntok = nullptr;
  double* scores = nullptr;
  int* dstatus = nullptr;
  GraphDev* gtab = nullptr;         // [B] per-stream graphs
  bool per_graph = false;           // gtab in use
  int* nn = nullptr;
  int* cnt = nullptr;
  long long* off = nullptr;
  int* dptr = nullptr;
  int4* arcs = nullptr;
  float* w = nullptr;
  double* pc = nullptr;
  int* rowctx = nullptr;
  double* alpha = nullptr;
  double* fw = nullptr;
  double* total = nullptr;
  int* status = nullptr;
  void* h = nullptr;                // joiner rows of one chunk of streams
  float* logits = nullptr;
  float2* stats = nullptr;
  // n-best scratch, for up to ncap paths
  int ncap = 0;
  int* seq = nullptr;
  int* pntok = nullptr;
  unsigned long long* hash = nullptr;
  int* first = nullptr;
  int* nuniq = nullptr;
  double* uscore = nullptr;
  double* dp = nullptr;
  size_t dp_lds = 0;
  int dp_grid = 0;
  hipEvent_t done = nullptr;        // the lattice's latest device work
  bool pending = false;

  LatticeDev dev() const {
    LatticeDev L;
    L.B = B;
    L.T = T;
    L.Ns = Ns;
    L.Nc = Nc;
    L.V = m->V;
    L.len = len;
    L.nodes = trace;
    L.graphs = per_graph ? gtab : nullptr;
    L.nn = nn;
    L.cnt = cnt;
    L.off = off;
    L.dptr = dptr;
    L.arcs = arcs;
    L.w = w;
    L.pc = pc;
    L.rowctx = rowctx;
    L.alpha = alpha;
    L.fw = fw;
    L.total = total;
    L.status = status;
    return L;
  }
  void free_nbest() {
    (void)hipFree(seq); (void)hipFree(pntok); (void)hipFree(hash); (void)hipFree(first); (void)hipFree(nuniq);
    (void)hipFree(uscore); (void)hipFree(dp);
    seq = pntok = first = nuniq = nullptr;
    hash = nullptr;
    uscore = dp = nullptr;
    ncap = 0;
  }
  void release() {
    if (done && pending) (void)hipEventSynchronize(done);
    free_nbest();
    (void)hipFree(len); (void)hipFree(trace); (void)hipFree(tokens); (void)hipFree(ntok); (void)hipFree(scores);
    (void)hipFree(dstatus); (void)hipFree(gtab); (void)hipFree(nn); (void)hipFree(cnt); (void)hipFree(off); (void)hipFree(dptr);
    (void)hipFree(arcs); (void)hipFree(w); (void)hipFree(pc); (void)hipFree(rowctx); (void)hipFree(alpha); (void)hipFree(fw); (void)hipFree(total);
    (void)hipFree(status); (void)hipFree(h); (void)hipFree(logits); (void)hipFree(stats);
    if (len_host) (void)hipHostFree(len_host);
    if (gtab_host) (void)hipHostFree(gtab_host);
    if (done) (void)hipEventDestroy(done);
  }
};

void lattice_free(tbs_lattice* L) {
  L->release();
  delete L;
}

namespace {

// Builds the lattice of a decode (tbs_lattice_create / tbs_lattice_create_graphs).
tbs_status lattice_create_impl(const tbs_model* model, const tbs_graph* graph,
                               const tbs_graph* const* graphs, const tbs_beam_params* params,
                               const float* encoder_out, const int32_t* lengths, int32_t B,
                               int32_t T, void* hip_stream, tbs_lattice** out, const char* who) {
  if (!out) return fail(TBS_EINVAL, "%s: out is NULL", who);
  *out = nullptr;
  if (B < 1 || T < 0) return fail(TBS_EINVAL, "%s: B must be >= 1 and T >= 0", who);
  GraphDev gd;
  tbs_status s = graph_set(model, graph, graphs, B, params, who, &gd);
  if (s != TBS_OK) return s;
  if (!lengths) return fail(TBS_EINVAL, "%s: lengths is NULL", who);
  for (int b = 0; b < B; ++b)
    if (lengths[b] < 0 || lengths[b] > T)
      return fail(TBS_EINVAL, "%s: lengths[%d] = %d outside [0, %d]", who, b, lengths[b], T);
  tbs_model* m = const_cast<tbs_model*>(model);
  hipStream_t st = (hipStream_t)hip_stream;
  const int Ns = params->max_states;
  const int Nc = params->max_contexts < Ns ? params->max_contexts : Ns;
  const size_t BN = (size_t)B * Ns, BT = (size_t)B * T;
  const int nvt = m->Vpad / kJoinerBN;
  const size_t esz = m->bf16 ? 2 : 4;
  // joiner rows per chunk of streams: whole streams, logits of at most 512 MiB
  const size_t per_stream = (size_t)T * Nc;
  size_t cap_rows = ((size_t)512 << 20) / ((size_t)m->Vpad * 4);
  if (cap_rows < per_stream) cap_rows = per_stream;
  const int chunk = per_stream == 0 ? B : (int)std::min<size_t>(B, cap_rows / per_stream);
  const size_t rows = per_stream * (size_t)chunk;
  // the buffers of the model's last destroyed lattice, when they are large enough
  tbs_lattice* L = nullptr;
  {
    std::lock_guard<std::mutex> lk(m->mu);
    L = m->lat_cache;
    m->lat_cache = nullptr;
  }
  if (L && !(B <= L->capB && T <= L->capT && Ns == L->capNs && Nc == L->capNc &&
             rows <= L->cap_rows)) {
    L->release();
    delete L;
    L = nullptr;
  }
  auto cleanup = [&](tbs_status st_) {
    L->release();
    delete L;
    return st_;
  };
  hipError_t e = hipSuccess;
  if (!L) {
    L = new tbs_lattice();
#define LAT_ALLOC(expr) \
  if (e == hipSuccess) e = (expr)
    LAT_ALLOC(dalloc(&L->len, B));
    LAT_ALLOC(dalloc(&L->trace, (size_t)(T + 1) * BN * 4));
    LAT_ALLOC(dalloc(&L->tokens, BT));
    LAT_ALLOC(dalloc(&L->ntok, B));
    LAT_ALLOC(dalloc(&L->scores, B));
    LAT_ALLOC(dalloc(&L->dstatus, B));
    LAT_ALLOC(dalloc(&L->gtab, B));
    LAT_ALLOC(dalloc(&L->nn, (size_t)B * (T + 1)));
    LAT_ALLOC(dalloc(&L->cnt, BT));
    LAT_ALLOC(dalloc(&L->off, BT + 1));
    LAT_ALLOC(dalloc(&L->dptr, BT * (Ns + 1)));
    LAT_ALLOC(dalloc(&L->rowctx, BT * Nc));
    LAT_ALLOC(dalloc(&L->alpha, (size_t)(T + 1) * BN));
    LAT_ALLOC(dalloc(&L->fw, BN));
    LAT_ALLOC(dalloc(&L->total, B));
    LAT_ALLOC(dalloc(&L->status, B));
    LAT_ALLOC(dalloc((char**)&L->h, rows * m->Kpad * esz));
    LAT_ALLOC(dalloc(&L->logits, rows * m->Vpad));
    LAT_ALLOC(dalloc(&L->stats, rows * nvt));
    LAT_ALLOC(hipHostMalloc((void**)&L->len_host, (size_t)B * 4, hipHostMallocDefault));
    LAT_ALLOC(hipHostMalloc((void**)&L->gtab_host, (size_t)B * sizeof(GraphDev),
                            hipHostMallocDefault));
    LAT_ALLOC(hipEventCreateWithFlags(&L->done, hipEventDisableTiming));
#undef LAT_ALLOC
    L->capB = B;
    L->capT = T;
    L->capNs = Ns;
    L->capNc = Nc;
    L->cap_rows = rows;
    if (e != hipSuccess) return cleanup(hip_fail(e, who));
  }
  L->m = m;
  L->gd = gd;
  L->B = B;
  L->T = T;
  L->Ns = Ns;
  L->Nc = Nc;
  L->A = 0;
  L->pending = false;
  std::memcpy(L->len_host, lengths, (size_t)B * 4);
  e = hipMemcpyAsync(L->len, L->len_host, (size_t)B * 4, hipMemcpyHostToDevice, st);
  if (graphs) {
    for (int b = 0; b < B; ++b) L->gtab_host[b] = graph_dev(graphs[b]);
    if (e == hipSuccess)
      e = hipMemcpyAsync(L->gtab, L->gtab_host, (size_t)B * sizeof(GraphDev),
                         hipMemcpyHostToDevice, st);
  }
  if (e != hipSuccess) return cleanup(hip_fail(e, who));
  L->per_graph = graphs != nullptr;
  // the search, with its survivor trace as the lattice nodes
  s = decode_impl(model, graph, graphs, params, encoder_out, lengths, B, T, L->tokens, L->ntok,
                  L->scores, L->dstatus, nullptr, L->trace, hip_stream, who);
  if (s != TBS_OK) return cleanup(s);
  const LatticeDev d0 = L->dev();
  // node counts: the count pass writes them; with no frames only the initial node exists
  e = T == 0 ? launch_fill_i32(L->nn, B, 1, st) : launch_lattice_count(d0, gd, st);
  if (e == hipSuccess) e = launch_lattice_scan(d0, st);
  if (e == hipSuccess)
    e = hipMemcpyAsync(&L->A, L->off + BT, sizeof(long long), hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e == hipSuccess && L->A > L->capA) {
    (void)hipFree(L->arcs);
    (void)hipFree(L->w);
    (void)hipFree(L->pc);
    L->arcs = nullptr;
    L->w = nullptr;
    L->pc = nullptr;
    L->capA = 0;
    e = dalloc(&L->arcs, (size_t)L->A);
    if (e == hipSuccess) e = dalloc(&L->w, (size_t)L->A);
    if (e == hipSuccess) e = dalloc(&L->pc, (size_t)L->A);
    if (e == hipSuccess) L->capA = L->A;
  }
  if (e != hipSuccess) return cleanup(hip_fail(e, who));
  const LatticeDev d = L->dev();
  const ModelDev md = model_dev(m);
  e = launch_lattice_fill(d, gd, st);
  for (int b0 = 0; e == hipSuccess && b0 < B; b0 += chunk)
    e = launch_lattice_weights(md, d, gd, encoder_out, b0, std::min(B, b0 + chunk), L->h,
                               L->logits, L->stats, m->ncu, st);
  if (e == hipSuccess) e = launch_lattice_forward(d, gd, st);
  if (e == hipSuccess) e = hipEventRecord(L->done, st);
  if (e != hipSuccess) return cleanup(hip_fail(e, who));
  L->pending = true;
  *out = L;
  return TBS_OK;
}

}  // namespace

extern "C" {

tbs_status tbs_decode(const tbs_model* model, const tbs_graph* graph,
                      const tbs_beam_params* params, const float* encoder_out,
                      const int32_t* lengths, int32_t B, int32_t T, int32_t* out_tokens,
                      int32_t* out_num_tokens, double* out_scores, int32_t* out_status,
                      int32_t* out_arcs, int32_t* trace, void* hip_stream) {
  if (!graph) return fail(TBS_EINVAL, "tbs_decode: graph is NULL");
  return decode_impl(model, graph, nullptr, params, encoder_out, lengths, B, T, out_tokens,
                     out_num_tokens, out_scores, out_status, out_arcs, trace, hip_stream,
                     "tbs_decode");
}

tbs_status tbs_decode_graphs(const tbs_model* model, const tbs_graph* const* graphs,
                             const tbs_beam_params* params, const float* encoder_out,
                             const int32_t* lengths, int32_t B, int32_t T, int32_t* out_tokens,
                             int32_t* out_num_tokens, double* out_scores, int32_t* out_status,
                             int32_t* out_arcs, int32_t* trace, void* hip_stream) {
  if (!graphs && B > 0) return fail(TBS_EINVAL, "tbs_decode_graphs: graphs is NULL");
  if (!model || !params) return fail(TBS_EINVAL, "tbs_decode_graphs: NULL model/params");
  return decode_impl(model, nullptr, graphs, params, encoder_out, lengths, B, T, out_tokens,
                     out_num_tokens, out_scores, out_status, out_arcs, trace, hip_stream,
                     "tbs_decode_graphs");
}

tbs_status tbs_decode_noalloc(const tbs_model* model, const tbs_graph* graph,
                              const tbs_beam_params* params, const float* encoder_out,
                              const int32_t* lengths, int32_t B, int32_t T, int32_t* out_tokens,
                              int32_t* out_num_tokens, double* out_scores, int32_t* out_status,
                              int32_t* out_arcs, int32_t* trace, void* hip_stream) {
  const char* who = "tbs_decode_noalloc";
  if (B < 0 || T < 0) return fail(TBS_EINVAL, "%s: B and T must be >= 0", who);
  tbs_status s = check_params(model, graph, params, who);
  if (s != TBS_OK || B == 0) return s;
  if (!lengths) return fail(TBS_EINVAL, "%s: lengths is NULL", who);
  if (T > 0 && !encoder_out) return fail(TBS_EINVAL, "%s: encoder_out is NULL", who);
  if (!out_num_tokens || !out_scores || (T > 0 && !out_tokens))
    return fail(TBS_EINVAL, "%s: NULL output pointer", who);
  const GraphDev gd = graph_dev(graph);
  const float beam = params->beam;
  const int Ns = params->max_states;
  const int Nc = params->max_contexts < Ns ? params->max_contexts : Ns;
  const int KT = (gd.trivial && Ns <= kMaxTopK) ? Ns : 0;
  tbs_model* m = const_cast<tbs_model*>(model);
  std::lock_guard<std::mutex> lk(m->mu);
  hipStream_t st = (hipStream_t)hip_stream;
  const ModelDev md = model_dev(m);
  const StreamPlan splan = plan_stream(md, Nc, KT, gd.trivial);
  bool per_stream = false;
  s = choose_schedule(m, splan, Ns, Nc, who, &per_stream);
  if (s != TBS_OK) return s;
  // the frame loop runs to T: lengths stay in device memory (no host copy)
  const int G = (per_stream && m->schedule != TBS_SCHEDULE_STREAM_SINGLE)
                    ? pick_group(m, splan, B, KT, T, gd.trivial)
                    : 1;
  const size_t xwords = G > 1 ? (size_t)B * G * 2 * group_words(Nc, KT) : 0;
  Workspace w;
  unsigned long long* xbuf = nullptr;
  const size_t need = carve_workspace(m, 0, B, T, Ns, Nc, KT, KT == 0, xwords, w, &xbuf);
  if (need > kScratchBytes)
    return fail(TBS_ECAPACITY,
                "%s: the workspace of this decode takes %zu bytes, more than the %zu-byte "
                "scratch array (use tbs_decode)",
                who, need, kScratchBytes);
  // the array's device address on this device, looked up once per device
  unsigned char* base = nullptr;
  {
    static std::mutex mu;
    static std::vector<std::pair<int, unsigned char*>> addr;
    int dev = 0;
    HIP_TRY(hipGetDevice(&dev), "hipGetDevice");
    std::lock_guard<std::mutex> al(mu);
    for (auto& a : addr)
      if (a.first == dev) base = a.second;
    if (!base) {
      void* p = nullptr;
      HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
      base = static_cast<unsigned char*>(p);
      addr.push_back({dev, base});
    }
  }
  carve_workspace(m, reinterpret_cast<uintptr_t>(base), B, T, Ns, Nc, KT, KT == 0, xwords, w,
                  &xbuf);
  HIP_TRY(model_wait(m, st), "hipStreamWaitEvent");
  HIP_TRY(launch_clamp_lengths(lengths, w.len, B, T, st), "launch(lengths)");
  const DecodeDev d = decode_dev(m, w, B, T, Ns, Nc, KT, encoder_out, w.len, nullptr, false);
  if (trace)
    HIP_TRY(launch_fill_i32(trace, (long long)(T + 1) * B * Ns * 4, -1, st), "fill(trace)");
  HIP_TRY(launch_init(md, d, gd, trace, st), "launch(init)");
  HIP_TRY(launch_fill_i32((int*)w.xerr, 1 + (long long)B + kXTickets, 0, st), "fill(exchange errors)");
  // the array keeps the last call's contents: the exchange words start at zero
  if (xbuf) HIP_TRY(launch_fill_i32((int*)xbuf, 2 * (long long)xwords, 0, st), "fill(exchange)");
  bool grouped = false;
  s = enqueue_frames(m, gd, beam, splan, per_stream, d, T, trace, w.xerr, xbuf, false, false, st,
                     &grouped);
  if (s != TBS_OK) return s;
  HIP_TRY(launch_final(gd, d, out_tokens, out_num_tokens, out_scores, out_status, out_arcs,
                       grouped ? w.xerr : nullptr, st),
          "launch(final)");
  HIP_TRY(model_mark(m, st), "hipEventRecord");
  return TBS_OK;
}

tbs_status tbs_state_create(const tbs_model* model, const tbs_graph* graph,
                            const tbs_beam_params* params, int32_t B, int32_t max_frames,
                            void* hip_stream, tbs_state** out) {
  if (!graph) {
    if (out) *out = nullptr;
    return fail(TBS_EINVAL, "tbs_state_create: graph is NULL");
  }
  return state_create_impl(model, graph, nullptr, params, B, max_frames, hip_stream, out,
                           "tbs_state_create");
}

tbs_status tbs_state_create_graphs(const tbs_model* model, const tbs_graph* const* graphs,
                                   const tbs_beam_params* params, int32_t B, int32_t max_frames,
                                   void* hip_stream, tbs_state** out) {
  if (!graphs || !model || !params) {
    if (out) *out = nullptr;
    return fail(TBS_EINVAL, "tbs_state_create_graphs: NULL model/graphs/params");
  }
  return state_create_impl(model, nullptr, graphs, params, B, max_frames, hip_stream, out,
                           "tbs_state_create_graphs");
}

tbs_status tbs_decode_chunk(tbs_state* S, const float* encoder_chunk,
                            const int32_t* chunk_lengths, int32_t Tc, int32_t* trace,
                            void* hip_stream) {
  if (!S) return fail(TBS_EINVAL, "tbs_decode_chunk: state is NULL");
  if (Tc < 0) return fail(TBS_EINVAL, "tbs_decode_chunk: Tc must be >= 0");
  if (!chunk_lengths) return fail(TBS_EINVAL, "tbs_decode_chunk: chunk_lengths is NULL");
  const int B = S->B;
  int maxlen = 0;
  for (int b = 0; b < B; ++b) {
    if (chunk_lengths[b] < 0 || chunk_lengths[b] > Tc)
      return fail(TBS_EINVAL, "tbs_decode_chunk: chunk_lengths[%d] = %d outside [0, %d]", b,
                  chunk_lengths[b], Tc);
    if ((long long)S->done[b] + chunk_lengths[b] > S->Tcap)
      return fail(TBS_ECAPACITY,
                  "tbs_decode_chunk: stream %d would reach %lld frames, beyond max_frames %d", b,
                  (long long)S->done[b] + chunk_lengths[b], S->Tcap);
    if (chunk_lengths[b] > maxlen) maxlen = chunk_lengths[b];
  }
  if (maxlen > 0 && !encoder_chunk)
    return fail(TBS_EINVAL, "tbs_decode_chunk: encoder_chunk is NULL");
  if (maxlen == 0) return TBS_OK;
  tbs_model* m = S->m;
  std::lock_guard<std::mutex> lk(m->mu);
  hipStream_t st = (hipStream_t)hip_stream;
  Workspace& w = S->w;
  HIP_TRY(model_wait(m, st), "hipStreamWaitEvent");
  if (w.pending) HIP_TRY(hipStreamWaitEvent(st, w.done, 0), "hipStreamWaitEvent");
  if (w.pending) HIP_TRY(hipEventSynchronize(w.done), "hipEventSynchronize");
  // chunk lengths and each stream's frame base, through the pinned staging buffer
  std::memcpy(w.len_host, chunk_lengths, (size_t)B * 4);
  std::memcpy(w.len_host + B, S->done.data(), (size_t)B * 4);
  HIP_TRY(hipMemcpyAsync(w.len, w.len_host, (size_t)2 * B * 4, hipMemcpyHostToDevice, st),
          "hipMemcpyAsync(lengths)");
  const DecodeDev d = decode_dev(m, w, B, Tc, S->Ns, S->Nc, S->KT, encoder_chunk, w.len,
                                 w.len + B, S->per_graph);
  HIP_TRY(launch_resume(model_dev(m), d, S->gd, trace, S->per_stream ? 0 : 1, st),
          "launch(resume)");
  bool grouped = false;
  tbs_status s = enqueue_frames(m, S->gd, S->beam, S->splan, S->per_stream, d, maxlen, trace,
                                S->w.xerr, nullptr, true, m->graphs, st, &grouped);
  if (s != TBS_OK) return s;
  HIP_TRY(hipEventRecord(w.done, st), "hipEventRecord");
  w.pending = true;
  HIP_TRY(model_mark(m, st), "hipEventRecord");
  for (int b = 0; b < B; ++b) S->done[b] += chunk_lengths[b];
  return TBS_OK;
}

tbs_status tbs_state_finish(tbs_state* S, int32_t* out_tokens, int32_t* out_num_tokens,
                            double* out_scores, int32_t* out_status, int32_t* out_arcs,
                            void* hip_stream) {
  if (!S) return fail(TBS_EINVAL, "tbs_state_finish: state is NULL");
  if (!out_tokens || !out_num_tokens || !out_scores)
    return fail(TBS_EINVAL, "tbs_state_finish: NULL output pointer");
  tbs_model* m = S->m;
  std::lock_guard<std::mutex> lk(m->mu);
  hipStream_t st = (hipStream_t)hip_stream;
  Workspace& w = S->w;
  if (w.pending) HIP_TRY(hipStreamWaitEvent(st, w.done, 0), "hipStreamWaitEvent");
  if (w.pending) HIP_TRY(hipEventSynchronize(w.done), "hipEventSynchronize");
  std::memcpy(w.len_host, S->done.data(), (size_t)S->B * 4);
  HIP_TRY(hipMemcpyAsync(w.len, w.len_host, (size_t)S->B * 4, hipMemcpyHostToDevice, st),
          "hipMemcpyAsync(lengths)");
  const DecodeDev d = decode_dev(m, w, S->B, S->Tcap, S->Ns, S->Nc, S->KT, nullptr, w.len,
                                 nullptr, S->per_graph);
  HIP_TRY(timed_launch(m, TBS_KERNEL_FINAL, st,
                       [&] {
                         return launch_final(S->gd, d, out_tokens, out_num_tokens,
                                             out_scores, out_status, out_arcs, S->w.xerr, st);
                       }),
          "launch(final)");
  HIP_TRY(hipEventRecord(w.done, st), "hipEventRecord");
  w.pending = true;
  return TBS_OK;
}

void tbs_state_destroy(tbs_state* S) {
  if (!S) return;
  {
    std::lock_guard<std::mutex> lk(S->m->mu);
    if (S->w.pending) (void)hipEventSynchronize(S->w.done);
    S->w.release();
  }
  delete S;
}

tbs_status tbs_joiner_logp(const tbs_model* model, const float* enc_rows, const int32_t* ctx,
                           int32_t R, float* out_logp, void* hip_stream) {
  if (!model) return fail(TBS_EINVAL, "tbs_joiner_logp: model is NULL");
  if (R < 0) return fail(TBS_EINVAL, "tbs_joiner_logp: R must be >= 0");
  if (R == 0) return TBS_OK;
  if (!enc_rows || !ctx || !out_logp) return fail(TBS_EINVAL, "tbs_joiner_logp: NULL pointer");
  tbs_model* m = const_cast<tbs_model*>(model);
  std::lock_guard<std::mutex> lk(m->mu);
  hipStream_t st = (hipStream_t)hip_stream;
  const int nvt = m->Vpad / kJoinerBN;
  const int Rpad = round_up(R, 64);
  if (Rpad > m->rows_cap) {
    HIP_TRY(hipStreamSynchronize(st), "hipStreamSynchronize");
    (void)hipFree(m->rows_h);
    (void)hipFree(m->rows_logits);
    (void)hipFree(m->rows_stats);
    m->rows_h = nullptr;
    m->rows_logits = nullptr;
    m->rows_stats = nullptr;
    m->rows_cap = 0;
    HIP_TRY(dalloc((char**)&m->rows_h, (size_t)Rpad * m->Kpad * (m->bf16 ? 2 : 4)),
            "hipMalloc(rows)");
    HIP_TRY(dalloc(&m->rows_logits, (size_t)Rpad * m->Vpad), "hipMalloc(rows)");
    HIP_TRY(dalloc(&m->rows_stats, (size_t)Rpad * nvt), "hipMalloc(rows)");
    m->rows_cap = Rpad;
  }
  HIP_TRY(launch_joiner_rows(model_dev(m), enc_rows, ctx, R, m->rows_h, m->rows_logits,
                             m->rows_stats, out_logp, m->ncu, st),
          "launch(joiner_rows)");
  return TBS_OK;
}

tbs_status tbs_model_set_schedule(tbs_model* model, int32_t schedule) {
  if (!model) return fail(TBS_EINVAL, "tbs_model_set_schedule: model is NULL");
  if (schedule != TBS_SCHEDULE_AUTO && schedule != TBS_SCHEDULE_FRAME &&
      schedule != TBS_SCHEDULE_STREAM && schedule != TBS_SCHEDULE_STREAM_SINGLE)
    return fail(TBS_EINVAL, "tbs_model_set_schedule: unknown schedule %d", schedule);
  std::lock_guard<std::mutex> lk(model->mu);
  model->schedule = schedule;
  return TBS_OK;
}

tbs_status tbs_model_set_graph_capture(tbs_model* model, int32_t enable) {
  if (!model) return fail(TBS_EINVAL, "tbs_model_set_graph_capture: model is NULL");
  std::lock_guard<std::mutex> lk(model->mu);
  model->graphs = enable != 0;
  return TBS_OK;
}

tbs_status tbs_model_graph_stats(const tbs_model* model, int32_t* captures, int32_t* replays) {
  if (!model || !captures || !replays)
    return fail(TBS_EINVAL, "tbs_model_graph_stats: NULL argument");
  tbs_model* m = const_cast<tbs_model*>(model);
  std::lock_guard<std::mutex> lk(m->mu);
  *captures = m->fg_captures;
  *replays = m->fg_replays;
  return TBS_OK;
}

tbs_status tbs_model_set_exchange_spin_limit(tbs_model* model, int32_t polls) {
  if (!model) return fail(TBS_EINVAL, "tbs_model_set_exchange_spin_limit: model is NULL");
  if (polls < 0) return fail(TBS_EINVAL, "tbs_model_set_exchange_spin_limit: polls %d < 0", polls);
  std::lock_guard<std::mutex> lk(model->mu);
  model->spin_limit = polls == 0 ? kDefaultSpinLimit : (unsigned)polls;
  return TBS_OK;
}

tbs_status tbs_model_set_profiling(tbs_model* model, int32_t enable) {
  if (!model) return fail(TBS_EINVAL, "tbs_model_set_profiling: model is NULL");
  std::lock_guard<std::mutex> lk(model->mu);
  prof_drop(model);
  for (auto& x : model->prof_acc) x = tbs_kernel_time{0, 0.0};
  model->prof = enable != 0;
  return TBS_OK;
}

tbs_status tbs_model_read_profile(tbs_model* model, tbs_kernel_time* out) {
  if (!model || !out) return fail(TBS_EINVAL, "tbs_model_read_profile: NULL argument");
  std::lock_guard<std::mutex> lk(model->mu);
  for (auto& x : model->prof_pending) {
    HIP_TRY(hipEventSynchronize(x.stop), "hipEventSynchronize");
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, x.start, x.stop), "hipEventElapsedTime");
    model->prof_acc[x.kernel].launches += 1;
    model->prof_acc[x.kernel].total_ms += ms;
  }
  prof_drop(model);
  for (int k = 0; k < TBS_KERNEL_COUNT; ++k) out[k] = model->prof_acc[k];
  return TBS_OK;
}


tbs_status tbs_lattice_create(const tbs_model* model, const tbs_graph* graph,
                              const tbs_beam_params* params, const float* encoder_out,
                              const int32_t* lengths, int32_t B, int32_t T, void* hip_stream,
                              tbs_lattice** out) {
  if (!graph) {
    if (out) *out = nullptr;
    return fail(TBS_EINVAL, "tbs_lattice_create: graph is NULL");
  }
  return lattice_create_impl(model, graph, nullptr, params, encoder_out, lengths, B, T,
                             hip_stream, out, "tbs_lattice_create");
}

tbs_status tbs_lattice_create_graphs(const tbs_model* model, const tbs_graph* const* graphs,
                                     const tbs_beam_params* params, const float* encoder_out,
                                     const int32_t* lengths, int32_t B, int32_t T,
                                     void* hip_stream, tbs_lattice** out) {
  if (!graphs || !model || !params) {
    if (out) *out = nullptr;
    return fail(TBS_EINVAL, "tbs_lattice_create_graphs: NULL model/graphs/params");
  }
  return lattice_create_impl(model, nullptr, graphs, params, encoder_out, lengths, B, T,
                             hip_stream, out, "tbs_lattice_create_graphs");
}

tbs_status tbs_lattice_num_arcs(const tbs_lattice* lat, int64_t* out) {
  if (!lat || !out) return fail(TBS_EINVAL, "tbs_lattice_num_arcs: NULL argument");
  *out = lat->A;
  return TBS_OK;
}

tbs_status tbs_lattice_export(const tbs_lattice* lat, int64_t* frame_off, int32_t* arcs,
                              float* weights, int32_t* nodes, double* alpha, double* final_w,
                              double* total, int32_t* status, void* hip_stream) {
  if (!lat) return fail(TBS_EINVAL, "tbs_lattice_export: lattice is NULL");
  tbs_lattice* L = const_cast<tbs_lattice*>(lat);
  std::lock_guard<std::mutex> lk(L->m->mu);
  hipStream_t st = (hipStream_t)hip_stream;
  if (L->pending) HIP_TRY(hipStreamWaitEvent(st, L->done, 0), "hipStreamWaitEvent");
  const size_t BT = (size_t)L->B * L->T, BN = (size_t)L->B * L->Ns;
  auto cp = [&](void* dst, const void* src, size_t bytes) {
    return dst && bytes ? hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, st)
                        : hipSuccess;
  };
  HIP_TRY(cp(frame_off, L->off, (BT + 1) * 8), "tbs_lattice_export");
  HIP_TRY(cp(arcs, L->arcs, (size_t)L->A * 16), "tbs_lattice_export");
  HIP_TRY(cp(weights, L->w, (size_t)L->A * 4), "tbs_lattice_export");
  HIP_TRY(cp(nodes, L->trace, (size_t)(L->T + 1) * BN * 16), "tbs_lattice_export");
  HIP_TRY(cp(alpha, L->alpha, (size_t)(L->T + 1) * BN * 8), "tbs_lattice_export");
  HIP_TRY(cp(final_w, L->fw, BN * 8), "tbs_lattice_export");
  HIP_TRY(cp(total, L->total, (size_t)L->B * 8), "tbs_lattice_export");
  HIP_TRY(cp(status, L->status, (size_t)L->B * 4), "tbs_lattice_export");
  HIP_TRY(hipEventRecord(L->done, st), "hipEventRecord");
  L->pending = true;
  return TBS_OK;
}

tbs_status tbs_lattice_nbest(tbs_lattice* lat, int32_t num_paths, const double* uniforms,
                             int32_t* out_tokens, int32_t* out_num_tokens, double* out_scores,
                             int32_t* out_num_unique, double* out_unique_scores,
                             int32_t* out_unique_first, int32_t* out_paths, void* hip_stream) {
  if (!lat) return fail(TBS_EINVAL, "tbs_lattice_nbest: lattice is NULL");
  if (num_paths < 1) return fail(TBS_EINVAL, "tbs_lattice_nbest: num_paths must be >= 1");
  if (!uniforms || !out_num_tokens || !out_scores || (lat->T > 0 && !out_tokens))
    return fail(TBS_EINVAL, "tbs_lattice_nbest: NULL uniforms or output pointer");
  tbs_lattice* L = lat;
  std::lock_guard<std::mutex> lk(L->m->mu);
  hipStream_t st = (hipStream_t)hip_stream;
  const int B = L->B, T = L->T, Ns = L->Ns;
  const size_t Bn = (size_t)B * num_paths;
  const int W = T / 2 + 1;  // widest band of the sequence DP
  if (num_paths > L->ncap) {
    if (L->pending) HIP_TRY(hipEventSynchronize(L->done), "hipEventSynchronize");
    L->free_nbest();
    hipError_t e = dalloc(&L->seq, Bn * (T > 0 ? T : 1));
    if (e == hipSuccess) e = dalloc(&L->pntok, Bn);
    if (e == hipSuccess) e = dalloc(&L->hash, Bn);
    if (e == hipSuccess) e = dalloc(&L->first, Bn);
    if (e == hipSuccess) e = dalloc(&L->nuniq, (size_t)B);
    if (e == hipSuccess) e = dalloc(&L->uscore, Bn);
    // the DP's two band buffers per sequence (four sequences per workgroup) live in LDS
    // (768 doubles per sequence) when the band fits; for shapes where a band may not
    // fit, a global scratch slice per sequence slot is allotted and the workgroups per
    // stream are capped at 1024 in all (grid-strided)
    const bool may_spill = 2 * (size_t)Ns * W > 768;
    L->dp_lds = may_spill ? 0 : 1;
    const int groups = (num_paths + 3) / 4;
    L->dp_grid = may_spill ? std::max(1, std::min(groups, 1024 / B)) : groups;
    if (e == hipSuccess && may_spill)
      e = dalloc(&L->dp, (size_t)L->dp_grid * B * 4 * 2 * Ns * W);
    if (e != hipSuccess) {
      L->free_nbest();
      return hip_fail(e, "tbs_lattice_nbest");
    }
    L->ncap = num_paths;
  }
  NBestDev N;
  N.n = num_paths;
  N.u = uniforms;
  N.paths = out_paths;
  N.seq = L->seq;
  N.ntok = L->pntok;
  N.hash = L->hash;
  N.first = L->first;
  N.nuniq = L->nuniq;
  N.score = L->uscore;
  N.dp = L->dp;
  N.dp_stride = W;
  if (L->pending) HIP_TRY(hipStreamWaitEvent(st, L->done, 0), "hipStreamWaitEvent");
  const int grid = std::min((num_paths + 3) / 4, L->dp_grid);
  HIP_TRY(launch_nbest(L->dev(), N, out_tokens, out_num_tokens, out_scores, out_num_unique,
                       out_unique_scores, out_unique_first, grid, L->dp_lds, st),
          "launch(nbest)");
  HIP_TRY(hipEventRecord(L->done, st), "hipEventRecord");
  L->pending = true;
  return TBS_OK;
}

void tbs_lattice_destroy(tbs_lattice* lat) {
  if (!lat) return;
  tbs_model* m = lat->m;
  std::lock_guard<std::mutex> lk(m->mu);
  if (lat->done && lat->pending) (void)hipEventSynchronize(lat->done);
  lat->pending = false;
  if (!m->lat_cache) {
    m->lat_cache = lat;  // its buffers serve the model's next lattice
    return;
  }
  lat->release();
  delete lat;
}


tbs_status tbs_hyp_search(const tbs_model* model, const tbs_hyp_params* params,
                          const float* encoder_out, const int32_t* lengths, int32_t B, int32_t T,
                          int32_t* out_tokens, int32_t* out_num_tokens, double* out_scores,
                          int32_t* trace, void* hip_stream) {
  if (!model || !params) return fail(TBS_EINVAL, "tbs_hyp_search: NULL model/params");
  const int N = params->beam_size;
  if (N < 1 || N > kMaxHyps)
    return fail(N < 1 ? TBS_EINVAL : TBS_ECAPACITY,
                "tbs_hyp_search: beam_size %d outside [1, %d]", N, kMaxHyps);
  if (params->merge != TBS_MERGE_MAX && params->merge != TBS_MERGE_LOGADD)
    return fail(TBS_EINVAL, "tbs_hyp_search: unknown merge %d", (int)params->merge);
  if (B < 0 || T < 0) return fail(TBS_EINVAL, "tbs_hyp_search: B and T must be >= 0");
  if (B == 0) return TBS_OK;
  if (!lengths) return fail(TBS_EINVAL, "tbs_hyp_search: lengths is NULL");
  int maxlen = 0;
  for (int b = 0; b < B; ++b) {
    if (lengths[b] < 0 || lengths[b] > T)
      return fail(TBS_EINVAL, "tbs_hyp_search: lengths[%d] = %d outside [0, %d]", b, lengths[b],
                  T);
    if (lengths[b] > maxlen) maxlen = lengths[b];
  }
  if (maxlen > 0 && !encoder_out) return fail(TBS_EINVAL, "tbs_hyp_search: encoder_out is NULL");
  if (!out_num_tokens || !out_scores || (T > 0 && !out_tokens))
    return fail(TBS_EINVAL, "tbs_hyp_search: NULL output pointer");
  tbs_model* m = const_cast<tbs_model*>(model);
  std::lock_guard<std::mutex> lk(m->mu);
  hipStream_t st = (hipStream_t)hip_stream;
  HypWork& w = m->hw;
  if (!(w.done && w.B >= B && w.T >= T && w.N == N)) {
    w.release();
    const size_t BN = (size_t)B * N;
    const int nvt = m->Vpad / kJoinerBN;
    hipError_t e = hipSuccess;
    for (int i = 0; i < 2 && e == hipSuccess; ++i) {
      e = dalloc(&w.hash[i], BN);
      if (e == hipSuccess) e = dalloc(&w.phash[i], BN);
      if (e == hipSuccess) e = dalloc(&w.n[i], BN);
      if (e == hipSuccess) e = dalloc(&w.ctx[i], BN);
      if (e == hipSuccess) e = dalloc(&w.score[i], BN);
      if (e == hipSuccess) e = dalloc(&w.nh[i], (size_t)B);
    }
    if (e == hipSuccess) e = dalloc(&w.len, (size_t)B);
    if (e == hipSuccess) e = dalloc(&w.rowctx, BN);
    if (e == hipSuccess) e = dalloc(&w.hrow, BN);
    if (e == hipSuccess) e = dalloc(&w.hist, (size_t)T * BN);
    if (e == hipSuccess) e = dalloc((char**)&w.h, BN * m->Kpad * (m->bf16 ? 2 : 4));
    if (e == hipSuccess) e = dalloc(&w.logits, BN * m->Vpad);
    if (e == hipSuccess) e = dalloc(&w.stats, BN * nvt);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&w.done, hipEventDisableTiming);
    if (e != hipSuccess) {
      w.release();
      return hip_fail(e, "tbs_hyp_search");
    }
    w.B = B;
    w.T = T;
    w.N = N;
  }
  HIP_TRY(model_wait(m, st), "hipStreamWaitEvent");
  if (w.pending) HIP_TRY(hipStreamWaitEvent(st, w.done, 0), "hipStreamWaitEvent");
  HIP_TRY(hipMemcpyAsync(w.len, lengths, (size_t)B * 4, hipMemcpyHostToDevice, st),
          "hipMemcpyAsync(lengths)");
  HypDev d;
  d.B = B;
  d.T = T;
  d.N = N;
  d.merge_logadd = params->merge == TBS_MERGE_LOGADD;
  d.len = w.len;
  for (int i = 0; i < 2; ++i) {
    d.hash[i] = w.hash[i];
    d.phash[i] = w.phash[i];
    d.n[i] = w.n[i];
    d.ctx[i] = w.ctx[i];
    d.score[i] = w.score[i];
    d.nh[i] = w.nh[i];
  }
  d.rowctx = w.rowctx;
  d.hrow = w.hrow;
  d.hist = w.hist;
  d.enc = encoder_out;
  d.h = w.h;
  const ModelDev md = model_dev(m);
  if (trace)
    HIP_TRY(launch_fill_i32(trace, (long long)(T + 1) * B * N * 2, -1, st), "fill(trace)");
  HIP_TRY(launch_hyp_init(md, d, st), "launch(hyp init)");
  for (int t = 0; t < maxlen; ++t) {
    HIP_TRY(timed_launch(m, TBS_KERNEL_JOINER, st,
                         [&] {
                           return launch_joiner_gemm(md, w.h, B * N, w.logits, w.stats, m->ncu,
                                                     st);
                         }),
            "launch(joiner)");
    HIP_TRY(timed_launch(m, TBS_KERNEL_HYP_STEP, st,
                         [&] { return launch_hyp_step(md, d, t, w.logits, w.stats, trace, st); }),
            "launch(hyp step)");
  }
  HIP_TRY(launch_hyp_final(d, out_tokens, out_num_tokens, out_scores, st), "launch(hyp final)");
  HIP_TRY(hipEventRecord(w.done, st), "hipEventRecord");
  w.pending = true;
  HIP_TRY(model_mark(m, st), "hipEventRecord");
  return TBS_OK;
}


tbs_status tbs_transducer_forward(int32_t kind, const float* blank, const float* label,
                                  const int32_t* lengths, int32_t B, int32_t T, int32_t U,
                                  double* out_total, float* out_alpha, int32_t* out_status,
                                  void* hip_stream) {
  if (kind != TBS_TRANSDUCER_STANDARD && kind != TBS_TRANSDUCER_MODIFIED &&
      kind != TBS_TRANSDUCER_CONSTRAINED)
    return fail(TBS_EINVAL, "tbs_transducer_forward: unknown kind %d", (int)kind);
  if (B < 0 || T < 1 || U < 0)
    return fail(TBS_EINVAL, "tbs_transducer_forward: need B >= 0, T >= 1, U >= 0");
  if (U + 1 > 64 * kTransducerMaxK)
    return fail(TBS_ECAPACITY, "tbs_transducer_forward: U = %d exceeds the limit %d", (int)U,
                64 * kTransducerMaxK - 1);
  if (B == 0) return TBS_OK;
  if (!blank || (U > 0 && !label) || !lengths || !out_total)
    return fail(TBS_EINVAL, "tbs_transducer_forward: NULL pointer");
  HIP_TRY(launch_transducer_forward(kind, blank, label, lengths, B, T, U, out_total, out_alpha,
                                    out_status, (hipStream_t)hip_stream),
          "launch(transducer)");
  return TBS_OK;
}

}  // extern "C"
