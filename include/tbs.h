/*
 * tbs.h -- C ABI of the MI355X (gfx950) library for batched FSA-based
 * one-symbol-per-frame transducer beam search.
 *
 * The method is the "FSA-based parallel beam search" of Kang et al., "Fast and
 * parallel decoding for transducer" (arXiv 2211.00484): Sec. 2.2 (stateless
 * transducer, two-label context), Sec. 2.3 (max-symbols decoding with S = 1),
 * Sec. 2.4 (on-the-fly composition with an epsilon-free decoding graph),
 * Sec. 2.5 (beam, max-states and max-contexts pruning) and Algorithm 1.
 *
 * Conventions shared by every entry point:
 *  - Every function returns a tbs_status; 0 is success, negative values are
 *    errors.  tbs_last_error() returns a message describing the last error of
 *    the calling thread.
 *  - All arguments are validated on the host before any device work is
 *    enqueued; a call that returns an error has written nothing.
 *  - Device pointers are plain HIP device addresses on the current device.
 *    Host pointers are ordinary CPU memory.  Each argument states which.
 *  - hip_stream is a hipStream_t (NULL = the null stream).  Device work is
 *    enqueued on it; calls return after enqueueing (stream-ordered), except
 *    where stated.
 *  - Graph and model handles are immutable after creation and may be shared
 *    between threads.  The decode workspace is cached in the model handle;
 *    decodes that share a model are serialised on it (host side by a mutex,
 *    device side by an event the next decode's stream waits on).
 *  - Blank is label 0.  Contexts are packed as ctx = a * V + b, where b is the
 *    most recent label (Sec. 2.4 footnote: the history fits one integer).
 */
#ifndef TBS_H
#define TBS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TBS_OK = 0,
  TBS_EINVAL = -1,        /* an argument is invalid; nothing was done            */
  TBS_ENOMEM = -2,        /* device or pinned-host allocation failed             */
  TBS_EDEVICE = -3,       /* a HIP call failed                                   */
  TBS_ECAPACITY = -4,     /* a size exceeds a documented library limit           */
  TBS_EUNSUPPORTED = -5   /* a valid but unsupported configuration               */
} tbs_status;

typedef struct tbs_graph tbs_graph;
typedef struct tbs_model tbs_model;

/*
 * Decoding graph: an epsilon-free FSA (Sec. 2.4) given as CSR arcs sorted by
 * source state.  All inputs are HOST arrays; the library copies them to the
 * device and the caller may free them when the call returns.
 *   num_states   S >= 1
 *   start_state  in [0, S)
 *   vocab_size   V in [2, 46340] (blank = 0 included; a context (a, b) is the
 *                int32 a * V + b, so V * V must stay below 2^31)
 *   row_ptr      host int32 [S+1]: row_ptr[0] = 0, non-decreasing; A = row_ptr[S]
 *   dest         host int32 [A]: destination state of each arc, in [0, S)
 *   label        host int32 [A]: label of each arc, in [1, V-1] (label 0 is
 *                rejected: the graph must be epsilon-free)
 *   score        host float [A]: finite log-domain arc weight (q in Sec. 2.4)
 *   final_score  host float [S] or NULL.  NULL: every state is final with
 *                weight 0.  Otherwise a finite value is the state's final
 *                weight and -INFINITY marks a non-final state.
 * Duplicate arcs are allowed; they merge by max during the search.
 * Errors: TBS_EINVAL on any violation above (with the offending index in the
 * message), TBS_ENOMEM / TBS_EDEVICE on allocation or copy failure.
 */
tbs_status tbs_graph_create(int32_t num_states, int32_t start_state, int32_t vocab_size,
                            const int32_t *row_ptr, const int32_t *dest,
                            const int32_t *label, const float *score,
                            const float *final_score, tbs_graph **out);

/*
 * The "trivial graph" of Table 6: one state (start and final, weight 0) with a
 * 0-weight self-loop for every non-blank label 1..V-1, in label order (so arc
 * id = label - 1).  The search over it is plain one-symbol-per-frame beam
 * search with (context) hypotheses.
 */
tbs_status tbs_graph_create_trivial(int32_t vocab_size, tbs_graph **out);
void tbs_graph_destroy(tbs_graph *graph);

typedef enum { TBS_JOINER_FP32 = 0, TBS_JOINER_BF16 = 1 } tbs_joiner_dtype;

/*
 * Transducer model pieces used by the search (Sec. 5.1 model; Algorithm 1
 * decoder and joiner):
 *   stateless decoder  dec(a, b) = ReLU(conv[:,0] * embed[a] + conv[:,1] * embed[b])
 *                      (embedding followed by a depthwise kernel-2 convolution
 *                      over the two most recent labels; tap 0 weights the older
 *                      label a; no bias);
 *   joiner             logits = w_out . tanh(enc + dec) + b_out, then log-softmax
 *                      over all V outputs, blank included.
 *   vocab_size V in [2, 46340] (contexts a * V + b are int32); dim C in [1, 2048];
 *   context_size must be 2
 *   (TBS_EUNSUPPORTED otherwise).
 *   embed  DEVICE float [V][C];  conv DEVICE float [C][2];
 *   w_out  DEVICE float [V][C] (torch Linear layout);  b_out DEVICE float [V] or NULL (= 0).
 *   dtype  TBS_JOINER_FP32: fp32 operands; TBS_JOINER_BF16: tanh output and
 *          w_out rounded to bfloat16 (nearest, ties to even), fp32 accumulation.
 * The library copies what it needs (and precomputes conv-tap-scaled embedding
 * tables) on hip_stream and synchronises that stream before returning, so the
 * caller may free the inputs afterwards.
 */
tbs_status tbs_model_create(int32_t vocab_size, int32_t dim, int32_t context_size,
                            const float *embed, const float *conv, const float *w_out,
                            const float *b_out, tbs_joiner_dtype dtype, void *hip_stream,
                            tbs_model **out);
void tbs_model_destroy(tbs_model *model);

/*
 * Pruning constraints of Sec. 2.5, applied per stream on every frame after
 * unpruned expansion and max-merge of equal (graph state, context) tuples:
 *   beam          log-domain beam >= 0 (INFINITY = off): keep tuples whose score
 *                 is >= best - beam (inclusive);
 *   max_states    in [1, 256]: together with the beam, keep at most this many
 *                 tuples, ranked by score descending, then (state, context)
 *                 ascending;
 *   max_contexts  >= 1: then keep the tuples of the max_contexts best contexts,
 *                 a context scoring the max over its tuples, ties by context
 *                 id ascending.
 */
typedef struct {
  float beam;
  int32_t max_states;
  int32_t max_contexts;
} tbs_beam_params;

/*
 * Batched decode (Algorithm 1 with the best path through the lattice, Sec. 2.5).
 *   encoder_out    DEVICE float [B][T][C], contiguous; frames t >= lengths[b] are ignored.
 *   lengths        HOST int32 [B], each in [0, T].
 *   B >= 0 (B = 0 is a no-op), T >= 0.
 *   out_tokens     DEVICE int32 [B][T]: the best path's non-blank labels, -1 padded
 *                  (one symbol per frame at most, so T slots suffice).
 *   out_num_tokens DEVICE int32 [B].
 *   out_scores     DEVICE double [B]: log-domain score of the best path, final
 *                  weight included.
 *   out_status     DEVICE int32 [B] or NULL: 0 = the path ends in a final state;
 *                  1 = no surviving tuple was final and the best non-final one
 *                  was used (its score then has no final weight); 2 = see
 *                  TBS_SCHEDULE_STREAM (device exchange timed out).
 *   out_arcs       DEVICE int32 [B][T] or NULL: per frame, the graph arc id taken
 *                  by the best path, -1 for blank, -2 for frames >= lengths[b].
 *   trace          DEVICE int32 [T+1][B][max_states][4] or NULL: for frame index
 *                  f, the surviving tuples of each stream as (ctx, state, parent,
 *                  label), in (ctx, state) ascending order, -1 padded; f = 0 is
 *                  the initial tuple (0, start, -1, -1).  Parents index the
 *                  previous frame's list.  For parity testing.
 * Scores are kept per stream in fp32 relative to the stream's best, plus an
 * fp64 per-stream offset, so long streams keep fp32 resolution.
 * All output buffers are caller-owned and fully written (including padding).
 * The workspace (sized by B, T, max_states, max_contexts and the vocabulary)
 * is allocated on first use and cached in the model.
 * Errors: TBS_EINVAL for NULL handles/pointers, a model/graph vocabulary
 * mismatch, a length outside [0, T], a NaN or negative beam or max_states /
 * max_contexts < 1; TBS_ECAPACITY if max_states > 256 or
 * max_states * (graph max out-degree + 1) >= 2^31; TBS_ENOMEM / TBS_EDEVICE.
 */
tbs_status tbs_decode(const tbs_model *model, const tbs_graph *graph,
                      const tbs_beam_params *params, const float *encoder_out,
                      const int32_t *lengths, int32_t B, int32_t T, int32_t *out_tokens,
                      int32_t *out_num_tokens, double *out_scores, int32_t *out_status,
                      int32_t *out_arcs, int32_t *trace, void *hip_stream);

/*
 * tbs_decode with one decoding graph per stream (Algorithm 1 takes the graph of
 * stream i from a vector of graphs): graphs is a HOST array of B graph handles
 * (entries may repeat); stream b searches graphs[b], and every output of stream b
 * is what tbs_decode gives for that stream alone with graph graphs[b].  Other
 * arguments, outputs and errors as for tbs_decode, with every graph checked
 * against the model and params (B >= 1 needs graphs != NULL).  The graphs must
 * stay alive until the decode has completed on hip_stream.  Every stream takes the
 * general search path (no trivial-graph fast path), so a batch of trivial graphs
 * decodes more slowly here than through tbs_decode.
 */
tbs_status tbs_decode_graphs(const tbs_model *model, const tbs_graph *const *graphs,
                             const tbs_beam_params *params, const float *encoder_out,
                             const int32_t *lengths, int32_t B, int32_t T, int32_t *out_tokens,
                             int32_t *out_num_tokens, double *out_scores, int32_t *out_status,
                             int32_t *out_arcs, int32_t *trace, void *hip_stream);

/*
 * tbs_decode without any allocation, for callers that cannot allocate: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  The decode workspace (survivors, history, joiner rows, softmax
 * partials, the grouped kernel's exchange words) is carved from a file-scope
 * device array of 64 MiB that each GPU the library runs on holds until the
 * process ends; the call makes no hipMalloc, hipFree, host allocation or
 * event creation, and ignores per-kernel profiling.
 * Differences from tbs_decode:
 *   lengths  DEVICE int32 [B] (not host), read on the device and clamped to
 *            [0, T]; the frame loop runs to T (frames past a stream's length
 *            do nothing for it).
 *   one shared graph (no per-stream graphs).
 * Every call on a GPU shares that GPU's array and leaves its contents behind
 * (each call clears what must start at zero).  Calls on the same model are
 * serialised like tbs_decode; calls on different models or threads that
 * overlap on one GPU race on the array and must be ordered by the caller.
 * Other arguments, outputs and errors as for tbs_decode; TBS_ECAPACITY when
 * the workspace of (B, T, max_states, max_contexts, vocabulary) exceeds the
 * array (nothing is enqueued then).
 */
tbs_status tbs_decode_noalloc(const tbs_model *model, const tbs_graph *graph,
                              const tbs_beam_params *params, const float *encoder_out,
                              const int32_t *lengths, int32_t B, int32_t T, int32_t *out_tokens,
                              int32_t *out_num_tokens, double *out_scores, int32_t *out_status,
                              int32_t *out_arcs, int32_t *trace, void *hip_stream);

/*
 * Streaming decode: tbs_decode split into chunks of frames (the decoding state of
 * Algorithm 1 carried across calls).  A decode state holds, for each of B streams,
 * the surviving tuples, the fp64 score offset and the back-pointers of every frame
 * decoded so far.  tbs_decode_chunk continues each stream from where it stopped;
 * tbs_state_finish traces the best paths back over all decoded frames.  Splitting
 * a stream's frames into chunks in any way gives the same outputs as tbs_decode
 * over all of them on the same schedule, bit for bit.
 *
 * tbs_state_create
 *   model, graph, params as for tbs_decode; the state keeps references to the
 *   model and graph, which must outlive it.  The model's schedule at this call
 *   applies to every chunk.  B >= 1 streams; max_frames >= 1 frames per stream
 *   at most (history capacity).  Initialisation is enqueued on hip_stream.
 *   Errors as for tbs_decode, TBS_EINVAL for B or max_frames < 1.
 * tbs_decode_chunk
 *   encoder_chunk  DEVICE float [B][Tc][C]: the next frames of every stream
 *                  (row t of stream b is its frame done_b + t);
 *   chunk_lengths  HOST int32 [B], each in [0, Tc]: frames of this chunk per
 *                  stream (0 = the stream does not advance);
 *   trace          DEVICE int32 [max_frames+1][B][max_states][4] or NULL: the
 *                  survivor trace of tbs_decode at absolute frame indices; only
 *                  kept tuples are written (fill the buffer with -1 first), and
 *                  frame 0 (the initial tuple) when a stream's first chunk runs.
 *   Errors: TBS_EINVAL for bad lengths or a NULL chunk, TBS_ECAPACITY when a
 *   stream would exceed max_frames (nothing is enqueued then).
 * tbs_state_finish
 *   outputs as for tbs_decode with T = max_frames.  The state stays valid: more
 *   chunks may follow, and finish may be called again.
 * Calls on one state are stream-ordered on the hip_stream of each call and
 * serialised with every other decode on the same model; a state must not be used
 * from two threads at once.
 */
typedef struct tbs_state tbs_state;

tbs_status tbs_state_create(const tbs_model *model, const tbs_graph *graph,
                            const tbs_beam_params *params, int32_t B, int32_t max_frames,
                            void *hip_stream, tbs_state **out);
/* tbs_state_create with one graph per stream (HOST array graphs[B], as for
 * tbs_decode_graphs); the state keeps references to the graphs. */
tbs_status tbs_state_create_graphs(const tbs_model *model, const tbs_graph *const *graphs,
                                   const tbs_beam_params *params, int32_t B, int32_t max_frames,
                                   void *hip_stream, tbs_state **out);
tbs_status tbs_decode_chunk(tbs_state *state, const float *encoder_chunk,
                            const int32_t *chunk_lengths, int32_t Tc, int32_t *trace,
                            void *hip_stream);
tbs_status tbs_state_finish(tbs_state *state, int32_t *out_tokens, int32_t *out_num_tokens,
                            double *out_scores, int32_t *out_status, int32_t *out_arcs,
                            void *hip_stream);
void tbs_state_destroy(tbs_state *state);

/*
 * Lattice output and label-sequence search (Sec. 2.5: the search's output is a lattice,
 * an FSA, from which the label sequence with the highest total probability is found by
 * sampling n paths, removing blanks, keeping the distinct sequences and scoring each by
 * composing it with the lattice -- the "LogAdd" rows of Tables 3 and 6).
 *
 * tbs_lattice_create
 *   Runs the search of tbs_decode (same arguments, schedule and kernels; B >= 1), then
 *   builds on the device, per stream, the lattice:
 *     nodes  the survivors of each frame f = 0..len_b (the survivor trace of tbs_decode);
 *     arcs   for each frame f < len_b, every expansion of a frame-f survivor -- blank, or
 *            a graph arc -- whose (state, context) survived frame f+1, whatever candidate
 *            won the max-merge; weight q + log P(label | context, f) (blank: log P(blank))
 *            in fp32, from the joiner and log-softmax recomputed for the survivors'
 *            contexts; ordered by (destination, source, arc position), blank first;
 *     final  per last-frame node the graph's final weight, or 0 for all of them if none
 *            is final (then status = 1, as out_status of tbs_decode).
 *   Forward scores and totals are computed in fp64.  Synchronises hip_stream once (the
 *   arc count sizes the arc arrays); the rest is enqueued.  The lattice keeps its own
 *   copies of everything it needs (the model and graphs must outlive it).  Errors as for
 *   tbs_decode; TBS_EINVAL for B < 1.
 * tbs_lattice_create_graphs: the same with one graph per stream (as tbs_decode_graphs).
 * tbs_lattice_num_arcs: total arcs A over all streams (host).
 * tbs_lattice_export: device copies (each pointer may be NULL):
 *   frame_off  int64 [B*T+1]: the arcs of frame f of stream b are
 *              [frame_off[b*T+f], frame_off[b*T+f+1]) (empty for f >= len_b);
 *   arcs       int32 [A][4]: (source node index within frame f, destination node index
 *              within frame f+1, label (0 = blank), graph arc id or -1);
 *   weights    float [A];
 *   nodes      int32 [T+1][B][max_states][4], the trace layout of tbs_decode;
 *   alpha      double [B][T+1][max_states]: log of the summed weight of the paths from
 *              the initial node to each node (-inf for empty slots and frames > len_b);
 *   final_w    double [B][max_states]; total double [B]: log of the summed weight of all
 *              complete paths, final weights included; status int32 [B].
 * tbs_lattice_nbest
 *   num_paths >= 1 paths per stream are sampled from the lattice's path distribution
 *   (probability proportional to exp(path weight + final weight)) by inversion, going
 *   backwards: uniforms (DEVICE double [B][num_paths][T+1], each in [0, 1)) entry len_b
 *   picks the final node, entry f < len_b the arc into the path's node of frame f+1;
 *   among K items of log weight v_k, the pick is the first k whose running sum of
 *   exp(v - max v) exceeds u times the full sum.  The blank-free label sequences of the
 *   paths, without repeats, in order of first occurrence, are each scored by the log of
 *   their total probability in the lattice (all paths with that label sequence, final
 *   weights included); the best (the first on ties) is returned:
 *   out_tokens int32 [B][T] (-1 padded), out_num_tokens [B], out_scores double [B];
 *   optional: out_num_unique int32 [B], out_unique_scores double [B][num_paths] and
 *   out_unique_first int32 [B][num_paths] (the sampled path that first gave each
 *   sequence; -inf / -1 padded), out_paths int32 [B][num_paths][T+1] (per path: the
 *   arc taken on frame f as an index within frame f's arcs, the final node at len_b,
 *   -1 after).  Scratch for num_paths is kept in the lattice.  Calls on one lattice are
 *   stream-ordered across streams.
 * tbs_lattice_destroy waits for the lattice's device work; its buffers then serve the
 *   model's next tbs_lattice_create when they are large enough (no allocation), and are
 *   freed with the model or when a larger lattice needs new ones.
 */
typedef struct tbs_lattice tbs_lattice;

tbs_status tbs_lattice_create(const tbs_model *model, const tbs_graph *graph,
                              const tbs_beam_params *params, const float *encoder_out,
                              const int32_t *lengths, int32_t B, int32_t T, void *hip_stream,
                              tbs_lattice **out);
tbs_status tbs_lattice_create_graphs(const tbs_model *model, const tbs_graph *const *graphs,
                                     const tbs_beam_params *params, const float *encoder_out,
                                     const int32_t *lengths, int32_t B, int32_t T,
                                     void *hip_stream, tbs_lattice **out);
tbs_status tbs_lattice_num_arcs(const tbs_lattice *lattice, int64_t *out);
tbs_status tbs_lattice_export(const tbs_lattice *lattice, int64_t *frame_off, int32_t *arcs,
                              float *weights, int32_t *nodes, double *alpha, double *final_w,
                              double *total, int32_t *status, void *hip_stream);
tbs_status tbs_lattice_nbest(tbs_lattice *lattice, int32_t num_paths, const double *uniforms,
                             int32_t *out_tokens, int32_t *out_num_tokens, double *out_scores,
                             int32_t *out_num_unique, double *out_unique_scores,
                             int32_t *out_unique_first, int32_t *out_paths, void *hip_stream);
void tbs_lattice_destroy(tbs_lattice *lattice);

/*
 * Full-sequence beam search with max-symbols 1: the comparison search of Table 5
 * ("beam search"), whose hypotheses are whole label sequences (footnote to Sec. 2.2)
 * instead of (context, graph state) tuples; no decoding graph.  On each frame every
 * hypothesis y expands to blank (y kept) and to every label c (y + c), weighted by
 * log P(label | last two labels of y, frame) with no blank factor; equal sequences
 * merge by max or by log-add (Table 3); the beam_size best by (score desc, first
 * candidate index asc) are kept, where candidate (i, c) of the i-th hypothesis has
 * index i * vocab_size + c (blank c = 0).  The result is the best hypothesis after
 * each stream's last frame.
 *   beam_size  in [1, 16] (TBS_ECAPACITY above); merge TBS_MERGE_MAX or TBS_MERGE_LOGADD.
 *   encoder_out, lengths, B, T, out_tokens, out_num_tokens, out_scores as tbs_decode
 *   (out_scores: the hypothesis score, fp64).
 *   trace  DEVICE int32 [T+1][B][beam_size][2] or NULL: per frame f >= 1 the kept
 *          hypotheses' (rank of the parent on frame f-1, label; 0 = blank), -1 padded.
 * Sequences are identified by 64-bit hashes (of y and of y without its last label)
 * plus their length; two distinct sequences with equal hashes would be merged.  The
 * workspace is cached in the model; calls on a model are serialised.
 */
typedef enum { TBS_MERGE_MAX = 0, TBS_MERGE_LOGADD = 1 } tbs_merge_op;

typedef struct {
  int32_t beam_size;
  int32_t merge;  /* tbs_merge_op */
} tbs_hyp_params;

tbs_status tbs_hyp_search(const tbs_model *model, const tbs_hyp_params *params,
                          const float *encoder_out, const int32_t *lengths, int32_t B, int32_t T,
                          int32_t *out_tokens, int32_t *out_num_tokens, double *out_scores,
                          int32_t *trace, void *hip_stream);

/*
 * Forward recursions of the transducer losses over the (frame t, labels emitted u) grid
 * (Sec. 3), on given log-probabilities:
 *   blank   DEVICE float [B][T][U+1]: log P(blank | frame t, u labels emitted);
 *   label   DEVICE float [B][T][U]: log P(label u+1 of the utterance | frame t, u labels);
 *   lengths DEVICE int32 [B][2]: each utterance's frames T_b in [1, T] and labels U_b in
 *           [0, U] (cells beyond them are not read);
 *   kind    TBS_TRANSDUCER_STANDARD, eq. (1): alpha(t, u) = log_add(alpha(t-1, u) +
 *             blank(t-1, u), alpha(t, u-1) + label(t, u-1)), likelihood
 *             alpha(T_b - 1, U_b) + blank(T_b - 1, U_b);
 *           TBS_TRANSDUCER_MODIFIED, eq. (2): a label also moves to the next frame,
 *             alpha(t, u) = log_add(alpha(t-1, u) + blank(t-1, u), alpha(t-1, u-1) +
 *             label(t-1, u-1)), likelihood alpha(T_b, U_b);
 *           TBS_TRANSDUCER_CONSTRAINED, eq. (3): as (2) with blank(t-1, u) added to the
 *             label term, likelihood alpha(T_b, U_b); alpha(0, 0) = 0 in all three.
 *   out_total  DEVICE double [B]: the log-likelihood (-inf if no path, e.g. U_b > T_b for
 *              (2) and (3)); NaN for an utterance whose lengths are out of range;
 *   out_alpha  DEVICE float [B][T+1][U+1] or NULL: alpha of the rows the recursion visits
 *              (t <= T_b for (2) and (3), t < T_b for (1)), -inf for u > U_b; other rows
 *              are not written;
 *   out_status DEVICE int32 [B] or NULL: 0, or 1 for out-of-range lengths.
 * Scores accumulate in fp64.  Errors: TBS_EINVAL (kind, sizes, NULL), TBS_ECAPACITY for
 * U > 1023.
 */
typedef enum {
  TBS_TRANSDUCER_STANDARD = 0,
  TBS_TRANSDUCER_MODIFIED = 1,
  TBS_TRANSDUCER_CONSTRAINED = 2
} tbs_transducer_kind;

tbs_status tbs_transducer_forward(int32_t kind, const float *blank, const float *label,
                                  const int32_t *lengths, int32_t B, int32_t T, int32_t U,
                                  double *out_total, float *out_alpha, int32_t *out_status,
                                  void *hip_stream);

/*
 * How tbs_decode drives the frame loop of Algorithm 1 (all schedules compute
 * the same search; results agree within the fp32 rounding of the joiner):
 *   TBS_SCHEDULE_FRAME   two kernels per frame over the whole batch: a joiner
 *                        GEMM over every active (stream, context) row, then a
 *                        search kernel with one workgroup per stream;
 *   TBS_SCHEDULE_STREAM_SINGLE
 *                        one persistent kernel, one workgroup per stream, that
 *                        runs joiner, log-softmax and search for every frame of
 *                        its stream on one compute unit (no per-frame launch or
 *                        global round trip).  Needs max_contexts (after
 *                        clamping to max_states) <= 16, vocab_size <= 512,
 *                        for the trivial graph max_states <= 16, and one
 *                        stream's joiner input and logit rows in LDS beside
 *                        the search state: tbs_decode returns
 *                        TBS_EUNSUPPORTED for shapes outside that;
 *   TBS_SCHEDULE_STREAM  as STREAM_SINGLE, except that for the trivial graph
 *                        with an fp32 joiner, when B x G workgroups fit the
 *                        device at once (G = 8, 4 or 2, each with 64 or 128
 *                        vocabulary columns), G workgroups share each stream:
 *                        each computes its columns of the joiner, they exchange
 *                        per-row normaliser terms and best labels every frame
 *                        through tagged words in device memory (device-scope
 *                        atomics; cooperative launch), and all run the same search.
 *                        A wait that exhausts its poll budget (which does not
 *                        happen while the whole grid is resident, as the
 *                        cooperative launch guarantees) makes every later wait
 *                        of the launch give up at once; each stream that gave up
 *                        returns out_status[b] = 2 and a NaN score (so the
 *                        failure shows even when out_status is NULL), and its
 *                        tokens are not valid;
 *   TBS_SCHEDULE_AUTO    (default) STREAM when it fits, the joiner weight
 *                        (V x dim) is at most 4 MiB and the joiner is bf16 or
 *                        max_contexts <= 4; else FRAME.
 * The setting is per model and applies to later tbs_decode calls; an unknown
 * value returns TBS_EINVAL.
 */
typedef enum {
  TBS_SCHEDULE_AUTO = 0,
  TBS_SCHEDULE_FRAME = 1,
  TBS_SCHEDULE_STREAM = 2,
  TBS_SCHEDULE_STREAM_SINGLE = 3
} tbs_schedule;

tbs_status tbs_model_set_schedule(tbs_model *model, int32_t schedule);

/*
 * Frame loop of TBS_SCHEDULE_FRAME in a HIP graph (Algorithm 1's loop over
 * frames without a host launch per kernel): when a decode's launch arguments
 * (graph, params, B, T, the workspace, encoder_out, trace, the longest length)
 * repeat those of the model's previous decode, the frame loop is captured once
 * into a HIP graph and replayed from then on; a decode with other arguments
 * launches directly (and becomes the candidate for the next capture).  Results
 * are identical either way.  enable = 0 turns capture off for later decodes
 * (default on); capture is skipped while per-kernel profiling is on.
 * tbs_model_graph_stats returns the number of captures and replays so far.
 */
tbs_status tbs_model_set_graph_capture(tbs_model *model, int32_t enable);
tbs_status tbs_model_graph_stats(const tbs_model *model, int32_t *captures, int32_t *replays);

/*
 * Poll budget of each exchange wait of the grouped per-stream kernel
 * (TBS_SCHEDULE_STREAM): polls >= 1, or 0 for the default (4,194,304).  A
 * diagnostic for the timeout path: a tiny budget makes waits give up while
 * the other workgroups are still busy, so that path can be exercised with
 * every kernel still finishing normally.  Per model, for later decodes;
 * polls < 0 returns TBS_EINVAL.
 */
tbs_status tbs_model_set_exchange_spin_limit(tbs_model *model, int32_t polls);

/*
 * Decoder + joiner + log-softmax alone (Algorithm 1: Decoder, IndexSelect,
 * joiner), for R (encoder row, context) pairs:
 *   enc_rows  DEVICE float [R][C];  ctx DEVICE int32 [R], each a * V + b with
 *             a, b in [0, V) (not checked on the device: the caller guarantees it);
 *   out_logp  DEVICE float [R][V]: log-probabilities.
 * R >= 0 (R = 0 is a no-op).
 */
tbs_status tbs_joiner_logp(const tbs_model *model, const float *enc_rows, const int32_t *ctx,
                           int32_t R, float *out_logp, void *hip_stream);

/*
 * Per-kernel timing, for benchmarks.  While enabled on a model, every decode
 * records a pair of HIP events for each kernel launch (joiner and search once
 * per frame, or the per-stream kernel once; final once per decode): inside the
 * launch's own dispatch packet, or for the cooperative grouped kernel on its
 * stream around the launch, and keeps them pending.  tbs_model_read_profile waits for those events, adds their elapsed
 * times into out[TBS_KERNEL_COUNT] (indexed by tbs_kernel_id; launches and
 * milliseconds since the last enable) and releases them.  Enabling resets the
 * counters; disabling drops pending events.
 */
typedef enum {
  TBS_KERNEL_JOINER = 0,
  TBS_KERNEL_SEARCH = 1,
  TBS_KERNEL_FINAL = 2,
  TBS_KERNEL_STREAM = 3, /* the persistent kernel, one workgroup per stream */
  TBS_KERNEL_STREAM_GROUP = 4, /* the persistent kernel, several workgroups per stream */
  TBS_KERNEL_HYP_STEP = 5, /* tbs_hyp_search: merge and selection of one frame */
  TBS_KERNEL_COUNT = 6
} tbs_kernel_id;

typedef struct {
  int32_t launches;
  double total_ms;
} tbs_kernel_time;

tbs_status tbs_model_set_profiling(tbs_model *model, int32_t enable);
tbs_status tbs_model_read_profile(tbs_model *model, tbs_kernel_time *out);

/* Message for the calling thread's last error ("" if none). */
const char *tbs_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* TBS_H */
