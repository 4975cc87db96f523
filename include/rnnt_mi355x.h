/*
 * rnnt_mi355x.h -- RNN-Transducer and W-Transducer loss and gradient over the
 * T x (U+1) alignment grid, for AMD Instinct MI355X (gfx950).
 *
 * Method: "Powerful and Extensible WFST Framework for RNN-Transducer Losses"
 * (Laptev, Bataev, Gitman, Ginsburg, ICASSP 2023).
 *   - Eq. 1: the loss of an utterance is the negative forward score of its
 *     training lattice, -ln P(Y | X), summed over every alignment.
 *   - Fig. 1 and Section 2.3 (Grid-Transducer): the lattice is a grid of nodes
 *     (t, u), 0 <= t < T, 0 <= u <= U.  A blank arc leaves (t, u) for (t+1, u)
 *     when t < T-1; a label arc carrying unit y_{u+1} leaves (t, u) for
 *     (t, u+1) when u < U; the closing blank leaves (T-1, U) for the final
 *     state.  Arc weights are selected from the log-softmax of the joint
 *     logits row (t, u) (Populate, Section 2.2).
 *   - Section 3.2 and Fig. 4 (W-Transducer, "force-final"): additional
 *     probability-one arcs from (0, 0) to every (t, 0), t >= 1, and from every
 *     (t, U), t <= T-2, to (T-1, U); the closing blank is still required.
 *   - Section 4.3 ("allow-ignore"): those final arcs go to the final state.
 *
 * Conventions shared by every entry point
 *   - All pointers are DEVICE pointers unless a comment says otherwise, and
 *     belong to the caller.  The library keeps no state between calls (apart
 *     from the per-GPU address of rnnt_loss_noalloc's static scratch) and
 *     never synchronises the stream: work is queued on `stream` and the call
 *     returns RNNT_OK before the results exist.
 *   - logits / grad are dense row-major (B, T_max, U_max+1, V), V innermost,
 *     16-byte aligned.  Element offsets are 64-bit (more than 2^31 elements
 *     are fine).
 *   - labels is dense (B, U_max) int32; row b is read for u < label_lens[b].
 *     logit_lens and label_lens are (B) int32.
 *   - Errors that the host can see (NULL pointer, bad shape, blank outside
 *     [0, V), unknown dtype or variant, workspace too small, misalignment)
 *     return a status and launch nothing.  Data errors that only the device
 *     can see (T_b outside [1, T_max], U_b outside [0, U_max], a label equal
 *     to blank or outside [0, V)) give loss NaN for that utterance and a zero
 *     gradient for all its rows; other utterances are unaffected.
 *   - Logits outside an utterance's valid rows (t >= T_b or u > U_b) are
 *     never used, so they may hold anything, NaN included.
 */
#ifndef RNNT_MI355X_H
#define RNNT_MI355X_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  RNNT_OK = 0,
  RNNT_ERR_NULL_PTR = 1,     /* a required pointer is NULL                       */
  RNNT_ERR_BAD_SHAPE = 2,    /* B < 1, T_max < 1, U_max < 0, V < 2, or too large */
  RNNT_ERR_BAD_BLANK = 3,    /* blank outside [0, V)                             */
  RNNT_ERR_BAD_DTYPE = 4,    /* unknown dtype, or grad_dtype not dtype / F32     */
  RNNT_ERR_BAD_VARIANT = 5,  /* unknown rnnt_variant_t                           */
  RNNT_ERR_WORKSPACE = 6,    /* workspace given but smaller than required        */
  RNNT_ERR_ALIGNMENT = 7,    /* logits or grad not 16-byte aligned               */
  RNNT_ERR_HIP = 8,          /* a HIP runtime call failed (launch, allocation)   */
  RNNT_ERR_UNSUPPORTED = 9,  /* shape outside what the library handles (U_max+1 > 2048,
                                T_max * (U_max+1) >= 2^27, or an arc-list lattice
                                beyond the sweep's limits)                          */
  RNNT_ERR_BAD_LATTICE = 10, /* an arc list that breaks the numbering rules of
                                rnnt_arc_plan, or a plan that does not match      */
  RNNT_ERR_SCRATCH = 11      /* rnnt_loss_noalloc: the shape needs more workspace
                                than the static scratch holds                     */
} rnnt_status_t;

typedef enum {
  RNNT_VARIANT_RNNT = 0,               /* Fig. 1, Section 2.3                      */
  RNNT_VARIANT_WRNNT = 1,              /* W-Transducer force-final, Section 3.2     */
  RNNT_VARIANT_WRNNT_ALLOW_IGNORE = 2  /* final wild-card arcs to the final state,  */
                                       /* Section 4.3                               */
} rnnt_variant_t;

typedef enum {
  RNNT_DTYPE_F32 = 0,   /* IEEE binary32 logits and gradient                       */
  RNNT_DTYPE_BF16 = 1,  /* bfloat16 logits and gradient, fp32 arithmetic inside    */
  RNNT_DTYPE_F16 = 2    /* IEEE binary16 logits and gradient, fp32 arithmetic      */
                        /* inside (the half-precision lattice of Section 4.2)      */
} rnnt_dtype_t;

/* Padded problem shape: logits are (B, T_max, U_max+1, V) of `dtype`; the
 * gradient has the same shape and element type `grad_dtype`, which must be
 * `dtype` itself or RNNT_DTYPE_F32 (a float32 gradient of half-precision
 * logits: the gradient is computed in float32 either way, this only decides
 * how it is stored). */
typedef struct {
  int32_t B;
  int32_t T_max;
  int32_t U_max;
  int32_t V;
  rnnt_dtype_t dtype;
  rnnt_dtype_t grad_dtype;
} rnnt_shape_t;

/* Bytes of device workspace that rnnt_loss needs for `shape` (0 if the shape
 * is invalid).  Host-only; touches no device. */
size_t rnnt_loss_workspace_bytes(rnnt_shape_t shape);

/*
 * Per-utterance loss -ln P(Y_b | X_b) (Eq. 1) and, if grad_out != NULL, the
 * gradient of sum_b loss_b with respect to the logits.
 *
 *   logits      (B, T_max, U_max+1, V) of shape.dtype; only rows t < T_b,
 *               u <= U_b are read.
 *   labels      (B, U_max) int32 units y_1..y_{U_b} per row.
 *   logit_lens  (B) int32 T_b;  label_lens (B) int32 U_b.
 *   blank       index of the blank symbol in [0, V).
 *   variant     rnnt_variant_t.
 *   loss_out    (B) float32: loss_b, no reduction (NaN for bad data).
 *   grad_out    NULL (loss only) or (B, T_max, U_max+1, V) of shape.grad_dtype:
 *               every element is written; rows outside t < T_b, u <= U_b and
 *               all rows of a bad utterance are exactly 0.  The gradient of
 *               row (t, u) is softmax * (g_blank + g_label) - g_blank at
 *               v = blank - g_label at v = y_{u+1}, where g_* are the arc
 *               posteriors; wild-card arcs carry no parameter.
 *   workspace   device buffer of at least rnnt_loss_workspace_bytes(shape)
 *               bytes, 256-byte aligned, or NULL: the library then takes and
 *               releases one with hipMallocAsync / hipFreeAsync on `stream`.
 *               Its contents need no initialisation and are not preserved.
 *   stream      HIP stream the work is ordered on.
 * Calls that overlap in time must not share a workspace.  Shapes with
 * U_max + 1 > 2048 or T_max * (U_max + 1) >= 2^27 return RNNT_ERR_UNSUPPORTED
 * (such lattices go through rnnt_arc_loss).
 */
rnnt_status_t rnnt_loss(const void* logits, rnnt_shape_t shape, const int32_t* labels,
                        const int32_t* logit_lens, const int32_t* label_lens, int32_t blank,
                        rnnt_variant_t variant, float* loss_out, void* grad_out, void* workspace,
                        size_t workspace_bytes, hipStream_t stream);

/* Bytes of the static device scratch of rnnt_loss_noalloc: one array of this
 * size on every GPU the library runs on, held until the process ends. */
#define RNNT_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

/*
 * rnnt_loss for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc.  Same
 * arguments (no workspace), kernels and results as rnnt_loss; the workspace is
 * the library's static device array of RNNT_NOALLOC_SCRATCH_BYTES bytes on the
 * GPU of `stream`.  No call allocates or frees memory (hipMalloc, hipFree,
 * stream-ordered or library allocations); the first call on a GPU looks up the
 * array's device address (hipGetSymbolAddress) and keeps it for later calls.
 *   - A shape whose workspace (rnnt_loss_workspace_bytes) exceeds the array
 *     returns RNNT_ERR_SCRATCH, checked on the host before any HIP call; the
 *     bpe-sized batch (B = 32, T_max = 250, U_max = 80) needs about 42 MB.
 *   - Every call on one GPU shares that GPU's array, which keeps the last
 *     call's contents.  Nothing in it needs to start at zero (each call writes
 *     every word it reads before reading it).  Calls that overlap in time on
 *     one GPU (other streams, other host threads) race on the array: order
 *     them on one stream or serialise them.
 *   - RNNT_ERR_HIP if the stream's device cannot be found or the address
 *     lookup fails.
 */
rnnt_status_t rnnt_loss_noalloc(const void* logits, rnnt_shape_t shape, const int32_t* labels,
                                const int32_t* logit_lens, const int32_t* label_lens, int32_t blank,
                                rnnt_variant_t variant, float* loss_out, void* grad_out, hipStream_t stream);

/*
 * rnnt_loss that also records timing events on `stream`: events[0] before the
 * first kernel, events[1] after kernel 1 (log-normaliser and gather),
 * events[2] after kernel 2 (forward / backward sweeps), events[3] after
 * kernel 2b (arc posteriors), events[4] after kernel 3 (gradient); without a
 * gradient, events[3] and events[4] follow events[2] directly.  `events` is a
 * HOST array of 5 events created by the caller (for example with
 * hipEventCreate); NULL behaves exactly like rnnt_loss.  Used to time each
 * kernel in place (hipEventElapsedTime between consecutive events).
 */
rnnt_status_t rnnt_loss_timed(const void* logits, rnnt_shape_t shape, const int32_t* labels,
                              const int32_t* logit_lens, const int32_t* label_lens, int32_t blank,
                              rnnt_variant_t variant, float* loss_out, void* grad_out, void* workspace,
                              size_t workspace_bytes, hipStream_t stream, hipEvent_t* events);

/*
 * Populate step alone (Section 2.2 Populate; Fig. 1 arc weights): for every
 * valid row (t < T_b, u <= U_b) of every good utterance
 *   lse[b,t,u]       = ln sum_v exp(logits[b,t,u,v])
 *   lp_blank[b,t,u]  = logits[b,t,u,blank] - lse
 *   lp_label[b,t,u]  = logits[b,t,u,y_{u+1}] - lse for u < U_b, -inf at u = U_b
 * as dense (B, T_max, U_max+1) float64 arrays.  Other entries are not written.
 * Label values are not validated here beyond the bounds needed to read safely
 * (an out-of-range label gives NaN in lp_label).
 */
rnnt_status_t rnnt_log_softmax_gather(const void* logits, rnnt_shape_t shape, const int32_t* labels,
                                      const int32_t* logit_lens, const int32_t* label_lens,
                                      int32_t blank, double* lse_out, double* lp_blank_out,
                                      double* lp_label_out, hipStream_t stream);

/*
 * Forward and backward scores on given lattice weights (Eq. 1's Fwd and its
 * backward counterpart), with no softmax: the lattice of Fig. 1 / Fig. 4 is
 * populated directly from
 *   lp_blank, lp_label  dense (B, T_max, U_max+1) float64 arc weights; entries
 *                       outside t < T_b, u <= U_b (and lp_label at u = U_b)
 *                       are never read.
 * Outputs (dense (B, T_max, U_max+1) float64 unless noted; any may be NULL):
 *   alpha_out           forward score of each node, -inf never written for
 *                       nodes outside the utterance (those entries untouched)
 *   beta_out            backward score of each node
 *   loss_out            (B) float64: -(forward score of the final state)
 *   loss_bwd_out        (B) float64: -beta(0, 0), computed by the backward sweep
 *   occ_blank_out       posterior of the blank arc leaving each node (0 where
 *                       absent)
 *   occ_label_out       posterior of the label arc leaving each node
 * label_lens/logit_lens as in rnnt_loss; shape.V, shape.dtype and
 * shape.grad_dtype are ignored (pass V >= 2).  A bad utterance (lengths out of range) gets NaN losses and
 * no other output.  Needs a workspace of rnnt_lattice_workspace_bytes(shape)
 * bytes or NULL (then allocated stream-ordered).
 */
size_t rnnt_lattice_workspace_bytes(rnnt_shape_t shape);
rnnt_status_t rnnt_lattice_scores(const double* lp_blank, const double* lp_label, rnnt_shape_t shape,
                                  const int32_t* logit_lens, const int32_t* label_lens,
                                  rnnt_variant_t variant, double* alpha_out, double* beta_out,
                                  double* loss_out, double* loss_bwd_out, double* occ_blank_out,
                                  double* occ_label_out, void* workspace, size_t workspace_bytes,
                                  hipStream_t stream);

/* Forced alignment: the single most probable path through the utterance's lattice
 * (the grid of Fig. 1, or the W-Transducer lattices of Section 3.2 / Fig. 4 and
 * Section 4.3 for variant = RNNT_VARIANT_WRNNT / RNNT_VARIANT_WRNNT_ALLOW_IGNORE),
 * the lattice serving forced alignment as it serves training (Section 2.2).
 *
 * Arguments as rnnt_loss for logits (any of the three dtypes; shape.grad_dtype is
 * ignored), labels, lengths, blank and variant.  Outputs, device memory owned by
 * the caller:
 *   score_out        (B) float: the best path's log-probability (natural log,
 *                    the closing blank included where the path takes it);
 *   label_frames_out (B, U_max) int32: entry [b, i] is the frame at which unit
 *                    y_{i+1} is emitted (the path takes the label arc
 *                    (t, i) -> (t, i+1)); -1 for i >= U_b;
 *   span_out         (B, 2) int32 or NULL: the first frame of the path (s > 0
 *                    when it enters (s, 0) by an initial wild-card arc) and the
 *                    last (e < T_b - 1 when it leaves (e, U_b) by a final
 *                    wild-card arc); (0, T_b - 1) for RNN-T.
 * Ties between equally probable paths are broken by a fixed order: at a node the
 * blank arc, then the label arc, then the initial wild-card arc, then the final
 * wild-card arcs (the earliest source frame) -- a later candidate wins only when
 * strictly more probable; at the end of the allow-ignore lattice the closing
 * blank wins a tie with the jump to the final state.  A bad utterance (as in
 * rnnt_loss) gets score NaN and frames / span -1.  Needs a workspace of
 * rnnt_viterbi_workspace_bytes(shape) bytes (256-byte aligned) or NULL (then
 * allocated stream-ordered).  U_max + 1 <= 2048 and T_max * (U_max + 1) < 2^27
 * (else RNNT_ERR_UNSUPPORTED).
 */
size_t rnnt_viterbi_workspace_bytes(rnnt_shape_t shape);
rnnt_status_t rnnt_viterbi(const void* logits, rnnt_shape_t shape, const int32_t* labels,
                           const int32_t* logit_lens, const int32_t* label_lens, int32_t blank,
                           rnnt_variant_t variant, float* score_out, int32_t* label_frames_out,
                           int32_t* span_out, void* workspace, size_t workspace_bytes, hipStream_t stream);

/* rnnt_viterbi, recording events[0..2] (caller-created hipEvent_t) on `stream`:
 * before the populate kernel, after it, and after the alignment kernel. */
rnnt_status_t rnnt_viterbi_timed(const void* logits, rnnt_shape_t shape, const int32_t* labels,
                                 const int32_t* logit_lens, const int32_t* label_lens, int32_t blank,
                                 rnnt_variant_t variant, float* score_out, int32_t* label_frames_out,
                                 int32_t* span_out, void* workspace, size_t workspace_bytes, hipStream_t stream,
                                 hipEvent_t* events);

/* ---------------------------------------------------------------------------
 * Lattices given as arc lists (Section 2.2: the lattice is built as a graph and
 * its arcs are filled in by indexed selection from X = log_softmax(logits) with
 * each arc's time index, unit index and label; the grid of Fig. 1 and the
 * W-Transducer lattices of Fig. 4 are particular arc lists, and a new loss is a
 * new graph, with no new kernel).
 *
 * An arc leaves state src for state dst and weighs (natural log)
 *     score + ln softmax(logits[b, t, u, :])[label]    when label >= 0,
 *     score                                            when label == -1 (an arc
 *                                                      that reads no logits).
 * Per utterance the states are numbered 0 .. n_b-1: 0 is the start, n_b-1 the
 * final state, and every arc goes from a lower to a higher number (n_b = 1 is
 * the lattice whose only path is empty).  Parallel arcs are separate entries
 * and their probabilities add.
 *     loss_b = -ln (sum over start -> final paths of exp(sum of arc weights)),
 * +inf when no path reaches the final state (then the gradient is 0);
 *     d loss_b / d logits[b, t, u, :] = sum over arcs a on row (t, u) of
 *                                       g_a (softmax(logits[b, t, u]) - onehot(label_a)),
 * g_a the arc's posterior.
 *
 * Work splits in two:
 *   rnnt_arc_plan (host only) rearranges a batch's arc lists for the device
 *     sweep -- topological levels, arcs grouped by destination level for the
 *     forward sweep and by source level for the backward one, arcs grouped by
 *     logits row for the gradient -- into one image of host memory, which the
 *     caller copies to device memory as it is (it holds no pointers).
 *   rnnt_arc_loss (device) computes the losses and the gradient of a batch of
 *     logits with that device image.  The plan depends on the lattices only, not
 *     on the logits or the lengths.
 */
typedef struct {
  int32_t src, dst; /* states of the utterance, 0 <= src < dst < n_b                 */
  int32_t t, u;     /* logits row read by the arc: 0 <= t < T_max, 0 <= u <= U_max  */
                    /* (ignored when label == -1)                                  */
  int32_t label;    /* vocabulary index in [0, V), or -1                            */
  float score;      /* natural-log weight added to the arc (finite)                 */
} rnnt_arc_t;

/* Descriptor of a plan (host memory, filled by rnnt_arc_plan).  The sizes are
 * informative; off[] and the chunk counts are read by rnnt_arc_loss. */
typedef struct {
  int32_t B, T_max, U_max, V, blank;
  int32_t num_states, num_levels, num_arcs, num_row_arcs, num_extra_rows;
  int32_t num_slots[2];             /* arc slots of the forward / backward sweep
                                       (the arcs plus padding)                   */
  int32_t max_level_states, max_level_arcs, max_in_degree, max_pins;
  int32_t state_chunks;             /* per-level register chunks of 64 states   */
  int32_t slots_per_state;          /* arc slots per state held in registers    */
  int64_t image_bytes;              /* bytes of the image to copy to the device */
  int64_t off[17];                  /* byte offsets of the image's arrays       */
} rnnt_arc_plan_t;

/* Upper bound of the image bytes rnnt_arc_plan writes for a batch with these
 * totals (0 if the arguments are out of range).  Host only. */
size_t rnnt_arc_plan_bytes_bound(int32_t B, int32_t T_max, int32_t U_max, int64_t num_states, int64_t num_arcs);

/* Plans a batch of B arc lists (host only; every pointer here is HOST memory).
 *   num_states  (B): n_b >= 1;
 *   arc_begin   (B+1): utterance b's arcs are arcs[arc_begin[b] .. arc_begin[b+1]),
 *               arc_begin[0] = 0, non-decreasing;
 *   arcs        the arc records, states local to their utterance;
 *   image       receives the device image (image_bytes >= the bound above is
 *               always enough); plan receives the descriptor.
 * The logits shape (T_max, U_max, V) and blank are those of the later loss calls
 * (blank decides how the gradient kernel groups a row's arcs).  Returns
 * RNNT_ERR_BAD_LATTICE for an arc list breaking the rules above,
 * RNNT_ERR_BAD_SHAPE / RNNT_ERR_BAD_BLANK for the shape, RNNT_ERR_WORKSPACE when
 * image_bytes is too small, and RNNT_ERR_UNSUPPORTED past the sweep's limits:
 * more than 4096 states on one topological level or 4096 arcs entering one, more
 * than 2048 states per utterance and direction whose scores must outlive the
 * sweep's 4096-state window (sources of arcs that span that many states), more
 * than 1024 label arcs on a row that carries two or more non-blank labels,
 * more than 2^27 states or arcs in one utterance, or batch totals of 2^31
 * states, arcs or logits rows. */
rnnt_status_t rnnt_arc_plan(int32_t B, int32_t T_max, int32_t U_max, int32_t V, int32_t blank,
                            const int32_t* num_states, const int64_t* arc_begin, const rnnt_arc_t* arcs,
                            void* image, size_t image_bytes, rnnt_arc_plan_t* plan);

/* Bytes of device workspace rnnt_arc_loss needs with this plan (0 if plan is NULL). */
size_t rnnt_arc_loss_workspace_bytes(const rnnt_arc_plan_t* plan);

/* Loss and gradient of a batch of arc-list lattices.
 *   logits, shape     as in rnnt_loss; (B, T_max, U_max, V) must equal the plan's;
 *   logit_lens, label_lens  (B) int32: the valid rows of utterance b are t < T_b,
 *                     u <= U_b; only those are read;
 *   plan              the descriptor (HOST memory) from rnnt_arc_plan;
 *   plan_image        the plan's image, copied to DEVICE memory (16-byte aligned);
 *   loss_out          (B) float32: loss_b, +inf when no path reaches the final state;
 *   grad_out          gradient as in rnnt_loss, or NULL for the loss alone.
 * Data errors seen on the device -- T_b outside [1, T_max], U_b outside
 * [0, U_max], an arc with a label that reads a row outside the utterance's valid
 * rows, or NaN logits on a row an arc reads -- give loss NaN and a zero gradient
 * for that utterance.  Workspace: rnnt_arc_loss_workspace_bytes(plan) bytes,
 * 256-byte aligned, or NULL (then allocated stream-ordered). */
rnnt_status_t rnnt_arc_loss(const void* logits, rnnt_shape_t shape, const int32_t* logit_lens,
                            const int32_t* label_lens, const rnnt_arc_plan_t* plan, const void* plan_image,
                            float* loss_out, void* grad_out, void* workspace, size_t workspace_bytes,
                            hipStream_t stream);

/* rnnt_arc_loss, recording events[0..5] (caller-created) on `stream`: before the
 * row normaliser, after it, after the arc populate kernel, after the sweep, after
 * the arc posteriors and row records, and after the gradient kernels. */
rnnt_status_t rnnt_arc_loss_timed(const void* logits, rnnt_shape_t shape, const int32_t* logit_lens,
                                  const int32_t* label_lens, const rnnt_arc_plan_t* plan, const void* plan_image,
                                  float* loss_out, void* grad_out, void* workspace, size_t workspace_bytes,
                                  hipStream_t stream, hipEvent_t* events);

/* Static description of a status code (never NULL). */
const char* rnnt_status_string(rnnt_status_t status);

/* Library version string, e.g. "rnnt_mi355x 0.1.0 gfx950". */
const char* rnnt_version(void);

#ifdef __cplusplus
}
#endif

#endif /* RNNT_MI355X_H */
