/*
 * softneuro.h -- C ABI of the MI355X routine-selection inference library.
 *
 * The calls follow the workflow of the SoftNeuro paper (Hilaga et al.,
 * arXiv 2110.06037): build a net of layers (Sec. III-B), profile every
 * routine of every layer on the device (Sec. III-C, unit profiling), select
 * the optimal routine path with dynamic programming over the layer graph
 * including adaptation costs (Sec. IV, Algorithm 1 "DPRS"), then run
 * inference with the selected routines (Sec. III-A, step 3).
 *
 * Terms.  A *routine* is one implementation of a layer: an algorithm
 * (direct, implicit GEMM, Winograd F(2x2,3x3)), a tensor layout, an element
 * type and a routine parameter (a tile configuration).  The *schema* of a
 * routine is its (element type, layout) pair: layouts NCHW, NHWC or NC8HW8
 * (channel blocks of 8, channels zero-padded to a multiple of 8), element
 * types float32, float16, bfloat16.  By default a graph computes in its run
 * dtype only, so schemas differ by layout alone; SN_OPT_DTYPES admits the
 * other element types (precision-hybrid tuning, Sec. IV-F).  Between two
 * layers whose routines have different schemas an *adapt* routine (a layout
 * converter, a cast, or both at once) runs.
 *
 * Conventions.
 *  - Every int-returning call returns SN_OK (0) or a negative sn_status.  No
 *    C++ exception crosses this boundary.  sn_last_error() returns a
 *    thread-local description of the last failure.
 *  - A graph is not thread-safe; separate graphs are independent.
 *  - State machine: create -> add_layer* -> (profile | set_costs) ->
 *    (select_path | set_path) -> run*.  A call out of order returns
 *    SN_E_STATE.  Adding a layer after selection is SN_E_STATE.
 *  - Device pointers (d_in, d_out) are caller-owned HIP device memory; the
 *    graph owns its weights, workspaces and intermediate tensors.
 *  - Streams are hipStream_t passed as void*; NULL means the null stream.
 *  - Element types: SN_F32 = IEEE binary32, SN_F16 = binary16, SN_BF16 =
 *    bfloat16 (passed as 16-bit patterns).  Biases are always float32.
 *    The user's input and output tensors and the weights passed in are in
 *    the graph's run dtype.  Accumulation is float32 in every routine;
 *    outputs are rounded to the routine's element type, and every cast
 *    (weights at graph build, tensors in adapt routines) rounds once, to
 *    nearest-even.
 */
#ifndef SOFTNEURO_H
#define SOFTNEURO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct sn_graph sn_graph;

typedef enum {
  SN_OK = 0,
  SN_E_INVALID = -1,     /* bad argument, unknown id, malformed JSON          */
  SN_E_SHAPE = -2,       /* inconsistent tensor shapes between layers          */
  SN_E_STATE = -3,       /* call out of order                                  */
  SN_E_UNSUPPORTED = -4, /* no routine for a layer / option not available      */
  SN_E_DEVICE = -5,      /* HIP error or no device (host-only graph)           */
  SN_E_NOMEM = -6,       /* caller buffer too small (required size reported)   */
  SN_E_INTERNAL = -7     /* consistency check failed inside the library        */
} sn_status;

typedef enum { SN_F32 = 0, SN_F16 = 1, SN_BF16 = 2 } sn_dtype;

/* Tensor layouts.  Values index bitmasks. */
typedef enum { SN_NCHW = 0, SN_NHWC = 1, SN_NC8HW8 = 2 } sn_layout;
#define SN_NUM_LAYOUTS 3
/* Schema index = dtype * SN_NUM_LAYOUTS + layout (0 .. 8); indexes the
 * adapt-cost matrices of the cost table. */
#define SN_NUM_SCHEMAS 9

/* Algorithms.  Non-convolution layers have one algorithm (SN_ALGO_DIRECT) per
 * layout; FC layers also have SN_ALGO_IGEMM, the paper's dense childnet
 * computed as a 1x1 convolution (Sec. III-D). */
typedef enum { SN_ALGO_DIRECT = 0, SN_ALGO_IGEMM = 1, SN_ALGO_WINOGRAD = 2 } sn_algo;
#define SN_NUM_ALGOS 3

typedef enum {
  SN_LAYER_INPUT = 0,  /* auxiliary input layer (id 0, created by sn_graph_create) */
  SN_LAYER_CONV2D = 1, /* 2-D cross-correlation, groups 1 (dense) or C (depthwise) */
  SN_LAYER_MAXPOOL = 2,
  SN_LAYER_GAP = 3,    /* global average pooling to N x C x 1 x 1 */
  SN_LAYER_ADD = 4,    /* residual merge of two inputs of equal shape */
  SN_LAYER_FC = 5,     /* y = act(W x + b) on an N x C x 1 x 1 input */
  SN_LAYER_OUTPUT = 6  /* auxiliary output layer (implicit, after the last layer) */
} sn_layer_type;

typedef enum { SN_ACT_NONE = 0, SN_ACT_RELU = 1, SN_ACT_RELU6 = 2 } sn_act;

/* Layer description.  Fields not used by a type are ignored.
 *   CONV2D : k = output channels, r x s kernel, stride, pad, groups, act;
 *            an optional second input is a residual of the output's shape
 *            (dense convolutions only): y = act(conv(x) + bias + residual),
 *            a residual add fused into the convolution that produces its
 *            other operand
 *   MAXPOOL: r (= s) window, stride, pad (padding never wins the max)
 *   GAP    : -
 *   ADD    : act
 *   FC     : k = output features, act                                    */
typedef struct {
  int32_t type;
  int32_t k;
  int32_t r, s;
  int32_t stride, pad;
  int32_t groups;
  int32_t act;
} sn_layer_desc;

typedef struct {
  int32_t id;        /* routine id, unique within the layer; ids enumerate
                        the run dtype first, then the other allowed dtypes
                        in sn_dtype order; within a dtype layout-major, then
                        algorithm, then parameter index                      */
  int32_t layout;    /* sn_layout                                            */
  int32_t algo;      /* sn_algo                                              */
  int32_t param;     /* routine-parameter index (tile configuration)         */
  int32_t dtype;     /* sn_dtype the routine computes and stores in          */
  int32_t schema;    /* dtype * SN_NUM_LAYOUTS + layout                      */
  int64_t cost_ns;   /* profiled time T(r) in ns, -1 if not profiled         */
  int64_t ws_bytes;  /* device workspace the routine needs beyond the layer's
                        input and output tensors (split reductions, the
                        three-kernel Winograd's transforms, a projection
                        stored for the two-launch routine), bytes           */
  char name[64];     /* descriptor, e.g. "nhwc/igemm:p41"; with several
                        dtypes allowed prefixed by the dtype, "f16:nhwc/..." */
} sn_routine_desc;

typedef enum {
  SN_SELECT_DPRS = 0,  /* optimal routine path by Algorithm 1 (layout, algo ignored) */
  SN_SELECT_FIXED = 1  /* one layout for the whole net and one convolution
                          algorithm wherever applicable (else implicit GEMM;
                          depthwise layers use their direct routine; FC layers
                          use igemm when algo is igemm, else direct); within
                          that, the fastest routine parameter */
} sn_select_mode;

typedef enum {
  SN_OPT_LAYOUTS = 0,   /* bitmask of allowed schemas (bit = sn_layout), default all */
  SN_OPT_ALGOS = 1,     /* bitmask of allowed algorithms (bit = sn_algo), default all */
  SN_OPT_PARAMS = 2,    /* 0: one routine parameter per algorithm; 1: all (default 1) */
  SN_OPT_HIPGRAPH = 3,  /* 1: sn_run replays a captured HIP graph (default 0)        */
  SN_OPT_SEED = 4,      /* seed of the profiler's scratch-tensor fill (default 1)    */
  SN_OPT_FLUSH = 5,     /* bytes written to a scratch buffer to evict the caches:
                           by sn_run_timed before each layer, and by sn_profile
                           before each timed run (cache-cold unit profiling);
                           0 = off, the default                                     */
  SN_OPT_KEEP = 6,      /* 1: the plan gives every intermediate tensor its own bytes
                           (no reuse by liveness), so sn_layer_output can read any
                           layer's stored output after a run (default 0)            */
  SN_OPT_DTYPES = 7,    /* bitmask of element types routines may compute in (bit =
                           sn_dtype), default the run dtype only; with more than one
                           every layer gets routines in each, and adapts cast
                           between them (precision-hybrid tuning, Sec. IV-F)        */
  SN_OPT_WS_LIMIT = 8   /* largest workspace (sn_routine_desc.ws_bytes) a routine
                           may use; routines above it are left out of every
                           layer's routine set, so selection optimises time under
                           that memory restriction (the restriction Sec. VI names
                           as future work; Winograd's transforms are its example).
                           -1 = no limit (the default); 0 = no workspace at all.
                           A layer left with no routine is refused by
                           sn_add_layer (SN_E_UNSUPPORTED).  A routine-set option:
                           set it before adding layers                               */
} sn_option;

/* Creates a graph whose auxiliary input layer (id 0) carries the user tensor
 * N x C x H x W in NCHW layout (Sec. IV-E: a zero-time single routine).
 * device >= 0 selects a HIP device; device = -1 creates a host-only graph on
 * which only the selection calls work (sn_set_costs, sn_select_path,
 * sn_set_path, queries) -- the graph used by GPU-free tests.
 * Errors: SN_E_INVALID (non-positive dims, unknown dtype), SN_E_UNSUPPORTED
 * (a tensor of 2 GiB or more: N * ceil8(C) * H * W * element size; every
 * kernel addresses a tensor with 32-bit byte offsets), SN_E_DEVICE. */
int sn_graph_create(int32_t dtype, int32_t n, int32_t c, int32_t h, int32_t w, int32_t device,
                    sn_graph** out);

/* Sets an sn_option.  Options that change the routine set (LAYOUTS, ALGOS,
 * PARAMS, DTYPES) are accepted only before the first sn_add_layer.
 * Errors: SN_E_INVALID (unknown option or value), SN_E_STATE. */
int sn_set_option(sn_graph* g, int32_t option, int64_t value);

/* Appends a layer (Sec. III-B: type, layer parameters, weights).  inputs
 * lists existing layer ids (so insertion order is a topological order,
 * Sec. IV-A); ADD takes two, CONV2D one or two (data, residual), the other
 * types one.  A CONV2D with a residual has the direct and implicit-GEMM
 * routines whose epilogue adds it (no Winograd, patch or small-channel
 * tiles).  weight: host memory in
 * the run dtype, OIHW for CONV2D ([K][C/groups][R][S]) and [K][C] for FC;
 * bias: host float32 [K] (may be NULL = zeros).  Both are copied.  The last
 * added layer is the net output.  *out_id receives the new id.
 * Errors: SN_E_INVALID (unknown input id, wrong arity, bad parameters),
 * SN_E_SHAPE (channel or size mismatch), SN_E_UNSUPPORTED (groups other than
 * 1 or C, or an output tensor of 2 GiB or more as for sn_graph_create),
 * SN_E_STATE (after selection), SN_E_DEVICE. */
int sn_add_layer(sn_graph* g, const sn_layer_desc* d, const int32_t* inputs, int32_t n_inputs,
                 const void* weight, const float* bias, int32_t* out_id);

/* Appends a dense convolution whose output also takes a projected shortcut:
 *   y = act(conv(x) + bias + conv1x1_stride(shortcut, shortcut_weight) + shortcut_bias)
 * with x = layer `input` (d describes the convolution: CONV2D, groups 1) and
 * the shortcut = layer `shortcut` (N x C2 x H2 x W2) read by a 1 x 1
 * convolution without padding at `shortcut_stride`, whose output has the
 * convolution's output shape.  This is the residual add of a bottleneck
 * block with a projection shortcut, folded together with the projection
 * into the convolution that produces the add's other operand (layer fusion,
 * Sec. III-A): one layer of two inputs whose routines compute both products
 * in one reduction (implicit GEMM on the LDS-DMA tiles, 16-bit channel-vector
 * layouts with C and C2 multiples of the tile depth) or, in any layout and
 * dtype, as the projection followed by the convolution with a residual
 * (direct routine, two launches and a workspace).  weight: OIHW [K][C][R][S],
 * shortcut_weight [K][C2] in the run dtype, host memory, copied; biases
 * float32 [K] or NULL = zeros (the two are summed in float64 and rounded
 * once to float32).
 * Errors: SN_E_INVALID (unknown ids, not CONV2D, groups != 1, stride < 1,
 * missing weights), SN_E_SHAPE (the shortcut projection does not give the
 * output's batch and size), SN_E_UNSUPPORTED, SN_E_STATE, SN_E_DEVICE as for
 * sn_add_layer. */
int sn_add_projected_conv(sn_graph* g, const sn_layer_desc* d, int32_t input, int32_t shortcut,
                          int32_t shortcut_stride, const void* weight, const float* bias,
                          const void* shortcut_weight, const float* shortcut_bias, int32_t* out_id);

/* Adds a further net input (multi-input nets, Sec. IV-E): an input layer
 * carrying the caller's tensor N x c x h x w (N of the graph, run dtype,
 * NCHW), with one routine of time 0.  The paper joins the inputs of such a
 * net with a zero-cost auxiliary input layer; layer 0 (the first input)
 * plays that role, joined to every further input by an edge that carries no
 * data and costs nothing.  Input k (0 = the graph's own) is the k-th tensor
 * of sn_run_mimo.  *out_id receives the layer id.
 * Errors: SN_E_INVALID (non-positive dims), SN_E_UNSUPPORTED (a tensor of
 * 2 GiB or more), SN_E_STATE (after selection), SN_E_DEVICE. */
int sn_add_input(sn_graph* g, int32_t c, int32_t h, int32_t w, int32_t* out_id);

/* Marks a layer as a net output (multi-output nets, Sec. IV-E); outputs are
 * numbered in marking order and delivered in NCHW, run dtype, by
 * sn_run_mimo.  Without any mark the last added layer is the one output.
 * The implicit auxiliary output layer merges all outputs; each output's edge
 * into it pays its conversion to the run-dtype NCHW schema.  Every layer
 * must reach an output (else selection fails with SN_E_INVALID).
 * Errors: SN_E_INVALID (unknown layer, an input layer, marked twice),
 * SN_E_STATE (after selection). */
int sn_mark_output(sn_graph* g, int32_t layer);

/* Number of net inputs and outputs (either pointer may be NULL). */
int sn_num_io(const sn_graph* g, int32_t* n_inputs, int32_t* n_outputs);

/* Unit profiling (Sec. III-C): times every routine of every layer on
 * scratch tensors of the layer's real shape, and every layout converter on
 * every edge (both directions of every schema pair), after warmup runs, as
 * the mean time of reps back-to-back runs.  HIP events are tied to the
 * start of the first run's first kernel dispatch and the end of the last
 * run's last one (hipExtLaunchKernelGGL), so host launch latency and the
 * events' own dispatch gaps are amortised over the block.  Identical layer
 * signatures and converter shapes are timed once.  With SN_OPT_FLUSH > 0 the
 * costs are cache-cold instead: before each of the reps runs an untimed
 * kernel writes that many bytes of scratch, each run is timed on its own, and
 * the cost is the median (warm and cold costs are cached apart).  Synchronous.
 * Errors: SN_E_STATE (no layers), SN_E_INVALID (reps < 1 or warmup < 0),
 * SN_E_DEVICE (host-only graph, HIP error). */
int sn_profile(sn_graph* g, int32_t warmup, int32_t reps, void* hip_stream);

/* Selects the routine path (Sec. IV) and compiles the execution plan
 * (buffers, converters, launch list).  See sn_select_mode.
 * Errors: SN_E_STATE (no costs), SN_E_UNSUPPORTED (a layer has no routine of
 * finite cost in any allowed schema), SN_E_INVALID (bad mode/layout/algo),
 * SN_E_INTERNAL (the dynamic program found inconsistent subpaths). */
int sn_select_path(sn_graph* g, int32_t mode, int32_t layout, int32_t algo);
/* (SN_SELECT_FIXED uses the run dtype, or the lowest allowed dtype when the
 * run dtype is not among SN_OPT_DTYPES.) */

/* Sets the routine path explicitly: routine_ids[i] is the routine id of
 * layer i for i = 0 .. n-1 (n = number of layers including the input).
 * Errors: SN_E_INVALID (wrong n or unknown id), SN_E_STATE. */
int sn_set_path(sn_graph* g, const int32_t* routine_ids, int32_t n);

/* Enqueues inference on the stream; asynchronous.  d_in: device tensor
 * N x C x H x W (NCHW, run dtype); d_out: device tensor of the output
 * layer's shape in NCHW (N x K for a net ending in FC or GAP).
 * Errors: SN_E_STATE (no plan), SN_E_INVALID (a net with several inputs or
 * outputs: use sn_run_mimo), SN_E_DEVICE (host-only graph, HIP error). */
int sn_run(sn_graph* g, const void* d_in, void* d_out, void* hip_stream);

/* sn_run for nets with several inputs and outputs: d_ins[k] is input k
 * (NCHW, run dtype, shape of its input layer), d_outs[k] output k (NCHW,
 * run dtype, shape of the k-th output layer); n_in and n_out must equal the
 * net's counts (sn_num_io).  Asynchronous on the stream.
 * Errors: SN_E_STATE (no plan), SN_E_INVALID (counts, null pointers),
 * SN_E_DEVICE. */
int sn_run_mimo(sn_graph* g, const void* const* d_ins, int32_t n_in, void* const* d_outs, int32_t n_out,
                void* hip_stream);

/* sn_run without allocation, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * it).  The same launches as sn_run on the same selected plan, with the
 * plan's intermediate tensors and workspaces (split-reduction partial sums,
 * Winograd transforms) placed in the library's static per-device region of
 * 64 MiB instead of the plan's own memory; the call itself allocates nothing
 * and enqueues nothing but kernels (no memset, no copy), so results are
 * identical to sn_run's.  Every call on one GPU shares that GPU's region, and
 * the region keeps the last call's contents (no routine relies on it being
 * zero): calls that overlap in time on one GPU (different streams, different
 * threads, or different graphs without ordering between them) race and give
 * undefined results.  d_in / d_out as for sn_run.
 * Errors: SN_E_STATE (no plan), SN_E_UNSUPPORTED (the plan needs more than
 * the 64 MiB region, e.g. ResNet-50 at batch 32: use sn_run), SN_E_DEVICE. */
int sn_run_noalloc(sn_graph* g, const void* d_in, void* d_out, void* hip_stream);

/* Like sn_run, but enqueues every layer's launches (its routine plus the
 * converters feeding it) reps times back to back, then synchronises and
 * writes each layer's mean time per repetition to layer_ms[0..n-1] (layer 0
 * gets 0).  HIP events are tied to the start of a layer's first kernel
 * dispatch and the end of its last (hipExtLaunchKernelGGL), so host launch
 * latency and the events' own dispatch gaps are amortised over reps.  Every
 * launch writes buffers distinct from the ones it reads, so d_out holds the
 * same result as after sn_run.  Used to attribute time per routine.  With
 * SN_OPT_FLUSH > 0 a device buffer of that many bytes is written before each
 * layer's repetitions (outside the timed launches), so with reps = 1 the
 * times are cache-cold ones; the buffer is allocated and freed by the call.
 * Errors: as sn_run; SN_E_INVALID if n is not the number of layers or reps
 * is outside 1..10000. */
int sn_run_timed(sn_graph* g, const void* d_in, void* d_out, void* hip_stream, int32_t reps,
                 float* layer_ms, int32_t n);

/* Copies the stored output of layer (1 .. n-1) as its selected routine wrote
 * it -- in the routine's layout (the schema of Sec. III-C), NC8HW8 with its
 * channels padded to a multiple of 8 -- from the plan's memory into the
 * caller's device buffer d_dst (cap bytes), as an asynchronous
 * device-to-device copy on the stream, with no arithmetic.  Read after an
 * sn_run on the same stream.  *bytes receives the stored size and *layout the
 * layout value (either may be NULL); d_dst = NULL only queries them.
 * Intermediate layers keep their output after the run only with SN_OPT_KEEP =
 * 1; the last layer's output stays until the next run.
 * Errors: SN_E_STATE (no plan, or an intermediate layer without
 * SN_OPT_KEEP), SN_E_INVALID (layer out of range), SN_E_NOMEM (cap smaller
 * than the stored size), SN_E_UNSUPPORTED (the layer stores straight into the
 * caller's output tensor of sn_run), SN_E_DEVICE. */
int sn_layer_output(const sn_graph* g, int32_t layer, void* d_dst, size_t cap, size_t* bytes,
                    int32_t* layout, void* hip_stream);

/* The kernel launches one sn_run of the selected plan makes, in order:
 * layer_of_launch[i] is the layer launch i belongs to (the adapt routines
 * feeding a layer count as that layer's; a routine may launch more than one
 * kernel).  Nothing is launched: the plan's steps are walked with launches
 * counted only.  Lets a kernel trace of sn_run (for instance per-dispatch
 * hardware counters) be attributed to layers.  *n receives the count;
 * layer_of_launch = NULL only queries it.
 * Errors: SN_E_STATE (no plan), SN_E_NOMEM (cap below the count),
 * SN_E_DEVICE (host-only graph). */
int sn_plan_launches(const sn_graph* g, int32_t* layer_of_launch, int32_t cap, int32_t* n);

/* Integrated profiling (Sec. III-C): the unit-profiled table filters the
 * routine patterns down to a short list of whole paths, and those are timed
 * end to end, which sees what a sum of isolated layer times misses (cache
 * reuse between layers, launch gaps).  Candidates, in this order, identical
 * paths kept once:
 *   1. the DPRS path over the allowed schemas (SN_OPT_LAYOUTS x SN_OPT_DTYPES);
 *   2. the DPRS path with layers restricted to each non-empty proper subset
 *      of the allowed layouts, subsets in increasing bitmask order;
 *   3. with several dtypes allowed, the DPRS path restricted to each one
 *      dtype (the single-precision tunings, in sn_dtype order);
 *   4. every fixed path (SN_SELECT_FIXED) of an allowed layout and algorithm
 *      (run dtype, or the lowest allowed dtype if it is not allowed).
 * A candidate that does not exist (some layer has no routine in the subset)
 * is skipped.  Each candidate's plan is compiled and run on a zero-filled
 * scratch input: warmup runs, then two rounds (candidate order, then
 * reverse) of reps back-to-back runs between HIP events on the stream; its
 * measured time is the smaller block mean.  The fastest candidate (the
 * earlier one on ties) is selected and its plan compiled, as after
 * sn_select_path.  Synchronous.  reps = 0 only enumerates the candidates
 * (measured time -1) and leaves the selection unchanged; this works on
 * host-only graphs.  *n_candidates (may be NULL) receives the count.
 * Errors: SN_E_STATE (no costs, no layers), SN_E_INVALID (warmup < 0, reps
 * outside 0..10000), SN_E_DEVICE (reps > 0 on a host-only graph, HIP
 * error); on an error during timing no path is selected. */
int sn_profile_integrated(sn_graph* g, int32_t warmup, int32_t reps, void* hip_stream,
                          int32_t* n_candidates);

/* Candidate idx of the last sn_profile_integrated: routine id per layer
 * (routine_ids may be NULL; else n = number of layers), model time T(S) under
 * the unit-profiled table, measured end-to-end ns per run (-1 if not
 * measured), and kind_ab[3] = {kind, a, b}: kind 0 = DPRS over the layout
 * bitmask a and the dtype bitmask b, kind 1 = fixed path of layout a and
 * algorithm b.  Any output
 * pointer may be NULL.
 * Errors: SN_E_INVALID (idx out of range, n mismatch). */
int sn_integrated_candidate(const sn_graph* g, int32_t idx, int32_t* routine_ids, int32_t n,
                            int64_t* model_ns, int64_t* measured_ns, int32_t* kind_ab);

/* In-path refinement of the selected path: integrated profiling (Sec.
 * III-C) applied one layer at a time.  A routine's unit-profiled time is
 * taken with its input and weights hot in the caches; inside the net its
 * input was just written by the layer before and its weights were last read
 * a whole run earlier, and near-tied routines can rank differently there.
 * For each layer, in order, the selected routine and the other routines of
 * its schema whose unit-profiled time is at most (1 + tol_permille / 1000)
 * times the selected one's (the max_alts fastest of them) are each run
 * inside the whole path with only that layer's routine swapped (adapts are
 * unchanged: the schema is the same), on a zero-filled scratch input; the
 * layer's time is read from HIP events tied to its first and last launch,
 * the median over reps runs after two warm-up runs.  The fastest routine,
 * when it beats the selected one by more than 2 % and does so again in a
 * second pair of timings, replaces it for the later layers' trials.  Finally the selected and the refined path are timed end to end
 * (four alternating rounds of 20 runs, block means, the median of each) and
 * the faster is kept; its plan is compiled, as after sn_select_path.
 * *n_changed (may be NULL) receives the number of layers whose routine
 * changed (0 when the refined path lost or nothing changed).  Synchronous.
 * Errors: SN_E_STATE (no costs, no selected path), SN_E_INVALID
 * (tol_permille outside 0..1000, max_alts outside 1..16, reps outside
 * 1..1000), SN_E_DEVICE (host-only graph, HIP error); after an error
 * during timing the previous path is selected again but has no plan (select
 * or set the path again before running). */
int sn_refine_in_path(sn_graph* g, int32_t tol_permille, int32_t max_alts, int32_t reps, void* hip_stream,
                      int32_t* n_changed);

/* Cost table as JSON (the profiling data of Sec. IV-A: T(r) per routine,
 * adapt times per edge and schema pair), all times int64 ns, -1 = no
 * routine / unavailable:
 *   {"dtype":..., "layers":[{"id":i,"type":t,"routines":[{"rid":..,"layout":..,
 *     "algo":..,"param":..,"dtype":..,"schema":..,"ns":..}]}],
 *    "edges":[{"from":j,"to":i,"ns":M}]}
 * M is 3 x 3, indexed by layout, when the graph computes in its run dtype
 * only, else 9 x 9, indexed by schema (dtype * 3 + layout).  The implicit
 * auxiliary output layer appears as the last layer with one NCHW routine (run
 * dtype) of time 0, with an edge from the net output layer.
 * A routine built from sub-layers (a childnet, Sec. III-D: the three-kernel
 * Winograd routine is wgenc -> wgconv -> wgdec, one wgconv sub-routine per
 * GEMM tile) also carries
 *   "child":{"layers":[names],"routines":[[names] per sub-layer],
 *            "ns":[[times] per sub-layer],"path":[chosen sub-routine per sub-layer]}
 * sn_profile times every sub-routine on its own, and the routine's "ns" is
 * the DPRS optimum over its sub-layers (Sec. IV-F: the algorithm is applied
 * to a childnet first).  sn_set_costs recomputes that optimum, and the path
 * the routine runs with, from "child" whenever any sub-routine time there is
 * known; with every one unknown (-1) the routine keeps the listed "ns".
 * sn_get_costs writes at most cap bytes including the terminating NUL; if
 * cap is too small it returns SN_E_NOMEM with *len = required size.
 * sn_set_costs replaces the table (host-only graphs included); it must list
 * exactly the graph's layers, routines and edges.
 * Errors: SN_E_INVALID (malformed or mismatched JSON), SN_E_NOMEM. */
int sn_get_costs(const sn_graph* g, char* json, size_t cap, size_t* len);
int sn_set_costs(sn_graph* g, const char* json);

/* Selected routine id per layer (n = number of layers) and the model time
 * T(S) = sum of routine and adapt times of the selected path (Definition 1).
 * Errors: SN_E_STATE (no path), SN_E_INVALID (n mismatch). */
int sn_get_path(const sn_graph* g, int32_t* routine_ids, int32_t n, int64_t* total_ns);

/* Number of layers including the input layer (the implicit output layer is
 * not counted). */
int sn_num_layers(const sn_graph* g, int32_t* n);

/* Number of routines of a layer, and their descriptions. */
int sn_num_routines(const sn_graph* g, int32_t layer, int32_t* count);
int sn_routine_info(const sn_graph* g, int32_t layer, int32_t idx, sn_routine_desc* out);

/* Output shape N, C, H, W of a layer (logical NCHW). */
int sn_layer_shape(const sn_graph* g, int32_t layer, int32_t* nchw);

/* Statistics of the last DPRS run for one layer: number of (schema,
 * constraint) states kept after the layer (Sec. IV-C, IV-D) and number of
 * candidate unions evaluated at it (the "fastest" terms of Eq. 3). */
int sn_dp_stats(const sn_graph* g, int32_t layer, int64_t* n_states, int64_t* n_candidates);

void sn_graph_destroy(sn_graph* g);
const char* sn_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SOFTNEURO_H */
