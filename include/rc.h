/* rc.h - C ABI of the schedule-parameterised contraction library (librc).
 *
 * The paper (Sec. 2, Eq. 1) states compiler optimisation as: an input
 * program P0 that is one layer of a network, a set M of semantics-preserving
 * transformations, a sequence of at most T of them, and an objective f
 * measured on the target.  This library is that statement for MI355X
 * (gfx950):
 *   - P0 is an operator descriptor (rc_op_desc): one of five dense
 *     contractions with fused epilogues, the layer kinds of Sec. 4.1
 *     (attention, MoE, convolution, gated MLP) plus the fp32 contraction of
 *     the App. A example module;
 *   - a program variant is a schedule (rc_schedule): one integer per knob;
 *   - a transformation (rc_transform) sets one knob, named after the
 *     transformation classes of App. A (TileSize, Parallel,
 *     ComputeLocation, Unroll) plus Vectorize and Layout (Sec. 1);
 *   - f is the measured throughput of the HIP kernels the schedule
 *     instantiates (rc_time), and the search of Sec. 3.2 runs over it
 *     (rc_search_*).
 *
 * Conventions for every call:
 *   - Functions return rc_status; RC_OK is 0.  On failure a thread-local
 *     message is available from rc_last_error().  No C++ exception and no
 *     abort crosses this interface.
 *   - Structs start with uint32_t struct_size, which callers set to
 *     sizeof(the struct) (rc_*_init helpers do it).
 *   - The library never allocates, frees or retains caller tensors.  Device
 *     pointers are caller-owned, must stay valid until the work queued on the
 *     stream has finished, must be 16-byte aligned and contiguous in the
 *     layout stated for the operator.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Launch calls only enqueue work; they never synchronise the host.
 *   - Illegal schedules are rejected on the host before any compilation or
 *     GPU work.
 */
#ifndef RC_H
#define RC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum rc_status {
    RC_OK = 0,
    RC_ERR_INVALID_ARGUMENT = 1,
    RC_ERR_ILLEGAL_SCHEDULE = 2,
    RC_ERR_UNSUPPORTED = 3,
    RC_ERR_COMPILE = 4,
    RC_ERR_HIP = 5,
    RC_ERR_OUT_OF_MEMORY = 6,
    RC_ERR_MISALIGNED = 7,
    RC_ERR_BUDGET = 8
} rc_status;

/* Human-readable name of a status code (static storage). */
const char *rc_status_str(rc_status s);
/* Detail text of the last failing call on this thread (empty if none). */
const char *rc_last_error(void);

/* ------------------------------------------------------------------ */
/* Operators: the input program P0 (Sec. 2; App. A)                    */
/* ------------------------------------------------------------------ */

typedef enum rc_op_kind {
    /* C[M][N] = A[M][K] B[K][N], fp32 in and out (the App. A contraction).
     * dim = {M, N, K}.  Inputs: in[0] = A [M][K]; in[1] = B stored [K][N]
     * (layout 0) or [N][K] (layout 1).  Output: out[0] = C [M][N]. */
    RC_OP_GEMM_F32 = 1,
    /* Softmax attention, bf16 Q/K/V/O [B][H][S][D], scale 1/sqrt(D), fp32
     * scores and softmax (the self-attention layers of Sec. 4.1).
     * dim = {B, H, S, D}; flags & RC_FLAG_CAUSAL selects the top-left aligned
     * causal mask (key j visible to query i iff j <= i).
     * in[0] = Q, in[1] = K, in[2] = V; out[0] = O. */
    RC_OP_ATTENTION = 2,
    /* Gated MLP (the MLP layer of Sec. 4.1):
     *   out = bf16( bf16( SiLU(X Wg) * (X Wu) ) Wd ), fp32 accumulation.
     * dim = {T, Hd, I}.  in[0] = X [T][Hd]; in[1] = Wg, in[2] = Wu stored
     * [Hd][I] (up.layout 0) or [I][Hd] (up.layout 1); in[3] = Wd stored
     * [I][Hd] (down.layout 0) or [Hd][I] (down.layout 1); out[0] = [T][Hd]. */
    RC_OP_GATED_MLP = 3,
    /* (Schedules of the gated MLP have the knobs up.tail / down.tail: with
     * 1, the column tiles of a last, partial round of workgroups run as a
     * second launch with half-height tiles; with 2, as full tiles whose K
     * range is cut in two, followed by a kernel that adds the two fp32
     * partial sums (and, for the gate/up GEMM, applies SiLU(g) * u).  The
     * knob down.split (1, 2, 4) cuts the down projection's K range over
     * that many workgroups per output tile, followed by a summing kernel.
     * rc_plan_kernels counts every launch.) */
    /* Routed mixture of gated-MLP experts (the MoE layer of Sec. 4.1):
     *   out[t] = bf16( sum_s w[t][s] * expert_{ids[t][s]}(X[t]) ),
     *   expert_e(x) = bf16( SiLU(x Wg[e]) * (x Wu[e]) ) Wd[e].
     * dim = {T, Hd, E, I, topk}.  in[0] = X [T][Hd] bf16; in[1] = ids
     * [T][topk] int32 in [0, E); in[2] = w [T][topk] fp32; in[3] = Wg,
     * in[4] = Wu stored [E][Hd][I] (up.layout 0) or [E][I][Hd] (1);
     * in[5] = Wd stored [E][I][Hd] (down.layout 0) or [E][Hd][I] (1);
     * out[0] = [T][Hd] bf16.  Routing (ids, w) is an input.
     * (Its schedules have the knobs up.skip / down.skip: with 1, an
     * expert's last, partial M tile skips the MFMAs of its empty row blocks;
     * the result is the same.) */
    RC_OP_MOE = 4,
    /* 2-D convolution, stride 1, zero padding, bias and SiLU (the
     * convolution layer of Sec. 4.1), as an implicit GEMM:
     *   y = bf16( SiLU( conv(x, w) + bias ) ),
     * or y = bf16( conv(x, w) + bias ) with flags & RC_FLAG_NO_ACT (the
     * same contraction without the activation; with 1 x 1 filters and no
     * padding it is a plain bf16 GEMM, and with integer-valued inputs every
     * output is exact in any accumulation order).
     * dim = {N, H, W, C, K, R, S, pad}.  in[0] = x [N][H][W][C] bf16;
     * in[1] = w stored [K][R][S][C] (layout 1) or [R][S][C][K] (layout 0)
     * bf16; in[2] = bias [K] fp32; out[0] = y [N][P][Q][K] bf16 with
     * P = H + 2 pad - R + 1, Q = W + 2 pad - S + 1. */
    RC_OP_CONV2D = 5
} rc_op_kind;

#define RC_FLAG_CAUSAL 1   /* RC_OP_ATTENTION only */
#define RC_FLAG_NO_ACT 2   /* RC_OP_CONV2D only: bias, no SiLU */
#define RC_MAX_DIMS 8

typedef struct rc_op_desc {
    uint32_t struct_size;
    int32_t kind;              /* rc_op_kind */
    int64_t dim[RC_MAX_DIMS];  /* meaning per kind, unused entries 0 */
    int32_t flags;
    int32_t reserved;
} rc_op_desc;

/* Fill *d for `kind` with `ndims` dimensions.  Checks the kind, the number
 * of dimensions, that every dimension is positive (pad may be 0) and that
 * `flags` holds only flags defined for the kind; RC_ERR_INVALID_ARGUMENT
 * otherwise. */
rc_status rc_op_init(rc_op_desc *d, int32_t kind, const int64_t *dims, int32_t ndims,
                     int32_t flags);

/* Algorithmic work of one execution of the operator.
 * FLOPs count 2 per multiply-add of the contraction only (for causal
 * attention only visible query/key pairs; for MoE only routed rows);
 * bytes count compulsory HBM traffic: each input read once and each output
 * written once.  Negative on an invalid descriptor. */
double rc_op_flops(const rc_op_desc *d);
double rc_op_bytes(const rc_op_desc *d);
/* Published MI355X peak that bounds the operator: fp32 MFMA (157.3 TFLOP/s)
 * for RC_OP_GEMM_F32, bf16 MFMA (2516.6 TFLOP/s) otherwise, in FLOP/s;
 * and HBM bandwidth (8.0e12 B/s). */
double rc_peak_flops(const rc_op_desc *d);
double rc_peak_bytes_per_s(void);

/* ------------------------------------------------------------------ */
/* Schedules and transformations (Sec. 2, Eq. 1; App. A)              */
/* ------------------------------------------------------------------ */

#define RC_MAX_KNOBS 32

typedef struct rc_schedule {
    uint32_t struct_size;
    int32_t nknobs;
    int32_t knob[RC_MAX_KNOBS];
} rc_schedule;

/* One transformation: set knob `knob` to `value`. */
typedef struct rc_transform {
    int32_t knob;
    int32_t value;
} rc_transform;

/* Knob table of an operator: the count, each knob's name ("tile_m",
 * "up.tile_n", ...), its transformation class ("TileSize", "Parallel",
 * "Vectorize", "Unroll", "ComputeLocation", "Layout") and its allowed
 * values.  Names point to static storage. */
int32_t rc_knob_count(const rc_op_desc *d);
const char *rc_knob_name(const rc_op_desc *d, int32_t knob);
const char *rc_knob_class(const rc_op_desc *d, int32_t knob);
rc_status rc_knob_values(const rc_op_desc *d, int32_t knob, int32_t *vals, int32_t cap,
                         int32_t *n);

/* The untransformed program P0: smallest tiles, one wave, one stage,
 * narrowest vectors, no unrolling, unfused epilogue, canonical layout.  It is
 * legal for every operator this library accepts, and it is the denominator
 * of reported speedups (Sec. 4.2). */
rc_status rc_default_schedule(const rc_op_desc *d, rc_schedule *out);

/* Legality check, host only.  Returns RC_OK or RC_ERR_ILLEGAL_SCHEDULE with
 * the first violated rule written to `why` (may be NULL).  Tiles may end
 * partially over the extents that vary with the input (every fp32 GEMM
 * dimension; the rows of the bf16 GEMMs: tokens, routed rows, output
 * pixels; the attention sequence length): such tiles are predicated, and a
 * tile twice the extent it covers is rejected as redundant.  Weight extents
 * (the N and K of the bf16 GEMMs, the channels of the convolution) must be
 * whole tiles.  (App. A's perfect-tile decisions.) */
rc_status rc_validate(const rc_op_desc *d, const rc_schedule *s, char *why, size_t why_len);

/* Apply one transformation: out = t(in).  If the result is illegal, returns
 * RC_ERR_ILLEGAL_SCHEDULE and leaves *out untouched.  in == out allowed. */
rc_status rc_apply(const rc_op_desc *d, const rc_schedule *in, const rc_transform *t,
                   rc_schedule *out);

/* The action set at a state: every transformation whose result is legal and
 * differs from `at`.  Writes min(count, cap) entries and the full count. */
rc_status rc_enumerate(const rc_op_desc *d, const rc_schedule *at, rc_transform *buf,
                       size_t cap, size_t *n);

/* Parse a textual transformation proposal such as "TileSize(up.tile_m=128)"
 * or "Unroll(unroll=2)".  Only a known class with one of its own knobs and
 * an allowed value is accepted (Sec. 3.1, proposal validation); anything
 * else returns RC_ERR_INVALID_ARGUMENT. */
rc_status rc_parse_transform(const rc_op_desc *d, const char *text, rc_transform *out);

/* "name=value,name=value,..." for logs; from_string accepts the same form
 * (missing knobs keep their default). */
rc_status rc_schedule_to_string(const rc_op_desc *d, const rc_schedule *s, char *buf,
                                size_t len);
rc_status rc_schedule_from_string(const rc_op_desc *d, const char *text, rc_schedule *out);
uint64_t rc_schedule_hash(const rc_schedule *s);

/* ------------------------------------------------------------------ */
/* Plans: a compiled program variant                                  */
/* ------------------------------------------------------------------ */

typedef struct rc_plan rc_plan;

/* Validate, generate the kernels' source for this schedule, compile them for
 * gfx950 with hipRTC (or load the cached code object) and load them on the
 * current device.  A variant whose kernels need scratch memory (register
 * spills) is rejected as RC_ERR_ILLEGAL_SCHEDULE ("spill").  The plan is
 * immutable and may be launched concurrently on different streams. */
rc_status rc_plan_create(const rc_op_desc *d, const rc_schedule *s, rc_plan **out);
void rc_plan_destroy(rc_plan *p);

/* Compile (without loading) the variants of n schedules into the code-object
 * cache using `nthreads` host threads; needs no GPU.  status[i] receives each
 * result (may be NULL). */
rc_status rc_precompile(const rc_op_desc *d, const rc_schedule *s, int32_t n, int32_t nthreads,
                        rc_status *status);

/* Directory of the on-disk code-object cache (set before the first compile;
 * NULL restores the default: $RC_CACHE_DIR, else the package's jit_cache). */
rc_status rc_set_cache_dir(const char *dir);

/* Bytes of device workspace a launch needs (0 if none).  The caller
 * allocates it; its contents need not be initialised. */
rc_status rc_plan_workspace(const rc_plan *p, size_t *bytes);
/* Number of kernels one launch enqueues, and the index of the one doing
 * most of the FLOPs (the contraction). */
rc_status rc_plan_kernels(const rc_plan *p, int32_t *nkernels, int32_t *dominant);

/* Algorithmic FLOPs of kernel `kernel` of a launch (2 per multiply-add of
 * the contraction it computes; 0 for routing, combine, reduction and
 * elementwise kernels).  The kernels' FLOPs add up to rc_op_flops. */
rc_status rc_plan_kernel_flops(const rc_plan *p, int32_t kernel, double *flops);

/* Byte offset and size of a named part of the workspace, so that a caller
 * can read intermediate results after a launch (each part starts on a
 * 256-byte boundary).  Parts by operator:
 *   RC_OP_MOE: "offsets" int32 [E + 1] (first permuted row of each expert,
 *     offsets[E] = T * topk); "perm" int32 [T * topk] (permuted row ->
 *     token * topk + slot, rows of one expert in increasing token * topk +
 *     slot order); "pos" int32 [T * topk] (the inverse of perm);
 *     "tile_up" / "tile_down" int32 [E + 1] (first M tile of each expert in
 *     the gate/up and down GEMMs: exclusive prefix sums of
 *     ceil(count_e / tile_m)); "hidden" bf16 [T * topk][I] (permuted
 *     rows); "expert_out" bf16 [T * topk][Hd] (permuted rows);
 *     "block_counts" int32 [ceil(T * topk / 1024)][E] (routed rows per
 *     block of 1024 consecutive rows and expert);
 *   RC_OP_GATED_MLP: "hidden" bf16 [T][I]; with K splits "down.partials"
 *     fp32 [down.split][T][Hd], "up.tail.gate" / "up.tail.up" fp32
 *     [2][T][tail columns], "down.tail.partials" fp32 [2][T][tail columns];
 *   unfused epilogues: "gate.f32", "up.f32" or "pre.f32" (fp32 [rows][cols]);
 *   RC_OP_ATTENTION with chunk > 0: "partials"; RC_OP_GEMM_F32 streaming
 *   stage with splits > 1: "splitk.partials".
 * RC_ERR_INVALID_ARGUMENT if the plan has no part of that name.  (The
 * routing preparation of the MoE layer of Sec. 4.1 is integer index work:
 * these parts let it be checked exactly.) */
rc_status rc_plan_buffer(const rc_plan *p, const char *name, size_t *offset, size_t *bytes);

/* Resources of one kernel of a variant, read from its gfx950 code object. */
typedef struct rc_kernel_info {
    uint32_t struct_size;
    char name[48];            /* kernel symbol */
    int32_t grid;             /* workgroups per launch */
    int32_t block;            /* threads per workgroup */
    int32_t lds_bytes;        /* static LDS per workgroup */
    int32_t vgprs;            /* VGPRs per lane, architectural + accumulation */
    int32_t agprs;            /* of which accumulation VGPRs (AGPRs) */
    int32_t sgprs;
    int32_t scratch_bytes;    /* private segment per lane (0 unless spilling) */
    int32_t waves_per_simd;   /* occupancy bound from registers and LDS */
} rc_kernel_info;

/* Compile (or fetch from the cache) the kernels of a schedule and report
 * their launch shape and resources, read from each kernel's own entry in
 * the code object's metadata; needs no GPU.  Writes min(count, cap)
 * entries and the count. */
rc_status rc_describe(const rc_op_desc *d, const rc_schedule *s, rc_kernel_info *buf,
                      int32_t cap, int32_t *n);

typedef struct rc_args {
    uint32_t struct_size;
    const void *in[8];
    void *out[2];
} rc_args;

/* Enqueue one execution of the operator on `stream`.  Checks pointers
 * (non-NULL, 16-byte aligned) and the workspace size; never synchronises. */
rc_status rc_launch(const rc_plan *p, const rc_args *a, void *workspace, size_t ws_bytes,
                    void *stream);

/* Enqueue one execution with a HIP event recorded before and after each
 * kernel: events[0..nkernels] (caller-created hipEvent_t, passed as void*).
 * The duration of kernel i is elapsed(events[i], events[i+1]). */
rc_status rc_launch_timed(const rc_plan *p, const rc_args *a, void *workspace,
                          size_t ws_bytes, void *stream, void **events, int32_t nevents);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): rc_launch
 * with the workspace taken from a static device array inside the library
 * instead of a caller buffer.  The caller still passes inputs and outputs.
 * The array holds rc_static_scratch_bytes() bytes (64 MiB) on each device
 * the library runs on, from the first call on that device until the process
 * ends; a plan whose workspace is larger is rejected with
 * RC_ERR_OUT_OF_MEMORY before any GPU work (use rc_launch).  The call
 * allocates nothing: no hipMalloc, hipFree or other allocating routine
 * (its first call on a device looks the array's address up once).  Every
 * call on one device shares that device's array and leaves its contents
 * behind; calls that overlap on one device (concurrent streams or host
 * threads) race, so the caller serialises them.  No kernel needs the
 * array cleared. */
rc_status rc_launch_static(const rc_plan *p, const rc_args *a, void *stream);
size_t rc_static_scratch_bytes(void);

typedef struct rc_time_opts {
    uint32_t struct_size;
    int32_t warmup;   /* untimed launches first (default 3) */
    int32_t repeat;   /* timed launches (default 20) */
    int32_t flush;    /* 1: overwrite a 512 MiB buffer before each timed
                         launch so no operand is cache-resident */
    int32_t reserved;
} rc_time_opts;

typedef struct rc_timing {
    uint32_t struct_size;
    int32_t nkernels;
    double median_ms, min_ms, mean_ms, q1_ms, q3_ms;
    double tflops;        /* rc_op_flops / median */
    double gbps;          /* rc_op_bytes / median */
    double frac_flops;    /* tflops / peak */
    double frac_bytes;    /* gbps / HBM peak */
    double kernel_ms[8];  /* median duration of each kernel (the first 8) */
} rc_timing;

void rc_time_opts_init(rc_time_opts *o);

/* Time a plan (the objective f of Sec. 2, measured on the target):
 * `warmup` launches, then `repeat` launches each bracketed by HIP events on
 * `stream`; with `flush`, a 512 MiB device buffer (twice the MI355X's
 * 256 MB last-level cache) is overwritten before each timed launch, outside
 * the brackets.  The flush buffer is allocated on the current device at its
 * first flushed timing and kept for later calls (rc_time_release frees it).
 * Returns the median, quartiles, minimum and mean of the timed launches,
 * the median duration of each kernel, and the derived rates against
 * rc_op_flops / rc_op_bytes and the peaks.  Synchronises the stream; every
 * event it created is destroyed on every path. */
rc_status rc_time(const rc_plan *p, const rc_args *a, void *workspace, size_t ws_bytes,
                  void *stream, const rc_time_opts *o, rc_timing *out);

/* Free the flush buffers rc_time allocated (on every device it used).  The
 * caller makes sure no rc_time call is running; a later flushed rc_time
 * allocates again. */
rc_status rc_time_release(void);

/* ------------------------------------------------------------------ */
/* Search (Sec. 3.2): UCT tree search, random sampling, exhaustive     */
/* ------------------------------------------------------------------ */

typedef enum rc_policy {
    RC_POLICY_RANDOM = 0,      /* random legal transformation sequences */
    RC_POLICY_UCT = 1,         /* MCTS with UCT selection (Sec. 3.2) */
    RC_POLICY_EXHAUSTIVE = 2   /* every legal schedule of the listed space */
} rc_policy;

/* Evaluate one schedule (the objective f).  Return 0 and set *reward (>= 0,
 * larger is better) for a valid sample; nonzero marks the schedule invalid
 * (compile failure, spill, launch error), which costs no budget. */
typedef int32_t (*rc_eval_fn)(void *user, const rc_schedule *s, double *reward);

/* Optional transformation proposer for expansion (Sec. 3.1): writes a
 * proposal text for the node `at` (whose ancestors' schedules are
 * parent/grandparent, NULL at the root).  The text holds alternatives
 * separated by ';' or newlines, tried in order; each alternative is one
 * transformation or a sequence of them joined by '+' (Sec. 3.1 proposes
 * sequences), parsed step by step with rc_parse_transform: steps that do
 * not parse are discarded, the others are applied in order (intermediate
 * schedules need not be legal) and the result becomes the new child if it
 * is legal and not yet in the tree.  When no alternative yields one, the
 * search samples a random legal transformation instead (a fallback). */
typedef int32_t (*rc_propose_fn)(void *user, const rc_schedule *at, const rc_schedule *parent,
                                 const rc_schedule *grandparent, char *buf, size_t len);

typedef struct rc_search_opts {
    uint32_t struct_size;
    int32_t policy;       /* rc_policy */
    int32_t budget;       /* valid samples to measure */
    int32_t horizon;      /* maximum sequence length T (default 12) */
    int32_t branching;    /* maximum children per node B (default 2) */
    double c;             /* UCT exploration constant (default sqrt(2)) */
    uint64_t seed;
    int32_t max_invalid;  /* stop after this many invalid samples (default 10 * budget) */
    int32_t reserved;
} rc_search_opts;

typedef struct rc_sample {
    rc_schedule schedule;
    double reward;
    int32_t valid;
    int32_t index;        /* valid-sample index (-1 if invalid) */
    double best_so_far;
} rc_sample;

typedef struct rc_search rc_search;

void rc_search_opts_init(rc_search_opts *o);
rc_status rc_search_create(const rc_op_desc *d, const rc_search_opts *o, rc_eval_fn eval,
                           void *eval_user, rc_search **out);
rc_status rc_search_set_proposer(rc_search *s, rc_propose_fn fn, void *user);
/* One iteration: select, expand, roll out, evaluate, back-propagate.
 * *done = 1 once the budget (or the space) is exhausted. */
rc_status rc_search_step(rc_search *s, int32_t *done);
rc_status rc_search_run(rc_search *s);
rc_status rc_search_best(const rc_search *s, rc_schedule *best, double *reward,
                         int32_t *sample_index);
/* All evaluations in order (valid and invalid). */
rc_status rc_search_history(const rc_search *s, rc_sample *buf, int32_t cap, int32_t *n);
/* Tree statistics of the root's children for tests: visits and cumulative
 * reward W of the node reached by applying t at the root (0s if absent). */
rc_status rc_search_node_stats(const rc_search *s, const rc_transform *path, int32_t len,
                               int32_t *visits, double *W);
/* Count of proposals that fell back to a random legal transformation. */
rc_status rc_search_fallbacks(const rc_search *s, int32_t *n);
void rc_search_destroy(rc_search *s);

#ifdef __cplusplus
}
#endif
#endif /* RC_H */
