/*
 * efsparse — error-feedback gradient sparsification on one AMD MI355X (gfx950).
 *
 * C ABI of the hot path of sparsified SGD with error feedback
 * (Foroutan Eghlidi & Jaggi, "Sparse Communication for Training Deep
 * Networks", Algorithm 1 and Section 3).  One worker step is
 *
 *     acc = g + e                      (Algorithm 1, accumulate step)
 *     q   = C(acc)                     (Algorithm 1, compress step; Section 3:
 *                                       top-k, random-k or block-random-k,
 *                                       layer-wise or global scope)
 *     e'  = acc with q's support set to +0.0
 *                                      (Section 3 worker steps / Algorithm 1:
 *                                       keep what was not sent)
 *
 * and the partner call sums W workers' messages into a dense vector in a fixed
 * worker order (Algorithm 1, aggregate step), averaged over W by default.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Sizes: d is the gradient length, 1 <= d < 2^31.  A layout splits [0, d)
 *    into n_seg contiguous segments (one per layer for layer-wise scope, one
 *    in total for global scope; Section 3, sparsification scope).
 *  - k per segment: k_l = clamp(floor(density * d_l + 0.5), 1, d_l), computed
 *    in IEEE double; K = sum of k_l.  Segment l's message entries occupy
 *    positions [P_l, P_l + k_l), P_l = k_0 + ... + k_{l-1}.
 *  - Sparse message (top-k, random-k): idx uint32[K] (global element indices,
 *    strictly ascending) and val float32[K] (acc at those indices, exact bits).
 *  - Block message (block-random-k): start uint32[n_seg] (segment-local start
 *    of the run) and val float32[K], val[P_l + t] = acc[o_l + (start_l + t)
 *    mod d_l], t = 0..k_l-1.
 *  - Memory: every pointer named g, e, acc, idx, val, start, out, ws is a
 *    device pointer owned by the caller; the library never allocates device
 *    memory and never synchronises the stream (ef_layout_bind excepted).
 *    g, e, acc and out must be 16-byte aligned (8-byte for a bf16 g); idx,
 *    val and start 4-byte aligned; ws 256-byte aligned.
 *  - Streams: `stream` is a hipStream_t (NULL = the null stream).  All work
 *    is enqueued on it, in order; results are ready when the stream is.
 *  - Aliasing: only where stated (acc may equal e in ef_accumulate; e may
 *    equal acc in ef_update).  Messages must not alias inputs.
 *  - Errors: argument errors are detected on the host before anything is
 *    enqueued and return a status below; launch failures return EF_EHIP.
 *    No call throws, exits or prints.
 *  - Threading: a bound layout is read-only and may be shared; concurrent
 *    calls need distinct workspaces (or the same stream).
 *  - Determinism: every output is bitwise reproducible for the same inputs,
 *    independent of launch timing (integer atomics only; no float atomics).
 */
#ifndef EFSPARSE_H
#define EFSPARSE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* status codes */
#define EF_OK 0
#define EF_EINVAL 1     /* null / misaligned pointer, bad dtype or kind, density outside (0,1],
                           block < 1, segment table not a strictly increasing partition of [0,d),
                           layout not bound */
#define EF_ERANGE 2     /* d == 0, d >= 2^31, n_seg < 1 or n_seg >= 2^24, W < 1 or W > 65535 */
#define EF_EWORKSPACE 3 /* ws_bytes smaller than ef_workspace_bytes() */
#define EF_EHIP 4       /* a HIP runtime or launch error */
#define EF_ENOMEM 5     /* host memory for a layout's tables (or the timing records) could not be
                           allocated; a layout whose ef_layout_tune failed this way is unusable */

/* gradient dtypes */
#define EF_F32 0
#define EF_BF16 1

/* workspace kinds for ef_workspace_bytes */
#define EF_OP_TOPK 0
#define EF_OP_RANDK 1
#define EF_OP_RANDBLOCK 2
#define EF_OP_AGG_SPARSE 3
#define EF_OP_AGG_BLOCK 4
#define EF_OP_AGG_SHARED 5
#define EF_OP_RANDK_PREP 6

/* message kinds */
#define EF_MSG_SPARSE 0
#define EF_MSG_BLOCK 1

/* tuning knobs for ef_layout_tune: they size the candidate sets and change speed only, never
   results (a segment whose candidates cannot contain the answer takes an exact whole-segment
   path) */
#define EF_TUNE_RANDK_SIGMA 0  /* random-k: candidate bound, standard deviations above k (default 6) */
#define EF_TUNE_RANDK_EXTRA 1  /* random-k: candidate bound, constant margin (default 32) */
#define EF_TUNE_TOPK_SIGMA 2   /* top-k: sampled threshold margin in standard deviations (default 6) */
#define EF_TUNE_TOPK_EXTRA 3   /* top-k: sampled threshold margin, constant part (default 8) */
#define EF_TUNE_TOPK_RETRY 4   /* top-k: 1 (default) lets a segment whose sampled candidates fall
                                  short re-collect them at a lower threshold over the whole device;
                                  0 sends it straight to the exact whole-segment path */
#define EF_TUNE_POOL 5         /* top-k / random-k workspace: scale (>= 0, default 1) of the
                                  candidate overflow pool and of the candidate lists, whose default
                                  sizes follow the expected candidate counts (O(K + rows), not
                                  O(d)).  Smaller saves workspace and sends more segments to the
                                  exact path; 0 keeps only each row's static slot.  A negative
                                  value is EF_EINVAL. */

typedef struct ef_layout ef_layout;

/* Human-readable name of a status code (static storage). */
const char* ef_status_string(int status);

/* The hipError_t behind the calling thread's most recent EF_EHIP (0 if none),
 * and its HIP description. */
int ef_last_hip_error(void);
const char* ef_last_hip_error_string(void);

/* Create a host-side layout (Section 3, sparsification scope).
 *   d            gradient length, 1 <= d < 2^31
 *   seg_offsets  host array of n_seg + 1 int64: 0 = o_0 < o_1 < ... < o_n_seg = d;
 *                segment l is [o_l, o_{l+1}).  Copied; the caller keeps ownership.
 *   density      k/d fraction in (0, 1] (Section 4.1 uses 1 %)
 *   block        random-block start alignment b >= 1; a segment with d_l <= b uses 1
 *   out          receives the new layout (unchanged on error)
 * Returns EF_OK, EF_EINVAL, EF_ERANGE or EF_ENOMEM.  Pure host code. */
int ef_layout_create(int64_t d, const int64_t* seg_offsets, int32_t n_seg, double density,
                     int64_t block, ef_layout** out);
int ef_layout_destroy(ef_layout* layout);

/* K = sum of k_l; -1 for a null layout. */
int64_t ef_layout_total_k(const ef_layout* layout);
int32_t ef_layout_num_segments(const ef_layout* layout);
/* Copies k_l for every segment into the host array k_out[n_seg]. */
int ef_layout_segment_k(const ef_layout* layout, int64_t* k_out);

/* Change a performance knob (EF_TUNE_*).  Unbinds the layout (bind it again before use).
 * Returns EF_ENOMEM, and leaves the layout unusable, if its tables cannot be rebuilt. */
int ef_layout_tune(ef_layout* layout, int knob, double value);

/* Bytes of device memory the layout's tables need. */
size_t ef_layout_device_bytes(const ef_layout* layout);
/* Upload the layout's tables into caller-owned device memory `dev_tables`
 * (>= ef_layout_device_bytes, 256-byte aligned), which must stay allocated
 * while the layout is used.  Synchronises `stream` once (setup call). */
int ef_layout_bind(ef_layout* layout, void* dev_tables, size_t bytes, void* stream);

/* Workspace bytes an entry point needs: EF_OP_TOPK for compress_topk /
 * ef_step_topk, EF_OP_RANDK for compress_randk / ef_step_randk,
 * EF_OP_AGG_SPARSE / EF_OP_AGG_BLOCK for decompress_aggregate and
 * decompress_aggregate_apply with W workers, EF_OP_AGG_SHARED for
 * decompress_aggregate_shared, EF_OP_RANDK_PREP for ef_randk_prepare and
 * ef_step_randk_prepared (W is ignored otherwise).  Random-block needs
 * none (returns 0).  Top-k and random-k workspaces grow with K and the
 * number of 4096-element rows (each row's static candidate slot, an overflow
 * pool, candidate lists), not with d (ResNet-50 at 0.1 % density: 16 MiB,
 * 0.65 bytes per element, in one segment); see EF_TUNE_POOL.  Their overflow counters are cleared by the
 * step's last kernel (top-k: also by its first), so a fresh workspace
 * needs no clearing (one holding garbage can send a random-k segment whose
 * row overflows its slot down the exact path once: same result).
 * Returns 0 for a null layout or unknown op. */
size_t ef_workspace_bytes(const ef_layout* layout, int op, int32_t W);

/* Algorithm 1, accumulate step: acc_i = fl32(g_i + e_i) for all i < d.
 *   g    f32[d] or bf16[d] (g_dtype EF_F32 / EF_BF16; bf16 widens exactly)
 *   e    f32[d];  acc  f32[d], may equal e (in place). */
int ef_accumulate(const ef_layout* layout, const void* g, int g_dtype, const float* e,
                  float* acc, void* stream);

/* Section 3, top-k: per segment, the k_l entries of acc with the largest
 * magnitude (key = float bits with the sign cleared; equal keys go to the
 * lower index), written as a sparse message (idx ascending, val = acc). */
int compress_topk(const ef_layout* layout, const float* acc, uint32_t* idx, float* val,
                  void* ws, size_t ws_bytes, void* stream);

/* Section 3, random-k: per segment, the k_l positions j with the smallest
 * Philox4x32-10 keys u_j (word j mod 4 of counter (j div 4, 0, step,
 * 0x01000000 | l) under key (seed lo, seed hi); equal keys: lower j), as a
 * sparse message.  Workers with equal seeds pick equal coordinates (the
 * allReduce mode of Section 3), distinct seeds the allGather mode. */
int compress_randk(const ef_layout* layout, const float* acc, uint64_t seed, uint32_t step,
                   uint32_t* idx, float* val, void* ws, size_t ws_bytes, void* stream);

/* Section 3, block-random-k: per segment one random start s_l (aligned to
 * b_l = b if d_l > b else 1; s_l = b_l * floor(r * n_l / 2^64), n_l =
 * ceil(d_l / b_l), r = x0 + 2^32 x1 of Philox counter (0, 0, step,
 * 0x02000000 | l)) and the k_l values that follow it, wrapping at the end of
 * the segment, as a block message.  Needs no workspace. */
int compress_randblock(const ef_layout* layout, const float* acc, uint64_t seed, uint32_t step,
                       uint32_t* start, float* val, void* stream);

/* Residual update (Section 3 worker steps; Algorithm 1): e_i = +0.0 where the
 * message (msg_kind EF_MSG_SPARSE: idx[K]; EF_MSG_BLOCK: start[n_seg]) sent
 * element i, else acc_i (bits unchanged).  e may equal acc. */
int ef_update(const ef_layout* layout, const float* acc, int msg_kind, const uint32_t* idx_or_start,
              float* e, void* stream);

/* Algorithm 1, aggregate step: out_i = fl32(sum over w = 0..W-1 in order of
 * the entries of message w at i, starting from +0.0), divided by W in IEEE
 * float32 when average != 0 (the plain sum of Algorithm 1 when 0).
 *   idx_or_start  uint32[W][K] (sparse) or uint32[W][n_seg] (block)
 *   val           float32[W][K]
 *   out           float32[d], written in full
 * Sparse messages must hold valid ascending indices as produced by the
 * compressors; entries that violate this are ignored, never written out of
 * bounds. */
int decompress_aggregate(const ef_layout* layout, int msg_kind, int32_t W,
                         const uint32_t* idx_or_start, const float* val, int average, float* out,
                         void* ws, size_t ws_bytes, void* stream);

/* Algorithm 1, the aggregate step fused with the parameter update
 * x_{t+1} = x_t - q_t that follows it, with the momentum and weight decay of
 * the paper's training setup (Section 4, experimental setup) as options: the
 * aggregate q of the W messages (as decompress_aggregate computes it) is
 * applied to the parameters in the same pass over d elements.  Per element:
 *   d = q + wd * x        (only when wd != 0; wd = learning rate x decay)
 *   m = beta * m + d, d = m   (only when mom is not null)
 *   x = x - d
 * each float32 operation rounded on its own (no fused multiply-add); the
 * learning rate is already inside q.  This is the order of a plain SGD step
 * with momentum (no dampening, no Nesterov) at learning rate 1.
 *   x     f32[d], updated in place;  mom  f32[d] or null (updated in place)
 *   out   f32[d] or null: also receives q
 * x, mom and out must be distinct buffers; beta and wd finite.  Workspace as
 * for decompress_aggregate (EF_OP_AGG_SPARSE for sparse messages). */
int decompress_aggregate_apply(const ef_layout* layout, int msg_kind, int32_t W,
                               const uint32_t* idx_or_start, const float* val, int average, float* x,
                               float* mom, float beta, float wd, float* out, void* ws, size_t ws_bytes,
                               void* stream);

/* decompress_aggregate for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same operation, arguments and result, bitwise, without a
 * workspace argument.  The sparse aggregate's tile-range table lives in a
 * static device array of ef_noalloc_scratch_bytes() bytes (16 MiB) that each
 * GPU the library runs on holds until the process ends; the call allocates
 * nothing (its first call on a device resolves that device's copy).
 *   Limit: ef_workspace_bytes(layout, EF_OP_AGG_SPARSE, W) must not exceed
 *   ef_noalloc_scratch_bytes() (W * (ceil(d / 1024) + 1) * 4 bytes, rounded
 *   up to 256), else EF_EWORKSPACE; block messages need no scratch.
 *   Every call on one GPU shares that GPU's array: calls that overlap on one
 *   GPU (on different streams or from different threads) race and must be
 *   ordered by the caller.  The stream must belong to the device whose memory
 *   the layout, messages and out live in. */
int decompress_aggregate_noalloc(const ef_layout* layout, int msg_kind, int32_t W,
                                 const uint32_t* idx_or_start, const float* val, int average,
                                 float* out, void* stream);
size_t ef_noalloc_scratch_bytes(void);

/* Algorithm 1's aggregate step when the workers share coordinates (Section
 * 3: equal seeds, the allReduce mode): every message has the same indices
 * (sparse) or block starts (block), given once:
 *   idx_or_start  uint32[K] (sparse) or uint32[n_seg] (block), as a message
 *   val           float32[W][K], the workers' values at those coordinates
 *   out           float32[d], written in full
 * The result is bitwise that of decompress_aggregate on the W messages
 * (coordinates repeated): the values are summed per coordinate in worker
 * order from +0.0, then placed like one message and divided by W.  Needs
 * ef_workspace_bytes(layout, EF_OP_AGG_SHARED, W) bytes of workspace. */
int decompress_aggregate_shared(const ef_layout* layout, int msg_kind, int32_t W,
                                const uint32_t* idx_or_start, const float* val, int average, float* out,
                                void* ws, size_t ws_bytes, void* stream);

/* Standard SGD's exchange, the paper's uncompressed baseline (Section 4,
 * results): out_i = fl32(sum over w = 0..W-1, in order, from +0.0, of
 * g[w][i]) divided by W in IEEE float32 when average != 0.
 *   g    float32[W][d] (the layout's d), contiguous
 *   out  float32[d] */
int ef_dense_average(const ef_layout* layout, int32_t W, const float* g, int average, float* out,
                     void* stream);

/* Fused worker steps: accumulate + compress + residual update in one call,
 * bitwise identical to ef_accumulate(g, e -> e), compress_*(e), ef_update(e, e).
 * e holds e_t on entry and e_{t+1} on return. */
int ef_step_topk(const ef_layout* layout, const void* g, int g_dtype, float* e, uint32_t* idx,
                 float* val, void* ws, size_t ws_bytes, void* stream);
int ef_step_randk(const ef_layout* layout, const void* g, int g_dtype, float* e, uint64_t seed,
                  uint32_t step, uint32_t* idx, float* val, void* ws, size_t ws_bytes, void* stream);
int ef_step_randblock(const ef_layout* layout, const void* g, int g_dtype, float* e, uint64_t seed,
                      uint32_t step, uint32_t* start, float* val, void* stream);

/* The fused top-k and random-k steps in phases, for callers that overlap
 * the steps of several workers (or gradient buckets) on more than one
 * stream.  Same operation and arguments as ef_step_topk / ef_step_randk,
 * plus `phases`, a nonzero OR of:
 *   EF_PHASE_PREPARE  top-k: the threshold sample of acc = g + e and the
 *                     candidate rule (reads g and e at the sample positions);
 *                     random-k: nothing (its keys do not depend on the data)
 *   EF_PHASE_STREAM   the streaming pass: acc = g + e written to e, the
 *                     candidates listed in the workspace
 *   EF_PHASE_FINISH   the exact threshold, the message and e = +0 where sent
 * Calling PREPARE, STREAM and FINISH in that order with the same arguments
 * and workspace (each call enqueued after the previous one has completed,
 * on one stream or ordered with events) is bitwise identical to the fused
 * step; EF_PHASE_ALL is the fused step itself.  Between the first and the
 * last phase, the workspace belongs to this step and g and e must not be
 * changed by other work.  Arguments are checked at every call; phases
 * outside EF_PHASE_ALL are EF_EINVAL. */
#define EF_PHASE_PREPARE 1u
#define EF_PHASE_STREAM 2u
#define EF_PHASE_FINISH 4u
#define EF_PHASE_ALL 7u
int ef_step_topk_phases(const ef_layout* layout, unsigned phases, const void* g, int g_dtype, float* e,
                        uint32_t* idx, float* val, void* ws, size_t ws_bytes, void* stream);
int ef_step_randk_phases(const ef_layout* layout, unsigned phases, const void* g, int g_dtype, float* e,
                         uint64_t seed, uint32_t step, uint32_t* idx, float* val, void* ws, size_t ws_bytes,
                         void* stream);

/* The fused top-k / random-k steps of W workers (or W gradient buckets of
 * one layout) in one call: with phases = EF_PHASE_ALL, bitwise W calls of
 * ef_step_topk / ef_step_randk.  The workers' streaming passes run back to
 * back and every selection kernel runs once for up to 64 workers (the worker
 * is the grid's second dimension), so the short latency-bound selection
 * steps are paid once per batch rather than once per worker.
 *   phases as for ef_step_*_phases, applied to all W workers: the phases of
 *         one batch called in order (ordered as there) give the same result
 *   g     host array of W device pointers: worker w's gradient, f32 or bf16[d]
 *   e     host array of W device pointers: worker w's residual f32[d], e_t on
 *         entry and e_{t+1} on return
 *   seeds random-k: host array of W seeds (worker w's seed); step as above
 *   idx   uint32[W][K], val float32[W][K]: worker w's message is row w
 *   ws    W workspaces, worker w's at ws + w * ws_stride; ws_stride a
 *         multiple of 256 and >= ef_workspace_bytes(layout, op, 1)
 * The host arrays are read during the call only.  (Each worker's g and e are
 * separate pointers: streaming over rows of two very large allocations
 * measured about 13 % slower here than over separate allocations.) */
int ef_step_topk_batch(const ef_layout* layout, unsigned phases, int32_t W, const void* const* g,
                       int g_dtype, float* const* e, uint32_t* idx, float* val, void* ws,
                       size_t ws_stride, void* stream);
int ef_step_randk_batch(const ef_layout* layout, unsigned phases, int32_t W, const void* const* g,
                        int g_dtype, float* const* e, const uint64_t* seeds, uint32_t step, uint32_t* idx,
                        float* val, void* ws, size_t ws_stride, void* stream);

/* Random-k with the selection prepared ahead (Section 3, random-k).  The
 * keys that choose the k_l coordinates of every segment depend only on the
 * seed, the step and the position, not on the gradient, so the message
 * indices can be computed before the gradient exists (for instance for step
 * t + 1 while step t runs, or during the backward pass); the step itself is
 * then one streaming pass.  ef_randk_prepare followed by
 * ef_step_randk_prepared gives bitwise the result of ef_step_randk.
 *
 * ef_randk_prepare: the message indices of (seed, step) and their tile table.
 *   idx   uint32[K], written: the indices, ascending within each segment
 *   ws    device, 256-byte aligned, ws_bytes >= ef_workspace_bytes(layout,
 *         EF_OP_RANDK_PREP, 1); on return it holds the tile table that
 *         ef_step_randk_prepared reads, valid until the next call on ws
 * ef_step_randk_prepared: the worker step given the prepared indices:
 *   acc = g + e; val[j] = acc[idx[j]]; e = acc with +0 at idx (e_{t+1}).
 *   idx, ws as written by ef_randk_prepare for this layout (read only);
 *   g, g_dtype, e, val as for ef_step_randk.
 * The _batch forms do W workers: seeds a host array of W seeds, idx and val
 * [W][K] (row w is worker w's), worker w's workspace at ws + w * ws_stride
 * (ws_stride a multiple of 256, >= the single worker's bytes), g and e host
 * arrays of W device pointers.  Errors are reported before anything is
 * enqueued, except that a batch checks all its arguments first and then
 * launches worker by worker. */
int ef_randk_prepare(const ef_layout* layout, uint64_t seed, uint32_t step, uint32_t* idx, void* ws,
                     size_t ws_bytes, void* stream);
int ef_randk_prepare_batch(const ef_layout* layout, int32_t W, const uint64_t* seeds, uint32_t step,
                           uint32_t* idx, void* ws, size_t ws_stride, void* stream);
int ef_step_randk_prepared(const ef_layout* layout, const void* g, int g_dtype, float* e, const uint32_t* idx,
                           float* val, const void* ws, size_t ws_bytes, void* stream);
int ef_step_randk_prepared_batch(const ef_layout* layout, int32_t W, const void* const* g, int g_dtype,
                                 float* const* e, const uint32_t* idx, float* val, const void* ws,
                                 size_t ws_stride, void* stream);

/* Diagnostics: byte offset inside a top-k / random-k workspace of a uint32
 * word whose bit 1 is set when, for at least one segment, the candidates could
 * not contain the answer, or did not fit the workspace, and the exact
 * whole-segment path ran instead (a slower path with the same result), bit 3 when a top-k segment's sampled
 * candidates fell short and were collected again at a lower threshold (a few
 * microseconds more, same result), and whose bit 2 is set if the per-row
 * winner counts of a segment did not add up to k_l (an internal consistency
 * check that should never fire; message writes stay inside the segment's
 * range regardless).  The word is only ever OR-ed: clear it to watch a given
 * call.  Returns (size_t)-1 for other ops. */
size_t ef_workspace_diag_offset(const ef_layout* layout, int op);

/* Per-kernel timing (diagnostics).  While enabled, every kernel the library
 * launches carries a start and a stop HIP event that the runtime binds to the
 * kernel's own dispatch on its stream (hipExtLaunchKernelGGL), so a launch's
 * duration is its execution time.
 * ef_timing_collect waits for the recorded events and adds each launch's
 * duration to a per-kernel total; ef_timing_get reads total i (kernel name in
 * static storage owned by the library, total milliseconds, launch count).
 * Process-wide; intended for benchmarks, not for hot loops. */
int ef_timing_enable(int enable);
int ef_timing_collect(void);
int ef_timing_count(void);
int ef_timing_get(int i, const char** name, double* total_ms, int64_t* launches);
int ef_timing_reset(void);

#ifdef __cplusplus
}
#endif

#endif /* EFSPARSE_H */
