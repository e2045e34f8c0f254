/*
 * rb.h - request batching for model serving on one MI355X (gfx950).
 *
 * The C boundary of the inter-request batching path of TensorFlow-Serving
 * (Olston et al., 2017), section 2.2.1 "Inter-Request Batching": requests for
 * a servable wait in that servable's batching queue; a batch is formed by
 * concatenating the requests' input tensors; queues share one device and are
 * served round-robin; the batched run is transparent to every caller, who
 * gets back exactly its own rows. Servables are opaque to the batching layer
 * (section 2, a servable is a black box behind a type-erased handle).
 *
 * Conventions
 *  - Every call returns rb_status: RB_OK (0) or a negative error code.
 *    Out-parameters are written only on RB_OK. No C++ exception crosses
 *    this boundary. rb_status_str() names a code (static string).
 *  - Host pointers are plain CPU memory; "device pointers" are addresses in
 *    the context's GPU memory (e.g. a torch CUDA tensor's data_ptr()).
 *  - Objects are created and destroyed by the caller; destroy calls accept
 *    NULL. Objects are not thread-safe: one host thread drives a scheduler.
 *  - Times are int64 nanoseconds of a simulated clock (see rb_sim_run).
 *  - All row-major. Floats are IEEE binary32; "bf16" storage is bfloat16
 *    rounded to nearest even, with fp32 accumulation.
 */
#ifndef RB_H
#define RB_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t rb_status;
#define RB_OK 0
#define RB_EINVAL (-1)  /* bad argument, shape or option */
#define RB_EBUSY (-2)   /* object still in use (bound queues, pending tasks) */
#define RB_EAGAIN (-3)  /* result not ready yet */
#define RB_EEMPTY (-4)  /* nothing to run */
#define RB_ESIZE (-5)   /* destination buffer too small */
#define RB_ENOENT (-6)  /* unknown or already collected request */
#define RB_EDEVICE (-7) /* HIP runtime error, or no device in this mode */
#define RB_ENOMEM (-8)  /* host or device allocation failed */
#define RB_ERANGE (-9)  /* the device found an id or length outside its bounds */

/* The name of a status code (a static string; "unknown status" for codes
 * not listed above): the outcome of the batching calls of paper section
 * 2.2.1, for messages. */
const char* rb_status_str(rb_status s);

typedef struct rb_ctx rb_ctx;
typedef struct rb_model rb_model;
typedef struct rb_sched rb_sched;
typedef struct rb_queue rb_queue;

/* ---------------------------------------------------------------- context */

/* The single shared device that the batching queues are scheduled onto
 * (paper section 2.2.1), with the manager thread that frees servable memory
 * off the inference path (section 2.1.2).
 * hip_device >= 0: bind to that GPU. hip_device < 0: host-only context; models
 * and schedulers created in it can only run in RB_MODE_NO_DEVICE.
 * *out is written on RB_OK and owned by the caller (rb_ctx_destroy).
 * RB_EINVAL if out is NULL; RB_EDEVICE if the device cannot be initialised. */
rb_status rb_ctx_create(int32_t hip_device, rb_ctx** out);
/* Ends the context's manager thread and frees it (paper section 2.1.2).
 * RB_EBUSY while models or schedulers created in it are alive. */
rb_status rb_ctx_destroy(rb_ctx* ctx);

/* ---------------------------------------------------------------- models */

enum { RB_MODEL_MLP = 0, RB_MODEL_RANKING = 1, RB_MODEL_SEQPOOL = 2 };
enum { RB_DT_F32 = 0, RB_DT_BF16 = 1 };
enum { RB_ACT_NONE = 0, RB_ACT_RELU = 1, RB_ACT_SIGMOID = 2, RB_ACT_SOFTMAX = 3 };

/* One dense layer y = act(x W^T + b). w: host [fan_out, fan_in] fp32,
 * b: host [fan_out] fp32. */
typedef struct {
  int32_t fan_in, fan_out, act;
  const float* w;
  const float* b;
} rb_layer_desc;

/* A servable's model (opaque to the queues and the scheduler).
 *   RB_MODEL_MLP      request rows of layers[0].fan_in floats -> layers.
 *   RB_MODEL_RANKING  per row: n_tables sum-pooled embedding bags of emb_dim
 *                     (one per table, in table order) followed by n_dense
 *                     floats -> layers; layers[0].fan_in must equal
 *                     n_tables*emb_dim + n_dense. Tables are host
 *                     [table_rows, emb_dim] fp32 arrays.
 *   RB_MODEL_SEQPOOL  per sequence: layers on every token, mean over the
 *                     sequence's tokens, then `head` (act RB_ACT_SOFTMAX or
 *                     RB_ACT_NONE).
 * dtype RB_DT_BF16 stores weights and tables as bf16 (rounded to nearest even
 * from the given fp32), rounds every layer input to bf16 and accumulates in
 * fp32; the last layer's output stays fp32. RB_DT_F32 keeps fp32 throughout.
 * RB_ACT_SIGMOID and RB_ACT_SOFTMAX are allowed only on the last layer (MLP
 * and ranking: sigmoid with fan_out 1) and on the head.
 * All host arrays are copied; the caller may free them when this returns.
 * RB_EINVAL on inconsistent shapes. */
typedef struct {
  int32_t kind, dtype;
  int32_t n_layers;
  const rb_layer_desc* layers;
  int32_t n_tables;
  int64_t table_rows;
  int32_t emb_dim;
  int32_t n_dense;
  const float* const* tables;
  rb_layer_desc head;
} rb_model_desc;

/* Load a servable version into device memory (a Loader's load, paper
 * section 2.1; the servable is a black box to the queues and the scheduler,
 * section 2.1). Safe to call on a thread of its own while a scheduler serves:
 * the upload runs on a private non-blocking stream, so loading is insulated
 * from inference (section 2.1.2, isolated load and inference threads).
 * *out is owned by the caller (rb_model_destroy). RB_EINVAL on inconsistent
 * shapes or NULL arguments; RB_ENOMEM / RB_EDEVICE on device failures. */
rb_status rb_model_create(rb_ctx* ctx, const rb_model_desc* desc, rb_model** out);
/* The servable's request interface (paper section 2.1: what a caller's
 * tensors must look like). d_in: floats per request row (tokens: per token);
 * d_out: floats per output row (seqpool: per sequence). RB_EINVAL on NULL. */
rb_status rb_model_info(const rb_model* m, int32_t* d_in, int32_t* d_out);
/* Unload a servable version (paper section 2.1.2: reference-counted servable
 * handles whose memory is freed in a manager thread, not an inference
 * thread). The caller's handle is invalid on return. RB_EBUSY while a queue
 * is bound to the model. Batches already dispatched to it keep references of
 * their own: its device memory is released by the context's deleter thread
 * once the last of them has finished, never on the caller's thread. */
rb_status rb_model_destroy(rb_model* m);

/* ---------------------------------------------------------------- scheduler */

enum { RB_MODE_DEVICE = 0, RB_MODE_NO_DEVICE = 1 };

typedef struct {
  int32_t mode;
  /* Device mode: dispatched batches are handed to the device in windows of
   * up to window_batches batches (>= 1); the batches of one model in a window
   * run in one launch chain (their rows stay in separate, separately padded
   * batches). 1 runs every batch on its own. */
  int32_t window_batches;
  /* Value written into padding rows (and padding tokens) before the forward
   * pass. 0 in production; NaN shows that padding never reaches an output. */
  float pad_value;
  /* 1: time every kernel launch with HIP events (rb_sched_kernel_stats);
   * 2: the same with cold caches: before each timed launch the scheduler
   * reads a 512 MB buffer on the launch stream (outside the timed events),
   * evicting L2 and the Infinity Cache; 0: no timing. */
  int32_t profile;
  /* Device mode: the launch chains of different models in a replay run on up
   * to n_streams HIP streams of their own (0 or 1: the scheduler's stream).
   * Each model keeps one stream, assigned in order of first use, so its
   * chains stay in order; outputs do not depend on this setting. */
  int32_t n_streams;
  /* Device mode, fp32 seqpool models: 1 packs the real tokens of a launch
   * group's sequences into consecutive rows (no time padding) for the
   * token-wise layers, then pools each sequence from its own rows (the
   * sub-graph batching the paper's Batch/Unbatch operations allow, section on
   * batching); 0 pads every sequence to its queue's bucket. Outputs are
   * identical either way. */
  int32_t seq_pack;
  /* Device mode, rb_sim_run: 0 runs the trace as a backlogged device would
   * (every launch window holds window_batches consecutive dispatched batches,
   * whatever the simulated clock did: the replay measures capacity); 1 runs
   * exactly the windows the simulated clock dispatched (see rb_sim_run). The
   * serving API always runs the clock's windows. */
  int32_t clocked_windows;
  /* Device mode, ranking models: 1 gathers each distinct table row of a
   * 64-row block's bags once (rb_k_embbag_dedup), 0 row by row (rb_k_embbag);
   * outputs are identical either way. */
  int32_t emb_dedup;
  /* Device mode, bf16 models whose last two hidden layers are ReLU layers of
   * 512 and 256 outputs ahead of a narrow head (the ranking MLP): 1 runs them
   * and the head as one kernel (rb_k_mlp_tail), 0 as three; outputs are
   * identical either way. */
  int32_t fuse_mlp_tail;
} rb_sched_opts;

/* The scheduler that serves the batching queues round-robin on one shared
 * device (paper section 2.2.1). It owns one HIP stream of the context's device
 * (device mode), plus opts->n_streams streams for concurrent launch chains in
 * replays, and a simulated clock (int64 ns) on which batches close, are
 * dispatched in launch windows and complete. *out is owned by the caller
 * (rb_sched_destroy). RB_EINVAL on a bad option; RB_EDEVICE when device mode
 * is asked of a host-only context or stream creation fails. */
rb_status rb_sched_create(rb_ctx* ctx, const rb_sched_opts* opts, rb_sched** out);
/* Frees the scheduler after waiting for its device work (paper section
 * 2.2.1). RB_EBUSY while queues exist. */
rb_status rb_sched_destroy(rb_sched* s);
/* Blocks until all device work of the scheduler has finished (the batched
 * Run() calls of paper section 2.2.1 have returned). RB_ERANGE if a kernel
 * found an id or a sequence length outside its request's bounds since the
 * last rb_sync (the offending values contributed nothing). */
rb_status rb_sync(rb_sched* s);
/* Kernel timings of a profiling scheduler since its creation (after rb_sync),
 * for measuring the batched Run() of paper section 2.2.1: kernel names are
 * those of rb_k_* without the prefix ("embbag", ...). RB_EINVAL on NULL. */
rb_status rb_sched_kernel_stats(rb_sched* s, const char* kernel, int64_t* launches, double* total_ms);
/* The scheduler's HIP stream (hipStream_t) on the shared device (paper
 * section 2.2.1), for callers that order their own work after the
 * scheduler's; NULL in RB_MODE_NO_DEVICE. RB_EINVAL on NULL. */
rb_status rb_sched_stream(rb_sched* s, void** stream);

/* ---------------------------------------------------------------- queues */

#define RB_MAX_BATCH_ROWS 4096
#define RB_MAX_STREAMS 16  /* rb_sched_opts.n_streams */

typedef struct {
  int32_t max_batch_size;            /* rows (sequences for seqpool) per batch, 1..RB_MAX_BATCH_ROWS */
  const int32_t* allowed_batch_sizes;/* strictly ascending, last == max_batch_size */
  int32_t n_allowed;                 /* 0: batches run at their real size */
  int64_t batch_timeout_ns;          /* > 0; INT64_MAX: batches close by count only */
  int32_t bucket_len;                /* seqpool: sequences up to this many tokens; else 0 */
  /* Simulated device time of a batch of padded size P is service_ns[P],
   * 0 <= P <= max_batch_size (n_service = max_batch_size + 1); NULL: 0. */
  const int64_t* service_ns;
  int32_t n_service;
  /* Simulated fixed device time of this queue's launch chain in a launch
   * window (>= 0): a window taking batches of this queue holds the device for
   * window_ns once plus service_ns[P] per batch. */
  int64_t window_ns;
  /* Simulated further time (>= 0) until that chain's results are complete
   * once the device has moved on to the next window (a chain's fixed latency
   * that the device overlaps with the next window's work). */
  int64_t window_tail_ns;
} rb_queue_opts;

/* A batching queue for one servable version (paper section 2.2.1: one queue
 * per servable or version, the set of queues dynamic as versions come and
 * go). Queues may be created and destroyed while the scheduler runs; queue
 * ids are assigned in creation order and round-robin follows them. The queue
 * binds m (rb_model_destroy then returns RB_EBUSY). *out is owned by the
 * caller (rb_queue_destroy). RB_EINVAL unless allowed_batch_sizes is strictly
 * ascending with last == max_batch_size (or empty), bucket_len is given
 * exactly for seqpool models, and the service table has max_batch_size + 1
 * non-negative entries. */
rb_status rb_queue_create(rb_sched* s, rb_model* m, const rb_queue_opts* opts, rb_queue** out);
/* Remove a queue (paper section 2.2.1, queues removed as versions go).
 * RB_EBUSY while the queue holds requests that have not run. */
rb_status rb_queue_destroy(rb_queue* q);
/* The queue's id, its place in the round-robin order (paper section 2.2.1).
 * RB_EINVAL on NULL. */
rb_status rb_queue_id(const rb_queue* q, int32_t* id);
/* Version transition (the version transition policies of the paper's
 * Aspired Versions Manager, section 2.1.2): batches the queue dispatches after
 * this call run model m. m must have the bound model's kind, dtype, input and
 * output widths and table count (RB_EINVAL otherwise); it may be created on
 * another thread while the scheduler serves (rb_model_create uploads on a
 * private non-blocking stream).
 *   Availability-preserving: load the new version, call this, then destroy
 *   the old one; with the old version's padded layer shapes the new one also
 *   takes over its launch stream and work buffers.
 *   Resource-preserving: m = NULL holds the queue (no version bound, so the
 *   old one can be destroyed before the new one is loaded): it keeps
 *   accepting requests and closing batches, validated against the old
 *   version's interface, but dispatches nothing (rb_run_next skips it;
 *   rb_sim_run refuses it with RB_EBUSY) until a version is set again.
 * RB_EBUSY while a launch window is being filled (only between rb_sim_run /
 * rb_run_next calls). The old model stays bound to any other queue that uses
 * it; once unbound, rb_model_destroy frees it off the inference path. */
rb_status rb_queue_set_model(rb_queue* q, rb_model* m);

/* ---------------------------------------------------------------- serving */

/* One request's input tensors (host memory; copied before rb_submit returns).
 *   MLP:      dense [n_rows, d_in]
 *   RANKING:  dense [n_rows, n_dense]; lens [n_rows, n_tables] ids per bag;
 *             ids [sum(lens)] table rows, row after row, bag after bag
 *   SEQPOOL:  n_rows sequences; lens [n_rows] tokens per sequence (>= 1);
 *             dense [sum(lens), d_in] tokens, sequence after sequence
 * n_dense/n_lens/n_ids are element counts. */
typedef struct {
  int32_t n_rows;
  const float* dense;
  int64_t n_dense;
  const int32_t* lens;
  int64_t n_lens;
  const int32_t* ids;
  int64_t n_ids;
} rb_request;

/* Enqueue one inference request on its servable's batching queue (paper
 * section 2.2.1: requests are merged into batches by concatenating their
 * input tensors; section 2.2: the caller's Run()). The payload is copied
 * before the call returns; the caller keeps ownership of r.
 * The simulated clock first runs its events before arrival_ns (timeouts, and
 * launch windows dispatched whenever the simulated device is free), then the
 * timeouts due at arrival_ns, then the arrival: next-fit in arrival order (the
 * open batch closes when the request would overflow it, the request opens the
 * next one, and a batch closes once full). Dispatches at arrival_ns wait for
 * rb_run_next / rb_run_window / rb_advance, so every request of one timestamp
 * should be submitted before those are called.
 * arrival_ns must be >= the clock (RB_EINVAL otherwise). RB_EINVAL if n_rows
 * < 1 or > max_batch_size, shapes mismatch, an id is outside its table, or a
 * sequence is longer than the queue's bucket. Request ids are dense per
 * scheduler, in submission order. */
rb_status rb_submit(rb_queue* q, const rb_request* r, int64_t arrival_ns, uint64_t* out_req_id);
/* Advance the simulated clock to now_ns, running its events up to and
 * including now_ns: batch timeouts (a batch must not wait unduly, paper
 * section 2.2.1) and the launch windows the simulated device dispatches.
 * RB_EINVAL if now_ns is before the clock. */
rb_status rb_advance(rb_sched* s, int64_t now_ns);
/* Close the queue's open batch at the current clock (no-op if empty; paper
 * section 2.2.1, the end of a stream of requests). RB_EINVAL on NULL. */
rb_status rb_flush(rb_queue* q);

typedef struct {
  uint64_t batch_id;
  int32_t queue;        /* queue id */
  int32_t real_rows;    /* s */
  int32_t padded_rows;  /* P */
  int32_t n_req;
  int64_t close_ns, dispatch_ns, done_ns;
  const uint64_t* req_ids; /* valid until the next rb_run_next */
} rb_batch_info;

/* Run one merged request (paper section 2.2.1: the batching wrapper forwards
 * the concatenated inputs to the wrapped Run() once). The clock first runs
 * its events up to and including the current time; then the next batch it
 * has dispatched (oldest launch window first, batches of a window in their
 * round-robin order) runs on its own: in device mode its payloads are staged
 * to the device and assemble -> forward -> split is enqueued on the
 * scheduler's stream (asynchronous; rb_collect waits for it). *out is valid
 * until the next rb_run_next / rb_run_window call. RB_EEMPTY if the clock has
 * dispatched nothing that has not run; RB_EDEVICE / RB_ENOMEM on device
 * failures. */
rb_status rb_run_next(rb_sched* s, rb_batch_info* out);

/* The batches of one launch window (valid until the next rb_run_next or
 * rb_run_window call). */
typedef struct {
  int32_t n_batches;
  const rb_batch_info* batches;
} rb_window_info;

/* Run the next launch window the simulated clock has dispatched (paper
 * section 2.2.1, several merged requests of the queues sharing the device):
 * the clock first runs its events up to and including the current time;
 * then all batches of the oldest dispatched window run, one launch chain per
 * queue, their payloads staged to the device in one copy and their outputs
 * copied back in one (asynchronous). *out is valid until the next
 * rb_run_next / rb_run_window call. RB_EEMPTY if nothing dispatched is
 * waiting; RB_EDEVICE / RB_ENOMEM on device failures. */
rb_status rb_run_window(rb_sched* s, rb_window_info* out);
/* Hand a caller its own part of a merged run (paper section 2.2.1: each
 * caller gets exactly its rows back): copy request req_id's output rows
 * ([n_rows, d_out] fp32, in the request's row order) to dst (host). Keyed by
 * the scheduler because request ids are dense per scheduler (a request keeps
 * its id while its queue changes version or is held). RB_EAGAIN if its batch
 * has not finished; RB_ESIZE if dst_bytes is too small; RB_ENOENT if unknown
 * or already collected; RB_EDEVICE without a device, or (once, after which
 * the id is unknown) when the run of its window failed. The library drops its
 * copy after a successful collect. */
rb_status rb_collect(rb_sched* s, uint64_t req_id, float* dst, size_t dst_bytes, int32_t* out_rows);

/* ---------------------------------------------------------------- trace replay */

/* A servable: its queues (one, or one per length bucket for seqpool; a request
 * goes to the smallest bucket that holds its longest sequence). */
typedef struct {
  int32_t n_queues;
  rb_queue* const* queues;
} rb_servable;

/* A whole request trace whose payloads are already in device memory.
 * Host arrays: servable, arrival_ns, n_rows, max_len (seqpool; else NULL),
 *   and the [n_requests + 1] element offsets *_off of each request's slice of
 *   the device arenas (the last entry is the arena's length).
 * Device arrays: dense (fp32), lens (i32), ids (i32) arenas laid out per
 *   request as in rb_request, and out, the fp32 output arena receiving
 *   request r's [n_rows, d_out] rows at out_off[r].
 * In RB_MODE_NO_DEVICE the device arrays may be NULL. */
typedef struct {
  int32_t n_requests;
  const int32_t* servable;
  const int64_t* arrival_ns;
  const int32_t* n_rows;
  const int32_t* max_len;
  const float* dense;
  const int64_t* dense_off;
  const int32_t* lens;
  const int64_t* lens_off;
  const int32_t* ids;
  const int64_t* ids_off;
  float* out;
  const int64_t* out_off;
} rb_trace;

/* Batch log of a replay (host arrays allocated by the caller).
 *   req_done_ns [n_requests], req_queue [n_requests] (queue id);
 *   per batch, in dispatch order, up to max_batches:
 *   b_queue, b_real, b_padded, b_close_ns, b_dispatch_ns, b_done_ns,
 *   b_req_begin [max_batches + 1] offsets into b_reqs [n_requests]. */
typedef struct {
  int64_t* req_done_ns;
  int32_t* req_queue;
  int64_t max_batches;
  int64_t n_batches; /* out */
  int32_t* b_queue;
  int32_t* b_real;
  int32_t* b_padded;
  int64_t* b_close_ns;
  int64_t* b_dispatch_ns;
  int64_t* b_done_ns;
  int64_t* b_req_begin;
  int32_t* b_reqs;
} rb_log;

/* Replay a whole request trace through the batching queues (paper section
 * 2.2.1: per-servable queues, merged requests, round-robin onto one device)
 * with the simulated clock, starting idle: events at one timestamp are
 * timeouts in queue-id order, then arrivals in request order, then the
 * end-of-trace close of count-only queues at the last arrival, then launch
 * windows dispatched while the simulated device is free. In device mode every
 * batch's device work is enqueued (asynchronous; rb_sync waits): in windows of
 * window_batches consecutive dispatched batches, or with clocked_windows in
 * the clock's own windows. The log is written by the caller's arrays.
 * RB_EBUSY if any queue of the scheduler still holds a request (open, closed
 * or dispatched but not run) or a queue of the replay is held; the replay
 * leaves its queues empty. RB_ESIZE if max_batches is too small; RB_EINVAL on
 * inconsistent arrays (shapes, offsets, arrival order, unknown servables). */
rb_status rb_sim_run(rb_sched* s, const rb_servable* servables, int32_t n_servables,
                     const rb_trace* trace, rb_log* log);

/* ---------------------------------------------------------------- kernel ABI */
/* Single kernels of the device path, for tests and measurement. All pointers
 * are device pointers, `stream` is a hipStream_t (NULL: the null stream), and
 * launches are asynchronous. The group descriptors (rb_k_req, rb_k_batch) are
 * device arrays too. */

/* A request of a launch group: [dense_off, dense_end) of the dense arena,
 * lens from lens_off, [ids_off, ids_end) of the ids arena, output at out_off;
 * tok_off (seqpool): the row of the request's first token among the group's
 * packed tokens (the requests' token counts summed in group order). */
typedef struct {
  int64_t dense_off, dense_end, lens_off, ids_off, ids_end, out_off;
  int32_t n_rows, tok_off;
} rb_k_req;

typedef struct {
  int32_t req_begin, n_req; /* requests [req_begin, req_begin + n_req) of the group */
  int32_t row_base;         /* first row of this batch in the group's row space */
  int32_t padded;           /* P */
  int32_t real;             /* s */
  int32_t seq_T;            /* seqpool: tokens per sequence slot (bucket), else 0 */
} rb_k_batch;

/* Per padded row: src = element offset of the row's dense input (-1: padding),
 * aux = ranking: offset of the row's first id; seqpool: sequence length,
 * lens = ranking: offset of the row's bag lengths; seqpool: the row of the
 * sequence's first token among the group's packed tokens (its request's
 * tok_off plus the tokens of the request's earlier sequences; -1 when the
 * request is rejected), out = offset of the row's output (-1: padding). */
typedef struct {
  int64_t src, aux, lens, out;
} rb_k_row;

/* ---------------------------------------------------------------- launch groups */

/* Run one merged request group of queue q's model (paper section 2.2.1: the
 * batching wrapper forwards the concatenated inputs of its callers to the
 * wrapped Run() once and hands each caller its part) on device-resident
 * inputs: route -> assemble | embedding bags -> layers -> head | pooling |
 * split, enqueued on `stream` (a hipStream_t; NULL: the scheduler's stream),
 * asynchronous. For callers that form their own batches.
 *   batches [n_batches] and reqs [n_reqs]: device arrays of rb_k_batch /
 *     rb_k_req (above) describing the group: batch b owns rows
 *     [row_base, row_base + padded) of the group's `slots` rows (its padded
 *     sizes summed; sequence slots for seqpool) and requests
 *     [req_begin, req_begin + n_req);
 *   tokens (seqpool with rb_sched_opts.seq_pack): the requests' real tokens
 *     summed (their dense extents over d_in), the rows of the token-wise
 *     layers; tok_off of each request its first packed row; else 0;
 *   dense / lens / ids: device payload arenas of dense_len / lens_len /
 *     ids_len elements; out: the fp32 output arena of out_len floats.
 * The queue's scheduler must be in device mode and the queue bound to a model
 * (RB_EBUSY while held); the queue's model and the scheduler's pad value and
 * seq_pack are used. Work buffers belong to the scheduler (one set per
 * servable lineage for these calls, grown by allocation as needed; growing
 * waits for `stream` and the scheduler's streams), so calls on one scheduler
 * must be ordered: on one stream, or each finished before the next. The
 * queue must stay bound and its model alive until the stream has run the
 * call. Rows no valid batch covers stay padding; payloads and descriptors are
 * bounds-checked on the device (RB_ERANGE from the scheduler's next rb_sync,
 * called once `stream` has finished). RB_EINVAL on NULL pointers, n_batches
 * < 1, slots < n_batches or negative extents; RB_EDEVICE without a device. */
rb_status rb_run_group(rb_queue* q, void* stream, const rb_k_batch* batches, int32_t n_batches,
                       const rb_k_req* reqs, int32_t n_reqs, int64_t slots, int64_t tokens, const float* dense, int64_t dense_len,
                       const int32_t* lens, int64_t lens_len, const int32_t* ids, int64_t ids_len, float* out,
                       int64_t out_len);

/* Size of the per-GPU scratch array of rb_run_group_static. */
#define RB_STATIC_SCRATCH_BYTES ((size_t)64 << 20)

/* rb_run_group for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation): the
 * same launch chain and arguments, with its work buffers (row map, assembled
 * input, two activation buffers and the last layer's fp32 output, each
 * rounded up to 256 bytes) carved from one file-scope device array of
 * RB_STATIC_SCRATCH_BYTES per GPU, which each GPU holds from the library's
 * load until the process ends. The call makes no device or pinned
 * allocation and no free; it launches kernels on `stream` only. A group whose
 * work buffers exceed the array returns RB_ESIZE before anything is launched
 * (one 1024-row batch of a 4096-8192-8192-4096 bf16 MLP fits; two do not).
 * Every call on one GPU shares that GPU's array and leaves its contents
 * behind: calls whose device work overlaps on one GPU (different streams, or
 * other schedulers) race and must be ordered by the caller. Nothing in the
 * array has to start at zero: each call writes its row map first, and every
 * value an output depends on is written by the call before it is read.
 * RB_EDEVICE if the array's address could not be looked up on the context's
 * GPU (at rb_ctx_create). */
rb_status rb_run_group_static(rb_queue* q, void* stream, const rb_k_batch* batches, int32_t n_batches,
                              const rb_k_req* reqs, int32_t n_reqs, int64_t slots, int64_t tokens,
                              const float* dense, int64_t dense_len, const int32_t* lens, int64_t lens_len,
                              const int32_t* ids, int64_t ids_len, float* out, int64_t out_len);

/* ---------------------------------------------------------------- single kernels */

/* Row routing (paper section 2.2.1, a merged request concatenates its
 * requests' input tensors; here as exclusive prefix scans of row counts and,
 * fused in the same kernel, of bag lengths or token counts): fills
 * rows[row_base .. row_base + P) of every batch (P <= RB_MAX_BATCH_ROWS; every
 * request has >= 1 row). kind = RB_MODEL_*; d_in floats per row (per token
 * for seqpool); d_out floats per output row; n_tables bags per ranking row.
 * Extents: reqs holds n_reqs requests, lens lens_len elements, rows
 * n_rows_total entries, and the output out_len floats. A batch whose rows or
 * requests fall outside them sets *err = 1 and writes no row. A request whose
 * payload does not match its n_rows (dense length, bag lengths vs ids,
 * sequence lengths outside [1, seq_T]), or whose lengths or output rows would
 * lie outside their extents, sets *err = 1, contributes no ids / no tokens and
 * gets no output rows (its rows' out = -1). */
rb_status rb_k_route(void* stream, int32_t kind, const rb_k_batch* batches, int32_t n_batches,
                     const rb_k_req* reqs, int32_t n_reqs, const int32_t* lens, int64_t lens_len, int32_t d_in,
                     int32_t d_out, int32_t n_tables, rb_k_row* rows, int32_t n_rows_total, int64_t out_len,
                     int32_t* err);
/* Concatenate and pad a batch (paper section 2.2.1, concatenating the input
 * tensors): gather rows into X [n_rows_total, ldx] (ldx >= d_in, columns
 * [d_in, ldx) zeroed), padding rows set to pad; out_bf16 != 0 writes bf16
 * (RNE), else fp32.
 * Seqpool (seq_T > 0): row r*T + t is token t of sequence slot r (pad past L).
 * seq_real_only == 1 (seqpool, fp32 out, n_rows_total a multiple of seq_T):
 * rows t >= L and every row of a padding slot are not written and keep
 * whatever X held; every layer maps row i to row i alone and the pooling reads
 * t < L only, so no value there reaches an output.
 * seq_real_only == 2: packed tokens: token t of slot r goes to row
 * rows[r].lens + t (n_rows_total / seq_T slots; those rows must lie below
 * n_rows_total, else *err = 1 and the sequence is not copied). */
rb_status rb_k_assemble(void* stream, const rb_k_row* rows, int32_t n_rows_total, int32_t seq_T,
                        int32_t seq_real_only, const float* dense, int64_t dense_len, int32_t d_in, void* X,
                        int32_t ldx, int32_t out_bf16, float pad, int32_t* err);
/* The ranking servable's input layer on a merged batch (paper section
 * 2.2.1, the wrapped Run() on the concatenated examples; section 2.2, the
 * examples' sparse features): X[r] = [bf16(sum of bag f of row r from table
 * f), f = 0..n_tables-1 |
 * bf16(dense) | 0 ...] with row stride ldx; tables: n_tables device pointers
 * (in a device array) to [table_rows, emb_dim] bf16. emb_dim must be 64,
 * n_dense <= 256. ids_len is the length of the ids arena (reads stay below it).
 * An id outside its table sets *err = 1 and contributes nothing. */
rb_status rb_k_embbag(void* stream, const rb_k_row* rows, int32_t n_rows_total, const int32_t* lens,
                      const int32_t* ids, int64_t ids_len, const void* const* tables, int32_t n_tables,
                      int64_t table_rows, int32_t emb_dim, const float* dense, int32_t n_dense, void* X,
                      int32_t ldx, float pad, int32_t* err);
/* rb_k_embbag with the ids of each block of 64 rows deduplicated per table
 * before the gathers (paper section 2.2: compressing away features common to
 * a batch of examples): every distinct table row of the block's bags is read
 * once into LDS, then each bag is summed from there. Same arguments, bounds
 * checks and outputs, bit for bit (the same fp32 additions in the same
 * order); table_rows must fit in 31 bits. */
rb_status rb_k_embbag_dedup(void* stream, const rb_k_row* rows, int32_t n_rows_total, const int32_t* lens,
                            const int32_t* ids, int64_t ids_len, const void* const* tables, int32_t n_tables,
                            int64_t table_rows, int32_t emb_dim, const float* dense, int32_t n_dense, void* X,
                            int32_t ldx, float pad, int32_t* err);
/* A dense layer of the served model run once on a merged batch (paper
 * section 2.2.1, the wrapped Run() on the concatenated inputs):
 * Y[M, N] = act(X[M, K] W[N, K]^T + b), bf16 X and W (row strides ldx, ldw,
 * ldx and ldw < 2^22), fp32 accumulation; Y bf16 (out_f32 == 0) or fp32, row
 * stride ldy (a multiple of 8; Y 16-byte aligned). K % 64 == 0, N % 128 == 0.
 * act: RB_ACT_NONE, RB_ACT_RELU or RB_ACT_SIGMOID. */
rb_status rb_k_gemm_bf16(void* stream, const void* X, int32_t ldx, const void* W, int32_t ldw,
                         const float* b, void* Y, int32_t ldy, int32_t M, int32_t N, int32_t K,
                         int32_t act, int32_t out_f32);
/* A dense layer on a merged batch (paper section 2.2.1), fp32 variant (fp32
 * MFMA, same k order for every M): K % 32 == 0, N % 64 == 0;
 * ldx, ldw and ldy multiples of 4 with X, W and Y 16-byte aligned; ldx and
 * ldw < 2^23. Optional tile skip for
 * sequence groups: with skip_rows (the per-slot row map, aux = sequence length)
 * X holds skip_T rows per slot (token t of slot e at row e*skip_T + t) and a
 * 64-row block starting at token t of slot e is neither computed nor stored
 * when t >= L_e or slot e is padding: it holds only padding tokens, which the
 * pooling never reads. skip_T % 64 == 0; skip_rows NULL computes every row. */
rb_status rb_k_gemm_f32(void* stream, const float* X, int32_t ldx, const float* W, int32_t ldw,
                        const float* b, float* Y, int32_t ldy, int32_t M, int32_t N, int32_t K, int32_t act,
                        const rb_k_row* skip_rows, int32_t skip_T);
/* The merged run's last layer handed back to the callers in the same launch
 * (paper section 2.2.1: each caller gets exactly its own rows): the layer of
 * rb_k_gemm_bf16 (bf16 X and W, out_f32) or rb_k_gemm_f32 (fp32 X and W, no
 * padding-token skip), with row r's first d_out fp32 outputs written to
 * out[rows[r].out, rows[r].out + d_out) when rows[r].out >= 0 instead of to a
 * Y matrix; padding rows and columns past d_out are never written. Same shape
 * rules as those calls; 1 <= d_out <= N. Bit-identical to the layer followed by
 * rb_k_split. RB_EINVAL on a bad shape, pointer or activation. */
rb_status rb_k_gemm_bf16_rows(void* stream, const void* X, int32_t ldx, const void* W, int32_t ldw, const float* b,
                              int32_t M, int32_t N, int32_t K, int32_t act, const rb_k_row* rows, int32_t d_out,
                              float* out);
/* The same for an fp32 layer (paper section 2.2.1, the split of the merged
 * run fused into its last layer): the layer of rb_k_gemm_f32 without the
 * padding-token skip, outputs through the row map as above. */
rb_status rb_k_gemm_f32_rows(void* stream, const float* X, int32_t ldx, const float* W, int32_t ldw, const float* b,
                             int32_t M, int32_t N, int32_t K, int32_t act, const rb_k_row* rows, int32_t d_out,
                             float* out);
/* The merged run's last layer handed back to the callers (paper section
 * 2.2.1: each caller gets its own rows): a narrow last layer fused with the
 * split, out[rows[r].out] = act(H[r, :K] . w + b)
 * for real rows (act RB_ACT_SIGMOID or RB_ACT_NONE); H bf16 [n_rows_total, ldh],
 * w bf16 [K]. */
rb_status rb_k_head(void* stream, const rb_k_row* rows, int32_t n_rows_total, const void* H, int32_t ldh,
                    const void* w, float b, int32_t K, int32_t act, float* out);
/* The merged run's last hidden layer and its narrow head in one launch (paper
 * section 2.2.1: one forward pass for the whole merged request, each caller
 * handed its own rows): for rows r < M, y_r = act(X[r, :K] W^T + b) with W bf16
 * [256, ldw] (256 outputs), rounded to bf16 as rb_k_gemm_bf16 stores it, then
 * out[rows[r].out] = head_act(y_r . w_head + b_head) for rows whose out >= 0
 * (head_act RB_ACT_SIGMOID or RB_ACT_NONE; w_head bf16 [256], 16-byte
 * aligned). X bf16 [M, ldx]; K a multiple of 64, ldx, ldw >= K and multiples
 * of 8. y never leaves the device's on-chip memory. Bit-identical to
 * rb_k_gemm_bf16 with N = 256 followed by rb_k_head with K = 256. RB_EINVAL on
 * a bad shape, alignment or activation. */
rb_status rb_k_gemm_head(void* stream, const void* X, int32_t ldx, const void* W, int32_t ldw, const float* b,
                         int32_t M, int32_t K, int32_t act, const rb_k_row* rows, const void* w_head, float b_head,
                         int32_t head_act, float* out);
/* The last two hidden layers and the narrow head of a bf16 MLP run once on a
 * merged batch (paper section 2.2.1) and handed back to the callers (each
 * caller gets its own rows), in one kernel per block of 128 rows:
 * Y2 = relu(H1[:, :K2] W2^T + b2) (512 outputs, bf16), Y3 = relu(Y2 W3^T +
 * b3) (256 outputs, bf16), out[rows[r].out] = act(Y3[r] . w4 + b4) for real
 * rows (act RB_ACT_SIGMOID or RB_ACT_NONE). H1 bf16 [n_rows_total, ldh1];
 * W2 bf16 [512, ldw2]; W3 bf16 [256, ldw3 >= 512]; w4 bf16 [256]; b2, b3 fp32.
 * K2 % 32 == 0; row strides multiples of 8 and operands 16-byte aligned.
 * Bit-identical to rb_k_gemm_bf16 twice and rb_k_head. */
rb_status rb_k_mlp_tail(void* stream, const rb_k_row* rows, int32_t n_rows_total, const void* H1, int32_t ldh1,
                        int32_t K2, const void* W2, int32_t ldw2, const float* b2, const void* W3, int32_t ldw3,
                        const float* b3, const void* w4, float b4, int32_t act, float* out);
/* A sequence model's pooling and head on a merged batch, unbatched per
 * sequence (paper section 2.2.1, sub-graph batching of sequence models with
 * Batch/Unbatch), fused with the split: per sequence slot r with L = rows[r].aux
 * real tokens (clamped to [0, seq_T]), pooled = mean of H[r*T + t, :D] over t < L (fp32; tokens past L
 * are never read), then out[rows[r].out + j] = act(Wh pooled + bh)[j], j < n_out
 * (act RB_ACT_SOFTMAX or RB_ACT_NONE; D <= 1024, n_out <= 16).
 * packed_rows > 0: packed tokens: token t of slot r is row rows[r].lens + t of
 * H [packed_rows, ldh]; a sequence whose rows would leave H pools nothing. */
rb_status rb_k_seqpool(void* stream, const rb_k_row* rows, int32_t n_seqs, int32_t seq_T, int64_t packed_rows,
                       const float* H, int32_t ldh, int32_t D, const float* Wh, const float* bh, int32_t n_out,
                       int32_t act, float* out);
/* Split a merged run's output back to its callers (paper section 2.2.1,
 * each caller gets exactly its own rows): out[rows[r].out + j] = Y[r, j] for
 * real rows, j < d_out; padding rows are never copied. */
rb_status rb_k_split(void* stream, const rb_k_row* rows, int32_t n_rows_total, const float* Y, int32_t ldy,
                     int32_t d_out, float* out);

#ifdef __cplusplus
}
#endif
#endif /* RB_H */
