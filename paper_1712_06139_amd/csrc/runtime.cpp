// Host runtime of the request-batching library: contexts, models, batching
// queues, the round-robin scheduler on a simulated clock, and the executor
// that turns dispatched batches into launch chains on a HIP stream.
//
// Paper, section 2.2.1: requests for each servable (version) wait in their own
// batching queue, are merged by concatenating their inputs, and the queues
// share one device in round-robin order; the set of queues changes as
// servables come and go. Section 2.1 (and the introduction): a big free of a
// servable's memory happens on a manager thread, never an inference thread.
//
// Formation, padding, clock and tie rules (the paper gives none):
//  - next-fit in arrival order: a batch closes when full, when the next
//    request would overflow it (that request opens the next batch), when its
//    timeout (from its first request's arrival) expires, or, in a replay, at
//    the last arrival for count-only queues;
//  - padded size = smallest allowed size >= real size (or the real size);
//  - one simulated serial device: when it is free, the first queue after the
//    last-served one (cyclic in queue-id order) holding a closed batch gets its
//    oldest closed batch dispatched, and the device is busy for the queue's
//    service time at that padded size;
//  - events at one timestamp: timeouts (queue-id order), arrivals (request
//    order), end-of-trace close, then dispatch.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <climits>
#include <cmath>
#include <condition_variable>
#include <cstdint>
#include <cstring>
#include <deque>
#include <map>
#include <memory>
#include <mutex>
#include <new>
#include <string>
#include <thread>
#include <vector>

#include "../../include/rb.h"

// kernels.hip: reads a buffer on the stream, leaving only its clean lines in the caches
void rb_scrub_caches(hipStream_t stream, const void* buf, size_t bytes, unsigned* sink);
// kernels.hip: sets n row-map entries to padding
void rb_fill_padding_rows(hipStream_t stream, rb_k_row* rows, int64_t n);
// kernels.hip: the per-device address of the static scratch array (set up once
// per device; nullptr before that succeeded)
rb_status rb_static_scratch_setup(int device);
void* rb_static_scratch(int device);

namespace {

constexpr int64_t NO_TIMEOUT = INT64_MAX;
constexpr int KPAD = 64;       // every contraction dimension is padded to a multiple of this
constexpr int NPAD_BF16 = 128; // output widths: the bf16 GEMM tile is 128 wide, the fp32 one 64
constexpr int NPAD_F32 = 64;
constexpr int N_SLOTS = 4;     // host/device staging slots in flight
constexpr int CHUNK_WINDOWS = 32;
constexpr size_t SCRUB_BYTES = (size_t)512 << 20;  // cold-cache profiling: more than L2 + Infinity Cache

inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

inline uint16_t host_f2bf(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

struct DevFree {  // device memory of a released model, for the deleter thread
  std::vector<void*> ptrs;
};

}  // namespace

// ---------------------------------------------------------------- objects

struct rb_ctx {
  int device = -1;
  int n_models = 0, n_scheds = 0;
  int64_t next_model_id = 1;
  // deleter thread: frees device memory after the events it waits on
  std::thread deleter;
  std::mutex mu;
  std::condition_variable cv;
  std::deque<DevFree> pending;
  bool stop = false;
};

struct DevLayer {
  int K = 0, N = 0, Kp = 0, Np = 0, act = 0;
  void* w = nullptr;   // [Np, Kp] bf16 or fp32, zero padded
  float* b = nullptr;  // [Np] zero padded
};

struct rb_model {
  rb_ctx* ctx = nullptr;
  int64_t id = 0;
  int kind = 0, dtype = 0;
  int d_in = 0, d_out = 0;
  std::vector<DevLayer> layers;
  bool head_last = false;  // last layer (fan_out 1, bf16) runs as the fused head
  float head_bias = 0.f;
  int n_tables = 0, emb_dim = 0, n_dense = 0;
  int64_t table_rows = 0;
  std::vector<void*> tables;
  void** tables_dev = nullptr;
  float* sp_w = nullptr;
  float* sp_b = nullptr;
  int sp_in = 0, sp_out = 0, sp_act = 0;
  std::atomic<int> bound{0};  // queues serving it
  // versions of one servable share a lineage: a scheduler keys its work
  // buffers and launch stream by lineage, so a new version takes them over
  // in stream order (rb_queue_set_model)
  int64_t lineage = 0;
  hipStream_t upload = nullptr;  // private non-blocking stream of rb_model_create
  std::vector<void*> allocs;
  // references: the caller's handle (until rb_model_destroy) and one per
  // staging slot whose device work runs the model (until the slot retires,
  // after that work has finished); the last one hands the device memory to
  // the context's deleter thread
  std::atomic<int64_t> refs{1};
};

namespace {

struct Batch {
  int64_t seq = 0;           // batch id in dispatch order
  std::vector<int64_t> reqs; // request indices (trace index, or serving request id)
  int s = 0, P = 0;
  int64_t close_ns = 0, dispatch_ns = 0, done_ns = 0;
};

// A batch the simulated clock dispatched, with its queue.
struct Disp {
  rb_queue* q = nullptr;
  Batch b;
};

// A served request submitted through rb_submit (host payload copied in).
struct HostReq {
  rb_queue* q = nullptr;
  int32_t n_rows = 0;
  int32_t d_out = 0;  // output width (its queue may change version or be held meanwhile)
  std::vector<float> dense;
  std::vector<int32_t> lens, ids;
  std::vector<float> out;
  int state = 0;      // 0 queued, 1 dispatched, 2 done, 3 collected, 4 failed (its window's launch failed)
  int slot = -1;      // staging slot holding its output while in flight
  int64_t out_off = 0;  // offset of its rows in the slot's output staging
};

struct Work {  // per (scheduler, model) device buffers, sized for the largest group seen
  int64_t rows_cap = 0, slots_cap = 0;
  void* X = nullptr;
  void* A = nullptr;
  void* B = nullptr;
  float* Y = nullptr;
  rb_k_row* rows = nullptr;
};

struct Group {  // the batches of one queue inside one window
  rb_queue* q = nullptr;
  std::vector<rb_k_batch> batches;
  std::vector<rb_k_req> reqs;
  int64_t slots = 0;   // sum of padded sizes
  int64_t tokens = 0;  // seqpool: real tokens of its requests (packed rows)
};


struct Slot {
  hipEvent_t ev = nullptr;
  bool busy = false;
  char* host = nullptr;
  char* dev = nullptr;
  size_t cap = 0;
  // models its device work runs (one reference each, dropped on retire)
  std::vector<rb_model*> models;
  // serving mode: payload arenas and the output staging of one batch
  std::vector<int64_t> serving_reqs;
  float* host_out = nullptr;
  size_t out_cap = 0;
};

struct Prof {
  std::string name;
  hipEvent_t a, b;
};

}  // namespace

// What requests of a queue must look like: the bound version's interface,
// kept while the queue is held between versions (no version bound).
struct QShape {
  int kind = 0, dtype = 0, d_in = 0, d_out = 0, n_dense = 0, n_tables = 0;
  int64_t table_rows = 0;
};

QShape shape_of(const rb_model* m) {
  return QShape{m->kind, m->dtype, m->d_in, m->d_out, m->n_dense, m->n_tables, m->table_rows};
}

struct rb_queue {
  rb_sched* s = nullptr;
  rb_model* m = nullptr;  // nullptr: held (resource-preserving transition)
  QShape shape;
  int id = 0;
  int B = 0;
  std::vector<int> allowed;
  int64_t T = NO_TIMEOUT;
  int bucket = 0;
  std::vector<int64_t> svc;
  // open batch
  std::vector<int64_t> open;
  int open_s = 0;
  int64_t open_t = 0;
  std::deque<Batch> closed;
  int64_t undispatched = 0;  // requests in the open batch or in closed batches
  int64_t window_ns = 0;     // simulated fixed device time of its launch chain in a window
  int64_t window_tail = 0;   // simulated further time until that chain's results are complete
  int64_t pending_run = 0;   // serving: batches the clock dispatched that have not run yet
};

struct rb_sched {
  rb_ctx* ctx = nullptr;
  rb_sched_opts opts{};
  hipStream_t stream = nullptr;
  // replay launch chains: one stream per model (lanes), or the main stream
  std::vector<hipStream_t> lanes;
  std::vector<hipEvent_t> lane_done;
  hipEvent_t ev_copy = nullptr;
  std::map<int64_t, int> lane_of;  // work key -> lane, in order of first use
  std::map<int64_t, int> pipe_next; // lineage -> work slot of its next launch chain
  // cold-cache profiling: written before every timed launch
  void* scrub = nullptr;
  std::vector<rb_queue*> queues;  // by id; null once destroyed
  int n_live_queues = 0;
  int64_t now = INT64_MIN;
  int64_t device_free = INT64_MIN;
  int last_served = -1;
  int64_t n_closed = 0;
  int64_t batch_seq = 0;
  int64_t window_seq = 0;  // simulated device dispatches (launch windows) so far
  // serving-mode requests, by request id
  std::vector<HostReq> hreqs;
  // serving: windows the clock dispatched whose batches have not run yet
  std::deque<std::vector<Disp>> ready;
  // what the last rb_run_next / rb_run_window returned (its pointers' targets)
  std::vector<uint64_t> last_req_ids;
  std::vector<rb_batch_info> last_infos;
  // executor
  std::map<int64_t, Work> work;
  std::vector<Group> window;     // current window, one group per queue
  int window_batches = 0;
  std::vector<std::vector<Group>> chunk;  // closed windows waiting for a flush
  Slot slots[N_SLOTS];
  int next_slot = 0;
  int* err_dev = nullptr;
  // trace replay arenas (device pointers of the current rb_sim_run)
  const float* a_dense = nullptr;
  int64_t a_dense_len = 0;
  const int32_t* a_lens = nullptr;
  int64_t a_lens_len = 0;
  const int32_t* a_ids = nullptr;
  int64_t a_ids_len = 0;
  float* a_out = nullptr;
  int64_t a_out_len = 0;
  // rb_run_group's work buffers, per servable lineage
  std::map<int64_t, Work> ext_work;
  // profiling
  std::vector<Prof> prof_pending;
  std::map<std::string, std::pair<int64_t, double>> prof;
  std::vector<hipEvent_t> ev_pool;
};

namespace {

bool hip_ok(hipError_t e) { return e == hipSuccess; }

void deleter_main(rb_ctx* c) {
  hipSetDevice(c->device);
  std::unique_lock<std::mutex> lk(c->mu);
  for (;;) {
    c->cv.wait(lk, [c] { return c->stop || !c->pending.empty(); });
    if (c->pending.empty() && c->stop) return;
    DevFree f = std::move(c->pending.front());
    c->pending.pop_front();
    lk.unlock();
    for (void* p : f.ptrs) hipFree(p);
    lk.lock();
  }
}

rb_status dev_alloc(rb_model* m, size_t bytes, void** out) {
  void* p = nullptr;
  if (!hip_ok(hipMalloc(&p, bytes))) return RB_ENOMEM;
  m->allocs.push_back(p);
  *out = p;
  return RB_OK;
}

// Host -> device copy of model data on the model's private non-blocking
// stream: a version loaded while a scheduler serves neither waits for nor
// holds up the scheduler's streams (the null stream would); only the loading
// thread waits, for its own copy.
bool copy_h2d(rb_model* m, void* dst, const void* src, size_t n) {
  return hip_ok(hipMemcpyAsync(dst, src, n, hipMemcpyHostToDevice, m->upload)) && hip_ok(hipStreamSynchronize(m->upload));
}

bool valid_hidden_act(int a) { return a == RB_ACT_NONE || a == RB_ACT_RELU; }
bool valid_last_act(int a) { return a == RB_ACT_NONE || a == RB_ACT_RELU || a == RB_ACT_SIGMOID; }

rb_status upload_layer(rb_model* m, const rb_layer_desc& L, DevLayer& d, bool bf16) {
  d.K = L.fan_in;
  d.N = L.fan_out;
  d.act = L.act;
  d.Kp = (int)round_up(L.fan_in, KPAD);
  d.Np = (int)round_up(L.fan_out, bf16 ? NPAD_BF16 : NPAD_F32);
  if (m->ctx->device < 0) return RB_OK;
  const size_t n = (size_t)d.Np * d.Kp;
  rb_status st;
  if (bf16) {
    std::vector<uint16_t> h(n, 0);
    for (int j = 0; j < d.N; ++j)
      for (int k = 0; k < d.K; ++k) h[(size_t)j * d.Kp + k] = host_f2bf(L.w[(size_t)j * d.K + k]);
    if ((st = dev_alloc(m, n * 2, &d.w)) != RB_OK) return st;
    if (!copy_h2d(m, d.w, h.data(), n * 2)) return RB_EDEVICE;
  } else {
    std::vector<float> h(n, 0.f);
    for (int j = 0; j < d.N; ++j) std::memcpy(&h[(size_t)j * d.Kp], L.w + (size_t)j * d.K, sizeof(float) * d.K);
    if ((st = dev_alloc(m, n * 4, &d.w)) != RB_OK) return st;
    if (!copy_h2d(m, d.w, h.data(), n * 4)) return RB_EDEVICE;
  }
  std::vector<float> hb(d.Np, 0.f);
  std::memcpy(hb.data(), L.b, sizeof(float) * d.N);
  void* pb = nullptr;
  if ((st = dev_alloc(m, (size_t)d.Np * 4, &pb)) != RB_OK) return st;
  d.b = (float*)pb;
  if (!copy_h2d(m, d.b, hb.data(), (size_t)d.Np * 4)) return RB_EDEVICE;
  return RB_OK;
}

void free_model_now(rb_model* m) {
  for (void* p : m->allocs) hipFree(p);
  m->allocs.clear();
}

void model_ref(rb_model* m) { m->refs.fetch_add(1, std::memory_order_relaxed); }

// Drop a reference; the last one hands the model's device memory to the
// context's deleter thread (never freed on the calling thread, which may be
// an inference thread) and frees the host object. Every device use of the
// model holds a reference until it has finished, so nothing waits here.
void model_unref(rb_model* m) {
  if (m->refs.fetch_sub(1, std::memory_order_acq_rel) != 1) return;
  rb_ctx* c = m->ctx;
  if (!m->allocs.empty()) {
    DevFree f;
    f.ptrs = std::move(m->allocs);
    {
      std::lock_guard<std::mutex> lk(c->mu);
      c->pending.push_back(std::move(f));
    }
    c->cv.notify_all();
  }
  delete m;
}

int padded_size(const rb_queue* q, int s) {
  if (q->allowed.empty()) return s;
  for (int a : q->allowed)
    if (a >= s) return a;
  return q->allowed.back();  // unreachable: s <= B == allowed.back()
}

int64_t service(const rb_queue* q, int P) {
  if (q->svc.empty()) return 0;
  return q->svc[std::min<size_t>((size_t)P, q->svc.size() - 1)];
}

void close_open(rb_queue* q, int64_t t) {
  Batch b;
  b.reqs.swap(q->open);
  b.s = q->open_s;
  b.P = padded_size(q, b.s);
  b.close_ns = t;
  q->closed.push_back(std::move(b));
  q->open_s = 0;
  q->s->n_closed++;
}

// Next-fit arrival of a request of n rows at time t.
void arrive(rb_queue* q, int64_t req, int n, int64_t t) {
  if (q->open_s > 0 && q->open_s + n > q->B) close_open(q, t);
  if (q->open_s == 0) q->open_t = t;
  q->open.push_back(req);
  q->open_s += n;
  q->undispatched++;
  if (q->open_s == q->B) close_open(q, t);
}

// Fire every timeout due at or before t (each queue's open batch closes at
// its own due time).
void fire_timeouts_upto(rb_sched* s, int64_t t) {
  for (rb_queue* q : s->queues)
    if (q && q->T != NO_TIMEOUT && q->open_s > 0 && q->open_t + q->T <= t) close_open(q, q->open_t + q->T);
}

// Timeouts due exactly at t, in queue-id order.
void fire_timeouts_at(rb_sched* s, int64_t t) {
  for (rb_queue* q : s->queues)
    if (q && q->T != NO_TIMEOUT && q->open_s > 0 && q->open_t + q->T == t) close_open(q, t);
}

int64_t next_timeout(const rb_sched* s) {
  int64_t best = INT64_MAX;
  for (const rb_queue* q : s->queues)
    if (q && q->T != NO_TIMEOUT && q->open_s > 0) best = std::min(best, q->open_t + q->T);
  return best;
}

rb_queue* pick_round_robin(rb_sched* s) {
  const int nq = (int)s->queues.size();
  for (int k = 1; k <= nq; ++k) {
    rb_queue* q = s->queues[(size_t)((s->last_served + k) % nq + nq) % nq];
    if (q && q->m && !q->closed.empty()) return q;  // held queues keep their batches
  }
  return nullptr;
}

// Some queue with a version bound holds a closed batch (held queues keep
// theirs until a version is set).
bool has_pickable(const rb_sched* s) {
  for (const rb_queue* q : s->queues)
    if (q && q->m && !q->closed.empty()) return true;
  return false;
}

// One dispatch of the simulated device at time t (the device is free): a
// launch window of up to window_batches closed batches, each the oldest
// closed batch of the next queue in round-robin order that holds one. The
// window holds the device for the window_ns of each queue it takes batches
// from plus service_ns[P] per batch; its batches complete the queues'
// window_tail later. Returns false when no queue holds a closed batch.
bool clock_dispatch(rb_sched* s, int64_t t, std::vector<Disp>& win) {
  win.clear();
  const int W = s->opts.window_batches;
  while ((int)win.size() < W) {
    rb_queue* q = pick_round_robin(s);
    if (!q) break;
    Disp d;
    d.q = q;
    d.b = std::move(q->closed.front());
    q->closed.pop_front();
    s->n_closed--;
    q->undispatched -= (int64_t)d.b.reqs.size();
    d.b.seq = s->batch_seq++;
    d.b.dispatch_ns = t;
    s->last_served = q->id;
    win.push_back(std::move(d));
  }
  if (win.empty()) return false;
  int64_t busy = 0, tail = 0;
  for (size_t i = 0; i < win.size(); ++i) {
    bool first = true;
    for (size_t j = 0; j < i && first; ++j) first = win[j].q != win[i].q;
    if (first) {
      busy += win[i].q->window_ns;
      tail += win[i].q->window_tail;
    }
    busy += service(win[i].q, win[i].b.P);
  }
  for (Disp& d : win) d.b.done_ns = t + busy + tail;
  s->device_free = t + busy;
  s->window_seq++;
  return true;
}

// Serving: run the simulated clock's events (timeouts, and device dispatches
// when the device is free and a batch waits) in time order, up to `limit`
// (exclusive, or inclusive with `incl`). Arrivals are not events here: every
// request submitted so far has been taken in at its arrival time, so a
// dispatch at time t sees every batch that closed at or before t. Dispatched
// windows wait in s->ready until rb_run_next / rb_run_window runs them.
void serve_until(rb_sched* s, int64_t limit, bool incl) {
  std::vector<Disp> win;
  for (;;) {
    int64_t e = next_timeout(s);
    if (has_pickable(s)) e = std::min(e, std::max(s->device_free, s->now));
    if (e == INT64_MAX || (incl ? e > limit : e >= limit)) break;
    fire_timeouts_at(s, e);
    s->now = std::max(s->now, e);
    while (s->device_free <= e && clock_dispatch(s, e, win)) {
      for (Disp& d : win) d.q->pending_run++;
      s->ready.push_back(std::move(win));
      win.clear();
    }
  }
}

// ---------------------------------------------------------------- executor

hipEvent_t ev_get(rb_sched* s) {
  if (!s->ev_pool.empty()) {
    hipEvent_t e = s->ev_pool.back();
    s->ev_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  hipEventCreate(&e);
  return e;
}

void prof_begin(rb_sched* s, hipStream_t st, hipEvent_t* a) {
  if (!s->opts.profile) return;
  if (s->scrub) rb_scrub_caches(st, s->scrub, SCRUB_BYTES, (unsigned*)s->err_dev);
  *a = ev_get(s);
  hipEventRecord(*a, st);
}

void prof_end(rb_sched* s, hipStream_t st, const char* name, hipEvent_t a) {
  if (!s->opts.profile) return;
  hipEvent_t b = ev_get(s);
  hipEventRecord(b, st);
  s->prof_pending.push_back(Prof{name, a, b});
}

void prof_collect(rb_sched* s) {
  for (Prof& p : s->prof_pending) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, p.a, p.b) == hipSuccess) {
      auto& e = s->prof[p.name];
      e.first += 1;
      e.second += ms;
    }
    s->ev_pool.push_back(p.a);
    s->ev_pool.push_back(p.b);
  }
  s->prof_pending.clear();
}

#define RB_LAUNCH(s, strm, name, call)         \
  do {                                         \
    hipEvent_t ev_a_ = nullptr;                \
    if (timed) prof_begin(s, strm, &ev_a_);    \
    rb_status st_ = (call);                    \
    if (timed) prof_end(s, strm, name, ev_a_); \
    if (st_ != RB_OK) return st_;              \
  } while (0)

int64_t group_rows(const rb_model* m, const rb_queue* q, int64_t slots) {
  return m->kind == RB_MODEL_SEQPOOL ? slots * q->bucket : slots;
}

// Drain every stream of the scheduler (main and lanes).
void sync_all(rb_sched* s) {
  hipStreamSynchronize(s->stream);
  for (hipStream_t l : s->lanes) hipStreamSynchronize(l);
}

// Stream of a model's launch chains in a replay.
// Work buffers and launch streams belong to (lineage, slot) pairs. When the
// lanes outnumber the lineages of a chunk at least PIPE_SLOTS times, a
// lineage's consecutive launch chains rotate over PIPE_SLOTS slots on their
// own lanes, so one window's gathers and another's GEMMs can run at once
// (with fewer lanes, each lineage keeps one slot and different models overlap
// instead); each slot's buffers are reused only on its own lane, in stream
// order.
constexpr int PIPE_SLOTS = 2;

int64_t work_key(const rb_model* m, int slot) { return m->lineage * PIPE_SLOTS + slot; }

int next_slot(rb_sched* s, const rb_model* m, bool pipe) {
  if (!pipe) return 0;
  int& n = s->pipe_next[m->lineage];
  const int k = n;
  n = (n + 1) % PIPE_SLOTS;
  return k;
}

hipStream_t lane_for(rb_sched* s, const rb_model* m, int slot) {
  if (s->lanes.empty()) return s->stream;
  const int64_t key = work_key(m, slot);
  auto it = s->lane_of.find(key);
  if (it == s->lane_of.end()) it = s->lane_of.emplace(key, (int)(s->lane_of.size() % s->lanes.size())).first;
  return s->lanes[(size_t)it->second];
}

// Bytes of a launch group's work buffers for R rows (padded batch rows, or
// sequence slots times the bucket) and S row-map entries: the row map, the
// assembled input X, two activation buffers A and B for the layers, and the
// fp32 output Y of the last layer.
struct WorkShape {
  size_t rows, x, ab, y;
};

WorkShape work_shape(const rb_model* m, int64_t R, int64_t S) {
  const size_t elt = m->dtype == RB_DT_BF16 ? 2 : 4;
  int maxN = 0;
  for (const DevLayer& L : m->layers) maxN = std::max(maxN, L.Np);
  return WorkShape{(size_t)S * sizeof(rb_k_row), (size_t)R * m->layers[0].Kp * elt, (size_t)R * maxN * elt,
                   (size_t)R * m->layers.back().Np * 4};
}

void free_work(Work& w) {
  hipFree(w.X);
  hipFree(w.A);
  hipFree(w.B);
  hipFree(w.Y);
  hipFree(w.rows);
  w = Work{};
}

// Grow work buffers to rows x slots (capacities only grow, both at once, so
// groups of different shapes never make the buffers shrink and grow back).
// The streams that may still use the old buffers are drained first.
rb_status grow_work(rb_sched* s, rb_model* m, Work& w, int64_t rows, int64_t slots, hipStream_t also) {
  if (rows <= w.rows_cap && slots <= w.slots_cap) return RB_OK;
  const int64_t R = std::max<int64_t>({rows, w.rows_cap, 64});
  const int64_t S = std::max<int64_t>({slots, w.slots_cap, 64});
  sync_all(s);
  if (also) hipStreamSynchronize(also);
  free_work(w);
  const WorkShape sh = work_shape(m, R, S);
  if (!hip_ok(hipMalloc(&w.X, sh.x)) || !hip_ok(hipMalloc(&w.A, sh.ab)) || !hip_ok(hipMalloc(&w.B, sh.ab)) ||
      !hip_ok(hipMalloc((void**)&w.Y, sh.y)) || !hip_ok(hipMalloc((void**)&w.rows, sh.rows))) {
    free_work(w);
    return RB_ENOMEM;
  }
  w.rows_cap = R;
  w.slots_cap = S;
  return RB_OK;
}

rb_status ensure_work(rb_sched* s, rb_model* m, int slot, int64_t rows, int64_t slots, Work** out) {
  Work& w = s->work[work_key(m, slot)];
  rb_status st = grow_work(s, m, w, rows, slots, nullptr);
  if (st != RB_OK) return st;
  *out = &w;
  return RB_OK;
}

// Launch chain of one group on stream st_h: route -> assemble | embbag ->
// layers -> head (alone or fused with the last hidden layer) | seqpool, or a
// last layer that writes the requests' outputs itself.
// A bf16 model whose last two hidden layers are ReLU layers of 512 and 256
// outputs ahead of a narrow head of 256 inputs: rb_k_mlp_tail runs them.
bool fused_tail(const rb_model* m) {
  if (m->dtype != RB_DT_BF16 || !m->head_last || m->layers.size() < 3) return false;
  const size_t nL = m->layers.size() - 1;
  const DevLayer& L2 = m->layers[nL - 2];
  const DevLayer& L3 = m->layers[nL - 1];
  const DevLayer& H = m->layers.back();
  return L2.Np == 512 && L2.act == RB_ACT_RELU && L2.Kp % 32 == 0 && L3.Np == 256 && L3.Kp == 512 &&
         L3.act == RB_ACT_RELU && H.K == 256;
}

// A bf16 model whose last hidden layer has 256 outputs ahead of a narrow
// head of 256 inputs: rb_k_gemm_head runs the two.
bool gemm_head(const rb_model* m) {
  if (m->dtype != RB_DT_BF16 || !m->head_last || m->layers.size() < 2) return false;
  const DevLayer& L = m->layers[m->layers.size() - 2];
  return L.N == 256 && L.Np == 256 && L.Kp % 64 == 0 && m->layers.back().K == 256;
}

// The chain of a group of n_batches batches of queue q holding `slots`
// padded rows (sequence slots) and `tokens` real tokens (seqpool), with work
// buffers w large enough for it; `timed`: HIP events around every launch when
// the scheduler profiles.
// Descriptors not built by this library start from a row map of padding
// (fill_rows).
rb_status run_chain(rb_sched* s, hipStream_t st_h, const rb_queue* q, int n_batches, int n_reqs, int64_t slots,
                    int64_t tokens, const Work* w, bool timed, bool fill_rows, const rb_k_batch* d_batches,
                    const rb_k_req* d_reqs, const float* dense, int64_t dense_len, const int32_t* lens,
                    int64_t lens_len, const int32_t* ids, int64_t ids_len, float* out, int64_t out_len) {
  const rb_model* m = q->m;
  const int64_t M = group_rows(m, q, slots);
  void* hs = (void*)st_h;
  const float pad = s->opts.pad_value;
  if (fill_rows) rb_fill_padding_rows(st_h, w->rows, slots);
  RB_LAUNCH(s, st_h, "route", rb_k_route(hs, m->kind, d_batches, n_batches, d_reqs, n_reqs, lens, lens_len, m->d_in,
                                         m->d_out, m->n_tables, w->rows, (int)slots, out_len, s->err_dev));
  const bool bf16 = m->dtype == RB_DT_BF16;
  const int Kp0 = m->layers[0].Kp;
  // sequence groups: padding tokens are not assembled and 64-token blocks of
  // them are not computed (every layer is row-wise and the pooling reads
  // tokens t < L only); with seq_pack the real tokens are packed into tokens
  // consecutive rows and the layers run on those rows alone
  const bool pack = m->kind == RB_MODEL_SEQPOOL && s->opts.seq_pack && !bf16;
  const bool seq_skip = m->kind == RB_MODEL_SEQPOOL && !pack && q->bucket % 64 == 0;
  const int64_t Ml = pack ? tokens : M;  // rows of the layers
  if (m->kind == RB_MODEL_RANKING) {
    auto emb = s->opts.emb_dedup ? rb_k_embbag_dedup : rb_k_embbag;
    RB_LAUNCH(s, st_h, "embbag", emb(hs, w->rows, (int)slots, lens, ids, ids_len, (const void* const*)m->tables_dev,
                                     m->n_tables, m->table_rows, m->emb_dim, dense, m->n_dense, w->X, Kp0, pad,
                                     s->err_dev));
  } else {
    RB_LAUNCH(s, st_h, "assemble", rb_k_assemble(hs, w->rows, (int)M, m->kind == RB_MODEL_SEQPOOL ? q->bucket : 0,
                                           pack ? 2 : (seq_skip ? 1 : 0), dense, dense_len, m->d_in, w->X, Kp0,
                                           bf16 ? 1 : 0, pad, s->err_dev));
  }
  const size_t nL = m->layers.size() - (m->head_last ? 1 : 0);
  // the last two hidden layers and the head in one kernel when they have its
  // shapes (bit-identical either way)
  const bool tail = fused_tail(m) && s->opts.fuse_mlp_tail;
  // otherwise a last hidden layer of 256 outputs and a 256-input head in one
  // kernel (bit-identical to the layer and the head run separately)
  const bool ghead = !tail && gemm_head(m);
  // a chain that ends in the split writes its last layer straight into the
  // requests' output rows (bit-identical to the layer and the split)
  const bool rows_out = !m->head_last && m->kind != RB_MODEL_SEQPOOL;
  void* h = w->X;
  int ldh = Kp0;
  for (size_t i = 0; i < nL - (tail ? 2 : 0) - (ghead ? 1 : 0); ++i) {
    const DevLayer& L = m->layers[i];
    const bool last = (i + 1 == nL) && !m->head_last;
    void* y = last ? (void*)w->Y : (i % 2 == 0 ? w->A : w->B);
    if (last && rows_out) {
      if (bf16)
        RB_LAUNCH(s, st_h, "gemm_bf16", rb_k_gemm_bf16_rows(hs, h, ldh, L.w, L.Kp, L.b, (int)Ml, L.Np, L.Kp, L.act,
                                                            w->rows, m->d_out, out));
      else
        RB_LAUNCH(s, st_h, "gemm_f32", rb_k_gemm_f32_rows(hs, (const float*)h, ldh, (const float*)L.w, L.Kp, L.b,
                                                          (int)Ml, L.Np, L.Kp, L.act, w->rows, m->d_out, out));
    } else if (bf16) {
      RB_LAUNCH(s, st_h, "gemm_bf16", rb_k_gemm_bf16(hs, h, ldh, L.w, L.Kp, L.b, y, L.Np, (int)Ml, L.Np, L.Kp, L.act,
                                               last ? 1 : 0));
    } else {
      RB_LAUNCH(s, st_h, "gemm_f32", rb_k_gemm_f32(hs, (const float*)h, ldh, (const float*)L.w, L.Kp, L.b, (float*)y,
                                             L.Np, (int)Ml, L.Np, L.Kp, L.act, seq_skip ? w->rows : nullptr,
                                             seq_skip ? q->bucket : 0));
    }
    h = y;
    ldh = L.Np;
  }
  if (tail) {
    const DevLayer& L2 = m->layers[nL - 2];
    const DevLayer& L3 = m->layers[nL - 1];
    const DevLayer& H = m->layers.back();
    RB_LAUNCH(s, st_h, "mlp_tail", rb_k_mlp_tail(hs, w->rows, (int)slots, h, ldh, L2.Kp, L2.w, L2.Kp, L2.b, L3.w,
                                                 L3.Kp, L3.b, H.w, m->head_bias, H.act, out));
  } else if (ghead) {
    const DevLayer& L3 = m->layers[nL - 1];
    const DevLayer& H = m->layers.back();
    RB_LAUNCH(s, st_h, "gemm_head", rb_k_gemm_head(hs, h, ldh, L3.w, L3.Kp, L3.b, (int)Ml, L3.Kp, L3.act, w->rows, H.w,
                                                   m->head_bias, H.act, out));
  } else if (m->head_last) {
    const DevLayer& L = m->layers.back();
    RB_LAUNCH(s, st_h, "head", rb_k_head(hs, w->rows, (int)slots, h, ldh, L.w, m->head_bias, L.K, L.act, out));
  } else if (m->kind == RB_MODEL_SEQPOOL) {
    RB_LAUNCH(s, st_h, "seqpool", rb_k_seqpool(hs, w->rows, (int)slots, q->bucket, pack ? std::max<int64_t>(Ml, 1) : 0,
                                         (const float*)h, ldh, m->sp_in, m->sp_w, m->sp_b, m->sp_out, m->sp_act,
                                         out));
  }
  return RB_OK;
}

// Launch chain of one group of a window on stream st_h, with the scheduler's
// work buffers of (lineage, slot).
rb_status run_group(rb_sched* s, hipStream_t st_h, int slot, const Group& g, const rb_k_batch* d_batches,
                    const rb_k_req* d_reqs, const float* dense, int64_t dense_len, const int32_t* lens,
                    int64_t lens_len, const int32_t* ids, int64_t ids_len, float* out, int64_t out_len) {
  rb_model* m = g.q->m;
  Work* w = nullptr;
  rb_status st = ensure_work(s, m, slot, group_rows(m, g.q, g.slots), g.slots, &w);
  if (st != RB_OK) return st;
  return run_chain(s, st_h, g.q, (int)g.batches.size(), (int)g.reqs.size(), g.slots, g.tokens, w, true, false,
                   d_batches, d_reqs, dense, dense_len, lens, lens_len, ids, ids_len, out, out_len);
}

// A slot whose work has finished: hand its serving outputs to their requests.
void retire_slot(rb_sched* s, Slot& sl) {
  for (int64_t id : sl.serving_reqs) {
    HostReq& r = s->hreqs[(size_t)id];
    const int64_t n = (int64_t)r.n_rows * r.d_out;
    r.out.assign(sl.host_out + r.out_off, sl.host_out + r.out_off + n);
    r.state = 2;
    r.slot = -1;
  }
  sl.serving_reqs.clear();
  for (rb_model* m : sl.models) model_unref(m);
  sl.models.clear();
  sl.busy = false;
}

// The slot's device work runs model m: hold a reference until it retires.
void slot_hold(Slot& sl, rb_model* m) {
  if (std::find(sl.models.begin(), sl.models.end(), m) != sl.models.end()) return;
  model_ref(m);
  sl.models.push_back(m);
}

// Reuse a staging slot: wait for its previous work, retire it, and make room
// for `bytes` of tables/payload and `out_bytes` of outputs.
rb_status acquire_slot(rb_sched* s, size_t bytes, size_t out_bytes, Slot** out) {
  Slot& sl = s->slots[s->next_slot];
  s->next_slot = (s->next_slot + 1) % N_SLOTS;
  if (sl.busy) {
    if (!hip_ok(hipEventSynchronize(sl.ev))) return RB_EDEVICE;
    retire_slot(s, sl);
  }
  if (bytes > sl.cap) {
    const size_t cap = std::max(bytes, sl.cap * 2);
    hipHostFree(sl.host);
    hipFree(sl.dev);
    sl.host = nullptr;
    sl.dev = nullptr;
    sl.cap = 0;
    if (!hip_ok(hipHostMalloc((void**)&sl.host, cap, hipHostMallocDefault))) return RB_ENOMEM;
    if (!hip_ok(hipMalloc((void**)&sl.dev, cap))) return RB_ENOMEM;
    sl.cap = cap;
  }
  if (out_bytes > sl.out_cap) {
    hipHostFree(sl.host_out);
    sl.host_out = nullptr;
    sl.out_cap = 0;
    if (!hip_ok(hipHostMalloc((void**)&sl.host_out, out_bytes, hipHostMallocDefault))) return RB_ENOMEM;
    sl.out_cap = out_bytes;
  }
  if (!sl.ev) hipEventCreateWithFlags(&sl.ev, hipEventDisableTiming);
  *out = &sl;
  return RB_OK;
}

// Flush the closed windows of a replay: one host->device copy of every
// group's batch and request tables, then each group's launch chain.
rb_status flush_chunk(rb_sched* s) {
  if (s->chunk.empty()) return RB_OK;
  size_t bytes = 0;
  for (auto& win : s->chunk)
    for (Group& g : win)
      bytes += round_up((int64_t)(g.batches.size() * sizeof(rb_k_batch)), 256) +
               round_up((int64_t)(g.reqs.size() * sizeof(rb_k_req)), 256);
  Slot* sl = nullptr;
  rb_status st = acquire_slot(s, bytes, 0, &sl);
  if (st != RB_OK) return st;
  size_t off = 0;
  std::vector<std::pair<size_t, size_t>> offs;
  for (auto& win : s->chunk)
    for (Group& g : win) {
      const size_t bb = g.batches.size() * sizeof(rb_k_batch), rr = g.reqs.size() * sizeof(rb_k_req);
      std::memcpy(sl->host + off, g.batches.data(), bb);
      const size_t o1 = off;
      off += round_up((int64_t)bb, 256);
      std::memcpy(sl->host + off, g.reqs.data(), rr);
      offs.push_back({o1, off});
      off += round_up((int64_t)rr, 256);
    }
  if (!hip_ok(hipMemcpyAsync(sl->dev, sl->host, off, hipMemcpyHostToDevice, s->stream))) return RB_EDEVICE;
  for (auto& win : s->chunk)
    for (Group& g : win) slot_hold(*sl, g.q->m);
  std::vector<int64_t> lin;
  for (auto& win : s->chunk)
    for (Group& g : win) lin.push_back(g.q->m->lineage);
  std::sort(lin.begin(), lin.end());
  const size_t n_lin = (size_t)(std::unique(lin.begin(), lin.end()) - lin.begin());
  const bool pipe = s->lanes.size() >= (size_t)PIPE_SLOTS * n_lin;
  // every group's work-buffer slot and launch stream, in launch order. A
  // chunk of one group runs on the main stream: nothing could overlap it, and
  // cross-stream events only add latency (its slot's earlier work on a lane
  // was joined into the main stream, and later lane work waits for a copy
  // enqueued after it, so the slot's buffers stay in stream order).
  std::vector<std::pair<int, hipStream_t>> where;
  for (auto& win : s->chunk)
    for (Group& g : win) {
      const int slot = next_slot(s, g.q->m, pipe);
      where.push_back({slot, lane_for(s, g.q->m, slot)});
    }
  if (where.size() == 1) where[0].second = s->stream;
  // the lanes this chunk launches on start after the copy; the main stream
  // (and the slot's event) after each of them. Lanes the chunk does not use
  // are left alone: their earlier work was joined by their own chunks.
  std::vector<size_t> used;
  if (!s->lanes.empty()) {
    for (const auto& w : where) {
      const size_t i = (size_t)(std::find(s->lanes.begin(), s->lanes.end(), w.second) - s->lanes.begin());
      if (i < s->lanes.size() && std::find(used.begin(), used.end(), i) == used.end()) used.push_back(i);
    }
    hipEventRecord(s->ev_copy, s->stream);
    for (size_t i : used) hipStreamWaitEvent(s->lanes[i], s->ev_copy, 0);
  }
  size_t gi = 0;
  for (auto& win : s->chunk) {
    for (Group& g : win) {
      st = run_group(s, where[gi].second, where[gi].first, g, (const rb_k_batch*)(sl->dev + offs[gi].first),
                     (const rb_k_req*)(sl->dev + offs[gi].second), s->a_dense, s->a_dense_len, s->a_lens,
                     s->a_lens_len, s->a_ids, s->a_ids_len, s->a_out, s->a_out_len);
      ++gi;
      if (st != RB_OK) break;
    }
    if (st != RB_OK) break;
  }
  // also after a failed launch: the copy out of the slot's host buffer and
  // any launched work stay fenced by the slot's event, so the buffer is not
  // rewritten and the models it holds are not released before they finish
  for (size_t i : used) {
    hipEventRecord(s->lane_done[i], s->lanes[i]);
    hipStreamWaitEvent(s->stream, s->lane_done[i], 0);
  }
  hipEventRecord(sl->ev, s->stream);
  sl->busy = true;
  s->chunk.clear();
  return st;
}

void close_window(rb_sched* s) {
  if (s->window.empty()) return;
  s->chunk.push_back(std::move(s->window));
  s->window.clear();
  s->window_batches = 0;
}

// Seqpool: give request r its first packed token row in group g and count its
// tokens (its dense extent over d_in, at most n_rows full buckets: a request
// whose extent is inconsistent is rejected by the routing, and the packed rows
// of the group never exceed its padded token rows).
void add_tokens(Group& g, const rb_model* m, rb_k_req& r) {
  r.tok_off = (int32_t)g.tokens;
  if (m->kind != RB_MODEL_SEQPOOL) return;
  const int64_t t = (r.dense_end - r.dense_off) / m->d_in;
  g.tokens += std::min<int64_t>(std::max<int64_t>(t, 0), (int64_t)r.n_rows * g.q->bucket);
}

// Add a dispatched batch (its requests already described) to the window.
void window_add(rb_sched* s, rb_queue* q, const Batch& b, std::vector<rb_k_req>& reqs) {
  Group* g = nullptr;
  for (Group& x : s->window)
    if (x.q == q) g = &x;
  if (!g) {
    s->window.push_back(Group{});
    g = &s->window.back();
    g->q = q;
  }
  rb_k_batch kb;
  kb.req_begin = (int32_t)g->reqs.size();
  kb.n_req = (int32_t)reqs.size();
  kb.row_base = (int32_t)g->slots;
  kb.padded = b.P;
  kb.real = b.s;
  kb.seq_T = q->m->kind == RB_MODEL_SEQPOOL ? q->bucket : 0;
  g->batches.push_back(kb);
  for (rb_k_req& r : reqs) add_tokens(*g, q->m, r);
  g->reqs.insert(g->reqs.end(), reqs.begin(), reqs.end());
  g->slots += b.P;
  s->window_batches++;
}

}  // namespace

// ================================================================== C ABI

extern "C" {

const char* rb_status_str(rb_status s) {
  switch (s) {
    case RB_OK: return "ok";
    case RB_EINVAL: return "invalid argument";
    case RB_EBUSY: return "busy";
    case RB_EAGAIN: return "not ready";
    case RB_EEMPTY: return "nothing to run";
    case RB_ESIZE: return "buffer too small";
    case RB_ENOENT: return "no such request";
    case RB_EDEVICE: return "device error";
    case RB_ENOMEM: return "out of memory";
    case RB_ERANGE: return "id or length out of range";
    default: return "unknown status";
  }
}

rb_status rb_ctx_create(int32_t hip_device, rb_ctx** out) {
  if (!out) return RB_EINVAL;
  rb_ctx* c = new (std::nothrow) rb_ctx();
  if (!c) return RB_ENOMEM;
  if (hip_device >= 0) {
    int n = 0;
    if (!hip_ok(hipGetDeviceCount(&n)) || hip_device >= n || !hip_ok(hipSetDevice(hip_device))) {
      delete c;
      return RB_EDEVICE;
    }
    c->device = hip_device;
    // the allocation-free entry point's scratch on this device: looked up
    // once, here (a failure makes only that entry point fail)
    (void)rb_static_scratch_setup(hip_device);
    c->deleter = std::thread(deleter_main, c);
  }
  *out = c;
  return RB_OK;
}

rb_status rb_ctx_destroy(rb_ctx* c) {
  if (!c) return RB_OK;
  if (c->n_models || c->n_scheds) return RB_EBUSY;
  if (c->deleter.joinable()) {
    {
      std::lock_guard<std::mutex> lk(c->mu);
      c->stop = true;
    }
    c->cv.notify_all();
    c->deleter.join();
  }
  delete c;
  return RB_OK;
}

rb_status rb_model_create(rb_ctx* ctx, const rb_model_desc* d, rb_model** out) {
  if (!ctx || !d || !out) return RB_EINVAL;
  if (d->kind < RB_MODEL_MLP || d->kind > RB_MODEL_SEQPOOL) return RB_EINVAL;
  if (d->dtype != RB_DT_F32 && d->dtype != RB_DT_BF16) return RB_EINVAL;
  if (d->n_layers < 1 || !d->layers) return RB_EINVAL;
  const bool dev = ctx->device >= 0;
  for (int i = 0; i < d->n_layers; ++i) {
    const rb_layer_desc& L = d->layers[i];
    if (L.fan_in < 1 || L.fan_out < 1) return RB_EINVAL;
    if (dev && (!L.w || !L.b)) return RB_EINVAL;
    if (i + 1 < d->n_layers && L.fan_out != d->layers[i + 1].fan_in) return RB_EINVAL;
    if (i + 1 < d->n_layers ? !valid_hidden_act(L.act) : !valid_last_act(L.act)) return RB_EINVAL;
  }
  const rb_layer_desc& last = d->layers[d->n_layers - 1];
  if (d->kind == RB_MODEL_RANKING) {
    if (d->dtype != RB_DT_BF16 || d->emb_dim != 64 || d->n_tables < 1 || d->n_tables > 64 || d->n_dense < 0 ||
        d->table_rows < 1 || d->table_rows > INT32_MAX)
      return RB_EINVAL;
    if (d->layers[0].fan_in != d->n_tables * d->emb_dim + d->n_dense) return RB_EINVAL;
    if (dev && !d->tables) return RB_EINVAL;
  }
  if (d->kind == RB_MODEL_SEQPOOL) {
    if (d->dtype != RB_DT_F32) return RB_EINVAL;
    if (d->head.fan_in != last.fan_out || d->head.fan_out < 1 || d->head.fan_out > 16 || d->head.fan_in > 1024)
      return RB_EINVAL;
    if (d->head.act != RB_ACT_SOFTMAX && d->head.act != RB_ACT_NONE) return RB_EINVAL;
    if (dev && (!d->head.w || !d->head.b)) return RB_EINVAL;
    if (last.act == RB_ACT_SIGMOID) return RB_EINVAL;
  }
  rb_model* m = new (std::nothrow) rb_model();
  if (!m) return RB_ENOMEM;
  m->ctx = ctx;
  {
    std::lock_guard<std::mutex> lk(ctx->mu);
    m->id = ctx->next_model_id++;
  }
  m->lineage = m->id;
  m->kind = d->kind;
  m->dtype = d->dtype;
  m->d_in = d->kind == RB_MODEL_RANKING ? d->n_dense : d->layers[0].fan_in;
  m->d_out = d->kind == RB_MODEL_SEQPOOL ? d->head.fan_out : last.fan_out;
  m->n_tables = d->kind == RB_MODEL_RANKING ? d->n_tables : 0;
  m->emb_dim = d->emb_dim;
  m->n_dense = d->n_dense;
  m->table_rows = d->table_rows;
  m->head_last = d->kind != RB_MODEL_SEQPOOL && d->dtype == RB_DT_BF16 && last.fan_out == 1 && d->n_layers >= 2 &&
                 (last.act == RB_ACT_SIGMOID || last.act == RB_ACT_NONE);
  if (dev) {
    hipSetDevice(ctx->device);
    if (!hip_ok(hipStreamCreateWithFlags(&m->upload, hipStreamNonBlocking))) {
      delete m;
      return RB_EDEVICE;
    }
  }
  m->layers.resize(d->n_layers);
  rb_status st = RB_OK;
  for (int i = 0; i < d->n_layers && st == RB_OK; ++i) {
    const rb_layer_desc& L = d->layers[i];
    if (i == d->n_layers - 1 && m->head_last) {
      // fused head: one bf16 weight row, bias kept on the host
      DevLayer& H = m->layers[i];
      H.K = L.fan_in;
      H.N = 1;
      H.Kp = (int)round_up(L.fan_in, KPAD);
      H.Np = 1;
      H.act = L.act;
      if (dev) {
        std::vector<uint16_t> h(H.Kp, 0);
        for (int k = 0; k < L.fan_in; ++k) h[k] = host_f2bf(L.w[k]);
        st = dev_alloc(m, (size_t)H.Kp * 2, &H.w);
        if (st == RB_OK && !copy_h2d(m, H.w, h.data(), (size_t)H.Kp * 2)) st = RB_EDEVICE;
        m->head_bias = L.b[0];
      }
    } else {
      st = upload_layer(m, L, m->layers[i], d->dtype == RB_DT_BF16);
    }
  }
  if (st == RB_OK && d->kind == RB_MODEL_RANKING && dev) {
    const size_t per = (size_t)d->table_rows * d->emb_dim;
    std::vector<uint16_t> h(per);
    for (int t = 0; t < d->n_tables && st == RB_OK; ++t) {
      if (!d->tables[t]) {
        st = RB_EINVAL;
        break;
      }
      for (size_t i = 0; i < per; ++i) h[i] = host_f2bf(d->tables[t][i]);
      void* p = nullptr;
      st = dev_alloc(m, per * 2, &p);
      if (st == RB_OK && !copy_h2d(m, p, h.data(), per * 2)) st = RB_EDEVICE;
      m->tables.push_back(p);
    }
    if (st == RB_OK) {
      void* p = nullptr;
      st = dev_alloc(m, sizeof(void*) * d->n_tables, &p);
      m->tables_dev = (void**)p;
      if (st == RB_OK &&
          !copy_h2d(m, m->tables_dev, m->tables.data(), sizeof(void*) * d->n_tables))
        st = RB_EDEVICE;
    }
  }
  if (st == RB_OK && d->kind == RB_MODEL_SEQPOOL) {
    m->sp_in = d->head.fan_in;
    m->sp_out = d->head.fan_out;
    m->sp_act = d->head.act;
    if (dev) {
      void *pw = nullptr, *pb = nullptr;
      const size_t nw = (size_t)m->sp_in * m->sp_out;
      st = dev_alloc(m, nw * 4, &pw);
      if (st == RB_OK) st = dev_alloc(m, (size_t)m->sp_out * 4, &pb);
      if (st == RB_OK && (!copy_h2d(m, pw, d->head.w, nw * 4) ||
                          !copy_h2d(m, pb, d->head.b, (size_t)m->sp_out * 4)))
        st = RB_EDEVICE;
      m->sp_w = (float*)pw;
      m->sp_b = (float*)pb;
    }
  }
  if (m->upload) hipStreamDestroy(m->upload);
  m->upload = nullptr;
  if (st != RB_OK) {
    free_model_now(m);
    delete m;
    return st;
  }
  {
    std::lock_guard<std::mutex> lk(ctx->mu);
    ctx->n_models++;
  }
  *out = m;
  return RB_OK;
}

rb_status rb_model_info(const rb_model* m, int32_t* d_in, int32_t* d_out) {
  if (!m || !d_in || !d_out) return RB_EINVAL;
  *d_in = m->d_in;
  *d_out = m->d_out;
  return RB_OK;
}

rb_status rb_model_destroy(rb_model* m) {
  if (!m) return RB_OK;
  if (m->bound) return RB_EBUSY;
  rb_ctx* c = m->ctx;
  {
    std::lock_guard<std::mutex> lk(c->mu);
    c->n_models--;
  }
  // the caller's reference; dispatched work may still hold others
  model_unref(m);
  return RB_OK;
}

rb_status rb_sched_create(rb_ctx* ctx, const rb_sched_opts* o, rb_sched** out) {
  if (!ctx || !o || !out) return RB_EINVAL;
  if (o->mode != RB_MODE_DEVICE && o->mode != RB_MODE_NO_DEVICE) return RB_EINVAL;
  if (o->mode == RB_MODE_DEVICE && ctx->device < 0) return RB_EDEVICE;
  if (o->window_batches < 1 || o->n_streams < 0 || o->n_streams > RB_MAX_STREAMS) return RB_EINVAL;
  if (o->seq_pack < 0 || o->seq_pack > 1) return RB_EINVAL;
  if (o->clocked_windows < 0 || o->clocked_windows > 1) return RB_EINVAL;
  if (o->emb_dedup < 0 || o->emb_dedup > 1) return RB_EINVAL;
  if (o->fuse_mlp_tail < 0 || o->fuse_mlp_tail > 1) return RB_EINVAL;
  if (o->profile < 0 || o->profile > 2) return RB_EINVAL;
  rb_sched* s = new (std::nothrow) rb_sched();
  if (!s) return RB_ENOMEM;
  s->ctx = ctx;
  s->opts = *o;
  if (o->mode == RB_MODE_DEVICE) {
    hipSetDevice(ctx->device);
    if (!hip_ok(hipStreamCreateWithFlags(&s->stream, hipStreamNonBlocking)) ||
        !hip_ok(hipMalloc((void**)&s->err_dev, sizeof(int))) || !hip_ok(hipMemset(s->err_dev, 0, sizeof(int)))) {
      if (s->stream) hipStreamDestroy(s->stream);
      delete s;
      return RB_EDEVICE;
    }
    bool ok = true;
    if (o->profile == 2) ok = hip_ok(hipMalloc(&s->scrub, SCRUB_BYTES)) && hip_ok(hipMemset(s->scrub, 0, SCRUB_BYTES));
    if (ok && o->n_streams > 1) {
      ok = hip_ok(hipEventCreateWithFlags(&s->ev_copy, hipEventDisableTiming));
      for (int i = 0; ok && i < o->n_streams; ++i) {
        hipStream_t l = nullptr;
        hipEvent_t e = nullptr;
        ok = hip_ok(hipStreamCreateWithFlags(&l, hipStreamNonBlocking));
        if (ok) s->lanes.push_back(l);
        ok = ok && hip_ok(hipEventCreateWithFlags(&e, hipEventDisableTiming));
        if (ok) s->lane_done.push_back(e);
      }
    }
    if (!ok) {
      if (s->scrub) hipFree(s->scrub);
      for (hipStream_t l : s->lanes) hipStreamDestroy(l);
      for (hipEvent_t e : s->lane_done) hipEventDestroy(e);
      if (s->ev_copy) hipEventDestroy(s->ev_copy);
      hipFree(s->err_dev);
      hipStreamDestroy(s->stream);
      delete s;
      return RB_EDEVICE;
    }
  }
  ctx->n_scheds++;
  *out = s;
  return RB_OK;
}

rb_status rb_sched_destroy(rb_sched* s) {
  if (!s) return RB_OK;
  if (s->n_live_queues) return RB_EBUSY;
  if (s->stream) {
    sync_all(s);
    // the device work is done: slots drop their model references
    for (Slot& sl : s->slots)
      if (sl.busy) retire_slot(s, sl);
    for (auto& kv : s->work) free_work(kv.second);
    for (auto& kv : s->ext_work) free_work(kv.second);
    for (Slot& sl : s->slots) {
      hipHostFree(sl.host);
      hipFree(sl.dev);
      hipHostFree(sl.host_out);
      if (sl.ev) hipEventDestroy(sl.ev);
    }
    for (Prof& p : s->prof_pending) {
      hipEventDestroy(p.a);
      hipEventDestroy(p.b);
    }
    for (hipEvent_t e : s->ev_pool) hipEventDestroy(e);
    hipFree(s->err_dev);
    if (s->scrub) hipFree(s->scrub);
    for (hipStream_t l : s->lanes) hipStreamDestroy(l);
    for (hipEvent_t e : s->lane_done) hipEventDestroy(e);
    if (s->ev_copy) hipEventDestroy(s->ev_copy);
    hipStreamDestroy(s->stream);
  }
  s->ctx->n_scheds--;
  delete s;
  return RB_OK;
}

rb_status rb_sync(rb_sched* s) {
  if (!s) return RB_EINVAL;
  if (!s->stream) return RB_OK;
  if (!hip_ok(hipStreamSynchronize(s->stream))) return RB_EDEVICE;
  for (hipStream_t l : s->lanes)
    if (!hip_ok(hipStreamSynchronize(l))) return RB_EDEVICE;
  for (Slot& sl : s->slots)
    if (sl.busy) retire_slot(s, sl);
  prof_collect(s);
  int err = 0;
  if (!hip_ok(hipMemcpy(&err, s->err_dev, sizeof(int), hipMemcpyDeviceToHost))) return RB_EDEVICE;
  if (err) {
    hipMemset(s->err_dev, 0, sizeof(int));
    return RB_ERANGE;
  }
  return RB_OK;
}

rb_status rb_sched_kernel_stats(rb_sched* s, const char* kernel, int64_t* launches, double* total_ms) {
  if (!s || !kernel || !launches || !total_ms) return RB_EINVAL;
  auto it = s->prof.find(kernel);
  *launches = it == s->prof.end() ? 0 : it->second.first;
  *total_ms = it == s->prof.end() ? 0.0 : it->second.second;
  return RB_OK;
}

rb_status rb_sched_stream(rb_sched* s, void** stream) {
  if (!s || !stream) return RB_EINVAL;
  *stream = (void*)s->stream;
  return RB_OK;
}

rb_status rb_queue_create(rb_sched* s, rb_model* m, const rb_queue_opts* o, rb_queue** out) {
  if (!s || !m || !o || !out || m->ctx != s->ctx) return RB_EINVAL;
  if (o->max_batch_size < 1 || o->max_batch_size > RB_MAX_BATCH_ROWS || o->n_allowed < 0 ||
      (o->n_allowed > 0 && !o->allowed_batch_sizes))
    return RB_EINVAL;
  if (o->batch_timeout_ns < 1) return RB_EINVAL;
  for (int i = 0; i < o->n_allowed; ++i) {
    const int a = o->allowed_batch_sizes[i];
    if (a < 1 || (i > 0 && a <= o->allowed_batch_sizes[i - 1])) return RB_EINVAL;
  }
  if (o->n_allowed > 0 && o->allowed_batch_sizes[o->n_allowed - 1] != o->max_batch_size) return RB_EINVAL;
  if (o->bucket_len < 0 || (m->kind == RB_MODEL_SEQPOOL) != (o->bucket_len > 0)) return RB_EINVAL;
  if (o->service_ns && o->n_service != o->max_batch_size + 1) return RB_EINVAL;
  if (o->service_ns)
    for (int i = 0; i < o->n_service; ++i)
      if (o->service_ns[i] < 0) return RB_EINVAL;
  if (o->window_ns < 0 || o->window_tail_ns < 0) return RB_EINVAL;
  rb_queue* q = new (std::nothrow) rb_queue();
  if (!q) return RB_ENOMEM;
  q->s = s;
  q->m = m;
  q->shape = shape_of(m);
  q->id = (int)s->queues.size();
  q->B = o->max_batch_size;
  q->allowed.assign(o->allowed_batch_sizes, o->allowed_batch_sizes + o->n_allowed);
  q->T = o->batch_timeout_ns;
  q->bucket = o->bucket_len;
  if (o->service_ns) q->svc.assign(o->service_ns, o->service_ns + o->n_service);
  q->window_ns = o->window_ns;
  q->window_tail = o->window_tail_ns;
  s->queues.push_back(q);
  s->n_live_queues++;
  m->bound++;
  *out = q;
  return RB_OK;
}

rb_status rb_queue_destroy(rb_queue* q) {
  if (!q) return RB_OK;
  if (q->undispatched || q->pending_run) return RB_EBUSY;
  rb_sched* s = q->s;
  // a queue with batches still in the unflushed window keeps them: flush first
  for (Group& g : s->window)
    if (g.q == q) return RB_EBUSY;
  s->queues[(size_t)q->id] = nullptr;
  s->n_live_queues--;
  if (q->m) q->m->bound--;
  delete q;
  return RB_OK;
}

rb_status rb_queue_set_model(rb_queue* q, rb_model* m) {
  if (!q) return RB_EINVAL;
  rb_model* o = q->m;
  if (m == o) return RB_OK;
  rb_sched* s = q->s;
  if (m) {
    const QShape a = shape_of(m), &b = q->shape;
    if (m->ctx != s->ctx || a.kind != b.kind || a.dtype != b.dtype || a.d_in != b.d_in || a.d_out != b.d_out ||
        a.n_dense != b.n_dense || a.n_tables != b.n_tables)
      return RB_EINVAL;
  }
  // batches dispatched into a window that has not been handed to the device
  // yet would run the new version: only swap between launches (serving:
  // after the batches the clock already dispatched from this queue have run)
  if (!s->window.empty() || !s->chunk.empty() || q->pending_run) return RB_EBUSY;
  // an unbound new version with the old one's padded layer shapes takes over
  // the old one's lineage: its launch chains follow the old version's on the
  // same stream and reuse its work buffers (no allocation and no device drain
  // when the first batch runs)
  if (m && o && m->bound.load() == 0 && m->lineage == m->id && m->layers.size() == o->layers.size() &&
      m->head_last == o->head_last && m->sp_in == o->sp_in) {
    bool same = true;
    for (size_t i = 0; same && i < m->layers.size(); ++i)
      same = m->layers[i].Kp == o->layers[i].Kp && m->layers[i].Np == o->layers[i].Np;
    if (same) m->lineage = o->lineage;
  }
  if (m) {
    m->bound++;
    q->shape.table_rows = m->table_rows;
  }
  if (o) o->bound--;
  q->m = m;
  return RB_OK;
}

rb_status rb_queue_id(const rb_queue* q, int32_t* id) {
  if (!q || !id) return RB_EINVAL;
  *id = q->id;
  return RB_OK;
}

// ---------------------------------------------------------------- serving

static rb_status validate_request(const rb_queue* q, const rb_request* r) {
  const QShape* m = &q->shape;
  if (r->n_rows < 1 || r->n_rows > q->B) return RB_EINVAL;
  const int64_t n = r->n_rows;
  if (r->n_dense < 0 || r->n_lens < 0 || r->n_ids < 0) return RB_EINVAL;
  if (r->n_dense > 0 && !r->dense) return RB_EINVAL;
  if (r->n_lens > 0 && !r->lens) return RB_EINVAL;
  if (r->n_ids > 0 && !r->ids) return RB_EINVAL;
  if (m->kind == RB_MODEL_MLP) {
    if (r->n_dense != n * m->d_in || r->n_lens || r->n_ids) return RB_EINVAL;
  } else if (m->kind == RB_MODEL_RANKING) {
    if (r->n_dense != n * m->n_dense || r->n_lens != n * m->n_tables) return RB_EINVAL;
    int64_t tot = 0;
    for (int64_t i = 0; i < r->n_lens; ++i) {
      if (r->lens[i] < 0) return RB_EINVAL;
      tot += r->lens[i];
    }
    if (tot != r->n_ids) return RB_EINVAL;
    for (int64_t i = 0; i < r->n_ids; ++i)
      if (r->ids[i] < 0 || r->ids[i] >= m->table_rows) return RB_EINVAL;
  } else {
    if (r->n_lens != n || r->n_ids) return RB_EINVAL;
    int64_t tot = 0;
    for (int64_t i = 0; i < n; ++i) {
      if (r->lens[i] < 1 || r->lens[i] > q->bucket) return RB_EINVAL;
      tot += r->lens[i];
    }
    if (r->n_dense != tot * m->d_in) return RB_EINVAL;
  }
  return RB_OK;
}

rb_status rb_submit(rb_queue* q, const rb_request* r, int64_t arrival_ns, uint64_t* out_req_id) {
  if (!q || !r || !out_req_id) return RB_EINVAL;
  rb_sched* s = q->s;
  if (arrival_ns < s->now) return RB_EINVAL;
  rb_status st = validate_request(q, r);
  if (st != RB_OK) return st;
  HostReq h;
  h.q = q;
  h.n_rows = r->n_rows;
  h.d_out = q->shape.d_out;
  try {
    h.dense.assign(r->dense, r->dense + r->n_dense);
    if (r->n_lens) h.lens.assign(r->lens, r->lens + r->n_lens);
    if (r->n_ids) h.ids.assign(r->ids, r->ids + r->n_ids);
    s->hreqs.push_back(std::move(h));
  } catch (...) {
    return RB_ENOMEM;
  }
  // the clock's events before the arrival, then the timeouts due at it,
  // then the arrival itself (dispatches at arrival_ns come after it)
  serve_until(s, arrival_ns, false);
  fire_timeouts_at(s, arrival_ns);
  s->now = arrival_ns;
  const int64_t id = (int64_t)s->hreqs.size() - 1;
  arrive(q, id, r->n_rows, arrival_ns);
  *out_req_id = (uint64_t)id;
  return RB_OK;
}

rb_status rb_advance(rb_sched* s, int64_t now_ns) {
  if (!s || now_ns < s->now) return RB_EINVAL;
  serve_until(s, now_ns, true);
  s->now = now_ns;
  return RB_OK;
}

rb_status rb_flush(rb_queue* q) {
  if (!q) return RB_EINVAL;
  if (q->open_s > 0) close_open(q, std::max<int64_t>(q->s->now, q->open_t));
  return RB_OK;
}

// Serving-mode device run of dispatched batches (one launch window): stage
// their payloads in one slot, run one launch chain per queue, copy the
// outputs back into the slot's pinned output buffer.
static rb_status run_serving_window(rb_sched* s, const std::vector<Disp>& win) {
  // one launch group per queue, in order of first appearance
  std::vector<Group> groups;
  std::vector<std::vector<int64_t>> greqs;  // each group's request ids
  for (const Disp& d : win) {
    size_t gi = 0;
    while (gi < groups.size() && groups[gi].q != d.q) ++gi;
    if (gi == groups.size()) {
      groups.push_back(Group{});
      groups.back().q = d.q;
      greqs.emplace_back();
    }
    Group& g = groups[gi];
    rb_k_batch kb{(int32_t)greqs[gi].size(), (int32_t)d.b.reqs.size(), (int32_t)g.slots, d.b.P, d.b.s,
                  d.q->m->kind == RB_MODEL_SEQPOOL ? d.q->bucket : 0};
    g.batches.push_back(kb);
    g.slots += d.b.P;
    greqs[gi].insert(greqs[gi].end(), d.b.reqs.begin(), d.b.reqs.end());
  }
  int64_t nd = 0, nl = 0, ni = 0, no = 0;
  size_t desc = 0;
  for (size_t gi = 0; gi < groups.size(); ++gi) {
    desc += round_up((int64_t)(groups[gi].batches.size() * sizeof(rb_k_batch)), 256) +
            round_up((int64_t)(greqs[gi].size() * sizeof(rb_k_req)), 256);
    for (int64_t id : greqs[gi]) {
      const HostReq& h = s->hreqs[(size_t)id];
      nd += (int64_t)h.dense.size();
      nl += (int64_t)h.lens.size();
      ni += (int64_t)h.ids.size();
      no += (int64_t)h.n_rows * h.d_out;
    }
  }
  const size_t o_dense = desc;
  const size_t o_lens = o_dense + round_up(nd * 4, 256);
  const size_t o_ids = o_lens + round_up(nl * 4, 256);
  const size_t o_out = o_ids + round_up(ni * 4, 256);
  const size_t total = o_out + round_up(no * 4, 256);
  Slot* sl = nullptr;
  rb_status st = acquire_slot(s, total, (size_t)std::max<int64_t>(no, 1) * 4, &sl);
  if (st != RB_OK) return st;
  int64_t cd = 0, cl = 0, ci = 0, co = 0;
  size_t off = 0;
  std::vector<std::pair<size_t, size_t>> offs;
  for (size_t gi = 0; gi < groups.size(); ++gi) {
    Group& g = groups[gi];
    const rb_model* m = g.q->m;
    for (int64_t id : greqs[gi]) {
      HostReq& h = s->hreqs[(size_t)id];
      rb_k_req kr{};
      kr.dense_off = cd;
      kr.dense_end = cd + (int64_t)h.dense.size();
      kr.lens_off = cl;
      kr.ids_off = ci;
      kr.ids_end = ci + (int64_t)h.ids.size();
      kr.out_off = co;
      kr.n_rows = h.n_rows;
      add_tokens(g, m, kr);
      std::memcpy(sl->host + o_dense + cd * 4, h.dense.data(), h.dense.size() * 4);
      if (!h.lens.empty()) std::memcpy(sl->host + o_lens + cl * 4, h.lens.data(), h.lens.size() * 4);
      if (!h.ids.empty()) std::memcpy(sl->host + o_ids + ci * 4, h.ids.data(), h.ids.size() * 4);
      h.out_off = co;
      h.slot = (int)(sl - s->slots);
      h.state = 1;
      cd += (int64_t)h.dense.size();
      cl += (int64_t)h.lens.size();
      ci += (int64_t)h.ids.size();
      co += (int64_t)h.n_rows * h.d_out;
      g.reqs.push_back(kr);
      sl->serving_reqs.push_back(id);
    }
    const size_t bb = g.batches.size() * sizeof(rb_k_batch), rr = g.reqs.size() * sizeof(rb_k_req);
    std::memcpy(sl->host + off, g.batches.data(), bb);
    const size_t o1 = off;
    off += round_up((int64_t)bb, 256);
    std::memcpy(sl->host + off, g.reqs.data(), rr);
    offs.push_back({o1, off});
    off += round_up((int64_t)rr, 256);
  }
  // a failure from here on: the window's requests fail (rb_collect reports
  // RB_EDEVICE for them), and whatever was enqueued stays fenced by the
  // slot's event, so its buffers are not reused before that work is done
  auto fail = [&](rb_status e) {
    for (int64_t id : sl->serving_reqs) {
      HostReq& h = s->hreqs[(size_t)id];
      h.state = 4;
      h.slot = -1;
    }
    sl->serving_reqs.clear();
    hipEventRecord(sl->ev, s->stream);
    sl->busy = true;
    return e;
  };
  for (Group& g : groups) slot_hold(*sl, g.q->m);
  if (!hip_ok(hipMemcpyAsync(sl->dev, sl->host, o_out, hipMemcpyHostToDevice, s->stream))) return fail(RB_EDEVICE);
  float* dout = (float*)(sl->dev + o_out);
  for (size_t gi = 0; gi < groups.size(); ++gi) {
    st = run_group(s, s->stream, 0, groups[gi], (const rb_k_batch*)(sl->dev + offs[gi].first),
                   (const rb_k_req*)(sl->dev + offs[gi].second), (const float*)(sl->dev + o_dense), nd,
                   (const int32_t*)(sl->dev + o_lens), nl, (const int32_t*)(sl->dev + o_ids), ni, dout, no);
    if (st != RB_OK) return fail(st);
  }
  if (!hip_ok(hipMemcpyAsync(sl->host_out, dout, (size_t)no * 4, hipMemcpyDeviceToHost, s->stream)))
    return fail(RB_EDEVICE);
  hipEventRecord(sl->ev, s->stream);
  sl->busy = true;
  return RB_OK;
}

// Run dispatched batches: on the device (asynchronous), or, without one,
// mark their requests done. Then describe them for the caller.
static rb_status run_dispatched(rb_sched* s, std::vector<Disp>& win) {
  for (Disp& d : win) d.q->pending_run--;
  if (s->stream) {
    rb_status st = run_serving_window(s, win);
    if (st != RB_OK) return st;
  } else {
    for (Disp& d : win)
      for (int64_t id : d.b.reqs) s->hreqs[(size_t)id].state = 2;
  }
  s->last_req_ids.clear();
  for (Disp& d : win) s->last_req_ids.insert(s->last_req_ids.end(), d.b.reqs.begin(), d.b.reqs.end());
  s->last_infos.clear();
  size_t k = 0;
  for (Disp& d : win) {
    rb_batch_info bi{};
    bi.batch_id = (uint64_t)d.b.seq;
    bi.queue = d.q->id;
    bi.real_rows = d.b.s;
    bi.padded_rows = d.b.P;
    bi.n_req = (int32_t)d.b.reqs.size();
    bi.close_ns = d.b.close_ns;
    bi.dispatch_ns = d.b.dispatch_ns;
    bi.done_ns = d.b.done_ns;
    bi.req_ids = s->last_req_ids.data() + k;
    k += d.b.reqs.size();
    s->last_infos.push_back(bi);
  }
  return RB_OK;
}

rb_status rb_run_next(rb_sched* s, rb_batch_info* out) {
  if (!s || !out) return RB_EINVAL;
  serve_until(s, s->now, true);
  if (s->ready.empty()) return RB_EEMPTY;
  std::vector<Disp> one;
  one.push_back(std::move(s->ready.front().front()));
  s->ready.front().erase(s->ready.front().begin());
  if (s->ready.front().empty()) s->ready.pop_front();
  rb_status st = run_dispatched(s, one);
  if (st != RB_OK) return st;
  *out = s->last_infos[0];
  return RB_OK;
}

rb_status rb_run_window(rb_sched* s, rb_window_info* out) {
  if (!s || !out) return RB_EINVAL;
  serve_until(s, s->now, true);
  if (s->ready.empty()) return RB_EEMPTY;
  std::vector<Disp> win = std::move(s->ready.front());
  s->ready.pop_front();
  rb_status st = run_dispatched(s, win);
  if (st != RB_OK) return st;
  out->n_batches = (int32_t)s->last_infos.size();
  out->batches = s->last_infos.data();
  return RB_OK;
}

rb_status rb_collect(rb_sched* s, uint64_t req_id, float* dst, size_t dst_bytes, int32_t* out_rows) {
  if (!s || !out_rows) return RB_EINVAL;
  if (req_id >= s->hreqs.size()) return RB_ENOENT;
  HostReq& h = s->hreqs[(size_t)req_id];
  if (h.state == 3) return RB_ENOENT;
  if (h.state == 0) return RB_EAGAIN;
  if (!s->stream) return RB_EDEVICE;  // no outputs without a device
  if (h.state == 4) {  // its window failed: reported once, then forgotten
    h.state = 3;
    std::vector<float>().swap(h.dense);
    std::vector<int32_t>().swap(h.lens);
    std::vector<int32_t>().swap(h.ids);
    return RB_EDEVICE;
  }
  if (h.state == 1) {
    Slot& sl = s->slots[h.slot];
    const hipError_t e = hipEventQuery(sl.ev);
    if (e == hipErrorNotReady) return RB_EAGAIN;
    if (e != hipSuccess) return RB_EDEVICE;
    retire_slot(s, sl);
  }
  const size_t need = h.out.size() * sizeof(float);
  if (!dst || dst_bytes < need) return RB_ESIZE;
  std::memcpy(dst, h.out.data(), need);
  *out_rows = h.n_rows;
  h.state = 3;
  std::vector<float>().swap(h.out);
  std::vector<float>().swap(h.dense);
  std::vector<int32_t>().swap(h.lens);
  std::vector<int32_t>().swap(h.ids);
  return RB_OK;
}

// ---------------------------------------------------------------- launch groups

// Checks of rb_run_group's arguments (the descriptors themselves are checked
// on the device).
static rb_status check_group(rb_queue* q, const rb_k_batch* batches, int32_t n_batches, const rb_k_req* reqs,
                             int32_t n_reqs, int64_t slots, int64_t tokens, const float* dense, int64_t dense_len,
                             const int32_t* lens, int64_t lens_len, const int32_t* ids, int64_t ids_len,
                             const float* out, int64_t out_len) {
  if (!q || !batches || !reqs || !out || !dense) return RB_EINVAL;
  if (n_batches < 1 || n_reqs < 1 || slots < n_batches || tokens < 0 || dense_len < 0 || lens_len < 0 ||
      ids_len < 0 || out_len < 0)
    return RB_EINVAL;
  if (!q->s->stream) return RB_EDEVICE;
  const rb_model* m = q->m;
  if (!m) return RB_EBUSY;
  if (m->kind != RB_MODEL_MLP && !lens) return RB_EINVAL;
  if (m->kind == RB_MODEL_RANKING && ids_len > 0 && !ids) return RB_EINVAL;
  if (group_rows(m, q, slots) > INT32_MAX || slots > INT32_MAX) return RB_EINVAL;
  if (tokens > group_rows(m, q, slots)) return RB_EINVAL;
  return RB_OK;
}

rb_status rb_run_group(rb_queue* q, void* stream, const rb_k_batch* batches, int32_t n_batches, const rb_k_req* reqs,
                       int32_t n_reqs, int64_t slots, int64_t tokens, const float* dense, int64_t dense_len,
                       const int32_t* lens, int64_t lens_len, const int32_t* ids, int64_t ids_len, float* out,
                       int64_t out_len) {
  rb_status st = check_group(q, batches, n_batches, reqs, n_reqs, slots, tokens, dense, dense_len, lens, lens_len,
                             ids, ids_len, out, out_len);
  if (st != RB_OK) return st;
  rb_sched* s = q->s;
  rb_model* m = q->m;
  hipStream_t hs = stream ? (hipStream_t)stream : s->stream;
  Work& w = s->ext_work[m->lineage];
  if ((st = grow_work(s, m, w, group_rows(m, q, slots), slots, hs)) != RB_OK) return st;
  return run_chain(s, hs, q, n_batches, n_reqs, slots, tokens, &w, false, true, batches, reqs, dense, dense_len, lens,
                   lens_len, ids, ids_len, out, out_len);
}

rb_status rb_run_group_static(rb_queue* q, void* stream, const rb_k_batch* batches, int32_t n_batches,
                              const rb_k_req* reqs, int32_t n_reqs, int64_t slots, int64_t tokens,
                              const float* dense, int64_t dense_len, const int32_t* lens, int64_t lens_len,
                              const int32_t* ids, int64_t ids_len, float* out, int64_t out_len) {
  rb_status st = check_group(q, batches, n_batches, reqs, n_reqs, slots, tokens, dense, dense_len, lens, lens_len,
                             ids, ids_len, out, out_len);
  if (st != RB_OK) return st;
  rb_sched* s = q->s;
  char* base = (char*)rb_static_scratch(s->ctx->device);
  if (!base) return RB_EDEVICE;
  // the group's work buffers carved from the scratch array: row map, X, A,
  // B, Y, each 256-byte aligned
  const WorkShape sh = work_shape(q->m, group_rows(q->m, q, slots), slots);
  const size_t parts[5] = {sh.rows, sh.x, sh.ab, sh.ab, sh.y};
  size_t off[5], end = 0;
  for (int i = 0; i < 5; ++i) {
    off[i] = end;
    end += (size_t)round_up((int64_t)parts[i], 256);
  }
  if (end > (size_t)RB_STATIC_SCRATCH_BYTES) return RB_ESIZE;
  Work w;
  w.rows = (rb_k_row*)(base + off[0]);
  w.X = base + off[1];
  w.A = base + off[2];
  w.B = base + off[3];
  w.Y = (float*)(base + off[4]);
  return run_chain(s, stream ? (hipStream_t)stream : s->stream, q, n_batches, n_reqs, slots, tokens, &w, false, true,
                   batches, reqs, dense, dense_len, lens, lens_len, ids, ids_len, out, out_len);
}

// ---------------------------------------------------------------- replay

rb_status rb_sim_run(rb_sched* s, const rb_servable* sv, int32_t n_sv, const rb_trace* tr, rb_log* log) {
  if (!s || !sv || n_sv < 1 || !tr || !log) return RB_EINVAL;
  const int64_t N = tr->n_requests;
  if (N < 0 || (N > 0 && (!tr->servable || !tr->arrival_ns || !tr->n_rows))) return RB_EINVAL;
  if (log->max_batches < N || (N > 0 && (!log->req_done_ns || !log->req_queue || !log->b_queue || !log->b_real ||
                                         !log->b_padded || !log->b_close_ns || !log->b_dispatch_ns ||
                                         !log->b_done_ns || !log->b_req_begin || !log->b_reqs)))
    return log->max_batches < N ? RB_ESIZE : RB_EINVAL;
  for (int32_t i = 0; i < n_sv; ++i) {
    if (sv[i].n_queues < 1 || !sv[i].queues) return RB_EINVAL;
    for (int32_t j = 0; j < sv[i].n_queues; ++j) {
      rb_queue* q = sv[i].queues[j];
      if (!q || q->s != s) return RB_EINVAL;
      if (!q->m) return RB_EBUSY;  // a held queue could not leave the replay empty
    }
  }
  // the replay runs the scheduler's clock over every queue it holds: any
  // request still waiting anywhere on it (open, closed or dispatched but not
  // run by the serving API) would be served as part of the replay
  if (!s->ready.empty()) return RB_EBUSY;
  for (const rb_queue* q : s->queues)
    if (q && (q->undispatched || !q->closed.empty() || q->pending_run)) return RB_EBUSY;
  const bool dev = s->stream != nullptr;
  if (dev && N > 0 && (!tr->dense || !tr->dense_off || !tr->out || !tr->out_off)) return RB_EINVAL;
  // route every request to its queue and validate it against that queue
  std::vector<rb_queue*> rq((size_t)N);
  for (int64_t r = 0; r < N; ++r) {
    const int32_t si = tr->servable[r];
    if (si < 0 || si >= n_sv) return RB_EINVAL;
    const rb_servable& v = sv[si];
    rb_queue* q = nullptr;
    if (v.n_queues == 1 && v.queues[0]->bucket == 0) {
      q = v.queues[0];
    } else {
      if (!tr->max_len) return RB_EINVAL;
      const int L = tr->max_len[r];
      for (int32_t j = 0; j < v.n_queues; ++j) {
        rb_queue* c = v.queues[j];
        if (c->bucket >= L && (!q || c->bucket < q->bucket)) q = c;
      }
      if (!q || L < 1) return RB_EINVAL;
    }
    if (tr->n_rows[r] < 1 || tr->n_rows[r] > q->B) return RB_EINVAL;
    if (r > 0 && tr->arrival_ns[r] < tr->arrival_ns[r - 1]) return RB_EINVAL;
    if (dev) {
      const QShape* m = &q->shape;
      const int64_t n = tr->n_rows[r];
      if (tr->out_off[r + 1] - tr->out_off[r] != n * m->d_out || tr->out_off[r] < 0) return RB_EINVAL;
      if (tr->dense_off[r] < 0 || tr->dense_off[r + 1] < tr->dense_off[r]) return RB_EINVAL;
      if (m->kind != RB_MODEL_SEQPOOL && tr->dense_off[r + 1] - tr->dense_off[r] != n * m->d_in) return RB_EINVAL;
      if (m->kind != RB_MODEL_MLP) {
        if (!tr->lens || !tr->lens_off) return RB_EINVAL;
        const int64_t want = m->kind == RB_MODEL_RANKING ? n * m->n_tables : n;
        if (tr->lens_off[r] < 0 || tr->lens_off[r + 1] - tr->lens_off[r] != want) return RB_EINVAL;
      }
      if (m->kind == RB_MODEL_RANKING) {
        if (!tr->ids || !tr->ids_off || tr->ids_off[r] < 0 || tr->ids_off[r + 1] < tr->ids_off[r]) return RB_EINVAL;
      }
    }
    rq[(size_t)r] = q;
  }
  if (dev) {
    s->a_dense = tr->dense;
    s->a_dense_len = N > 0 ? tr->dense_off[N] : 0;
    s->a_lens = tr->lens;
    s->a_lens_len = (N > 0 && tr->lens_off) ? tr->lens_off[N] : 0;
    s->a_ids = tr->ids;
    s->a_ids_len = (N > 0 && tr->ids_off) ? tr->ids_off[N] : 0;
    s->a_out = tr->out;
    s->a_out_len = N > 0 ? tr->out_off[N] : 0;
  }
  // a replay runs on its own simulated clock, starting idle
  s->now = INT64_MIN;
  s->device_free = INT64_MIN;
  s->last_served = -1;
  // event loop
  int64_t nb = 0, nreq_logged = 0;
  const int64_t end_t = N > 0 ? tr->arrival_ns[N - 1] : 0;
  bool flushed = N == 0;
  int64_t nxt = 0;
  std::vector<rb_k_req> kreqs;
  rb_status st = RB_OK;
  std::vector<Disp> win;
  const bool clocked = s->opts.clocked_windows != 0;
  auto dispatch_at = [&](int64_t t) -> rb_status {
    while (s->device_free <= t && clock_dispatch(s, t, win)) {
      for (Disp& d : win) {
        rb_queue* q = d.q;
        const Batch& b = d.b;
        log->b_queue[nb] = q->id;
        log->b_real[nb] = b.s;
        log->b_padded[nb] = b.P;
        log->b_close_ns[nb] = b.close_ns;
        log->b_dispatch_ns[nb] = b.dispatch_ns;
        log->b_done_ns[nb] = b.done_ns;
        log->b_req_begin[nb] = nreq_logged;
        for (int64_t r : b.reqs) {
          log->b_reqs[nreq_logged++] = (int32_t)r;
          log->req_done_ns[r] = b.done_ns;
          log->req_queue[r] = q->id;
        }
        ++nb;
        if (!dev) continue;
        kreqs.clear();
        for (int64_t r : b.reqs) {
          rb_k_req k{};
          k.dense_off = tr->dense_off[r];
          k.dense_end = tr->dense_off[r + 1];
          k.lens_off = tr->lens_off ? tr->lens_off[r] : 0;
          k.ids_off = tr->ids_off ? tr->ids_off[r] : 0;
          k.ids_end = tr->ids_off ? tr->ids_off[r + 1] : 0;
          k.out_off = tr->out_off[r];
          k.n_rows = tr->n_rows[r];
          kreqs.push_back(k);
        }
        window_add(s, q, b, kreqs);
        // a backlogged device runs window_batches consecutive batches per
        // launch window; clocked replays run the clock's own windows
        if (!clocked && s->window_batches >= s->opts.window_batches) {
          close_window(s);
          if ((int)s->chunk.size() >= CHUNK_WINDOWS) {
            rb_status e = flush_chunk(s);
            if (e != RB_OK) return e;
          }
        }
      }
      if (dev && clocked) {
        close_window(s);
        if ((int)s->chunk.size() >= CHUNK_WINDOWS) {
          rb_status e = flush_chunk(s);
          if (e != RB_OK) return e;
        }
      }
    }
    return RB_OK;
  };
  for (;;) {
    int64_t t = INT64_MAX;
    if (nxt < N) t = std::min(t, tr->arrival_ns[nxt]);
    t = std::min(t, next_timeout(s));
    if (!flushed && nxt >= N) t = std::min(t, end_t);
    if (has_pickable(s)) t = std::min(t, s->device_free);
    if (t == INT64_MAX) break;
    fire_timeouts_at(s, t);
    while (nxt < N && tr->arrival_ns[nxt] == t) {
      arrive(rq[(size_t)nxt], nxt, tr->n_rows[nxt], t);
      ++nxt;
    }
    if (!flushed && nxt >= N && t == end_t) {
      for (rb_queue* q : s->queues)
        if (q && q->T == NO_TIMEOUT && q->open_s > 0) close_open(q, t);
      flushed = true;
    }
    s->now = std::max(s->now, t);
    if ((st = dispatch_at(t)) != RB_OK) break;
  }
  if (st == RB_OK && dev) {
    close_window(s);
    st = flush_chunk(s);
  }
  log->n_batches = nb;
  if (N > 0) log->b_req_begin[nb] = nreq_logged;
  return st;
}

}  // extern "C"
