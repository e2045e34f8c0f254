// Drives every host-only path of the batching library's C ABI (host-only
// context, no-device schedulers) for sanitizer builds of the host runtime:
// model and queue life cycles, option validation, trace replays on the
// simulated clock with launch windows, the serving calls with version
// transitions and dynamic queues, and, with --threads, models created and
// destroyed on loader threads while the main thread serves and swaps them in.
// Exits non-zero (or the sanitizer aborts) on any failure.
#include <atomic>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <thread>
#include <vector>

#include "rb.h"

namespace {

int failures = 0;
int64_t replayed_batches = 0, served_requests = 0, transitions = 0, queue_churn = 0;

#define CHECK(cond)                                                  \
  do {                                                               \
    if (!(cond)) {                                                   \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
      ++failures;                                                    \
    }                                                                \
  } while (0)

struct Rng {  // 64-bit linear congruential generator (Knuth's MMIX constants)
  uint64_t s;
  explicit Rng(uint64_t seed) : s(seed * 2 + 1) {}
  uint32_t next() {
    s = s * 6364136223846793005ull + 1442695040888963407ull;
    return (uint32_t)(s >> 33);
  }
  int range(int lo, int hi) { return lo + (int)(next() % (uint32_t)(hi - lo + 1)); }  // inclusive
};

rb_model* make_mlp(rb_ctx* ctx, int d_in, int d_out) {
  rb_layer_desc L[2] = {{d_in, 8, RB_ACT_RELU, nullptr, nullptr}, {8, d_out, RB_ACT_NONE, nullptr, nullptr}};
  rb_model_desc d{};
  d.kind = RB_MODEL_MLP;
  d.dtype = RB_DT_F32;
  d.n_layers = 2;
  d.layers = L;
  rb_model* m = nullptr;
  CHECK(rb_model_create(ctx, &d, &m) == RB_OK);
  return m;
}

void model_validation(rb_ctx* ctx) {
  rb_layer_desc bad[2] = {{4, 8, RB_ACT_RELU, nullptr, nullptr}, {7, 3, RB_ACT_NONE, nullptr, nullptr}};
  rb_model_desc d{};
  d.kind = RB_MODEL_MLP;
  d.dtype = RB_DT_F32;
  d.n_layers = 2;
  d.layers = bad;
  rb_model* m = nullptr;
  CHECK(rb_model_create(ctx, &d, &m) == RB_EINVAL);
  // ranking: 3 tables of 64 + 5 dense
  rb_layer_desc rl[2] = {{3 * 64 + 5, 16, RB_ACT_RELU, nullptr, nullptr}, {16, 1, RB_ACT_SIGMOID, nullptr, nullptr}};
  rb_model_desc r{};
  r.kind = RB_MODEL_RANKING;
  r.dtype = RB_DT_BF16;
  r.n_layers = 2;
  r.layers = rl;
  r.n_tables = 3;
  r.table_rows = 100;
  r.emb_dim = 64;
  r.n_dense = 5;
  CHECK(rb_model_create(ctx, &r, &m) == RB_OK);
  int32_t di = 0, dout = 0;
  CHECK(rb_model_info(m, &di, &dout) == RB_OK && di == 5 && dout == 1);
  CHECK(rb_model_destroy(m) == RB_OK);
  r.emb_dim = 32;
  CHECK(rb_model_create(ctx, &r, &m) == RB_EINVAL);
  // seqpool with a softmax head
  rb_layer_desc sl[1] = {{6, 6, RB_ACT_RELU, nullptr, nullptr}};
  rb_model_desc q{};
  q.kind = RB_MODEL_SEQPOOL;
  q.dtype = RB_DT_F32;
  q.n_layers = 1;
  q.layers = sl;
  q.head = {6, 2, RB_ACT_SOFTMAX, nullptr, nullptr};
  CHECK(rb_model_create(ctx, &q, &m) == RB_OK);
  CHECK(rb_model_destroy(m) == RB_OK);
  q.head.fan_out = 40;
  CHECK(rb_model_create(ctx, &q, &m) == RB_EINVAL);
}

struct QCfg {
  int B;
  std::vector<int32_t> allowed;
  int64_t T;
  std::vector<int64_t> svc;
  int64_t wns, tail;
};

QCfg random_queue(Rng& g) {
  QCfg c;
  c.B = g.range(1, 40);
  if (c.B > 2 && g.range(0, 1)) {
    int a = g.range(1, c.B - 1);
    c.allowed = {a, c.B};
  }
  c.T = g.range(0, 3) == 0 ? INT64_MAX : g.range(1, 400);
  for (int p = 0; p <= c.B; ++p) c.svc.push_back(g.range(0, 150));
  c.wns = g.range(0, 100);
  c.tail = g.range(0, 200);
  return c;
}

rb_queue* make_queue(rb_sched* s, rb_model* m, const QCfg& c) {
  rb_queue_opts o{};
  o.max_batch_size = c.B;
  o.allowed_batch_sizes = c.allowed.empty() ? nullptr : c.allowed.data();
  o.n_allowed = (int32_t)c.allowed.size();
  o.batch_timeout_ns = c.T;
  o.service_ns = c.svc.data();
  o.n_service = (int32_t)c.svc.size();
  o.window_ns = c.wns;
  o.window_tail_ns = c.tail;
  rb_queue* q = nullptr;
  CHECK(rb_queue_create(s, m, &o, &q) == RB_OK);
  return q;
}

void replays(rb_ctx* ctx, uint64_t seed) {
  Rng g(seed);
  rb_model* m = make_mlp(ctx, 4, 3);
  for (int it = 0; it < 20; ++it) {
    rb_sched_opts so{};
    so.mode = RB_MODE_NO_DEVICE;
    so.window_batches = g.range(1, 9);
    rb_sched* s = nullptr;
    CHECK(rb_sched_create(ctx, &so, &s) == RB_OK);
    const int nq = g.range(1, 5);
    std::vector<QCfg> cfg;
    std::vector<rb_queue*> qs;
    for (int i = 0; i < nq; ++i) {
      cfg.push_back(random_queue(g));
      qs.push_back(make_queue(s, m, cfg.back()));
    }
    const int N = g.range(0, 400);
    std::vector<int32_t> serv(N), rows(N);
    std::vector<int64_t> arr(N);
    int64_t t = 0;
    for (int r = 0; r < N; ++r) {
      t += g.range(0, 30);
      arr[r] = t;
      serv[r] = g.range(0, nq - 1);
      rows[r] = g.range(1, cfg[serv[r]].B);
    }
    std::vector<rb_servable> sv(nq);
    for (int i = 0; i < nq; ++i) sv[i] = rb_servable{1, &qs[i]};
    rb_trace tr{};
    tr.n_requests = N;
    tr.servable = serv.data();
    tr.arrival_ns = arr.data();
    tr.n_rows = rows.data();
    std::vector<int64_t> done(N), b_close(N), b_disp(N), b_done(N), b_beg(N + 1);
    std::vector<int32_t> rq(N), b_queue(N), b_real(N), b_pad(N), b_reqs(N);
    rb_log lg{done.data(), rq.data(), N, 0, b_queue.data(), b_real.data(), b_pad.data(),
              b_close.data(), b_disp.data(), b_done.data(), b_beg.data(), b_reqs.data()};
    CHECK(rb_sim_run(s, sv.data(), nq, &tr, &lg) == RB_OK);
    std::vector<int> seen(N, 0);
    replayed_batches += lg.n_batches;
    for (int64_t b = 0; b < lg.n_batches; ++b) {
      CHECK(b_close[b] <= b_disp[b] && b_disp[b] <= b_done[b]);
      for (int64_t k = b_beg[b]; k < b_beg[b + 1]; ++k) seen[b_reqs[k]]++;
    }
    for (int r = 0; r < N; ++r) CHECK(seen[r] == 1);
    // too small a log
    if (N > 1) {
      lg.max_batches = N - 1;
      CHECK(rb_sim_run(s, sv.data(), nq, &tr, &lg) == RB_ESIZE);
    }
    for (rb_queue* q : qs) CHECK(rb_queue_destroy(q) == RB_OK);
    CHECK(rb_sched_destroy(s) == RB_OK);
  }
  CHECK(rb_model_destroy(m) == RB_OK);
}

// The serving calls in random order, with version transitions and queues
// coming and going; every submitted request must come out of exactly one
// dispatched batch.
void serving(rb_ctx* ctx, uint64_t seed) {
  Rng g(seed);
  rb_sched_opts so{};
  so.mode = RB_MODE_NO_DEVICE;
  so.window_batches = g.range(1, 6);
  rb_sched* s = nullptr;
  CHECK(rb_sched_create(ctx, &so, &s) == RB_OK);
  std::vector<rb_model*> models;
  std::vector<rb_queue*> qs;
  std::vector<QCfg> cfg;
  for (int i = 0; i < 3; ++i) {
    models.push_back(make_mlp(ctx, 4, 3));
    cfg.push_back(random_queue(g));
    qs.push_back(make_queue(s, models.back(), cfg.back()));
  }
  std::vector<int> ran;  // per request id: times it came out of a batch
  std::vector<float> x(4 * 64, 0.f);
  int64_t now = 0;
  auto count = [&](const rb_batch_info& b) {
    for (int i = 0; i < b.n_req; ++i) {
      CHECK(b.req_ids[i] < ran.size());
      if (b.req_ids[i] < ran.size()) ran[b.req_ids[i]]++;
    }
  };
  for (int step = 0; step < 3000; ++step) {
    const int op = g.range(0, 9);
    const int qi = g.range(0, (int)qs.size() - 1);
    rb_queue* q = qs[qi];
    if (op <= 4) {
      now += g.range(0, 20);
      rb_request r{};
      r.n_rows = g.range(1, cfg[qi].B + (g.range(0, 9) == 0 ? 3 : 0));
      r.dense = x.data();
      r.n_dense = (int64_t)r.n_rows * 4;
      uint64_t id = 0;
      const rb_status st = rb_submit(q, &r, now, &id);
      if (r.n_rows > cfg[qi].B || r.n_rows > 64) {
        CHECK(st == RB_EINVAL);
      } else {
        CHECK(st == RB_OK);
        if (st == RB_OK) {
          CHECK(id == ran.size());
          ran.push_back(0);
        }
      }
    } else if (op == 5) {
      now += g.range(0, 200);
      CHECK(rb_advance(s, now) == RB_OK);
      CHECK(rb_advance(s, now - 1) == RB_EINVAL || now == 0);
    } else if (op == 6) {
      CHECK(rb_flush(q) == RB_OK);
    } else if (op == 7) {
      rb_batch_info b{};
      const rb_status st = rb_run_next(s, &b);
      CHECK(st == RB_OK || st == RB_EEMPTY);
      if (st == RB_OK) count(b);
    } else if (op == 8) {
      rb_window_info w{};
      const rb_status st = rb_run_window(s, &w);
      CHECK(st == RB_OK || st == RB_EEMPTY);
      if (st == RB_OK) {
        CHECK(w.n_batches >= 1 && w.n_batches <= so.window_batches);
        for (int i = 0; i < w.n_batches; ++i) count(w.batches[i]);
      }
    } else {
      // a version transition: swap in a new model, or hold and resume
      rb_model* nm = make_mlp(ctx, 4, 3);
      rb_status st = rb_queue_set_model(q, nullptr);
      CHECK(st == RB_OK || st == RB_EBUSY);
      if (st == RB_OK) {
        rb_model* old = models[qi];
        bool shared = false;
        for (size_t j = 0; j < qs.size(); ++j)
          if ((int)j != qi && models[j] == old) shared = true;
        CHECK(rb_model_destroy(old) == (shared ? RB_EBUSY : RB_OK));
        CHECK(rb_queue_set_model(q, nm) == RB_OK);
        models[qi] = nm;
        ++transitions;
      } else {
        CHECK(rb_model_destroy(nm) == RB_OK);
      }
      // a queue goes away once empty and a new one takes its place
      if (g.range(0, 3) == 0) {
        const rb_status dst = rb_queue_destroy(q);
        CHECK(dst == RB_OK || dst == RB_EBUSY);
        if (dst == RB_OK) {
          cfg[qi] = random_queue(g);
          qs[qi] = make_queue(s, models[qi], cfg[qi]);
          ++queue_churn;
        }
      }
    }
  }
  // drain everything, then collect: no device, so no outputs
  for (size_t i = 0; i < qs.size(); ++i) CHECK(rb_flush(qs[i]) == RB_OK);
  CHECK(rb_advance(s, now + ((int64_t)1 << 40)) == RB_OK);
  for (;;) {
    rb_window_info w{};
    const rb_status st = rb_run_window(s, &w);
    if (st != RB_OK) {
      CHECK(st == RB_EEMPTY);
      break;
    }
    for (int i = 0; i < w.n_batches; ++i) count(w.batches[i]);
  }
  for (size_t r = 0; r < ran.size(); ++r) CHECK(ran[r] == 1);
  served_requests += (int64_t)ran.size();
  if (!ran.empty()) {
    float out[3 * 64];
    int32_t n = 0;
    CHECK(rb_collect(s, 0, out, sizeof(out), &n) == RB_EDEVICE);
    CHECK(rb_collect(s, ran.size() + 5, out, sizeof(out), &n) == RB_ENOENT);
  }
  for (rb_queue* q : qs) CHECK(rb_queue_destroy(q) == RB_OK);
  CHECK(rb_sched_destroy(s) == RB_OK);
  for (rb_model* m : models) CHECK(rb_model_destroy(m) == RB_OK);
}

// Loader threads build and drop models on the shared host-only context while
// the main thread serves and swaps their models in (the handoff of a model
// between threads goes through a mutex of the caller's, as the ABI asks).
void loaders(rb_ctx* ctx) {
  std::mutex mu;
  std::vector<rb_model*> ready;
  std::atomic<bool> stop{false};
  std::vector<std::thread> th;
  for (int k = 0; k < 4; ++k)
    th.emplace_back([&, k] {
      Rng g(1000 + k);
      while (!stop.load()) {
        rb_model* m = make_mlp(ctx, 4, 3);
        if (g.range(0, 1)) {
          CHECK(rb_model_destroy(m) == RB_OK);
          continue;
        }
        std::lock_guard<std::mutex> lk(mu);
        if (ready.size() < 8) ready.push_back(m);
        else CHECK(rb_model_destroy(m) == RB_OK);
      }
    });
  rb_sched_opts so{};
  so.mode = RB_MODE_NO_DEVICE;
  so.window_batches = 4;
  rb_sched* s = nullptr;
  CHECK(rb_sched_create(ctx, &so, &s) == RB_OK);
  rb_model* cur = make_mlp(ctx, 4, 3);
  Rng g(77);
  QCfg c = random_queue(g);
  rb_queue* q = make_queue(s, cur, c);
  std::vector<float> x(4 * 64, 0.f);
  int64_t now = 0;
  for (int it = 0; it < 4000; ++it) {
    rb_request r{};
    r.n_rows = g.range(1, c.B);
    r.dense = x.data();
    r.n_dense = (int64_t)r.n_rows * 4;
    uint64_t id = 0;
    now += g.range(0, 10);
    CHECK(rb_submit(q, &r, now, &id) == RB_OK);
    rb_window_info w{};
    while (rb_run_window(s, &w) == RB_OK) {
    }
    rb_model* nm = nullptr;
    {
      std::lock_guard<std::mutex> lk(mu);
      if (!ready.empty()) {
        nm = ready.back();
        ready.pop_back();
      }
    }
    if (nm) {
      const rb_status st = rb_queue_set_model(q, nm);
      CHECK(st == RB_OK || st == RB_EBUSY);
      if (st == RB_OK) {
        CHECK(rb_model_destroy(cur) == RB_OK);
        cur = nm;
        ++transitions;
      } else {
        CHECK(rb_model_destroy(nm) == RB_OK);
      }
    }
  }
  stop.store(true);
  for (std::thread& t : th) t.join();
  for (rb_model* m : ready) CHECK(rb_model_destroy(m) == RB_OK);
  CHECK(rb_flush(q) == RB_OK);
  CHECK(rb_advance(s, now + ((int64_t)1 << 40)) == RB_OK);
  rb_window_info w{};
  while (rb_run_window(s, &w) == RB_OK) {
  }
  CHECK(rb_queue_destroy(q) == RB_OK);
  CHECK(rb_sched_destroy(s) == RB_OK);
  CHECK(rb_model_destroy(cur) == RB_OK);
}

}  // namespace

int main(int argc, char** argv) {
  const bool threads = argc > 1 && std::strcmp(argv[1], "--threads") == 0;
  rb_ctx* ctx = nullptr;
  CHECK(rb_ctx_create(-1, &ctx) == RB_OK);
  if (threads) {
    loaders(ctx);
  } else {
    model_validation(ctx);
    for (uint64_t seed = 0; seed < 4; ++seed) replays(ctx, seed);
    for (uint64_t seed = 0; seed < 8; ++seed) serving(ctx, seed);
    rb_sched_opts bad{};
    bad.mode = RB_MODE_DEVICE;
    bad.window_batches = 1;
    rb_sched* s = nullptr;
    CHECK(rb_sched_create(ctx, &bad, &s) == RB_EDEVICE);
  }
  CHECK(rb_ctx_destroy(ctx) == RB_OK);
  if (failures) std::fprintf(stderr, "%d checks failed\n", failures);
  else
    std::printf("host paths ok%s: %lld replayed batches, %lld served requests, %lld version transitions, "
                "%lld queues replaced\n",
                threads ? " (loader threads)" : "", (long long)replayed_batches, (long long)served_requests,
                (long long)transitions, (long long)queue_churn);
  return failures ? 1 : 0;
}
