// Host runtime of libconvtune: device set-up, the pool of CU-masked streams,
// the timing protocol (profile stage of the tuning loop) with its timeout
// watchdog, registered references, tuning clients on disjoint CU masks (the
// thread machinery is in clients.cpp), one client over several CU slots,
// cross-evaluation and the probes.
#include <hip/hip_runtime.h>
#include <cstdio>
#include <cstdlib>

#include <algorithm>
#include <array>
#include <atomic>
#include <chrono>
#include <cmath>
#include <condition_variable>
#include <cstring>
#include <functional>
#include <map>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "ct_internal.h"
#include "k_util.h"

namespace ct {

int launch_max_error(const float* y, const float* ref, int64_t n, unsigned* out2, hipStream_t st);
int launch_cu_probe(int* out, int nblocks, hipStream_t st);
int launch_empty(int nblocks, hipStream_t st);
int launch_copy(const void* src, void* dst, int64_t bytes, int nblocks, hipStream_t st);

static int hip_fail(const char* what, hipError_t e) {
  set_error(std::string(what) + ": " + hipGetErrorString(e));
  return CT_E_HIP;
}
#define HIP_TRY(call)                                  \
  do {                                                 \
    hipError_t e_ = (call);                            \
    if (e_ != hipSuccess) return hip_fail(#call, e_);  \
  } while (0)

// ------------------------------------------------------------------ device
static std::mutex g_mu;  // guards the device state, the stream pool and the references
static int g_device = -1;
static int g_num_cus = 0;

// Split partial sums of conv2d_run_noalloc: a static array in device memory,
// one copy on every device the library runs on, held until the process ends.
// Host code never uses its name as an address: ct_init looks up the device
// address of the initialised device's copy (g_scratch_dev) and the launches
// take that.
constexpr int kMaxDevices = 64;
static __device__ __align__(256) float scratch[CT_SCRATCH_FLOATS];
static float* g_scratch_dev[kMaxDevices] = {};

using MaskKey = std::array<uint32_t, CT_MASK_WORDS>;

// Completion signal of a stream's work: a host function enqueued after the
// work sets it (see wait_events).
struct DrainSignal {
  std::mutex mu;
  std::condition_variable cv;
  bool done = true;
};

// One CU-masked stream with everything a measurement needs on it. A context
// is held by one call at a time (in_use) and returned to the pool after it.
struct StreamCtx {
  MaskKey key{};
  DrainSignal sig;
  bool in_use = false;
  bool abandoned = false;  // a wait on it was given up: never reused or synchronised
  hipStream_t stream = nullptr;
  std::vector<hipEvent_t> events;
  float* ws = nullptr;
  int64_t ws_floats = 0;
  unsigned* err = nullptr;  // 2 words per candidate of a batch
  int err_slots = 0;
  int* probe = nullptr;
  int probe_len = 0;
};

static std::vector<StreamCtx*> g_pool;  // every context, for reuse and ct_shutdown

// A context held for the duration of a call (or of a tuning client).
class Lease {
 public:
  Lease() = default;
  Lease(const Lease&) = delete;
  Lease& operator=(const Lease&) = delete;
  ~Lease() { release(); }
  StreamCtx* get() const { return c_; }
  void set(StreamCtx* c) { c_ = c; }
  void release() {
    if (!c_) return;
    std::lock_guard<std::mutex> g(g_mu);
    c_->in_use = false;
    c_ = nullptr;
  }

 private:
  StreamCtx* c_ = nullptr;
};

static int check_init() {
  if (g_device < 0) {
    set_error("ct_init has not succeeded");
    return CT_E_NOINIT;
  }
  return CT_OK;
}

static int mask_words_needed() { return (g_num_cus + 31) / 32; }

static int make_key(const uint32_t* mask, int words, MaskKey* key) {
  key->fill(0);
  if (!mask) {  // all CUs
    for (int b = 0; b < g_num_cus; ++b) (*key)[b / 32] |= 1u << (b % 32);
    return CT_OK;
  }
  if (words < mask_words_needed() || words > 64) {
    set_error("CU mask has the wrong number of words");
    return CT_E_ARG;
  }
  int bits = 0;
  for (int i = 0; i < words; ++i) {
    for (int b = 0; b < 32; ++b) {
      if (!(mask[i] >> b & 1u)) continue;
      const int cu = 32 * i + b;
      if (cu >= g_num_cus) {
        set_error("CU mask names a CU the device does not have");
        return CT_E_ARG;
      }
      (*key)[i] |= 1u << b;
      ++bits;
    }
  }
  if (!bits) {
    set_error("CU mask is empty");
    return CT_E_ARG;
  }
  return CT_OK;
}

// Slot j of the partition of the device into k = num_cus / m blocks of m
// contiguous mask bits, when the mask is one (the slots ct_build_cu_mask makes).
static bool partition_slot(const MaskKey& key, int* m, int* j) {
  int first = -1, last = -1, bits = 0;
  for (int b = 0; b < g_num_cus; ++b)
    if (key[b / 32] >> (b % 32) & 1u) {
      if (first < 0) first = b;
      last = b;
      ++bits;
    }
  if (bits == 0 || last - first + 1 != bits || g_num_cus % bits || first % bits) return false;
  *m = bits;
  *j = first / bits;
  return true;
}

static MaskKey slot_key(int m, int j) {
  MaskKey k;
  k.fill(0);
  for (int b = j * m; b < (j + 1) * m; ++b) k[b / 32] |= 1u << (b % 32);
  return k;
}

static std::mutex g_create_mu;  // stream creation, one at a time

// Takes an idle context of the mask from the pool, or creates one.
//
// The device deals hardware queues out to its dispatch pipes in the order the
// queues are created (measured: four CU-masked streams, one per 64-CU slot,
// run side by side with 3-9 % latency inflation when created one after the
// other, and with 2-3x when two of them were created four queues apart, which
// puts them on one pipe: a kernel waiting for CUs of its own slot then holds
// back the dispatch of the other slot's kernels). So the first use of any slot
// of a partition into at most 8 equal contiguous slots creates the streams of
// every slot of that partition at once, in slot order: the clients of one
// share get consecutive queues, on distinct pipes for up to 4 slots.
static int acquire(const MaskKey& key, Lease* lease) {
  int rc = check_init();
  if (rc) return rc;
  HIP_TRY(hipSetDevice(g_device));
  auto take_idle = [&]() -> bool {
    std::lock_guard<std::mutex> g(g_mu);
    for (StreamCtx* c : g_pool)
      if (!c->in_use && !c->abandoned && c->key == key) {
        c->in_use = true;
        lease->set(c);
        return true;
      }
    return false;
  };
  if (take_idle()) return CT_OK;
  std::lock_guard<std::mutex> cg(g_create_mu);
  if (take_idle()) return CT_OK;  // another thread created it meanwhile
  std::vector<MaskKey> todo;
  int m = 0, j = 0;
  if (partition_slot(key, &m, &j) && g_num_cus / m <= 8) {
    std::lock_guard<std::mutex> g(g_mu);
    for (int s = 0; s < g_num_cus / m; ++s) {
      const MaskKey ks = slot_key(m, s);
      bool have = false;
      for (StreamCtx* c : g_pool) have = have || (c->key == ks && !c->abandoned);
      if (!have || ks == key) todo.push_back(ks);
    }
  } else {
    todo.push_back(key);
  }
  StreamCtx* mine = nullptr;
  for (const MaskKey& k : todo) {
    StreamCtx* c = new StreamCtx();
    c->key = k;
    c->in_use = (k == key && !mine);
    hipError_t e = hipExtStreamCreateWithCUMask(&c->stream, (uint32_t)mask_words_needed(), k.data());
    if (e != hipSuccess) {
      delete c;
      return hip_fail("hipExtStreamCreateWithCUMask", e);
    }
    if (c->in_use) mine = c;
    std::lock_guard<std::mutex> g(g_mu);
    g_pool.push_back(c);
  }
  lease->set(mine);
  return CT_OK;
}

static int acquire_mask(const uint32_t* mask, int words, Lease* lease) {
  MaskKey key;
  int rc = check_init();
  if (rc || (rc = make_key(mask, words, &key))) return rc;
  return acquire(key, lease);
}

static int ensure_events(StreamCtx* c, size_t n) {
  while (c->events.size() < n) {
    hipEvent_t ev;
    HIP_TRY(hipEventCreate(&ev));
    c->events.push_back(ev);
  }
  return CT_OK;
}

static int ensure_ws(StreamCtx* c, int64_t floats) {
  if (floats <= c->ws_floats) return CT_OK;
  if (c->ws) {
    HIP_TRY(hipStreamSynchronize(c->stream));
    HIP_TRY(hipFree(c->ws));
    c->ws = nullptr;
    c->ws_floats = 0;
  }
  if (hipMalloc((void**)&c->ws, sizeof(float) * floats) != hipSuccess) {
    c->ws = nullptr;
    set_error("workspace allocation failed");
    return CT_E_OOM;
  }
  c->ws_floats = floats;
  return CT_OK;
}

static int ensure_err(StreamCtx* c, int slots) {
  if (slots <= c->err_slots) return CT_OK;
  if (c->err) {
    HIP_TRY(hipStreamSynchronize(c->stream));
    HIP_TRY(hipFree(c->err));
  }
  c->err = nullptr;
  c->err_slots = 0;
  HIP_TRY(hipMalloc((void**)&c->err, sizeof(unsigned) * 2 * slots));
  c->err_slots = slots;
  return CT_OK;
}

// Teardown is best effort: a failing release leaves nothing else to undo, so
// the return codes are dropped on purpose.
static void destroy_ctx(StreamCtx* c) {
  if (c->abandoned) return;  // work may still be queued on it: leave it alone
  if (c->stream) (void)hipStreamSynchronize(c->stream);
  for (hipEvent_t e : c->events) (void)hipEventDestroy(e);
  if (c->ws) (void)hipFree(c->ws);
  if (c->err) (void)hipFree(c->err);
  if (c->probe) (void)hipFree(c->probe);
  if (c->stream) (void)hipStreamDestroy(c->stream);
  delete c;
}

// ------------------------------------------------------------------ references
using OpKey = std::array<int32_t, sizeof(ct_op) / sizeof(int32_t)>;
struct RefBuf {
  float* d = nullptr;
  int64_t n = 0;
  float tol = 0.f;
};
static std::map<OpKey, RefBuf> g_refs;

static OpKey op_key(const ct_op& op) {
  OpKey k;
  std::memcpy(k.data(), &op, sizeof(ct_op));
  return k;
}

// The reference a measurement checks against: the explicit one, else the op's
// registered one, else none.
static void resolve_ref(const OpX& x, const ct_verify* v, const float** ref, float* tol) {
  *ref = nullptr;
  *tol = 0.f;
  if (v && v->y_ref) {
    *ref = v->y_ref;
    *tol = v->tol;
    return;
  }
  std::lock_guard<std::mutex> g(g_mu);
  auto it = g_refs.find(op_key(x.op));
  if (it != g_refs.end() && it->second.n == x.ny) {
    *ref = it->second.d;
    *tol = it->second.tol;
  }
}

// ------------------------------------------------------------------ launch
static int launch_once(const OpX& x, const ct_schedule& s, const Geom& g, const void* xin, const void* w,
                       void* y, float* ws, hipStream_t st) {
  switch (s.family) {
    case CT_FAM_DIRECT_F32: return launch_direct_f32(x, s, g, xin, w, y, ws, st);
    case CT_FAM_DEPTHWISE_F32: return launch_depthwise_f32(x, s, g, xin, w, y, ws, st);
    case CT_FAM_IGEMM_BF16: return launch_igemm_bf16(x, s, g, xin, w, y, ws, st);
    case CT_FAM_IGEMM_F32: return launch_igemm_f32(x, s, g, xin, w, y, ws, st);
  }
  return -1;
}

static bool opts_ok(const ct_measure_opts* o) {
  return o && o->warmup >= 0 && o->repeats >= 1 && o->repeats <= 64 && o->launches >= 1 &&
         o->launches <= 100000 && o->batch >= 1 && o->timeout_ms > 0.f;
}

static float median_of(std::vector<float> v) {
  std::sort(v.begin(), v.end());
  const size_t n = v.size();
  if (n % 2) return v[n / 2];
  return (float)(((double)v[n / 2 - 1] + (double)v[n / 2]) / 2.0);
}

// ------------------------------------------------------------------ watchdog
constexpr double kSlackS = 0.05;
constexpr double kDrainMinS = 2.0;
constexpr double kDrainMaxS = 60.0;

// Events recorded on one stream since the last wait, in enqueue order.
struct EventLog {
  std::vector<hipEvent_t> ev;
  std::vector<int32_t> runs;   // runs enqueued since the previous event
  std::vector<int32_t> owner;  // candidate whose runs end at the event
  int pending = 0;
  hipError_t err = hipSuccess;  // the first failed record since the last clear
  void clear() {
    ev.clear();
    runs.clear();
    owner.clear();
    pending = 0;
    err = hipSuccess;
  }
  void record(hipEvent_t e, hipStream_t st, int who) {
    const hipError_t r = hipEventRecord(e, st);
    if (r != hipSuccess && err == hipSuccess) err = r;
    ev.push_back(e);
    runs.push_back(pending);
    owner.push_back(who);
    pending = 0;
  }
};

static void on_drain(void* p) {
  DrainSignal* d = static_cast<DrainSignal*>(p);
  {
    std::lock_guard<std::mutex> g(d->mu);
    d->done = true;
  }
  d->cv.notify_all();
}

// Waits for every event of the log with the watchdog. A host function enqueued
// after the last event signals completion, so the host sleeps instead of
// polling; an event is queried only once its deadline has passed (querying an
// event the device has not reached makes the runtime submit extra work to
// flush the queue, which would disturb the streams being timed). Returns CT_OK
// (and the owner of a missed deadline in *late, -1 if none), CT_E_TIMEOUT when
// the stream did not drain (the context is then abandoned; the signal it still
// points to is never freed), or CT_E_HIP.
static int wait_events(StreamCtx* c, const EventLog& lg, double run_limit_s, int* late) {
  *late = -1;
  const int n = (int)lg.ev.size();
  {
    std::lock_guard<std::mutex> g(c->sig.mu);
    c->sig.done = false;
  }
  const hipError_t he = hipLaunchHostFunc(c->stream, on_drain, &c->sig);
  if (he != hipSuccess) {
    std::lock_guard<std::mutex> g(c->sig.mu);
    c->sig.done = true;
    return hip_fail("hipLaunchHostFunc", he);
  }
  auto done = [&](int k) -> int {
    const hipError_t e = hipEventQuery(lg.ev[k]);
    if (e == hipSuccess) return 1;
    if (e == hipErrorNotReady) return 0;
    return hip_fail("hipEventQuery", e);
  };
  auto wait_until = [&](double t) -> bool {
    using clk = std::chrono::steady_clock;
    const auto tp = clk::time_point(std::chrono::duration_cast<clk::duration>(std::chrono::duration<double>(t)));
    std::unique_lock<std::mutex> l(c->sig.mu);
    return c->sig.cv.wait_until(l, tp, [&] { return c->sig.done; });
  };
  int64_t total_runs = 0;
  for (int32_t r : lg.runs) total_runs += r;
  const double drain = std::min(kDrainMaxS, std::max(kDrainMinS, 4.0 * run_limit_s * (double)total_runs));
  const WatchResult w = watch_events(n, lg.runs.data(), run_limit_s, kSlackS, drain, done, wait_until, now_s);
  if (w.rc) return w.rc;
  if (w.expired >= 0) *late = lg.owner[w.expired];
  if (!w.drained) {
    {
      std::lock_guard<std::mutex> g(g_mu);
      c->abandoned = true;
    }
    set_error("a candidate ran past its time limit and the stream did not drain within " + std::to_string(drain) +
              " s; the stream is abandoned");
    return CT_E_TIMEOUT;
  }
  return CT_OK;
}

// The profile step: time n candidates on one stream with protocol o.
// skip (optional): candidates that are not measured (their lat/status are the
// caller's). on_batch (optional): called with each group [i0, i1) once its
// results are final; returning false stops the measurement (CT_E_STOPPED).
static int measure_impl(const OpX& x, const ct_schedule* s, int n, StreamCtx* c, const ct_measure_opts& o,
                        const ct_verify* v, const void* xin, const void* w, void* y, float* lat, int32_t* status,
                        float* rep, const uint8_t* skip = nullptr,
                        const std::function<bool(int, int)>& on_batch = nullptr) {
  std::vector<Geom> geo(n);
  std::vector<char> live(n, 0);
  int64_t maxws = 0;
  for (int i = 0; i < n; ++i) {
    if (skip && skip[i]) continue;
    lat[i] = INFINITY;
    status[i] = CT_S_INVALID;
    if (rep)
      for (int r = 0; r < o.repeats; ++r) rep[(int64_t)i * o.repeats + r] = INFINITY;
    if (compute_geom(x, s[i], &geo[i], nullptr) == CT_OK) {
      live[i] = 1;
      status[i] = CT_S_OK;
      maxws = std::max(maxws, geo[i].ws_floats);
    }
  }
  int rc = ensure_ws(c, maxws);
  if (rc) return rc;
  const float* ref = nullptr;
  float tol = 0.f;
  resolve_ref(x, v, &ref, &tol);
  const int batch = std::min(o.batch, std::max(n, 1));
  if (ref && (rc = ensure_err(c, batch))) return rc;
  const int R = o.repeats, L = o.launches;
  if ((rc = ensure_events(c, (size_t)2 * R * batch + 1))) return rc;
  hipStream_t st = c->stream;
  const double limit_s = (double)o.timeout_ms * 1e-3;
  EventLog lg;

  auto run = [&](int i) -> bool {  // one run of candidate i; false on launch failure
    ++lg.pending;
    if (launch_once(x, s[i], geo[i], xin, w, y, c->ws, st) != 0) {
      live[i] = 0;
      status[i] = CT_S_LAUNCH;
      return false;
    }
    return true;
  };
  auto timed = [&](int i, int slot, int r) {
    lg.record(c->events[(size_t)2 * (slot * R + r)], st, i);
    for (int l = 0; l < L && live[i]; ++l) run(i);
    lg.record(c->events[(size_t)2 * (slot * R + r) + 1], st, i);
  };
  // candidates left unmeasured when a call gives up on its stream
  auto abandon_rest = [&](int from) {
    for (int i = from; i < n; ++i)
      if (live[i]) status[i] = CT_S_TIMEOUT;
  };

  std::vector<float> reps(R);
  for (int b0 = 0; b0 < n; b0 += batch) {
    const int b1 = std::min(n, b0 + batch);
    lg.clear();
    for (int i = b0; i < b1; ++i)
      for (int k = 0; k < o.warmup && live[i]; ++k) run(i);
    if (o.interleave) {
      for (int r = 0; r < R; ++r)
        for (int i = b0; i < b1; ++i)
          if (live[i]) timed(i, i - b0, r);
    } else {
      for (int i = b0; i < b1; ++i)
        if (live[i])
          for (int r = 0; r < R; ++r) timed(i, i - b0, r);
    }
    int late = -1;
    if (lg.err != hipSuccess) return hip_fail("hipEventRecord", lg.err);
    if (!lg.ev.empty()) {
      rc = wait_events(c, lg, limit_s, &late);
      if (rc == CT_E_TIMEOUT) {
        if (late >= 0) status[late] = CT_S_TIMEOUT;
        abandon_rest(b0);
      }
      if (rc) return rc;
    }
    for (int i = b0; i < b1; ++i) {
      if (!live[i]) continue;
      for (int r = 0; r < R; ++r) {
        float ms = 0.f;
        HIP_TRY(hipEventElapsedTime(&ms, c->events[(size_t)2 * ((i - b0) * R + r)],
                                    c->events[(size_t)2 * ((i - b0) * R + r) + 1]));
        reps[r] = ms * 1000.0f / (float)L;
        if (rep) rep[(int64_t)i * R + r] = reps[r];
      }
      lat[i] = median_of(reps);
      if (i == late || lat[i] > o.timeout_ms * 1000.0f) status[i] = CT_S_TIMEOUT;
    }
    if (ref) {
      // Re-run every live candidate once more, each followed by its check, so
      // the compared output is the candidate's own whatever the timing order.
      lg.clear();
      for (int i = b0; i < b1; ++i) {
        if (!live[i]) continue;
        if (!run(i)) continue;
        if (launch_max_error((const float*)y, ref, x.ny, c->err + 2 * (i - b0), st) != 0)
          return hip_fail("verification launch", hipGetLastError());
      }
      std::vector<unsigned> h(2 * (size_t)(b1 - b0));
      HIP_TRY(hipMemcpyAsync(h.data(), c->err, sizeof(unsigned) * h.size(), hipMemcpyDeviceToHost, st));
      lg.record(c->events[(size_t)2 * R * batch], st, -1);
      if (lg.err != hipSuccess) return hip_fail("hipEventRecord", lg.err);
      int late2 = -1;
      rc = wait_events(c, lg, limit_s, &late2);
      if (rc == CT_E_TIMEOUT) abandon_rest(b0);
      if (rc) return rc;
      HIP_TRY(hipStreamSynchronize(st));  // the copy into pageable memory has landed
      for (int i = b0; i < b1; ++i) {
        if (!live[i] || status[i] != CT_S_OK) continue;
        float e, m;
        std::memcpy(&e, &h[2 * (i - b0)], 4);
        std::memcpy(&m, &h[2 * (i - b0) + 1], 4);
        if (!(e <= tol * m)) status[i] = CT_S_WRONG_ANSWER;
      }
    }
    for (int i = b0; i < b1; ++i)
      if (!(skip && skip[i]) && status[i] != CT_S_OK && status[i] != CT_S_TIMEOUT &&
          status[i] != CT_S_WRONG_ANSWER)
        lat[i] = INFINITY;
    if (on_batch && !on_batch(b0, b1)) {
      set_error("measurement stopped by its caller");
      return CT_E_STOPPED;
    }
  }
  return CT_OK;
}

static int derive_checked(const ct_op* op, OpX* x) {
  if (!op) {
    set_error("null op");
    return CT_E_ARG;
  }
  std::string why;
  if (!derive_op(*op, x, &why)) {
    set_error(why);
    return CT_E_ARG;
  }
  return CT_OK;
}

// ------------------------------------------------------------------ tuning
// Stage 1 on all candidates, then stage 2 on the top_t and the tie rule.
static int tune_job(ct_tune_job* j, StreamCtx* c, const ct_measure_opts& o1, const ct_measure_opts& o2, float eps,
                    RecordSink* sink) {
  OpX x;
  int rc = derive_checked(&j->op, &x);
  if (rc) return rc;
  j->t_start_s = now_s();
  j->n_top = 0;
  j->winner_pos = -1;
  j->winner_lat_us = INFINITY;
  std::function<bool(int, int)> on_batch;
  if (sink) on_batch = [&](int i0, int i1) { return sink->candidates(*j, i0, i1); };
  rc = measure_impl(x, j->cands, j->n_cands, c, o1, &j->verify, j->x, j->w, j->y, j->lat1_us, j->status1, nullptr,
                    j->skip, on_batch);
  if (rc) return rc;
  ct_measure_opts o = o2;
  o.interleave = 1;
  rc = select_job(j, eps, [&](const int32_t* pos, int nt, float* lat2) {
    std::vector<ct_schedule> s2(nt);
    for (int i = 0; i < nt; ++i) s2[i] = j->cands[pos[i]];
    std::vector<int32_t> st2(nt);
    int r = measure_impl(x, s2.data(), nt, c, o, nullptr, j->x, j->w, j->y, lat2, st2.data(), nullptr);
    if (r) return r;
    for (int i = 0; i < nt; ++i)
      if (st2[i] != CT_S_OK) lat2[i] = INFINITY;
    return CT_OK;
  });
  j->t_end_s = now_s();
  return rc;
}

static int check_jobs(const ct_tune_job* jobs, int n_jobs) {
  for (int i = 0; i < n_jobs; ++i) {
    const ct_tune_job& j = jobs[i];
    if (!j.cands || j.n_cands < 0 || !j.lat1_us || !j.status1 || j.top_t < 1 || !j.top_pos || !j.lat2_us ||
        !j.x || !j.w || !j.y) {
      set_error("tune job " + std::to_string(i) + ": bad arrays");
      return CT_E_ARG;
    }
  }
  return CT_OK;
}

// Runs the clients on the device: each holds one context of its mask for all
// of its jobs.
static int run_device_clients(ct_client* clients, int n_clients, const std::vector<JobSource>& src,
                              const ct_measure_opts* o1, const ct_measure_opts* o2, float eps) {
  std::vector<Lease> leases(n_clients);  // slot i is touched by client thread i only
  JobFn fn = [&](int ci, ct_tune_job* j, RecordSink* sink) -> int {
    if (!leases[ci].get()) {
      const int rc = acquire_mask(clients[ci].cu_mask, CT_MASK_WORDS, &leases[ci]);
      if (rc) return rc;
    }
    return tune_job(j, leases[ci].get(), *o1, *o2, eps, sink);
  };
  ClientEndFn end = [&](int ci) { leases[ci].release(); };
  return run_clients(clients, n_clients, src, fn, end, -1);
}

}  // namespace ct

// ================================================================= C ABI
using namespace ct;

extern "C" {

int ct_init(int device) {
  std::lock_guard<std::mutex> g(g_mu);
  if (g_device >= 0) {
    if (device == g_device) return CT_OK;
    set_error("ct_init: already initialised for another device");
    return CT_E_ARG;
  }
  int count = 0;
  hipError_t e = hipGetDeviceCount(&count);
  if (e != hipSuccess || count <= 0) {
    set_error("ct_init: no HIP device");
    return CT_E_NODEV;
  }
  if (device < 0 || device >= count) {
    set_error("ct_init: device index out of range");
    return CT_E_ARG;
  }
  HIP_TRY(hipSetDevice(device));
  hipDeviceProp_t p;
  HIP_TRY(hipGetDeviceProperties(&p, device));
  if (std::strncmp(p.gcnArchName, "gfx950", 6) != 0) {
    set_error(std::string("ct_init: device is ") + p.gcnArchName + ", the kernels are built for gfx950");
    return CT_E_NODEV;
  }
  if (p.multiProcessorCount <= 0 || p.multiProcessorCount > 32 * CT_MASK_WORDS) {
    set_error("ct_init: unexpected CU count");
    return CT_E_NODEV;
  }
  if (device >= kMaxDevices) {
    set_error("ct_init: device index beyond the library's table");
    return CT_E_ARG;
  }
  if (!g_scratch_dev[device]) {  // this device's copy of the static scratch array
    float* ptr = nullptr;
    HIP_TRY(hipGetSymbolAddress((void**)&ptr, HIP_SYMBOL(scratch)));
    g_scratch_dev[device] = ptr;
  }
  g_num_cus = p.multiProcessorCount;
  g_device = device;
  return CT_OK;
}

int ct_num_cus(void) {
  if (check_init()) return CT_E_NOINIT;
  return g_num_cus;
}

void ct_shutdown(void) {
  std::lock_guard<std::mutex> g(g_mu);
  if (g_device < 0 && g_pool.empty() && g_refs.empty()) return;  // nothing to release (a second call)
  if (g_device >= 0) (void)hipSetDevice(g_device);  // teardown: best effort
  for (StreamCtx* c : g_pool) destroy_ctx(c);
  g_pool.clear();
  for (auto& kv : g_refs) (void)hipFree(kv.second.d);
  g_refs.clear();
  g_device = -1;
  g_num_cus = 0;
}

int ct_stream_count(void) {
  std::lock_guard<std::mutex> g(g_mu);
  return (int)g_pool.size();
}

int ct_cu_mask(double fraction, int slot, uint32_t* mask, int words) {
  int rc = check_init();
  if (rc) return rc;
  return ct_build_cu_mask(g_num_cus, fraction, slot, mask, words);
}

int ct_set_reference(const ct_op* op, const double* y_ref_host) {
  OpX ox;
  int rc = derive_checked(op, &ox);
  if (rc || (rc = check_init())) return rc;
  const OpKey key = op_key(*op);
  float* d = nullptr;
  if (y_ref_host) {
    std::vector<float> h((size_t)ox.ny);
    for (int64_t i = 0; i < ox.ny; ++i) h[(size_t)i] = (float)y_ref_host[i];
    HIP_TRY(hipSetDevice(g_device));
    if (hipMalloc((void**)&d, sizeof(float) * (size_t)ox.ny) != hipSuccess) {
      set_error("ct_set_reference: allocation failed");
      return CT_E_OOM;
    }
    const hipError_t e = hipMemcpy(d, h.data(), sizeof(float) * (size_t)ox.ny, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
      (void)hipFree(d);
      return hip_fail("ct_set_reference: upload", e);
    }
  }
  float* old = nullptr;
  {
    std::lock_guard<std::mutex> g(g_mu);
    auto it = g_refs.find(key);
    if (it != g_refs.end()) {
      old = it->second.d;
      g_refs.erase(it);
    }
    if (d) g_refs[key] = RefBuf{d, ox.ny, op->dtype == CT_DT_BF16 ? 2e-2f : 1e-4f};
  }
  if (old) HIP_TRY(hipFree(old));
  return CT_OK;
}

int conv2d_run(const ct_op* op, const ct_schedule* s, const void* x, const void* w, void* y,
               const uint32_t* cu_mask, int words) {
  OpX ox;
  int rc = derive_checked(op, &ox);
  if (rc) return rc;
  if (!s || !x || !w || !y) {
    set_error("conv2d_run: null argument");
    return CT_E_ARG;
  }
  Geom g;
  std::string why;
  if (compute_geom(ox, *s, &g, &why) != CT_OK) {
    set_error("conv2d_run: invalid schedule: " + why);
    return CT_E_ARG;
  }
  Lease lease;
  if ((rc = acquire_mask(cu_mask, words, &lease))) return rc;
  StreamCtx* c = lease.get();
  if ((rc = ensure_ws(c, g.ws_floats))) return rc;
  const int lrc = launch_once(ox, *s, g, x, w, y, c->ws, c->stream);
  if (lrc == -2) return CT_E_ARG;  // the launcher refused the arguments (reason already set)
  if (lrc != 0) return hip_fail("conv2d_run launch", hipGetLastError());
  HIP_TRY(hipStreamSynchronize(c->stream));
  return CT_OK;
}

int conv2d_run_noalloc(const ct_op* op, const ct_schedule* s, const void* x, const void* w, void* y,
                       void* stream) {
  OpX ox;
  int rc = derive_checked(op, &ox);
  if (rc) return rc;
  if (!s || !x || !w || !y) {
    set_error("conv2d_run_noalloc: null argument");
    return CT_E_ARG;
  }
  if ((rc = check_init())) return rc;
  Geom g;
  std::string why;
  if (compute_geom(ox, *s, &g, &why) != CT_OK) {
    set_error("conv2d_run_noalloc: invalid schedule: " + why);
    return CT_E_ARG;
  }
  if (g.ws_floats > (int64_t)CT_SCRATCH_FLOATS) {
    set_error("conv2d_run_noalloc: the schedule's split partial sums need " + std::to_string(g.ws_floats) +
              " floats; the static scratch array holds " + std::to_string((int64_t)CT_SCRATCH_FLOATS));
    return CT_E_ARG;
  }
  float* ws = g_scratch_dev[g_device];
  if (!ws) {
    set_error("conv2d_run_noalloc: no scratch address for the device");
    return CT_E_NOINIT;
  }
  const int lrc = launch_once(ox, *s, g, x, w, y, ws, (hipStream_t)stream);
  if (lrc == -2) return CT_E_ARG;  // the launcher refused the arguments (reason already set)
  if (lrc != 0) return hip_fail("conv2d_run_noalloc launch", hipGetLastError());
  return CT_OK;
}

int measure_candidates_mask(const ct_op* op, const ct_schedule* s, int n, const uint32_t* cu_mask, int words,
                            const ct_measure_opts* o, const ct_verify* v, const void* x, const void* w, void* y,
                            float* lat_us, int32_t* status, float* rep_us) {
  OpX ox;
  int rc = derive_checked(op, &ox);
  if (rc) return rc;
  if (n < 0 || (n > 0 && (!s || !lat_us || !status)) || !x || !w || !y || !opts_ok(o)) {
    set_error("measure_candidates: bad argument");
    return CT_E_ARG;
  }
  Lease lease;
  if ((rc = acquire_mask(cu_mask, words, &lease))) return rc;
  return measure_impl(ox, s, n, lease.get(), *o, v, x, w, y, lat_us, status, rep_us);
}

int measure_candidates(const ct_op* op, const ct_schedule* s, int n, double cu_fraction,
                       const ct_measure_opts* o, const void* x, const void* w, void* y, float* lat_us,
                       int32_t* status) {
  int rc = check_init();
  if (rc) return rc;
  uint32_t mask[CT_MASK_WORDS];
  if ((rc = ct_build_cu_mask(g_num_cus, cu_fraction, 0, mask, CT_MASK_WORDS))) return rc;
  return measure_candidates_mask(op, s, n, mask, CT_MASK_WORDS, o, nullptr, x, w, y, lat_us, status, nullptr);
}

int ct_tune_clients(ct_client* clients, int n_clients, const ct_measure_opts* stage1,
                    const ct_measure_opts* stage2, float eps) {
  int rc = check_init();
  if (rc) return rc;
  if (!clients || n_clients < 1 || n_clients > 64 || !opts_ok(stage1) || !opts_ok(stage2) || !(eps >= 0.f)) {
    set_error("ct_tune_clients: bad argument");
    return CT_E_ARG;
  }
  std::vector<JobSource> src(n_clients);
  for (int i = 0; i < n_clients; ++i) {
    if (clients[i].n_jobs < 0 || (clients[i].n_jobs > 0 && !clients[i].jobs) ||
        (rc = check_jobs(clients[i].jobs, clients[i].n_jobs))) {
      if (!rc) set_error("ct_tune_clients: bad job list");
      return rc ? rc : CT_E_ARG;
    }
    src[i] = {clients[i].jobs, clients[i].n_jobs, nullptr, nullptr};
  }
  return run_device_clients(clients, n_clients, src, stage1, stage2, eps);
}

int ct_tune_shared(ct_client* clients, int n_clients, ct_tune_job* jobs, int n_jobs,
                   const ct_measure_opts* stage1, const ct_measure_opts* stage2, float eps,
                   int32_t* job_client) {
  int rc = check_init();
  if (rc) return rc;
  if (!clients || n_clients < 1 || n_clients > 64 || n_jobs < 0 || (n_jobs > 0 && !jobs) || !opts_ok(stage1) ||
      !opts_ok(stage2) || !(eps >= 0.f)) {
    set_error("ct_tune_shared: bad argument");
    return CT_E_ARG;
  }
  if ((rc = check_jobs(jobs, n_jobs))) return rc;
  if (job_client)
    for (int i = 0; i < n_jobs; ++i) job_client[i] = -1;
  std::atomic<int> next{0};
  std::vector<JobSource> src(n_clients, JobSource{jobs, n_jobs, &next, job_client});
  return run_device_clients(clients, n_clients, src, stage1, stage2, eps);
}

int ct_tune_split(ct_tune_job* job, const uint32_t* masks, int k, int words, void* const* y_slots,
                  const ct_measure_opts* stage1, const ct_measure_opts* stage2, float eps, double* screen_s) {
  int rc = check_init();
  if (rc) return rc;
  if (!job || !masks || k < 1 || k > 64 || !y_slots || !opts_ok(stage1) || !opts_ok(stage2) || !(eps >= 0.f)) {
    set_error("ct_tune_split: bad argument");
    return CT_E_ARG;
  }
  for (int j = 0; j < k; ++j)
    if (!y_slots[j]) {
      set_error("ct_tune_split: null output buffer");
      return CT_E_ARG;
    }
  if ((rc = check_jobs(job, 1))) return rc;
  OpX x;
  if ((rc = derive_checked(&job->op, &x))) return rc;
  job->t_start_s = now_s();
  job->n_top = 0;
  job->winner_pos = -1;
  job->winner_lat_us = INFINITY;
  const int n = job->n_cands;
  std::vector<int> rcs(k, CT_OK);
  std::vector<std::string> errs(k);
  auto screen = [&](int j) {
    const int b = (int)((int64_t)n * j / k), e = (int)((int64_t)n * (j + 1) / k);
    Lease lease;
    int r = acquire_mask(masks + (size_t)j * words, words, &lease);
    if (!r && e > b)
      r = measure_impl(x, job->cands + b, e - b, lease.get(), *stage1, &job->verify, job->x, job->w, y_slots[j],
                       job->lat1_us + b, job->status1 + b, nullptr, job->skip ? job->skip + b : nullptr);
    rcs[j] = r;
    if (r) errs[j] = last_error();
  };
  const double t0 = now_s();
  {
    std::vector<std::thread> th;
    for (int j = 0; j < k; ++j) th.emplace_back(screen, j);
    for (auto& t : th) t.join();
  }
  if (screen_s) *screen_s = now_s() - t0;
  for (int j = 0; j < k; ++j)
    if (rcs[j]) {
      set_error("ct_tune_split: slot " + std::to_string(j) + ": " + errs[j]);
      return job->rc = rcs[j];
    }
  Lease lease0;
  if ((rc = acquire_mask(masks, words, &lease0))) return job->rc = rc;
  ct_measure_opts o2 = *stage2;
  o2.interleave = 1;
  rc = select_job(job, eps, [&](const int32_t* pos, int nt, float* lat2) {
    std::vector<ct_schedule> s2(nt);
    for (int i = 0; i < nt; ++i) s2[i] = job->cands[pos[i]];
    std::vector<int32_t> st2(nt);
    int r = measure_impl(x, s2.data(), nt, lease0.get(), o2, nullptr, job->x, job->w, y_slots[0], lat2, st2.data(),
                         nullptr);
    if (r) return r;
    for (int i = 0; i < nt; ++i)
      if (st2[i] != CT_S_OK) lat2[i] = INFINITY;
    return CT_OK;
  });
  job->t_end_s = now_s();
  return job->rc = rc;
}

int ct_cross_eval(const ct_op* op, const ct_schedule* s, int n_sched, const uint32_t* masks, int n_masks,
                  int words, const ct_measure_opts* o, const void* x, const void* w, void* y, float* M) {
  OpX ox;
  int rc = derive_checked(op, &ox);
  if (rc) return rc;
  if (!s || n_sched < 1 || !masks || n_masks < 1 || !M || !opts_ok(o) || !x || !w || !y) {
    set_error("ct_cross_eval: bad argument");
    return CT_E_ARG;
  }
  if ((rc = check_init())) return rc;
  ct_measure_opts oo = *o;
  oo.interleave = 1;
  std::vector<float> lat(n_sched);
  std::vector<int32_t> st(n_sched);
  for (int j = 0; j < n_masks; ++j) {
    Lease lease;
    if ((rc = acquire_mask(masks + (size_t)j * words, words, &lease))) return rc;
    if ((rc = measure_impl(ox, s, n_sched, lease.get(), oo, nullptr, x, w, y, lat.data(), st.data(), nullptr)))
      return rc;
    for (int i = 0; i < n_sched; ++i) M[(size_t)i * n_masks + j] = st[i] == CT_S_OK ? lat[i] : INFINITY;
  }
  return CT_OK;
}

int ct_test_xcd_band(int tiles, int32_t* tile_of_block) {
  if (tiles < 1 || !tile_of_block) {
    set_error("ct_test_xcd_band: bad argument");
    return CT_E_ARG;
  }
  for (int b = 0; b < tiles; ++b) tile_of_block[b] = xcd_band_tile(b, tiles);
  return CT_OK;
}

int ct_probe_cus(const uint32_t* cu_mask, int words, int blocks, int32_t* out, int cap, int32_t* n_out) {
  int rc;
  if (blocks < 1 || blocks > (1 << 20) || !n_out) {
    set_error("ct_probe_cus: bad argument");
    return CT_E_ARG;
  }
  Lease lease;
  if ((rc = acquire_mask(cu_mask, words, &lease))) return rc;
  StreamCtx* c = lease.get();
  if (c->probe_len < blocks) {
    if (c->probe) HIP_TRY(hipFree(c->probe));
    c->probe = nullptr;
    c->probe_len = 0;
    HIP_TRY(hipMalloc((void**)&c->probe, sizeof(int) * blocks));
    c->probe_len = blocks;
  }
  if (launch_cu_probe(c->probe, blocks, c->stream) != 0) return hip_fail("cu probe launch", hipGetLastError());
  std::vector<int> h(blocks);
  HIP_TRY(hipMemcpyAsync(h.data(), c->probe, sizeof(int) * blocks, hipMemcpyDeviceToHost, c->stream));
  HIP_TRY(hipStreamSynchronize(c->stream));
  std::sort(h.begin(), h.end());
  h.erase(std::unique(h.begin(), h.end()), h.end());
  *n_out = (int32_t)h.size();
  for (int i = 0; i < (int)h.size() && i < cap && out; ++i) out[i] = h[i];
  return CT_OK;
}

static int probe_timed(const uint32_t* cu_mask, int words, const ct_measure_opts* o, float* us,
                       const std::function<int(hipStream_t)>& body) {
  int rc;
  if (!opts_ok(o) || !us) {
    set_error("probe: bad argument");
    return CT_E_ARG;
  }
  Lease lease;
  if ((rc = acquire_mask(cu_mask, words, &lease))) return rc;
  StreamCtx* c = lease.get();
  if ((rc = ensure_events(c, (size_t)2 * o->repeats))) return rc;
  for (int k = 0; k < o->warmup; ++k)
    if (body(c->stream)) return hip_fail("probe launch", hipGetLastError());
  for (int r = 0; r < o->repeats; ++r) {
    HIP_TRY(hipEventRecord(c->events[2 * r], c->stream));
    for (int l = 0; l < o->launches; ++l)
      if (body(c->stream)) return hip_fail("probe launch", hipGetLastError());
    HIP_TRY(hipEventRecord(c->events[2 * r + 1], c->stream));
  }
  HIP_TRY(hipStreamSynchronize(c->stream));
  std::vector<float> v(o->repeats);
  for (int r = 0; r < o->repeats; ++r) {
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, c->events[2 * r], c->events[2 * r + 1]));
    v[r] = ms * 1000.0f / (float)o->launches;
  }
  *us = median_of(v);
  return CT_OK;
}

int ct_probe_empty(const uint32_t* cu_mask, int words, int blocks, const ct_measure_opts* o, float* us) {
  if (blocks < 1 || blocks > (1 << 20)) {
    set_error("ct_probe_empty: bad block count");
    return CT_E_ARG;
  }
  return probe_timed(cu_mask, words, o, us, [&](hipStream_t st) { return launch_empty(blocks, st); });
}

int ct_probe_copy(const uint32_t* cu_mask, int words, const void* src, void* dst, int64_t bytes,
                  const ct_measure_opts* o, float* gbps) {
  if (!src || !dst || bytes <= 0 || ((uintptr_t)src % 16) || ((uintptr_t)dst % 16) || !gbps) {
    set_error("ct_probe_copy: bad argument (buffers must be 16-byte aligned)");
    return CT_E_ARG;
  }
  int rc = check_init();
  if (rc) return rc;
  MaskKey key;
  if ((rc = make_key(cu_mask, words, &key))) return rc;
  int cus = 0;
  for (uint32_t v : key) cus += __builtin_popcount(v);
  const int blocks = cus * 8;
  float us = 0.f;
  rc = probe_timed(cu_mask, words, o, &us, [&](hipStream_t st) { return launch_copy(src, dst, bytes, blocks, st); });
  if (rc) return rc;
  *gbps = (float)(2.0 * (double)bytes / ((double)us * 1e-6) / 1e9);
  return CT_OK;
}

}  // extern "C"
