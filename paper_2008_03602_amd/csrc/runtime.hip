// Host runtime of libconvtune: device set-up, per-thread CU-masked streams,
// the timing protocol (profile stage of the tuning loop), tuning clients on
// disjoint CU masks, cross-evaluation and the probes.
#include <hip/hip_runtime.h>
#include <cstdio>
#include <cstdlib>
#include <pthread.h>
#include <sched.h>

#include <algorithm>
#include <array>
#include <atomic>
#include <chrono>
#include <cmath>
#include <cstring>
#include <functional>
#include <map>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "ct_internal.h"

namespace ct {

int launch_max_error(const float* y, const float* ref, int64_t n, unsigned* out2, hipStream_t st);
int launch_cu_probe(int* out, int nblocks, hipStream_t st);
int launch_empty(int nblocks, hipStream_t st);
int launch_copy(const void* src, void* dst, int64_t bytes, int nblocks, hipStream_t st);

// ------------------------------------------------------------------ errors
static thread_local std::string t_err;
void set_error(const std::string& msg) { t_err = msg; }

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
static std::mutex g_mu;
static int g_device = -1;
static int g_num_cus = 0;
static std::atomic<int> g_generation{0};

using MaskKey = std::array<uint32_t, CT_MASK_WORDS>;

// One CU-masked stream with everything a measurement needs on it.
struct StreamCtx {
  hipStream_t stream = nullptr;
  std::vector<hipEvent_t> events;
  float* ws = nullptr;
  int64_t ws_floats = 0;
  unsigned* err = nullptr;  // 2 words per candidate of a batch
  int err_slots = 0;
  int* probe = nullptr;
  int probe_len = 0;
};

static std::vector<StreamCtx*> g_all;  // every context, for ct_shutdown

struct ThreadState {
  int generation = -1;
  std::map<MaskKey, StreamCtx*> ctx;
};
static thread_local ThreadState t_state;

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

// The calling thread's stream context for a mask (created on first use).
static int get_ctx(const MaskKey& key, StreamCtx** out) {
  int rc = check_init();
  if (rc) return rc;
  HIP_TRY(hipSetDevice(g_device));
  const int gen = g_generation.load();
  if (t_state.generation != gen) {
    t_state.ctx.clear();
    t_state.generation = gen;
  }
  auto it = t_state.ctx.find(key);
  if (it != t_state.ctx.end()) {
    *out = it->second;
    return CT_OK;
  }
  StreamCtx* c = new StreamCtx();
  hipError_t e = hipExtStreamCreateWithCUMask(&c->stream, (uint32_t)mask_words_needed(), key.data());
  if (e != hipSuccess) {
    delete c;
    return hip_fail("hipExtStreamCreateWithCUMask", e);
  }
  {
    std::lock_guard<std::mutex> g(g_mu);
    g_all.push_back(c);
  }
  t_state.ctx[key] = c;
  *out = c;
  return CT_OK;
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

static void release_ctx(StreamCtx* c) {
  if (c->stream) hipStreamSynchronize(c->stream);
  for (hipEvent_t e : c->events) hipEventDestroy(e);
  if (c->ws) hipFree(c->ws);
  if (c->err) hipFree(c->err);
  if (c->probe) hipFree(c->probe);
  if (c->stream) hipStreamDestroy(c->stream);
  delete c;
}

static double now_s() {
  return std::chrono::duration<double>(std::chrono::steady_clock::now().time_since_epoch()).count();
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

// The profile step: time n candidates on one stream with protocol o.
static int measure_impl(const OpX& x, const ct_schedule* s, int n, StreamCtx* c, const ct_measure_opts& o,
                        const ct_verify* v, const void* xin, const void* w, void* y, float* lat,
                        int32_t* status, float* rep) {
  std::vector<Geom> geo(n);
  std::vector<char> live(n, 0);
  int64_t maxws = 0;
  for (int i = 0; i < n; ++i) {
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
  const bool verify = v && v->y_ref;
  const int batch = std::min(o.batch, std::max(n, 1));
  if (verify && (rc = ensure_err(c, batch))) return rc;
  const int R = o.repeats, L = o.launches;
  if ((rc = ensure_events(c, (size_t)2 * R * batch))) return rc;
  hipStream_t st = c->stream;

  auto run = [&](int i) -> bool {  // one run of candidate i; false on launch failure
    if (launch_once(x, s[i], geo[i], xin, w, y, c->ws, st) != 0) {
      live[i] = 0;
      status[i] = CT_S_LAUNCH;
      return false;
    }
    return true;
  };
  auto timed = [&](int i, int slot, int r) {
    hipEventRecord(c->events[(size_t)2 * (slot * R + r)], st);
    for (int l = 0; l < L && live[i]; ++l) run(i);
    hipEventRecord(c->events[(size_t)2 * (slot * R + r) + 1], st);
  };

  std::vector<float> reps(R);
  for (int b0 = 0; b0 < n; b0 += batch) {
    const int b1 = std::min(n, b0 + batch);
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
    HIP_TRY(hipStreamSynchronize(st));
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
      if (lat[i] > o.timeout_ms * 1000.0f) status[i] = CT_S_TIMEOUT;
    }
    if (verify) {
      // Re-run every live candidate once more, each followed by its check, so
      // the compared output is the candidate's own whatever the timing order.
      for (int i = b0; i < b1; ++i) {
        if (!live[i]) continue;
        if (!run(i)) continue;
        if (launch_max_error((const float*)y, v->y_ref, x.ny, c->err + 2 * (i - b0), st) != 0)
          return hip_fail("verification launch", hipGetLastError());
      }
      std::vector<unsigned> h(2 * (size_t)(b1 - b0));
      HIP_TRY(hipMemcpyAsync(h.data(), c->err, sizeof(unsigned) * h.size(), hipMemcpyDeviceToHost, st));
      HIP_TRY(hipStreamSynchronize(st));
      for (int i = b0; i < b1; ++i) {
        if (!live[i] || status[i] != CT_S_OK) continue;
        float e, m;
        std::memcpy(&e, &h[2 * (i - b0)], 4);
        std::memcpy(&m, &h[2 * (i - b0) + 1], 4);
        if (!(e <= v->tol * m)) status[i] = CT_S_WRONG_ANSWER;
      }
    }
  }
  for (int i = 0; i < n; ++i)
    if (status[i] != CT_S_OK && status[i] != CT_S_TIMEOUT && status[i] != CT_S_WRONG_ANSWER) lat[i] = INFINITY;
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

// ------------------------------------------------------------------ clients
static void pin_to_core(int core) {
  if (core < 0 || core >= CPU_SETSIZE) return;
  cpu_set_t set;
  CPU_ZERO(&set);
  CPU_SET(core, &set);
  pthread_setaffinity_np(pthread_self(), sizeof(set), &set);  // best effort
}

static int tune_job(ct_tune_job* j, StreamCtx* c, const ct_measure_opts& o1, const ct_measure_opts& o2,
                    float eps) {
  OpX x;
  int rc = derive_checked(&j->op, &x);
  if (rc) return rc;
  if (!j->cands || j->n_cands < 0 || !j->lat1_us || !j->status1 || j->top_t < 1 || !j->top_pos ||
      !j->lat2_us) {
    set_error("tune job: bad arrays");
    return CT_E_ARG;
  }
  j->t_start_s = now_s();
  j->n_top = 0;
  j->winner_pos = -1;
  j->winner_lat_us = INFINITY;
  rc = measure_impl(x, j->cands, j->n_cands, c, o1, &j->verify, j->x, j->w, j->y, j->lat1_us, j->status1,
                    nullptr);
  if (rc) return rc;
  int32_t n_top = 0;
  rc = ct_top_t(j->lat1_us, j->status1, j->n_cands, j->top_t, j->top_pos, &n_top);
  if (rc) return rc;
  j->n_top = n_top;
  if (n_top > 0) {
    std::vector<ct_schedule> s2(n_top);
    for (int i = 0; i < n_top; ++i) s2[i] = j->cands[j->top_pos[i]];
    std::vector<int32_t> st2(n_top);
    ct_measure_opts o = o2;
    o.interleave = 1;
    rc = measure_impl(x, s2.data(), n_top, c, o, nullptr, j->x, j->w, j->y, j->lat2_us, st2.data(), nullptr);
    if (rc) return rc;
    for (int i = 0; i < n_top; ++i)
      if (st2[i] != CT_S_OK) j->lat2_us[i] = INFINITY;
    int32_t wi = -1;
    rc = ct_select_winner(j->lat2_us, j->top_pos, n_top, eps, &wi);
    if (rc) return rc;
    if (wi >= 0) {
      j->winner_pos = j->top_pos[wi];
      j->winner_lat_us = j->lat2_us[wi];
    }
  }
  j->t_end_s = now_s();
  return CT_OK;
}

// The jobs a client runs: its own list in order, or (next != nullptr) the
// next unclaimed job of a queue shared by all clients.
struct JobSource {
  ct_tune_job* jobs;
  int n;
  std::atomic<int>* next;
  int32_t* owner;  // shared queue: owner[i] = index of the client that ran job i
};

static void run_client(ct_client* cl, int index, JobSource src, const ct_measure_opts* o1,
                       const ct_measure_opts* o2, float eps) {
  pin_to_core(cl->host_core);
  cl->rc = CT_OK;
  cl->n_measured = 0;
  cl->t_start_s = now_s();
  cl->t_end_s = cl->t_start_s;
  try {
    MaskKey key;
    int rc = make_key(cl->cu_mask, CT_MASK_WORDS, &key);
    StreamCtx* c = nullptr;
    if (!rc) rc = get_ctx(key, &c);
    // CT_PROGRESS set in the environment: one line on stderr per finished job
    const bool progress = getenv("CT_PROGRESS") != nullptr;
    for (int k = 0; !rc; ++k) {
      int i = k;
      if (src.next) i = src.next->fetch_add(1);
      if (i >= src.n) break;
      if (src.owner) src.owner[i] = index;
      rc = tune_job(&src.jobs[i], c, *o1, *o2, eps);
      if (!rc) cl->n_measured += src.jobs[i].n_cands;
      if (progress)
        fprintf(stderr, "[ct] client %d: job %d of %d done, rc %d, %.1f s\n", index, i + 1, src.n, rc,
                now_s() - cl->t_start_s);
    }
    cl->rc = rc;
  } catch (...) {
    set_error("tuning client: unexpected exception");
    cl->rc = CT_E_ARG;
  }
  cl->t_end_s = now_s();
}

static int run_clients(ct_client* clients, int n_clients, const std::vector<JobSource>& src,
                       const ct_measure_opts* stage1, const ct_measure_opts* stage2, float eps) {
  std::vector<std::thread> th;
  th.reserve(n_clients);
  for (int i = 0; i < n_clients; ++i) th.emplace_back(run_client, &clients[i], i, src[i], stage1, stage2, eps);
  for (auto& t : th) t.join();
  for (int i = 0; i < n_clients; ++i)
    if (clients[i].rc) {
      set_error("tuning client " + std::to_string(i) + " failed with code " + std::to_string(clients[i].rc));
      return clients[i].rc;
    }
  return CT_OK;
}

}  // namespace ct

// ================================================================= C ABI
using namespace ct;

extern "C" {

const char* ct_last_error(void) { return t_err.c_str(); }

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
  if (g_device >= 0) hipSetDevice(g_device);
  for (StreamCtx* c : g_all) release_ctx(c);
  g_all.clear();
  g_generation.fetch_add(1);
  g_device = -1;
  g_num_cus = 0;
}

int ct_cu_mask(double fraction, int slot, uint32_t* mask, int words) {
  int rc = check_init();
  if (rc) return rc;
  return ct_build_cu_mask(g_num_cus, fraction, slot, mask, words);
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
  MaskKey key;
  if ((rc = check_init()) || (rc = make_key(cu_mask, words, &key))) return rc;
  StreamCtx* c = nullptr;
  if ((rc = get_ctx(key, &c))) return rc;
  if ((rc = ensure_ws(c, g.ws_floats))) return rc;
  const int lrc = launch_once(ox, *s, g, x, w, y, c->ws, c->stream);
  if (lrc == -2) return CT_E_ARG;  // the launcher refused the arguments (reason already set)
  if (lrc != 0) return hip_fail("conv2d_run launch", hipGetLastError());
  HIP_TRY(hipStreamSynchronize(c->stream));
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
  MaskKey key;
  if ((rc = check_init()) || (rc = make_key(cu_mask, words, &key))) return rc;
  StreamCtx* c = nullptr;
  if ((rc = get_ctx(key, &c))) return rc;
  return measure_impl(ox, s, n, c, *o, v, x, w, y, lat_us, status, rep_us);
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
  for (int i = 0; i < n_clients; ++i) src[i] = {clients[i].jobs, clients[i].n_jobs, nullptr, nullptr};
  return run_clients(clients, n_clients, src, stage1, stage2, eps);
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
  if (job_client)
    for (int i = 0; i < n_jobs; ++i) job_client[i] = -1;
  std::atomic<int> next{0};
  std::vector<JobSource> src(n_clients, JobSource{jobs, n_jobs, &next, job_client});
  return run_clients(clients, n_clients, src, stage1, stage2, eps);
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
    MaskKey key;
    if ((rc = make_key(masks + (size_t)j * words, words, &key))) return rc;
    StreamCtx* c = nullptr;
    if ((rc = get_ctx(key, &c))) return rc;
    if ((rc = measure_impl(ox, s, n_sched, c, oo, nullptr, x, w, y, lat.data(), st.data(), nullptr))) return rc;
    for (int i = 0; i < n_sched; ++i) M[(size_t)i * n_masks + j] = st[i] == CT_S_OK ? lat[i] : INFINITY;
  }
  return CT_OK;
}

int ct_probe_cus(const uint32_t* cu_mask, int words, int blocks, int32_t* out, int cap, int32_t* n_out) {
  int rc;
  MaskKey key;
  if (blocks < 1 || blocks > (1 << 20) || !n_out) {
    set_error("ct_probe_cus: bad argument");
    return CT_E_ARG;
  }
  if ((rc = check_init()) || (rc = make_key(cu_mask, words, &key))) return rc;
  StreamCtx* c = nullptr;
  if ((rc = get_ctx(key, &c))) return rc;
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
  MaskKey key;
  if (!opts_ok(o) || !us) {
    set_error("probe: bad argument");
    return CT_E_ARG;
  }
  if ((rc = check_init()) || (rc = make_key(cu_mask, words, &key))) return rc;
  StreamCtx* c = nullptr;
  if ((rc = get_ctx(key, &c))) return rc;
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
