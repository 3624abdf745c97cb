// Host side of the tuning clients (section 3.1.1: several tuning clients share
// the GPU, each with its own log; a model's operators are sharded over the
// clients and their logs merged): client threads, the shared job queue, the
// per-client JSON-lines logs, stage-2 selection of a job, throughput, and the
// host-logic test hooks. Nothing here touches the device: the device work of a
// job is the JobFn that runtime.hip passes in, so this unit also builds and
// runs under a host thread sanitizer on its own.
#include <pthread.h>
#include <sched.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <stdexcept>
#include <string>
#include <thread>
#include <vector>

#include "ct_internal.h"

namespace ct {

// ------------------------------------------------------------------ errors
static thread_local std::string t_err;
void set_error(const std::string& msg) { t_err = msg; }
const std::string& last_error() { return t_err; }

double now_s() {
  return std::chrono::duration<double>(std::chrono::steady_clock::now().time_since_epoch()).count();
}

// ------------------------------------------------------------------ logs
static void put_float(std::string* s, float v) {
  if (!std::isfinite(v)) {
    *s += "null";
    return;
  }
  char b[32];
  std::snprintf(b, sizeof b, "%.9g", (double)v);
  *s += b;
}

// One client's append-only log. Records of a group are written with one
// fwrite and flushed, so a killed process leaves whole lines only (the last
// line may be cut, and readers skip a line that does not parse).
class ClientLog : public RecordSink {
 public:
  ClientLog(const char* path, std::atomic<int64_t>* total, int64_t stop_after)
      : total_(total), stop_after_(stop_after) {
    if (path && *path) f_ = std::fopen(path, "a");
  }
  ~ClientLog() override {
    if (f_) std::fclose(f_);
  }
  bool open_failed(const char* path) const { return path && *path && !f_; }

  bool candidates(const ct_tune_job& j, int i0, int i1) override {
    std::string s;
    int64_t wrote = 0;
    for (int i = i0; i < i1; ++i) {
      if (j.skip && j.skip[i]) continue;
      const ct_schedule& c = j.cands[i];
      const FamilyDef* f = family_def(c.family);
      s += "{\"kind\":\"cand\",\"layer\":" + std::to_string(j.layer_id) + ",\"pos\":" + std::to_string(i) +
           ",\"family\":" + std::to_string(c.family) + ",\"knobs\":[";
      for (int k = 0; f && k < f->nknobs; ++k) s += (k ? "," : "") + std::to_string(c.knob[k]);
      s += "],\"lat_us\":";
      put_float(&s, j.lat1_us[i]);
      s += ",\"status\":" + std::to_string(j.status1[i]) + "}\n";
      ++wrote;
    }
    if (f_ && !s.empty()) {
      std::fwrite(s.data(), 1, s.size(), f_);
      std::fflush(f_);
    }
    const int64_t t = total_->fetch_add(wrote) + wrote;
    return stop_after_ < 0 || t < stop_after_;
  }

  void job_done(const ct_tune_job& j) override {
    if (!f_) return;
    std::string s = "{\"kind\":\"job\",\"layer\":" + std::to_string(j.layer_id) +
                    ",\"n_cands\":" + std::to_string(j.n_cands) + ",\"winner_pos\":" + std::to_string(j.winner_pos) +
                    ",\"winner_lat_us\":";
    put_float(&s, j.winner_lat_us);
    s += ",\"top_pos\":[";
    for (int i = 0; i < j.n_top; ++i) s += (i ? "," : "") + std::to_string(j.top_pos[i]);
    s += "],\"lat2_us\":[";
    for (int i = 0; i < j.n_top; ++i) {
      if (i) s += ",";
      put_float(&s, j.lat2_us[i]);
    }
    s += "],\"rc\":" + std::to_string(j.rc) + "}\n";
    std::fwrite(s.data(), 1, s.size(), f_);
    std::fflush(f_);
  }

 private:
  FILE* f_ = nullptr;
  std::atomic<int64_t>* total_;
  int64_t stop_after_;
};

// ------------------------------------------------------------------ selection
int select_job(ct_tune_job* j, float eps, const std::function<int(const int32_t*, int, float*)>& remeasure) {
  int32_t n_top = 0;
  int rc = ct_top_t(j->lat1_us, j->status1, j->n_cands, j->top_t, j->top_pos, &n_top);
  if (rc) return rc;
  j->n_top = n_top;
  j->winner_pos = -1;
  j->winner_lat_us = INFINITY;
  if (n_top == 0) return CT_OK;
  if ((rc = remeasure(j->top_pos, n_top, j->lat2_us))) return rc;
  int32_t wi = -1;
  if ((rc = ct_select_winner(j->lat2_us, j->top_pos, n_top, eps, &wi))) return rc;
  if (wi >= 0) {
    j->winner_pos = j->top_pos[wi];
    j->winner_lat_us = j->lat2_us[wi];
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

static void run_client(ct_client* cl, int index, JobSource src, const JobFn& fn, const ClientEndFn& on_end,
                       std::atomic<int64_t>* records, int64_t stop_after, std::string* err) {
  pin_to_core(cl->host_core);
  cl->rc = CT_OK;
  cl->n_measured = 0;
  cl->cands_per_s = 0.0;
  cl->t_start_s = now_s();
  cl->t_end_s = cl->t_start_s;
  const bool progress = std::getenv("CT_PROGRESS") != nullptr;
  int rc = CT_OK;
  ct_tune_job* cur = nullptr;  // the job running, for the exception handlers
  try {
    ClientLog log(cl->log_path, records, stop_after);
    if (log.open_failed(cl->log_path)) {
      set_error(std::string("cannot open the client log ") + cl->log_path);
      rc = CT_E_ARG;
    }
    for (int k = 0; !rc; ++k) {
      const int i = src.next ? src.next->fetch_add(1) : k;
      if (i >= src.n) break;
      if (src.owner) src.owner[i] = index;
      ct_tune_job* j = &src.jobs[i];
      cur = j;
      j->rc = CT_OK;
      rc = fn(index, j, &log);
      j->rc = rc;
      cur = nullptr;
      if (!rc) {
        for (int c = 0; c < j->n_cands; ++c) cl->n_measured += (j->skip && j->skip[c]) ? 0 : 1;
        log.job_done(*j);
      }
      if (progress)
        std::fprintf(stderr, "[ct] client %d: job %d of %d done, rc %d, %.1f s\n", index, i + 1, src.n, rc,
                     now_s() - cl->t_start_s);
    }
  } catch (const std::exception& e) {
    set_error(std::string("tuning client: ") + e.what());
    rc = CT_E_CLIENT;
  } catch (...) {
    set_error("tuning client: unknown exception");
    rc = CT_E_CLIENT;
  }
  if (cur) cur->rc = rc;
  cl->rc = rc;
  if (rc) *err = last_error();
  if (on_end) on_end(index);
  cl->t_end_s = now_s();
  const double span = cl->t_end_s - cl->t_start_s;
  cl->cands_per_s = span > 0 ? (double)cl->n_measured / span : 0.0;
}

int run_clients(ct_client* clients, int n_clients, const std::vector<JobSource>& src, const JobFn& fn,
                const ClientEndFn& on_end, int64_t stop_after_records) {
  std::vector<std::thread> th;
  std::vector<std::string> errs(n_clients);
  std::atomic<int64_t> records{0};
  th.reserve(n_clients);
  for (int i = 0; i < n_clients; ++i)
    th.emplace_back(run_client, &clients[i], i, src[i], std::cref(fn), std::cref(on_end), &records,
                    stop_after_records, &errs[i]);
  for (auto& t : th) t.join();
  for (int i = 0; i < n_clients; ++i)
    if (clients[i].rc) {
      set_error("tuning client " + std::to_string(i) + " failed with code " + std::to_string(clients[i].rc) +
                ": " + errs[i]);
      return clients[i].rc;
    }
  return CT_OK;
}

// Checks a client array and its jobs; the jobs' result arrays must exist.
static int check_jobs(const ct_tune_job* jobs, int n_jobs) {
  for (int i = 0; i < n_jobs; ++i) {
    const ct_tune_job& j = jobs[i];
    if (!j.cands || j.n_cands < 0 || !j.lat1_us || !j.status1 || j.top_t < 1 || !j.top_pos || !j.lat2_us) {
      set_error("tune job " + std::to_string(i) + ": bad arrays");
      return CT_E_ARG;
    }
  }
  return CT_OK;
}

}  // namespace ct

// ================================================================= C ABI
using namespace ct;

extern "C" {

const char* ct_last_error(void) { return t_err.c_str(); }

int ct_throughput(const ct_client* clients, int n_clients, double* cands_per_s) {
  if (!clients || n_clients < 1 || !cands_per_s) {
    set_error("ct_throughput: bad argument");
    return CT_E_ARG;
  }
  double t0 = INFINITY, t1 = -INFINITY;
  int64_t n = 0;
  for (int i = 0; i < n_clients; ++i) {
    t0 = std::min(t0, clients[i].t_start_s);
    t1 = std::max(t1, clients[i].t_end_s);
    n += clients[i].n_measured;
  }
  *cands_per_s = t1 > t0 ? (double)n / (t1 - t0) : 0.0;
  return CT_OK;
}

int ct_test_run_clients(ct_client* clients, int n_clients, ct_tune_job* jobs, int n_jobs, const ct_test_hooks* hooks,
                        int32_t* job_client) {
  if (!clients || n_clients < 1 || n_clients > 64 || n_jobs < 0 || (n_jobs > 0 && !jobs) || !hooks ||
      hooks->delay_us < 0) {
    set_error("ct_test_run_clients: bad argument");
    return CT_E_ARG;
  }
  int rc = check_jobs(jobs, n_jobs);
  if (rc) return rc;
  if (job_client)
    for (int i = 0; i < n_jobs; ++i) job_client[i] = -1;
  const ct_test_hooks h = *hooks;
  std::vector<int> started(n_clients, 0);  // jobs started per client (each slot touched by its own thread only)
  auto fake_lat = [](const ct_tune_job& j, int i) {
    const uint64_t v = ((uint64_t)(uint32_t)j.layer_id * 7919u + (uint64_t)i) * 2654435761ull % 1000u;
    return 1.0f + (float)v / 100.0f;
  };
  JobFn fn = [&](int ci, ct_tune_job* j, RecordSink* sink) -> int {
    if (ci == h.throw_client && started[ci] == h.throw_after_jobs) throw std::runtime_error("test hook raised");
    ++started[ci];
    j->t_start_s = now_s();
    for (int i = 0; i < j->n_cands; ++i) {
      if (j->skip && j->skip[i]) continue;
      if (h.delay_us) std::this_thread::sleep_for(std::chrono::microseconds(h.delay_us));
      j->lat1_us[i] = fake_lat(*j, i);
      j->status1[i] = CT_S_OK;
      if (!sink->candidates(*j, i, i + 1)) {
        set_error("client stopped by the test hook");
        return CT_E_STOPPED;
      }
    }
    const int r = select_job(j, 0.01f, [&](const int32_t* pos, int n, float* lat2) {
      for (int i = 0; i < n; ++i) lat2[i] = fake_lat(*j, pos[i]);
      return CT_OK;
    });
    j->t_end_s = now_s();
    return r;
  };
  std::atomic<int> next{0};
  std::vector<JobSource> src(n_clients, JobSource{jobs, n_jobs, &next, job_client});
  return run_clients(clients, n_clients, src, fn, nullptr, h.stop_after_records);
}

int ct_test_watchdog(int n_events, const int32_t* runs, const double* done_at_s, double run_limit_s, double slack_s,
                     double drain_cap_s, int32_t* expired_event, int32_t* drained) {
  if (n_events < 0 || (n_events > 0 && (!runs || !done_at_s)) || !expired_event || !drained || !(run_limit_s > 0) ||
      !(slack_s >= 0) || !(drain_cap_s >= 0)) {
    set_error("ct_test_watchdog: bad argument");
    return CT_E_ARG;
  }
  // simulated clock in whole milliseconds; a wait advances it 1 ms at a time
  int64_t ms = 0;
  auto t = [&]() { return (double)ms * 1e-3; };
  auto done = [&](int k) { return done_at_s[k] >= 0.0 && t() >= done_at_s[k] ? 1 : 0; };
  auto wait_until = [&](double until) {
    for (;;) {
      if (n_events == 0 || done(n_events - 1)) return true;
      if (t() >= until) return false;
      ++ms;
    }
  };
  const WatchResult r = watch_events(n_events, runs, run_limit_s, slack_s, drain_cap_s, done, wait_until, t);
  *expired_event = r.expired;
  *drained = r.drained ? 1 : 0;
  return r.rc;
}

}  // extern "C"
