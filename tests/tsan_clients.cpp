// Thread-sanitizer driver of the library's host-only client machinery
// (clients.cpp with schedule.cpp): four client threads on one shared job
// queue, with per-client logs, a delayed stand-in measurement, a client that
// raises, and clients stopped after a number of records. Built with
// -fsanitize=thread by tests/test_host_tsan.py; a data race makes it exit 66.
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "convtune.h"

namespace {

struct Jobs {
  std::vector<ct_schedule> cands;
  std::vector<std::vector<float>> lat1, lat2;
  std::vector<std::vector<int32_t>> st1, top;
  std::vector<ct_tune_job> jobs;
};

void make(Jobs* J, int n_jobs, int n_cands) {
  J->cands.resize(n_cands);
  for (int i = 0; i < n_cands; ++i) ct_grid_decode(CT_FAM_DIRECT_F32, 1000 + 37 * i, &J->cands[i]);
  J->lat1.assign(n_jobs, std::vector<float>(n_cands));
  J->st1.assign(n_jobs, std::vector<int32_t>(n_cands));
  J->top.assign(n_jobs, std::vector<int32_t>(4));
  J->lat2.assign(n_jobs, std::vector<float>(4));
  J->jobs.assign(n_jobs, ct_tune_job{});
  for (int j = 0; j < n_jobs; ++j) {
    ct_tune_job& b = J->jobs[j];
    b.cands = J->cands.data();
    b.n_cands = n_cands;
    b.lat1_us = J->lat1[j].data();
    b.status1 = J->st1[j].data();
    b.top_t = 4;
    b.top_pos = J->top[j].data();
    b.lat2_us = J->lat2[j].data();
    b.layer_id = j;
  }
}

int run(const char* what, int n_clients, const ct_test_hooks& h, const std::string& dir, int expect_rc) {
  Jobs J;
  make(&J, 24, 20);
  std::vector<ct_client> cl(n_clients);
  std::vector<std::string> paths(n_clients);
  for (int c = 0; c < n_clients; ++c) {
    std::memset(&cl[c], 0, sizeof(ct_client));
    cl[c].host_core = -1;
    paths[c] = dir + "/" + what + "_" + std::to_string(c) + ".jsonl";
    cl[c].log_path = paths[c].c_str();
  }
  std::vector<int32_t> owner(J.jobs.size());
  const int rc = ct_test_run_clients(cl.data(), n_clients, J.jobs.data(), (int)J.jobs.size(), &h, owner.data());
  double agg = 0;
  ct_throughput(cl.data(), n_clients, &agg);
  std::printf("%s: rc %d (expected %d), %.0f candidates/s\n", what, rc, expect_rc, agg);
  return rc == expect_rc ? 0 : 1;
}

}  // namespace

int main(int argc, char** argv) {
  const std::string dir = argc > 1 ? argv[1] : ".";
  int bad = 0;
  bad += run("plain", 4, ct_test_hooks{50, -1, 0, -1}, dir, CT_OK);
  bad += run("raise", 4, ct_test_hooks{50, 2, 1, -1}, dir, CT_E_CLIENT);
  bad += run("stop", 4, ct_test_hooks{50, -1, 0, 100}, dir, CT_E_STOPPED);
  int32_t ex = 0, dr = 0;
  const int32_t runs[3] = {1, 10, 10};
  const double done[3] = {0.0, 0.005, 0.5};
  ct_test_watchdog(3, runs, done, 0.001, 0.0, 1.0, &ex, &dr);
  bad += (ex == 2 && dr == 1) ? 0 : 1;
  std::printf("watchdog: expired %d drained %d\n", ex, dr);
  return bad ? 1 : 0;
}
