// Address- and undefined-behaviour-sanitizer driver of the library's
// host-only units (schedule.cpp, search.cpp): for every op listed in the
// input file, every valid schedule through the validator, the launch shape,
// the kernel name and the grid encoding; both samplers; top-t and winner
// selection on stand-in latencies; CU masks; and a whole guided search over a
// stand-in measurement. Built with -fsanitize=address,undefined by
// tests/test_host_asan.py; any report ends the run with a non-zero status.
//
// Input: one op per line, "n c h w k r s stride_h stride_w pad_h pad_w dil_h
// dil_w groups dtype layout". Output: one summary line per op, then "done".
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "convtune.h"

namespace {

// a deterministic stand-in latency (us) from a schedule's knobs
float fake_latency(const ct_schedule& s) {
  uint64_t h = 1469598103934665603ull ^ (uint64_t)s.family;
  for (int i = 0; i < CT_MAX_KNOBS; ++i) h = (h ^ (uint64_t)(uint32_t)s.knob[i]) * 1099511628211ull;
  return 5.0f + (float)(h % 10000) / 100.0f;
}

int fail(const char* what, const ct_op& op) {
  std::printf("FAIL %s on op %dx%dx%dx%d k%d r%ds%d: %s\n", what, op.n, op.c, op.h, op.w, op.k, op.r, op.s,
              ct_last_error());
  return 1;
}

}  // namespace

// The device measurement that ct_search calls, replaced by the stand-in
// latencies: every candidate the validator accepts is "measured" OK.
extern "C" int measure_candidates_mask(const ct_op* op, const ct_schedule* s, int n, const uint32_t*, int,
                                       const ct_measure_opts*, const ct_verify*, const void*, const void*, void*,
                                       float* lat_us, int32_t* status, float* rep_us) {
  for (int i = 0; i < n; ++i) {
    const bool ok = ct_validate(op, &s[i]) == 0;
    lat_us[i] = ok ? fake_latency(s[i]) : INFINITY;
    status[i] = ok ? CT_S_OK : CT_S_INVALID;
    if (rep_us) rep_us[i] = lat_us[i];
  }
  return 0;
}

int main(int argc, char** argv) {
  if (argc < 2) return 2;
  FILE* f = std::fopen(argv[1], "r");
  if (!f) return 2;
  int bad = 0, n_ops = 0;
  ct_op op{};
  while (std::fscanf(f, "%d %d %d %d %d %d %d %d %d %d %d %d %d %d %d %d", &op.n, &op.c, &op.h, &op.w, &op.k, &op.r,
                     &op.s, &op.stride_h, &op.stride_w, &op.pad_h, &op.pad_w, &op.dil_h, &op.dil_w, &op.groups,
                     &op.dtype, &op.layout) == 16) {
    ++n_ops;
    int64_t count = 0;
    if (ct_valid_space(&op, nullptr, 0, &count)) { bad += fail("ct_valid_space(count)", op); continue; }
    std::vector<ct_schedule> all((size_t)count);
    int64_t got = 0;
    if (count && ct_valid_space(&op, all.data(), count, &got)) { bad += fail("ct_valid_space", op); continue; }
    int64_t per_family = 0;
    for (int fam = 1; fam <= 4; ++fam) {
      int64_t nf = 0;
      if (ct_grid_size(&op, fam, &nf)) { bad += fail("ct_grid_size", op); break; }
      per_family += nf;
    }
    if (per_family != count) { std::printf("FAIL family sizes %lld != %lld\n", (long long)per_family, (long long)count); ++bad; }
    char name[256];
    for (const ct_schedule& s : all) {
      int32_t lds = 0, threads = 0, kernels = 0;
      int64_t blocks = 0, index = -1;
      ct_schedule back{};
      if (ct_validate(&op, &s) != 0) { bad += fail("a listed schedule is invalid", op); break; }
      if (ct_launch_shape(&op, &s, &lds, &threads, &blocks, &kernels)) { bad += fail("ct_launch_shape", op); break; }
      if (threads < 1 || blocks < 1 || kernels < 1 || kernels > 2 || lds < 0) { bad += fail("launch shape range", op); break; }
      if (ct_kernel_name(&op, &s, name, (int)sizeof name)) { bad += fail("ct_kernel_name", op); break; }
      if (ct_grid_encode(&s, &index) || ct_grid_decode(s.family, index, &back) ||
          std::memcmp(&back, &s, sizeof s) != 0) { bad += fail("grid encode/decode round trip", op); break; }
    }
    // both samplers, then top-t and the winner on stand-in latencies
    std::vector<ct_schedule> cand(256);
    int32_t n_cand = 0;
    if (ct_sample(&op, 7, 2, n_ops, 256, cand.data(), &n_cand)) { bad += fail("ct_sample", op); continue; }
    int32_t n_uni = 0;
    std::vector<ct_schedule> uni(256);
    if (ct_sample_uniform(&op, 7, 2, n_ops, 256, uni.data(), &n_uni)) { bad += fail("ct_sample_uniform", op); continue; }
    if (n_cand) {
      std::vector<float> lat(n_cand);
      std::vector<int32_t> st(n_cand), top(8), pos(8);
      for (int i = 0; i < n_cand; ++i) {
        lat[i] = fake_latency(cand[i]);
        st[i] = i % 17 == 3 ? CT_S_INVALID : CT_S_OK;
      }
      int32_t n_top = 0, winner = -1;
      if (ct_top_t(lat.data(), st.data(), n_cand, 8, top.data(), &n_top)) { bad += fail("ct_top_t", op); continue; }
      std::vector<float> lat2(n_top);
      for (int i = 0; i < n_top; ++i) {
        lat2[i] = lat[top[i]];
        pos[i] = top[i];
      }
      if (n_top && ct_select_winner(lat2.data(), pos.data(), n_top, 0.01f, &winner)) {
        bad += fail("ct_select_winner", op);
        continue;
      }
    }
    // a whole guided search against the stand-in measurement
    if (count) {
      ct_search_opts so{};
      so.seed = 11;
      so.batch = 16;
      so.budget = 96;
      so.patience = 48;
      so.sa_chains = 4;
      so.sa_steps = 24;
      so.explore = 0.25f;
      so.eps = 0.01f;
      so.sa_temp = 1.0f;
      ct_measure_opts o{1, 1, 1, 8, 1000.0f, 0};
      uint32_t mask[8];
      if (ct_build_cu_mask(256, 0.25, 1, mask, 8)) { bad += fail("ct_build_cu_mask", op); continue; }
      std::vector<ct_schedule> measured(so.budget);
      std::vector<float> lat(so.budget);
      std::vector<int32_t> st(so.budget);
      ct_search_result res{};
      if (ct_search(&op, &so, mask, 8, &o, &o, 4, 0.01f, nullptr, nullptr, nullptr, measured.data(), lat.data(),
                    st.data(), &res)) {
        bad += fail("ct_search", op);
        continue;
      }
      if (res.n_measured < 1 || res.winner < 0) { bad += fail("ct_search found nothing", op); continue; }
    }
    std::printf("op %d: %lld valid, %d + %d sampled\n", n_ops, (long long)count, n_cand, n_uni);
  }
  std::fclose(f);
  for (double fr : {0.125, 0.25, 0.5, 1.0})
    for (int slot = 0; slot < 8; ++slot) {
      uint32_t mask[8];
      const int rc = ct_build_cu_mask(256, fr, slot, mask, 8);
      (void)rc;  // slots past the share count are refused; only the sanitizers judge this loop
    }
  std::printf("%s: %d ops, %d failures\n", bad ? "failed" : "done", n_ops, bad);
  return bad ? 1 : 0;
}
