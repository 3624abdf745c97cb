// Guided search (section 2.1, stage 4 "search strategy"): an exploration
// algorithm, simulated annealing, walks the schedule space guided by a cost
// model trained on the configurations profiled so far and proposes the next
// batch to profile; early stopping ends the search once newly profiled
// configurations stop improving the best latency (section 2.1 on the TVM
// explorer, section 2.2.1 on tuning until early stop).
//
// The cost model is this library's own, not the paper's gradient-boosted
// trees: per kernel family, ridge regression of log latency on a one-hot
// code of every knob value plus launch-geometry features (grid size against
// the CUs of the share being tuned, block size, LDS bytes, padded work),
// which carry the knob interactions that matter most.
// Everything here is host code and deterministic for a given seed and given
// measurements.
#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <unordered_map>
#include <unordered_set>
#include <vector>

#include "ct_internal.h"

namespace ct {
namespace {

constexpr int kGeomFeatures = 7;
constexpr double kRidge = 0.3;

struct Space {
  OpX x;
  std::vector<ct_schedule> all;  // every valid schedule, families in order, grid order within
  std::unordered_map<uint64_t, int32_t> pos;  // key -> index in all
  std::vector<std::vector<int32_t>> fam;       // per applicable family: its indices in all
};

// Value index of every knob (the mixed-radix digits of the grid encoding).
bool digits_of(const FamilyDef& f, const ct_schedule& s, int* d) {
  for (int i = 0; i < f.nknobs; ++i) {
    d[i] = -1;
    for (int j = 0; j < f.knobs[i].nvals; ++j)
      if (f.knobs[i].vals[j] == s.knob[i]) d[i] = j;
    if (d[i] < 0) return false;
  }
  return true;
}

uint64_t key_of(const ct_schedule& s) {
  const FamilyDef* f = family_def(s.family);
  if (!f) return ~0ull;
  int d[CT_MAX_KNOBS];
  if (!digits_of(*f, s, d)) return ~0ull;
  uint64_t idx = 0;
  for (int i = 0; i < f->nknobs; ++i) idx = idx * (uint64_t)f->knobs[i].nvals + (uint64_t)d[i];
  return (uint64_t)s.family << 48 | idx;
}

int build_space(const ct_op& op, Space* sp) {
  std::string why;
  if (!derive_op(op, &sp->x, &why)) { set_error(why); return CT_E_ARG; }
  Geom g;
  for (int fam = 1; fam <= CT_NUM_FAMILIES; ++fam) {
    if (!family_applies(fam, sp->x)) continue;
    const int64_t n = family_grid_size(*family_def(fam));
    std::vector<int32_t> mine;
    ct_schedule s;
    for (int64_t i = 0; i < n; ++i) {
      ct_grid_decode(fam, i, &s);
      if (compute_geom(sp->x, s, &g, nullptr) == CT_OK) {
        sp->pos.emplace((uint64_t)fam << 48 | (uint64_t)i, (int32_t)sp->all.size());
        mine.push_back((int32_t)sp->all.size());
        sp->all.push_back(s);
      }
    }
    if (!mine.empty()) sp->fam.push_back(std::move(mine));
  }
  if (sp->all.empty()) { set_error("search: no schedule applies to this op"); return CT_E_ARG; }
  return CT_OK;
}

int feature_count(const FamilyDef& f) {
  int n = kGeomFeatures;
  for (int i = 0; i < f.nknobs; ++i) n += f.knobs[i].nvals;
  return n;
}

// Output elements the grid of a schedule computes, padding included (the
// tiles times their sizes): against the op's own output volume this is the
// work a tile shape wastes on ragged edges.
double padded_outputs(const OpX& x, const ct_schedule& s, const Geom& g) {
  const ct_op& o = x.op;
  switch (s.family) {
    case CT_FAM_DIRECT_F32:
      return (double)(g.tiles_h * s.knob[direct_knob::TOH]) * (double)(g.tiles_w * s.knob[direct_knob::TOW]) *
             (double)(g.tiles_k * s.knob[direct_knob::TK]) * (double)o.n;
    case CT_FAM_DEPTHWISE_F32:
      return (double)(g.tiles_h * s.knob[dw_knob::TOH]) * (double)(g.tiles_w * s.knob[dw_knob::TOW]) *
             (double)(g.tiles_c * s.knob[dw_knob::TC]) * (double)(g.tiles_n * s.knob[dw_knob::NB]);
    case CT_FAM_IGEMM_BF16:
      return (double)(g.tiles_h * g.bm) * (double)(g.tiles_k * g.bn);
    default:
      return (double)o.n * (double)(g.tiles_h * g.tph) * (double)(g.tiles_w * g.tpw) * (double)(g.tiles_k * g.bm);
  }
}

// Features of a valid schedule on a share of `cus` CUs (false if it does not
// validate).
bool features(const OpX& x, const ct_schedule& s, int cus, std::vector<double>* out) {
  const FamilyDef& f = *family_def(s.family);
  Geom g;
  if (compute_geom(x, s, &g, nullptr) != CT_OK) return false;
  int d[CT_MAX_KNOBS];
  if (!digits_of(f, s, d)) return false;
  out->assign(feature_count(f), 0.0);
  int o = 0;
  for (int i = 0; i < f.nknobs; ++i) {
    (*out)[o + d[i]] = 1.0;
    o += f.knobs[i].nvals;
  }
  const double lb = std::log2((double)std::max<int64_t>(g.blocks, 1));
  const double waves = std::log2((double)std::max<int64_t>(g.blocks * ((g.threads + 63) / 64), 1));
  const double bpc = (double)std::max<int64_t>(g.blocks, 1) / (double)std::max(cus, 1);  // blocks per CU
  (*out)[o + 0] = lb;
  (*out)[o + 1] = std::log2(bpc) * std::log2(bpc) / 8.0;  // distance from one block per CU of the share
  (*out)[o + 2] = std::log2((double)std::max(g.threads, 1));
  (*out)[o + 3] = g.lds_bytes / 65536.0;
  (*out)[o + 4] = waves;
  // the last round of blocks: ceil(bpc) rounds for bpc rounds of work
  (*out)[o + 5] = std::log2(std::ceil(bpc) / bpc);
  (*out)[o + 6] = std::log2(std::max(padded_outputs(x, s, g) / (double)x.ny, 1.0));  // padded work
  return true;
}

// Solves (A + ridge I) b = r by Cholesky; A is n x n, symmetric positive semidefinite.
bool ridge_solve(std::vector<double>& A, std::vector<double>& r, int n, std::vector<double>* b) {
  for (int i = 0; i < n; ++i) A[(size_t)i * n + i] += kRidge;
  for (int j = 0; j < n; ++j) {
    double s = A[(size_t)j * n + j];
    for (int k = 0; k < j; ++k) s -= A[(size_t)j * n + k] * A[(size_t)j * n + k];
    if (!(s > 0.0)) return false;
    const double l = std::sqrt(s);
    A[(size_t)j * n + j] = l;
    for (int i = j + 1; i < n; ++i) {
      double t = A[(size_t)i * n + j];
      for (int k = 0; k < j; ++k) t -= A[(size_t)i * n + k] * A[(size_t)j * n + k];
      A[(size_t)i * n + j] = t / l;
    }
  }
  b->assign(n, 0.0);
  for (int i = 0; i < n; ++i) {  // L z = r
    double t = r[i];
    for (int k = 0; k < i; ++k) t -= A[(size_t)i * n + k] * (*b)[k];
    (*b)[i] = t / A[(size_t)i * n + i];
  }
  for (int i = n - 1; i >= 0; --i) {  // L^T b = z
    double t = (*b)[i];
    for (int k = i + 1; k < n; ++k) t -= A[(size_t)k * n + i] * (*b)[k];
    (*b)[i] = t / A[(size_t)i * n + i];
  }
  return true;
}

// Cost model: per family, mean log latency plus a ridge fit on the features.
struct Model {
  double global_mean = 0.0;
  bool any = false;
  struct Fam { bool fitted = false; double mean = 0.0; std::vector<double> beta; };
  Fam fam[CT_NUM_FAMILIES + 1];

  void fit(const OpX& x, int cus, const ct_schedule* s, const float* lat, const int32_t* st, int n) {
    double sum = 0.0;
    int cnt = 0;
    for (int i = 0; i < n; ++i)
      if (st[i] == CT_S_OK && std::isfinite(lat[i]) && lat[i] > 0.0f) { sum += std::log((double)lat[i]); ++cnt; }
    any = cnt > 0;
    global_mean = any ? sum / cnt : 0.0;
    for (int f = 1; f <= CT_NUM_FAMILIES; ++f) {
      const FamilyDef* fd = family_def(f);
      const int dim = feature_count(*fd);
      std::vector<std::vector<double>> X;
      std::vector<double> y;
      std::vector<double> feat;
      for (int i = 0; i < n; ++i) {
        if (s[i].family != f || st[i] != CT_S_OK || !std::isfinite(lat[i]) || !(lat[i] > 0.0f)) continue;
        if (!features(x, s[i], cus, &feat)) continue;
        X.push_back(feat);
        y.push_back(std::log((double)lat[i]));
      }
      Fam& m = fam[f];
      m.fitted = false;
      if (y.empty()) continue;
      double my = 0.0;
      for (double v : y) my += v;
      my /= (double)y.size();
      m.mean = my;
      std::vector<double> A((size_t)dim * dim, 0.0), r(dim, 0.0);
      for (size_t i = 0; i < y.size(); ++i) {
        const double yi = y[i] - my;
        for (int a = 0; a < dim; ++a) {
          if (X[i][a] == 0.0) continue;
          r[a] += X[i][a] * yi;
          for (int b = 0; b < dim; ++b) A[(size_t)a * dim + b] += X[i][a] * X[i][b];
        }
      }
      m.fitted = ridge_solve(A, r, dim, &m.beta);
    }
  }

  // Predicted log latency of a valid schedule.
  double predict(const OpX& x, int cus, const ct_schedule& s, std::vector<double>* feat) const {
    const Fam& m = fam[s.family];
    if (!m.fitted) return any ? global_mean : 0.0;
    if (!features(x, s, cus, feat)) return INFINITY;
    double p = m.mean;
    for (size_t i = 0; i < feat->size(); ++i) p += (*feat)[i] * m.beta[i];
    return p;
  }
};

double uniform01(uint64_t* st) { return (double)(splitmix64_next(st) >> 11) * (1.0 / 9007199254740992.0); }

// One neighbour of s: one knob moved to an adjacent value (or, one time in
// four, to any other value) such that the result validates; s itself if
// eight tries find none.
ct_schedule neighbour(const OpX& x, const ct_schedule& s, uint64_t* st) {
  const FamilyDef& f = *family_def(s.family);
  int movable[CT_MAX_KNOBS], nm = 0;
  for (int i = 0; i < f.nknobs; ++i)
    if (f.knobs[i].nvals > 1) movable[nm++] = i;
  if (!nm) return s;
  int d[CT_MAX_KNOBS];
  if (!digits_of(f, s, d)) return s;
  Geom g;
  for (int t = 0; t < 8; ++t) {
    const int k = movable[splitmix64_next(st) % (uint64_t)nm];
    const int nv = f.knobs[k].nvals;
    int v;
    if (splitmix64_next(st) % 4 == 0) {
      v = (int)(splitmix64_next(st) % (uint64_t)(nv - 1));
      if (v >= d[k]) ++v;
    } else {
      v = d[k] + ((splitmix64_next(st) & 1) ? 1 : -1);
      if (v < 0) v = 1;
      if (v >= nv) v = nv - 2;
    }
    ct_schedule c = s;
    c.knob[k] = f.knobs[k].vals[v];
    if (compute_geom(x, c, &g, nullptr) == CT_OK) return c;
  }
  return s;
}

// A uniformly drawn valid schedule of the draw-th family in turn: families
// get equal shares of the random draws whatever the sizes of their spaces,
// so a small family (often the matrix-core one) is explored as much as a
// large one.
const ct_schedule& draw(const Space& sp, uint64_t draw_no, uint64_t* st) {
  const std::vector<int32_t>& f = sp.fam[draw_no % sp.fam.size()];
  return sp.all[(size_t)f[splitmix64_next(st) % f.size()]];
}

int propose(const Space& sp, const ct_schedule* meas, const float* lat, const int32_t* st, int n,
            const ct_search_opts& so, int round, ct_schedule* out, int want) {
  std::unordered_set<uint64_t> seen;
  for (int i = 0; i < n; ++i) seen.insert(key_of(meas[i]));
  uint64_t rng = so.seed ^ 0x5A17E5EA5C4ull ^ (0x9E3779B97F4A7C15ull * (uint64_t)(round + 1));
  splitmix64_next(&rng);
  std::vector<std::pair<double, uint64_t>> picked;  // (predicted, key), in selection order
  std::unordered_set<uint64_t> chosen;

  Model model;
  const int cus = so.cus > 0 ? so.cus : 256;
  model.fit(sp.x, cus, meas, lat, st, n);
  int n_model = 0;
  if (model.any) {
    n_model = want - (int)std::floor(so.explore * want + 0.5);
    n_model = std::max(0, std::min(want, n_model));
  }
  if (n_model > 0) {
    // chains start from the best measured schedules of each family in turn
    // (half of them) and from random ones (the other half)
    const size_t nf = sp.fam.size();
    std::vector<std::vector<int>> ok(nf);
    for (int i = 0; i < n; ++i) {
      if (st[i] != CT_S_OK || !std::isfinite(lat[i])) continue;
      for (size_t f = 0; f < nf; ++f)
        if (sp.all[(size_t)sp.fam[f][0]].family == meas[i].family) ok[f].push_back(i);
    }
    for (auto& v : ok)
      std::sort(v.begin(), v.end(), [&](int a, int b) { return lat[a] < lat[b] || (lat[a] == lat[b] && a < b); });
    std::unordered_map<uint64_t, double> pool;
    std::vector<double> feat;
    const int chains = std::max(1, so.sa_chains);
    const int steps = std::max(1, so.sa_steps);
    for (int c = 0; c < chains; ++c) {
      const std::vector<int>& best = ok[(size_t)c % nf];
      ct_schedule s = (c < chains / 2 && !best.empty()) ? meas[best[((size_t)c / nf) % best.size()]]
                                                         : draw(sp, (uint64_t)c, &rng);
      double e = model.predict(sp.x, cus, s, &feat);
      for (int t = 0; t < steps; ++t) {
        const double temp = so.sa_temp * (1.0 - (double)t / steps);
        const ct_schedule c2 = neighbour(sp.x, s, &rng);
        const double e2 = model.predict(sp.x, cus, c2, &feat);
        if (e2 <= e || (temp > 0.0 && uniform01(&rng) < std::exp(-(e2 - e) / temp))) {
          s = c2;
          e = e2;
        }
        const uint64_t k = key_of(s);
        if (!seen.count(k)) pool.emplace(k, e);
      }
    }
    std::vector<std::pair<double, uint64_t>> ranked;
    ranked.reserve(pool.size());
    for (const auto& kv : pool) ranked.emplace_back(kv.second, kv.first);
    std::sort(ranked.begin(), ranked.end());
    for (const auto& pk : ranked) {
      if ((int)picked.size() >= n_model) break;
      picked.push_back(pk);
      chosen.insert(pk.second);
    }
  }
  // exploration: uniform draws over the unmeasured space, families in turn
  const uint64_t size = sp.all.size();
  int guard = 0;
  const uint64_t turn0 = splitmix64_next(&rng);
  while ((int)picked.size() < want && guard < 64 * want) {
    const ct_schedule& s = draw(sp, turn0 + (uint64_t)guard, &rng);
    ++guard;
    const uint64_t k = key_of(s);
    if (seen.count(k) || chosen.count(k)) continue;
    picked.emplace_back(NAN, k);
    chosen.insert(k);
  }
  if ((int)picked.size() < want) {  // nearly exhausted: scan from a random start
    const uint64_t start = splitmix64_next(&rng) % size;
    for (uint64_t i = 0; i < size && (int)picked.size() < want; ++i) {
      const uint64_t k = key_of(sp.all[(start + i) % size]);
      if (seen.count(k) || chosen.count(k)) continue;
      picked.emplace_back(NAN, k);
      chosen.insert(k);
    }
  }
  int m = 0;
  for (const auto& pk : picked) {
    auto it = sp.pos.find(pk.second);  // every state visited validates, so it is in the space
    if (it != sp.pos.end()) out[m++] = sp.all[(size_t)it->second];
  }
  return m;
}

bool opts_ok(const ct_search_opts* so) {
  return so && so->batch > 0 && so->budget > 0 && so->patience >= 0 && so->sa_chains >= 0 && so->sa_steps >= 0 &&
         so->explore >= 0.0f && so->explore <= 1.0f && so->eps >= 0.0f && so->sa_temp >= 0.0f && so->cus >= 0;
}

}  // namespace
}  // namespace ct

using namespace ct;

extern "C" {

int ct_search_propose(const ct_op* op, const ct_schedule* measured, const float* lat_us, const int32_t* status,
                      int n_measured, const ct_search_opts* so, int32_t round, ct_schedule* out, int32_t cap,
                      int32_t* n_out) {
  if (!op || !out || !n_out || cap < 0 || n_measured < 0 || !opts_ok(so) ||
      (n_measured > 0 && (!measured || !lat_us || !status))) {
    set_error("ct_search_propose: bad argument");
    return CT_E_ARG;
  }
  for (int i = 0; i < n_measured; ++i)
    if (key_of(measured[i]) == ~0ull) { set_error("ct_search_propose: measured schedule outside the knob tables"); return CT_E_ARG; }
  Space sp;
  int rc = build_space(*op, &sp);
  if (rc) return rc;
  *n_out = propose(sp, measured, lat_us, status, n_measured, *so, round, out, std::min(cap, so->batch));
  return CT_OK;
}

int ct_search(const ct_op* op, const ct_search_opts* so, const uint32_t* cu_mask, int words,
              const ct_measure_opts* stage1, const ct_measure_opts* stage2, int32_t top_t, float eps,
              const void* x, const void* w, void* y, ct_schedule* measured, float* lat_us, int32_t* status,
              ct_search_result* res) {
  if (!op || !opts_ok(so) || !stage1 || !stage2 || top_t < 1 || !(eps >= 0.0f) || !measured || !lat_us ||
      !status || !res) {
    set_error("ct_search: bad argument");
    return CT_E_ARG;
  }
  std::memset(res, 0, sizeof(*res));
  res->winner = -1;
  res->winner_lat_us = INFINITY;
  Space sp;
  int rc = build_space(*op, &sp);
  if (rc) return rc;
  const bool progress = std::getenv("CT_PROGRESS") != nullptr;
  // the cost model scores grids against the CUs of the share being tuned
  ct_search_opts sopt = *so;
  if (sopt.cus == 0) {
    int c = 0;
    for (int i = 0; cu_mask && i < words; ++i) c += __builtin_popcount(cu_mask[i]);
    sopt.cus = c > 0 ? c : 256;
  }
  int n = 0, since = 0;
  double best = INFINITY;
  while (n < so->budget) {
    const int want = std::min(so->batch, so->budget - n);
    double t0 = now_s();
    const int got = propose(sp, measured, lat_us, status, n, sopt, res->rounds, measured + n, want);
    double t1 = now_s();
    res->propose_s += t1 - t0;
    if (got == 0) break;
    rc = measure_candidates_mask(op, measured + n, got, cu_mask, words, stage1, nullptr, x, w, y, lat_us + n,
                                 status + n, nullptr);
    res->measure_s += now_s() - t1;
    if (rc) return rc;
    for (int i = n; i < n + got; ++i) {
      if (status[i] == CT_S_OK && std::isfinite(lat_us[i]) && (double)lat_us[i] < best * (1.0 - (double)so->eps)) {
        best = lat_us[i];
        since = 0;
      } else {
        ++since;
      }
    }
    n += got;
    ++res->rounds;
    if (progress)
      std::fprintf(stderr, "[search] round %d: %d measured, best %.2f us, %d since improvement\n", res->rounds, n,
                   best, since);
    if (so->patience > 0 && since >= so->patience) {
      res->stopped_early = 1;
      break;
    }
  }
  res->n_measured = n;
  std::vector<int32_t> top(top_t);
  int32_t n_top = 0;
  ct_top_t(lat_us, status, n, top_t, top.data(), &n_top);
  if (n_top == 0) return CT_OK;
  std::vector<ct_schedule> ts(n_top);
  for (int i = 0; i < n_top; ++i) ts[i] = measured[top[i]];
  std::vector<float> lat2(n_top);
  std::vector<int32_t> st2(n_top);
  const double t2 = now_s();
  rc = measure_candidates_mask(op, ts.data(), n_top, cu_mask, words, stage2, nullptr, x, w, y, lat2.data(),
                               st2.data(), nullptr);
  res->measure_s += now_s() - t2;
  if (rc) return rc;
  for (int i = 0; i < n_top; ++i)
    if (st2[i] != CT_S_OK) lat2[i] = INFINITY;
  int32_t wi = -1;
  ct_select_winner(lat2.data(), top.data(), n_top, eps, &wi);
  if (wi >= 0) {
    res->winner = top[wi];
    res->winner_lat_us = lat2[wi];
  }
  return CT_OK;
}

}  // extern "C"
