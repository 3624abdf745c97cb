// Internal declarations of libconvtune: knob tables, derived op facts and the
// launch geometry of each kernel family. The validator and the launchers both
// derive a schedule's geometry from the functions declared here, so a
// schedule that validates is launched exactly as it was checked.
#pragma once

#include <atomic>
#include <cstdint>
#include <functional>
#include <string>
#include <vector>

#include "convtune.h"

namespace ct {

constexpr int kMaxLdsBytes = 160 * 1024;  // per-block LDS budget (the gfx950 workgroup maximum)
constexpr int kMaxThreads = 1024;
constexpr int kMinThreads = 32;
constexpr int kMaxLoadsPerThread = 8;     // register staging bound of the GEMM loaders
// fp32 MFMA family, stages 3 (four loader waves): the largest accumulator
// tile in registers that still leaves room, two waves per SIMD, for the copy
// plan the loaders keep across the chunk loop (no spills up to here)
constexpr int kLoaderMaxAcc = 32;

// ---- derived facts of one op ----
struct OpX {
  ct_op op;
  int64_t oh, ow;
  int64_t cg, kg;
  int64_t kred;        // Cg * R * S
  int64_t npix;        // N * OH * OW
  int64_t nx, nw, ny;  // element counts
  int elem_bytes;      // of x and w
};

// Fills x from op; returns false (with a reason) if the op itself is malformed.
bool derive_op(const ct_op& op, OpX* x, std::string* why);

// ---- knob tables ----
struct KnobDef {
  const char* name;
  int nvals;
  int32_t vals[12];
};
struct FamilyDef {
  int family;
  const char* name;
  int nknobs;
  KnobDef knobs[CT_MAX_KNOBS];
};
const FamilyDef* family_def(int family);  // nullptr for an unknown family
int64_t family_grid_size(const FamilyDef& f);

// Which families apply to an op (layout, dtype and grouping contract).
bool family_applies(int family, const OpX& x);

// ---- per-family geometry ----
// Knob positions of each family, in table order.
namespace direct_knob { enum { TOH, TOW, TK, MK, MW, LDS, CT, SPLIT, UNR, COUNT }; }
namespace dw_knob { enum { TC, TOH, TOW, VEC, RPT, LDS, NB, ORDER, Q4, COUNT }; }
namespace bf16_knob { enum { MF, TM, TN, WM, WN, KC, LDS, SPLIT, SWZ, COUNT }; }
namespace f32g_knob { enum { MF, TM, TN, WM, WN, WS, TPW, CPC, STAGES, SPLIT, COUNT }; }

// Filter/stride specialisation chosen from the op (not a knob).
enum Spec { SPEC_GENERIC = 0, SPEC_1X1_S1 = 1, SPEC_1X1_S2 = 2, SPEC_3X3_S1 = 3, SPEC_3X3_S2 = 4 };
Spec op_spec(const OpX& x);

struct Geom {
  int family;
  Spec spec;
  int threads;        // per block
  int lds_bytes;      // dynamic LDS per block
  int64_t blocks;     // main kernel
  int split;          // >1: partial sums to workspace + reduction kernel
  int kernels;        // launches per run (1 or 2)
  int64_t ws_floats;  // workspace floats needed (split * ny)
  // family-specific derived values
  int64_t tiles_h, tiles_w, tiles_k, tiles_c, tiles_n;  // grid factors
  int ih_t, iw_t;     // input halo tile (direct, depthwise)
  int bm, bn;         // GEMM block tile (rows x cols)
  int chunks;         // reduction chunks in total
  int chunks_per_split;
  int a_loads, b_loads;  // per-thread staged loads per chunk (GEMM families)
  int kc, kcp;           // reduction rows per chunk, and padded to whole k-steps
  int cpcp, lda, tph, tpw;  // fp32 MFMA family: padded channels per chunk, filter row pitch, pixel rectangle
  int xs_pad, f_nseg;       // fp32 MFMA family: halo words per stage, 64-word segments per filter row
  int hpp, hrw, hshift;     // fp32 MFMA family: LDS words per halo channel / row, column shift
  int vec_h, vec_f;         // fp32 MFMA family: 16-byte copies of the halo / filter
};

// Validates s on x and fills g. Returns CT_OK or CT_S_INVALID (reason in why).
int compute_geom(const OpX& x, const ct_schedule& s, Geom* g, std::string* why);

// ---- kernel launchers (one per family, in the .hip files) ----
// Return 0, -1 on a HIP launch error, or -2 when the arguments are refused
// (reason given to set_error).
// ws: workspace of at least g.ws_floats floats when g.split > 1.
int launch_direct_f32(const OpX& x, const ct_schedule& s, const Geom& g, const void* xin,
                      const void* w, void* y, float* ws, void* stream);
int launch_depthwise_f32(const OpX& x, const ct_schedule& s, const Geom& g, const void* xin,
                         const void* w, void* y, float* ws, void* stream);
int launch_igemm_bf16(const OpX& x, const ct_schedule& s, const Geom& g, const void* xin,
                      const void* w, void* y, float* ws, void* stream);
int launch_igemm_f32(const OpX& x, const ct_schedule& s, const Geom& g, const void* xin,
                     const void* w, void* y, float* ws, void* stream);
// Sums split partial outputs in split order: y[i] = sum_j ws[j * n + i].
int launch_split_reduce(const float* ws, float* y, int64_t n, int split, void* stream);

// ---- host rules shared by the C ABI ----
void set_error(const std::string& msg);
const std::string& last_error();
uint64_t splitmix64_next(uint64_t* state);
double now_s();  // steady clock, seconds

// ---- tuning clients (clients.cpp, host only) ----
// Receives a job's per-candidate results as they become final, and the job's
// end. Returns false when the client has to stop (a test hook).
class RecordSink {
 public:
  virtual ~RecordSink() = default;
  virtual bool candidates(const ct_tune_job& j, int i0, int i1) = 0;
  virtual void job_done(const ct_tune_job& j) = 0;
};

// Runs one job for client `ci`; returns CT_OK or a CT_E_* code.
using JobFn = std::function<int(int ci, ct_tune_job* j, RecordSink* sink)>;
// Called once per client thread after its last job (releases per-client state).
using ClientEndFn = std::function<void(int ci)>;

// The jobs a client runs: its own list in order, or (next != nullptr) the
// next unclaimed job of a queue shared by all clients.
struct JobSource {
  ct_tune_job* jobs;
  int n;
  std::atomic<int>* next;
  int32_t* owner;  // shared queue: owner[i] = index of the client that ran job i
};

// One host thread per client; returns CT_OK or the first failing client's code.
int run_clients(ct_client* clients, int n_clients, const std::vector<JobSource>& src, const JobFn& fn,
                const ClientEndFn& on_end, int64_t stop_after_records);

// Stage 2 and selection of a job whose stage-1 results are in place:
// remeasure(positions, n, lat2) fills lat2 (+inf where not OK).
int select_job(ct_tune_job* j, float eps,
               const std::function<int(const int32_t* pos, int n, float* lat2)>& remeasure);

// ---- timeout watchdog ----
// Waits for n events of one in-order stream without polling them while the
// stream keeps pace: runs[k] kernel runs were enqueued between event k-1 (or
// the start) and event k, each may take at most run_limit_s, so event k is due
// run_limit_s * runs[k] + slack_s after event k-1 was found complete.
// wait_until(t) blocks until every event has completed (returns true) or the
// clock reaches t (returns false); only when a deadline passes is the progress
// read, with done(k) (1 complete, 0 not, negative on failure). On the first
// event found past its deadline the watchdog records it and waits up to
// drain_cap_s more for the whole stream.
struct WatchResult {
  int rc = 0;            // 0, or a negative code from done()
  int expired = -1;      // first event past its deadline, -1 if none
  bool drained = true;   // every event completed
};
template <class DoneFn, class WaitFn, class ClockFn>
WatchResult watch_events(int n, const int32_t* runs, double run_limit_s, double slack_s,
                         double drain_cap_s, DoneFn done, WaitFn wait_until, ClockFn now) {
  WatchResult r;
  if (n <= 0) return r;
  double t_prev = now();
  int k = 0;
  for (;;) {
    if (k >= n) {  // every event has completed: only the completion signal is left
      if (!wait_until(now() + drain_cap_s)) r.drained = false;
      return r;
    }
    if (wait_until(t_prev + run_limit_s * (double)runs[k] + slack_s)) return r;
    const int k0 = k;
    while (k < n) {
      const int d = done(k);
      if (d < 0) { r.rc = d; return r; }
      if (!d) break;
      ++k;
    }
    if (k == k0) {  // no progress since the deadline of event k was set
      r.expired = k;
      break;
    }
    t_prev = now();
  }
  if (!wait_until(now() + drain_cap_s)) r.drained = false;
  return r;
}

}  // namespace ct
