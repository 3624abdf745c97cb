/*
 * convtune.h -- C ABI of the MI355X conv2d tuning library (libconvtune.so).
 *
 * The library implements the measurement side of the paper's autotuning loop
 * (section 2.1, Fig. 1a: select candidate configurations, build, profile on
 * the target device, search) for one DNN operator, conv2d, on gfx950:
 *
 *   - a schedule-parametrised conv2d kernel family (direct and depthwise fp32
 *     on the vector ALU, implicit GEMM on MFMA in fp32 and bf16);
 *   - "profile": run a candidate on a stream restricted to a fixed share of
 *     the compute units and time it with HIP events (section 2.2: a fixed GPU
 *     share per profiling process isolates it and gives predictable latency;
 *     here the share is a CU mask, hipExtStreamCreateWithCUMask);
 *   - several tuning clients at once on disjoint CU shares (section 3.1.1:
 *     profiling servers with distinct GPU shares, and the operators of a model
 *     sharded over tuning clients);
 *   - cross-evaluation: a schedule tuned at one share re-run at another
 *     (section 2.2.1, Tables 1 and 2).
 *
 * Conventions for every entry point:
 *   - All functions are extern "C", thread-safe, and never throw.
 *   - Return value: 0 on success, or a negative CT_E_* code; the message of
 *     the last failure on the calling thread is in ct_last_error().
 *   - Device pointers (x, w, y, references) are caller-owned HIP device
 *     memory, contiguous, in the layout and dtype that ct_op states. The
 *     library never frees caller memory; it owns its streams, events and
 *     split-reduction workspaces and releases them in ct_shutdown().
 *   - Host arrays (latencies, status, masks, schedules) are caller-owned.
 *   - Calls from different threads run concurrently on different HIP streams;
 *     two threads with the same CU mask still get separate streams.
 *
 * Operator (the reading of conv2d used throughout, since the paper names the
 * operator but does not write it out): cross-correlation with zero padding,
 * floor output size and grouped channels,
 *   OH = floor((H + 2 ph - dh (R-1) - 1) / sh) + 1,
 *   y[n,k,p,q] = sum_{c<C/g, r<R, t<S} x[n, (k div K/g) C/g + c, p sh - ph + r dh,
 *                                       q sw - pw + t dw] * w[k,c,r,t].
 */
#ifndef CONVTUNE_H
#define CONVTUNE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- error codes (return values) ---- */
#define CT_OK          0
#define CT_E_ARG      -1   /* bad argument: null pointer, bad shape, bad size   */
#define CT_E_HIP      -2   /* a HIP call failed; its message is in ct_last_error */
#define CT_E_NOINIT   -3   /* ct_init() has not succeeded                        */
#define CT_E_OOM      -4   /* workspace allocation failed                        */
#define CT_E_NODEV    -5   /* no usable gfx950 device                            */
#define CT_E_TIMEOUT  -6   /* a candidate ran past its time limit and its stream */
                           /* did not drain within the grace period: the call    */
                           /* gave up waiting (its stream is never reused)        */
#define CT_E_CLIENT   -7   /* a tuning client thread stopped on an exception     */
#define CT_E_STOPPED  -8   /* a client was stopped by a test hook (host tests)   */

/* ---- per-candidate status codes (status[] outputs) ---- */
#define CT_S_OK           0
#define CT_S_INVALID      1  /* rejected by the validator; never launched, latency +inf */
#define CT_S_LAUNCH       2  /* the launch itself failed                                */
#define CT_S_TIMEOUT      3  /* a run took longer than the protocol's time limit        */
#define CT_S_WRONG_ANSWER 4  /* output differs from the reference beyond tolerance      */

/* ---- kernel families ---- */
#define CT_FAM_DIRECT_F32     1  /* NCHW fp32, groups 1, vector-ALU direct convolution       */
#define CT_FAM_DEPTHWISE_F32  2  /* NCHW fp32, groups = C = K, vector-ALU depthwise           */
#define CT_FAM_IGEMM_BF16     3  /* NHWC bf16 in, fp32 out, 1x1 stride 1: MFMA implicit GEMM  */
#define CT_FAM_IGEMM_F32      4  /* NCHW fp32, groups 1, any filter: fp32 MFMA implicit GEMM  */
#define CT_NUM_FAMILIES       4

#define CT_DT_F32   0
#define CT_DT_BF16  1
#define CT_LAYOUT_NCHW 0  /* x N,C,H,W; w K,C/g,R,S; y N,K,OH,OW                 */
#define CT_LAYOUT_NHWC 1  /* x N,H,W,C; w K,R,S,C/g (K,C for 1x1); y N,OH,OW,K   */

#define CT_MASK_WORDS 8   /* CU masks are 8 x 32 bits: bit i of word j = CU 32 j + i */
#define CT_MAX_KNOBS  15

/* One conv2d task (the paper's tuning task: one operator at one shape). */
typedef struct ct_op {
    int32_t n, c, h, w, k, r, s;
    int32_t stride_h, stride_w, pad_h, pad_w, dil_h, dil_w, groups;
    int32_t dtype;   /* CT_DT_*; x and w in this type, y always fp32 */
    int32_t layout;  /* CT_LAYOUT_* */
} ct_op;

/* One candidate configuration (the paper's "configuration": tiles, loop
 * order, caching in LDS, unrolling, threading, matrix units -- section 2.1).
 * knob[] holds the family's knob values in the order below; unused slots are
 * 0. ct_knob_values lists each knob's values and ct_grid_decode gives
 * encodings of the grid (the validator decides which run on an op).
 *   CT_FAM_DIRECT_F32: toh, tow (output tile), tk (output channels per
 *     block), mk, mw (channels and columns per thread), lds (stage halo and
 *     filter in LDS), ct (channels per chunk), split (reduction split),
 *     unroll (channels unrolled together).
 *   CT_FAM_DEPTHWISE_F32: tc (channels per block), toh, tow, vec, rpt
 *     (columns and rows per thread), lds, nb (images per block), order
 *     (block numbering: tiles fastest or channel groups fastest), q4 (4
 *     consecutive columns per thread from 16-byte row loads).
 *   CT_FAM_IGEMM_BF16: mfma (16 or 32: the MFMA tile), tm, tn (MFMA tiles
 *     per wave), wm, wn (waves per block), kc (input channels per chunk),
 *     lds (stage operands in LDS), split, swizzle (XCD-band block order).
 *   CT_FAM_IGEMM_F32: mfma, tm, tn, wm, wn, ws (reduction groups per
 *     block), tpw (pixel tile width), cpc (channels per chunk), stages (1:
 *     one LDS stage; 2: two; 3: two, with four loader waves issuing every
 *     copy), split. */
typedef struct ct_schedule {
    int32_t family;
    int32_t knob[CT_MAX_KNOBS];
} ct_schedule;

/* Timing protocol. Each candidate: `warmup` untimed runs, then `repeats`
 * repeats of (event record; `launches` back-to-back runs; event record).
 * Latency = median over repeats of (elapsed / launches). Candidates are
 * enqueued in groups of `batch`; the host then sleeps until a host function
 * enqueued after the group signals that the stream has reached it. Deadlines
 * bound the wait: the runs enqueued before an event may take at most
 * timeout_ms each (plus 50 ms of slack for the host's own scheduling), counted
 * from when the previous event was found complete; the events themselves are
 * examined only when a deadline passes.
 * A candidate whose runs pass that deadline, or whose median latency exceeds
 * timeout_ms, gets CT_S_TIMEOUT. Kernels already enqueued cannot be recalled:
 * after a deadline passes the host waits for the stream to drain for
 * max(2 s, 4 x the remaining runs x timeout_ms), at most 60 s; if it drains
 * the other candidates keep their measurements, otherwise the call returns
 * CT_E_TIMEOUT and the stream is abandoned. */
typedef struct ct_measure_opts {
    int32_t warmup;
    int32_t repeats;     /* 1..64 */
    int32_t launches;    /* >= 1  */
    int32_t batch;       /* >= 1; candidates per synchronisation */
    float   timeout_ms;
    int32_t interleave;  /* 1: repeats run round-robin across the candidates */
} ct_measure_opts;

/* Optional correctness check during measurement: after each candidate's
 * last timed run, the device compares y with y_ref (fp32, same layout as y)
 * and sets CT_S_WRONG_ANSWER when max|y - y_ref| > tol * max|y_ref|. */
typedef struct ct_verify {
    const float *y_ref;  /* device pointer, or NULL for no check */
    float tol;
} ct_verify;

/* ---- set-up and device facts ---- */

/* Select HIP device `device`, check that it is gfx950, read its CU count and
 * build the per-process state. Idempotent for the same device. */
int ct_init(int device);
/* Compute units of the initialised device (256 on MI355X), or CT_E_NOINIT. */
int ct_num_cus(void);
/* Release streams, events and workspaces of every thread. */
void ct_shutdown(void);
/* Message of the last failure on the calling thread ("" if none). The
 * pointer stays valid until the thread's next library call. */
const char *ct_last_error(void);

/* ---- CU masks (section 2.2: a fixed share of the device per process) ---- */

/* Mask for `slot` of the share `fraction` on a device with num_cus CUs:
 * m = round(num_cus * fraction) CUs, slot j = bits [j m, (j+1) m). A
 * contiguous bit block spreads evenly over the XCDs because the driver
 * deals consecutive mask bits out to the XCDs in turn. Pure host function.
 * Returns CT_E_ARG if m = 0, words < num_cus/32, or the slot does not fit. */
int ct_build_cu_mask(int num_cus, double fraction, int slot, uint32_t *mask, int words);
/* Same, for the initialised device. */
int ct_cu_mask(double fraction, int slot, uint32_t *mask, int words);

/* ---- knob grids and validation (host only) ---- */

/* Number of knobs of a family and the raw grid size (product of the value
 * counts). */
int ct_grid_info(int family, int32_t *num_knobs, int64_t *grid_size);
/* Value list of knob `knob` of `family`: writes up to cap values, sets *count. */
int ct_knob_values(int family, int knob, int32_t *values, int32_t cap, int32_t *count);
/* Number of schedules of `family` that the validator accepts for op (0 if the
 * family does not apply to op's layout, dtype or grouping). */
int ct_grid_size(const ct_op *op, int family, int64_t *n);
/* Mixed-radix decode/encode: the first knob is the most significant digit. */
int ct_grid_decode(int family, int64_t index, ct_schedule *out);
int ct_grid_encode(const ct_schedule *s, int64_t *index);
/* 0 if schedule s may run on op, CT_S_INVALID if the validator rejects it
 * (reason in ct_last_error), CT_E_ARG for a malformed op or schedule.
 * Every schedule that passes is safe to launch: all its global accesses are
 * bounds-checked and its LDS, thread and grid sizes fit the device. */
int ct_validate(const ct_op *op, const ct_schedule *s);
/* LDS bytes, threads per block and blocks of one run of s on op (for
 * reports); the schedule must be valid. */
int ct_launch_shape(const ct_op *op, const ct_schedule *s, int32_t *lds_bytes,
                    int32_t *threads, int64_t *blocks, int32_t *kernels);

/* Name of the kernel template instance a schedule launches on op (its main
 * kernel, as a profiler lists it, e.g. "igemm_f32_kernel<32, 1, 1, 2, 3>"),
 * NUL-terminated in buf. For reports and for matching profiler traces. */
int ct_kernel_name(const ct_op *op, const ct_schedule *s, char *buf, int cap);

/* ---- candidate generation (section 2.1 stage 1: with no history, pick
 *      random candidates from the search space) ---- */

/* The candidate space of op is the concatenation, in ascending family order,
 * of each applicable family's valid grid indices in ascending order. Writes
 * up to cap schedules of it in that order; *count = its full size. */
int ct_valid_space(const ct_op *op, ct_schedule *out, int64_t cap, int64_t *count);
/* Seeded sample of n candidates without replacement, stratified by kernel
 * family (a family is a schedule template, which a TVM-style tuner tunes as a
 * task of its own). The valid space (ct_valid_space order: family by family,
 * grid order within) is split by family; family f gets a quota q_f: equal
 * shares of min(n, |V|), the remainder to the first families, and a family
 * with fewer valid schedules than its share hands the rest on, in rounds,
 * until the total is reached. Within family f, a partial Fisher-Yates shuffle
 * of its schedules driven by splitmix64 from state
 *   seed ^ (0x9E3779B97F4A7C15 * (1 + config_id)) ^ (0xC0FFEE << 32) ^ layer_id
 *        ^ (0xD1B54A32D192ED03 * family)
 * (first output discarded): for i < q_f, j = i + next() mod (|V_f| - i), swap.
 * out[] interleaves the families: the k-th pick of each family in family
 * order, then the (k+1)-th, so every prefix of the list is balanced.
 * out[i] is the candidate at sample position i. If |V| < n, all |V| are
 * returned. *n_out = number written. */
int ct_sample(const ct_op *op, uint64_t seed, int32_t config_id, int32_t layer_id,
              int32_t n, ct_schedule *out, int32_t *n_out);

/* The same without family quotas: the first n positions of one seeded partial
 * Fisher-Yates shuffle of the whole valid space (ct_valid_space order),
 * splitmix64 from state seed ^ (0x9E3779B97F4A7C15 * (1 + config_id)) ^
 * (0xC0FFEE << 32) ^ layer_id, first output discarded; j = i + next() mod
 * (|V| - i). Every valid schedule is equally likely, so a family's share of
 * the sample follows the size of its knob grid. */
int ct_sample_uniform(const ct_op *op, uint64_t seed, int32_t config_id, int32_t layer_id,
                      int32_t n, ct_schedule *out, int32_t *n_out);

/* ---- running and timing (section 2.1 stage 3, "profile") ---- */

/* Run schedule s once on op: y = conv2d(x, w). cu_mask = NULL uses all CUs.
 * Returns after the run has completed. CT_E_ARG if s is invalid for op, or
 * if s copies 16 bytes per lane (IGEMM_F32 on suitable shapes) and x or w is
 * not 16-byte aligned; measurement entry points report the latter as
 * CT_S_LAUNCH for that candidate. */
int conv2d_run(const ct_op *op, const ct_schedule *s, const void *x, const void *w, void *y,
               const uint32_t *cu_mask, int words);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops that forbid hipMalloc): conv2d_run's work, y =
 * conv2d(x, w) with schedule s, enqueued on the caller's HIP stream (a
 * hipStream_t; NULL = the null stream) and returned without waiting. A
 * schedule that splits its reduction keeps the partial sums in a static
 * device array of CT_SCRATCH_FLOATS floats (64 MiB) that the library holds
 * on each device until the process ends; schedules needing more than that
 * (split * N*K*OH*OW floats) are refused with CT_E_ARG. No device memory is
 * allocated or freed, and no stream is created. The array is shared by every
 * call on a device and keeps the last call's contents (each split schedule
 * overwrites every partial it reads, so nothing needs clearing): calls that
 * overlap on one device (two streams, or two threads) race on it and must be
 * serialised by the caller. Needs ct_init; x and w as for conv2d_run. */
#define CT_SCRATCH_FLOATS (1 << 24)
int conv2d_run_noalloc(const ct_op *op, const ct_schedule *s, const void *x, const void *w, void *y,
                       void *stream);

/* Time n candidates on slot 0 of the share cu_fraction, with the protocol o.
 * lat_us[i] = median latency in microseconds (+inf unless status OK),
 * status[i] = CT_S_*. rep_us (optional, n * o->repeats) receives every
 * repeat's per-run time. y is overwritten. Returns 0 even if some
 * candidates fail; a negative code means the call itself failed. */
int measure_candidates(const ct_op *op, const ct_schedule *s, int n, double cu_fraction,
                       const ct_measure_opts *o, const void *x, const void *w, void *y,
                       float *lat_us, int32_t *status);
/* Same with an explicit CU mask, optional verification and repeat output. */
int measure_candidates_mask(const ct_op *op, const ct_schedule *s, int n,
                            const uint32_t *cu_mask, int words, const ct_measure_opts *o,
                            const ct_verify *v, const void *x, const void *w, void *y,
                            float *lat_us, int32_t *status, float *rep_us);

/* Register the exact output of op for later measurements (the runner's
 * correctness check): y_ref_host is N*OH*OW*K fp64 values in op's output
 * layout (host memory, read during the call only). The library rounds them
 * to fp32 and keeps one device copy per op (ops compare field by field).
 * From then on every measurement of that op without an explicit ct_verify
 * reference re-runs each candidate once after its timed runs and sets
 * CT_S_WRONG_ANSWER when max|y - ref| > tol * max|ref| (tol 1e-4 for fp32 ops,
 * 2e-2 for bf16 ops). The reference holds only for the x and w it was
 * computed from: the caller keeps them. y_ref_host = NULL removes the op's
 * reference. Released by ct_shutdown. */
int ct_set_reference(const ct_op *op, const double *y_ref_host);

/* ---- selection (stage 4 of the loop; the best configuration is the one
 *      with the lowest measured latency, as the early-stop rule implies) ---- */

/* Order of stage-1 screening: indices of the t fastest OK candidates, by
 * (latency, sample position) ascending. Writes min(t, #OK) indices. */
int ct_top_t(const float *lat_us, const int32_t *status, int n, int t, int32_t *top, int32_t *n_top);
/* Winner among the re-measured candidates: the lowest sample position among
 * those whose latency is within (1 + eps) of the minimum. pos[i] is the sample
 * position of candidate i. Returns the index i of the winner in *winner. */
int ct_select_winner(const float *lat_us, const int32_t *pos, int n, float eps, int32_t *winner);

/* ---- tuning clients (section 3.1.1) ---- */

/* One layer to tune: the candidate list (in sample order), its buffers and
 * the result fields the library fills. */
typedef struct ct_tune_job {
    ct_op op;
    const void *x, *w;  void *y;        /* device buffers for this layer       */
    const ct_schedule *cands;  int32_t n_cands;
    ct_verify verify;                   /* optional correctness check          */
    /* outputs */
    float   *lat1_us;  int32_t *status1; /* caller arrays [n_cands]: screening  */
    int32_t top_t;                       /* in: re-measure this many (>= 1)     */
    int32_t *top_pos;  float *lat2_us;   /* caller arrays [top_t]: re-measure   */
    int32_t n_top;                       /* out: entries used in top_pos/lat2   */
    int32_t winner_pos;                  /* out: sample position of the winner, -1 if none */
    float   winner_lat_us;               /* out */
    double  t_start_s, t_end_s;          /* out: steady-clock seconds           */
    int32_t layer_id;                    /* in: the layer's id, written to logs */
    const uint8_t *skip;                 /* in, optional [n_cands]: candidates  */
                                         /* with skip[i] != 0 are not measured; */
                                         /* lat1_us[i] / status1[i] must hold   */
                                         /* their recorded values (resume)      */
    int32_t rc;                          /* out: 0, or the CT_E_* code that     */
                                         /* stopped this job                    */
} ct_tune_job;

/* One tuning client: a host thread that owns a CU-masked stream and tunes
 * its jobs in order (screen all candidates, re-measure the top_t with the
 * stage-2 protocol interleaved across them, select the winner). */
typedef struct ct_client {
    uint32_t cu_mask[CT_MASK_WORDS];
    int32_t host_core;                   /* pin the thread to this core; -1 = no pinning */
    ct_tune_job *jobs;  int32_t n_jobs;
    int32_t rc;                          /* out: 0 or a CT_E_* code             */
    double t_start_s, t_end_s;           /* out: first job start, last job end  */
    int64_t n_measured;                  /* out: candidates screened            */
    const char *log_path;                /* in, optional: append-only JSON-lines */
                                         /* log of this client (below); NULL =  */
                                         /* none                                */
    double cands_per_s;                  /* out: n_measured / (t_end - t_start) */
} ct_client;

/* Run n_clients clients concurrently, one host thread each, and wait for all.
 * Clients with overlapping masks are allowed but then share CUs. With the
 * environment variable CT_PROGRESS set, each client writes one line to stderr
 * per finished job.
 *
 * Logs (section 3.1.1: each tuning client keeps its own log and the logs are
 * merged per model). A client with log_path appends one JSON object per line
 * and flushes after each group of measured candidates:
 *   {"kind":"cand","layer":L,"pos":P,"family":F,"knobs":[...],"lat_us":X,"status":S}
 * for every screened candidate (X is null when not finite), and after a job
 * {"kind":"job","layer":L,"n_cands":N,"winner_pos":P,"winner_lat_us":X,
 *  "top_pos":[...],"lat2_us":[...],"rc":R}.
 * Candidate lists are a pure function of (seed, configuration, layer), so a
 * run is resumed by passing the recorded candidates through the job's skip
 * array. A client that fails (rc < 0) stops; the others keep taking jobs. An
 * exception inside a client thread is caught and reported as CT_E_CLIENT. */
int ct_tune_clients(ct_client *clients, int n_clients, const ct_measure_opts *stage1,
                    const ct_measure_opts *stage2, float eps);

/* The same clients fed from one queue: the jobs are taken in array order, each
 * by whichever client is idle first, so a model's layers spread over the
 * clients by their actual cost (list them longest first for the shortest
 * makespan). The clients' jobs / n_jobs fields are ignored; their other
 * fields are used as above. job_client (out, may be NULL) receives, per job,
 * the index of the client that ran it (-1 if none did). Returns 0, or the
 * code of the first client that failed (the other clients keep taking jobs). */
int ct_tune_shared(ct_client *clients, int n_clients, ct_tune_job *jobs, int n_jobs,
                   const ct_measure_opts *stage1, const ct_measure_opts *stage2, float eps,
                   int32_t *job_client);

/* Aggregate throughput of clients that have run: the sum of n_measured over
 * (latest t_end_s - earliest t_start_s), the conservative "time taken to
 * finish all of them" reading of the paper's throughput. Host only. */
int ct_throughput(const ct_client *clients, int n_clients, double *cands_per_s);

/* One client, one layer, k tuning server instances (section 3.1.1, Fig. 7a):
 * the job's candidate list is split into k contiguous parts, part j =
 * sample positions [n j / k, n (j + 1) / k), screened concurrently (one host
 * thread per part) on masks[j] (words words each) with output buffer
 * y_slots[j]; the k results are merged in place in lat1_us / status1, the
 * job's top_t are re-measured with stage2 on masks[0] (into y_slots[0]) and
 * the winner selected as in ct_tune_clients. y_slots holds k device buffers
 * the size of y (distinct, so that concurrent parts do not write the same
 * output); y_slots[0] may be job->y. screen_s (optional out) = wall seconds
 * of the concurrent screening. The job's verify reference (or the op's
 * registered one) checks every part. */
int ct_tune_split(ct_tune_job *job, const uint32_t *masks, int k, int words, void *const *y_slots,
                  const ct_measure_opts *stage1, const ct_measure_opts *stage2, float eps,
                  double *screen_s);

/* ---- cross-evaluation (section 2.2.1, Tables 1-2: tuned at f, run at g) ---- */

/* M[i * n_masks + j] = stage-2 latency of schedule s[i] run on mask j. The
 * repeats of all (i, j) cells are interleaved round-robin per mask. */
int ct_cross_eval(const ct_op *op, const ct_schedule *s, int n_sched,
                  const uint32_t *masks, int n_masks, int words,
                  const ct_measure_opts *o, const void *x, const void *w, void *y, float *M);

/* ---- guided search (section 2.1, stage 4: an exploration algorithm steered
 *      by a cost model trained on the profiled configurations; early stop) ---- */

typedef struct ct_search_opts {
    uint64_t seed;       /* all random choices derive from it (splitmix64)            */
    int32_t batch;       /* candidates proposed and measured per round (>= 1)         */
    int32_t budget;      /* most candidates measured in total (>= 1)                  */
    int32_t patience;    /* stop after this many measured candidates in a row that do */
                         /* not improve the best stage-1 latency by more than eps;    */
                         /* 0 = never stop early                                       */
    int32_t sa_chains;   /* simulated-annealing chains per round                      */
    int32_t sa_steps;    /* steps per chain per round                                 */
    float explore;       /* share of each batch drawn at random from the unmeasured   */
                         /* space (the rest: the cost model's best unmeasured states) */
    float eps;           /* relative improvement that resets the patience count       */
    float sa_temp;       /* starting temperature, in units of log latency; it falls   */
                         /* linearly to 0 over a chain                                 */
    int32_t cus;         /* CUs of the share being tuned, for the cost model's grid   */
                         /* features; 0 = ct_search counts the mask (all 256 for      */
                         /* ct_search_propose)                                        */
} ct_search_opts;

typedef struct ct_search_result {
    int32_t n_measured;     /* candidates measured (<= budget)                        */
    int32_t rounds;
    int32_t stopped_early;  /* 1 if the patience rule ended the search                */
    int32_t winner;         /* index into the measured list, -1 if none measured OK   */
    float winner_lat_us;    /* the winner's stage-2 latency                           */
    float pad_;
    double propose_s;       /* host seconds spent proposing                           */
    double measure_s;       /* host seconds spent in measurement calls                */
} ct_search_result;

/* Next batch of a guided search (host only, no device work). The cost model
 * is fitted on the n_measured schedules measured so far (status CT_S_OK ones
 * only): per kernel family, ridge regression of log latency on a one-hot code
 * of the knob values plus launch-geometry features. so->sa_chains annealing
 * chains of so->sa_steps steps each (half start at the best measured
 * schedules of each family in turn, half at random valid ones; a step moves
 * one knob to a neighbouring value) walk the predicted latency; the
 * best-predicted unmeasured states they visit fill the batch, except a share
 * so->explore of it (all of it when nothing has been measured OK yet) drawn
 * at random: the applicable kernel families in turn, uniformly within each,
 * so a small family is explored as much as a large one. Random draws that hit
 * measured schedules are redrawn. Writes min(cap, so->batch) distinct valid
 * schedules not among `measured` (fewer once the space runs out) to out,
 * count in *n_out. Same inputs and round give the same output. */
int ct_search_propose(const ct_op *op, const ct_schedule *measured, const float *lat_us, const int32_t *status,
                      int n_measured, const ct_search_opts *so, int32_t round, ct_schedule *out, int32_t cap,
                      int32_t *n_out);

/* Guided tuning of one op on a CU mask: rounds of ct_search_propose and
 * stage-1 measurement until so->budget candidates are measured, the space
 * runs out, or the patience rule fires; then the top_t by stage-1 latency are
 * re-measured with stage2 and the winner chosen by ct_select_winner with eps
 * (position = index in the measured list). measured, lat_us and status are
 * caller arrays of so->budget entries and receive every measured candidate in
 * order. With CT_PROGRESS set, one line per round goes to stderr. */
int ct_search(const ct_op *op, const ct_search_opts *so, const uint32_t *cu_mask, int words,
              const ct_measure_opts *stage1, const ct_measure_opts *stage2, int32_t top_t, float eps,
              const void *x, const void *w, void *y, ct_schedule *measured, float *lat_us, int32_t *status,
              ct_search_result *res);

/* ---- probes (support for masks and rooflines) ---- */

/* Launch `blocks` one-wave blocks on the mask; each records the hardware
 * (XCC, SE, SH, CU) of the CU it ran on. out[i] = packed id
 * (xcc << 12 | se << 8 | sh << 4 | cu) of the i-th distinct CU seen,
 * *n_out = number of distinct CUs (<= cap written). */
int ct_probe_cus(const uint32_t *cu_mask, int words, int blocks, int32_t *out, int cap, int32_t *n_out);
/* Median time per launch of an empty kernel with `blocks` blocks on the mask
 * (the dispatch floor of the timing protocol). */
int ct_probe_empty(const uint32_t *cu_mask, int words, int blocks, const ct_measure_opts *o, float *us);
/* Achieved copy bandwidth (read + write bytes / time) of a bytes-sized
 * device-to-device copy kernel on the mask, in GB/s. Buffers are the caller's. */
int ct_probe_copy(const uint32_t *cu_mask, int words, const void *src, void *dst, int64_t bytes,
                  const ct_measure_opts *o, float *gbps);

/* Number of CU-masked streams the library holds. A stream is reused by later
 * calls with the same mask once the call holding it returns, so the count is
 * bounded by the most calls that ran at once on one mask (diagnostic). */
int ct_stream_count(void);

/* ---- host-logic test hooks (no device work) ----
 * These drive the library's own host code -- client threads, the shared job
 * queue, logs, resume, top-t selection and the timeout watchdog -- with a
 * stand-in for the device, so that failure handling is tested on a machine
 * without a GPU. They never compute a convolution. */

typedef struct ct_test_hooks {
    int32_t delay_us;           /* host sleep per stand-in measurement              */
    int32_t throw_client;       /* client that raises an exception (-1: none) ...   */
    int32_t throw_after_jobs;   /* ... when it starts its job number k (0-based)    */
    int64_t stop_after_records; /* every client stops (CT_E_STOPPED) once this many */
                                /* candidate records are logged in total (-1: never) */
} ct_test_hooks;

/* ct_tune_shared with the stand-in measurement: candidate i of a job gets
 * status CT_S_OK and latency 1 + ((layer_id * 7919 + i) * 2654435761 mod 1000)
 * / 100 microseconds after hooks->delay_us of host sleep; the re-measure
 * repeats the same latency. Needs no ct_init. */
int ct_test_run_clients(ct_client *clients, int n_clients, ct_tune_job *jobs, int n_jobs,
                        const ct_test_hooks *hooks, int32_t *job_client);

/* The timeout watchdog on a simulated stream: event k completes at
 * done_at_s[k] seconds (< 0: never); runs[k] runs precede it; the host polls
 * every millisecond of simulated time. Outputs the first event whose
 * deadline passed (-1: none) and whether the stream drained afterwards. */
int ct_test_watchdog(int n_events, const int32_t *runs, const double *done_at_s, double run_limit_s,
                     double slack_s, double drain_cap_s, int32_t *expired_event, int32_t *drained);

/* The XCD-band block renumbering (each XCD takes one contiguous band of
 * tiles) that the bf16 pointwise family applies under its swizzle knob and
 * the fp32 MFMA family always, computed by the same function the kernels
 * use: tile_of_block[b] for b < tiles. */
int ct_test_xcd_band(int tiles, int32_t *tile_of_block);

#ifdef __cplusplus
}
#endif
#endif /* CONVTUNE_H */
