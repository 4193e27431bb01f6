// Internal layout shared by the HIP kernels and the host side of libaladdin.
//
// Worker state (one "scenario" = one pool of workers with one latency model;
// ald_place_stream uses one scenario, ald_sweep_scenarios many):
//
//   Each worker owns a slot range [slot_base, slot_base + cap] of five int32
//   arrays.  Requests are kept in absolute decode-iteration form so that a
//   heartbeat (one decode iteration of every worker) only increments tau:
//       e = r + tau   (iteration at which the request emits its last token)
//       s = c - tau   (context minus tau; c = s + tau at any tau)
//   Slots [head, n) hold the live requests sorted by e ascending; slots before
//   head hold finished requests (e < tau) that are dropped lazily.
//
//   With P_k = sum_{j >= k} (s_j + e_k)  (the KV demand at the end point of
//   request k counted over the requests at or after slot k; it equals the
//   demand at iteration r_k whenever k is the first of its tie group, and is
//   below it otherwise), the summaries, kept together in one int4 per slot
//   (pms = {pme, sm, ss, n - k}), are
//       ss[k]  = sum_{j >= k} s_j                     (ss[n] = 0)
//       pme[k] = max_{head <= j < k} (P_j + e_j)       (pme[head] = PME_NONE)
//       sm[k]  = max_{j >= k} P_j                     (sm[n] = NEG)
//   For a query with sq = l_in - tau, eq = l_pred + tau and
//   l = first live slot with e >= eq, the demand peak with the query added is
//       max( pme[l] + sq,  sm[l],  ss[l] + (n - l) * eq + sq + eq ).
//   All of these are tau-free: a heartbeat leaves them valid except that
//   requests whose e fell below tau must leave the live range.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/aladdin.h"

namespace ald {

constexpr int TOPK = 4;            // feasible candidates kept per query
constexpr int EVAL_THREADS = 256;  // threads per pair-evaluation block
constexpr int EVAL_QPT = 4;        // queries per pair-evaluation thread
constexpr int EVAL_Q = EVAL_THREADS * EVAL_QPT;  // queries per pair-evaluation block
constexpr int EVAL_WPB_MAX = 64;  // workers per pair-evaluation block at most
constexpr int STAGE_MAX = 768;     // live requests of a worker the evaluation stages in LDS (fewer than)
constexpr int SORT_MIN_TILE = 16384;  // one-scenario tiles at least this long are evaluated in l_pred order
constexpr int SEL_THREADS = 256;   // queries per selection block
constexpr int COMMIT_THREADS = 64;  // the arrival-order commit runs as one wave
constexpr int HOT = 8192;          // most request slots per worker (commit keeps one worker in LDS)
constexpr int BUILD_THREADS = 256;
constexpr int MAX_DIRTY = 64;      // workers changed within one tile before the tile is cut
constexpr int COMMIT_CACHE_W = 2048;  // workers of a scenario whose scan rows the commit can keep in LDS
#ifndef ALD_STALE_CUT
#define ALD_STALE_CUT 24
#endif
// exact re-scans of changed workers (infeasible ones, or for diagnostics) after
// which the commit cuts its tile; a build-time option
constexpr int STALE_CUT = ALD_STALE_CUT;
constexpr int32_t NEG = INT32_MIN;
// pme with no slot before it: far below every demand, yet pme + sq cannot wrap
// in 32 bits (|sq| < 2^28)
constexpr int32_t PME_NONE = -(1 << 30);
constexpr int LB_MAX = 2048;       // l_pred range of a worker's breakpoint table
constexpr int LB_SLOTS = 4096;     // workers with fewer live requests have a breakpoint table

// error codes raised on the device (mirrors ALD_E* in aladdin.h)
constexpr int32_t DEV_EINVAL = -1;
constexpr int32_t DEV_ESLOTS = -3;
constexpr int32_t DEV_EOVERFLOW = -5;

struct Scen {
    double c1, k1, k1q, c3, c2, k2, ttft, tdec, theta;
    int32_t gn, gs;
    int32_t W;          // workers in this scenario
    int32_t wbase;      // first global worker index
    int32_t wpb;        // workers per pair-evaluation block
    int32_t nblk;       // worker blocks (ceil(W / wpb))
    int32_t eval_blk0;  // first pair-evaluation block of this scenario
    int32_t sel_blk0;   // first selection block
    int32_t fin_blk0;   // the scenario's commit block
    int32_t sel_g;      // waves of a selection block that share one 64-query group (1, 2 or 4)
    int32_t uniform_M;  // every worker has the same capacity: empty workers are interchangeable
    int32_t mono;       // k1, k1q >= 0: the TTFT of a pair grows with l_in (integer thresholds apply)
    int32_t ntint;      // with mono: every near-tie band spans at most 64 integer values (bound
                        // from the coefficients), so near-tie margins have integer forms too
    int32_t use_d;      // the residents' decode history is known: constraint (d) is checked
    int64_t bits_off;   // uint64 words into bits_feas / bits_nt
    int64_t part_off;   // int4 entries into part (worker block major: part_off + wb * pstride + query)
    int64_t pstride;    // queries per tile rounded up to whole evaluation chunks
    int64_t qsum_off;   // QSum entries into qsum
    int64_t out_off;    // offset into out_worker
    // The scenario's query i is entry qmap[i] of the call's query arrays (and
    // of out_worker after out_off, and of out_diag), or entry i when qmap is
    // null; grouped placement lists each group's queries this way.  out_add
    // is added to the worker index written (a group's first worker; 0
    // elsewhere).  hb[i] (null: none) = decode iterations (heartbeats) that run
    // before the scenario's query i; the control block's hb_next points at
    // the next i > start with hb[i] > 0.
    const int32_t* qmap;
    const int32_t* hb;
    int32_t out_add;
    int32_t gpw;        // GPUs per worker (a sweep's answer counts n_workers * gpw GPUs)
};

__host__ __device__ inline int64_t q_at(const Scen& sc, int32_t i) { return sc.qmap ? (int64_t)sc.qmap[i] : (int64_t)i; }

// Per-scenario control block.  Written by the commit kernel's sequential block
// only; every other kernel only reads it (kernel boundaries order the accesses).
struct Ctl {
    int32_t start;      // next query to process
    int32_t Q;          // queries in this call
    int32_t T;          // tile length
    int32_t H;          // heartbeat period (0 = none)
    int32_t since_hb;   // processed queries since the last heartbeat
    int32_t tau;        // decode iterations run so far (absolute time offset)
    int32_t hb_index;   // heartbeat counter (stamps the TTFT sums)
    int32_t rebuild;    // 1: every worker's summaries must be rebuilt (tau moved)
    int32_t err;        // first device error (0 = none)
    int32_t n_rej;      // rejected queries
    int32_t first_rej;  // first rejected query (INT32_MAX = none)
    int32_t aborts;     // tiles cut short (statistics)
    int32_t round;      // rounds run
    int32_t commits;    // placements made
    int32_t ndirty;     // workers the last commit round changed (their summaries are stale)
    int32_t hb_next;    // with per-query heartbeats: the next query (> start) that heartbeats
                        // precede, Q if none; 0 otherwise
    int32_t fallbacks;  // decisions that scanned the untouched workers' bit words (statistics)
    int32_t stale_cuts; // tiles cut on the stale-scan budget (statistics)
    int32_t call;       // the placement call the block belongs to (State::call); kernels
                        // launched for another call leave it alone
};

// The outcome of a one-scenario placement call as the ALD_* code its
// synchronous form returns (control block `c`, after the call's rounds).
__host__ __device__ inline int32_t ctl_status(const Ctl& c)
{
    if (c.err == DEV_ESLOTS) return ALD_ESLOTS;
    if (c.err == DEV_EOVERFLOW) return ALD_EOVERFLOW;
    if (c.err == DEV_EINVAL) return ALD_EINVAL;
    if (c.err != 0) return ALD_EHIP;
    return c.start < c.Q ? ALD_EINCOMPLETE : ALD_OK;
}

// Tile description published by the selection kernel for the commit kernel.
struct TileInfo {
    int32_t start, end, parity, pad;
    int32_t first_pc[2];  // first query of the tile with a feasible worker (by round parity)
};

// Per-query result of the selection kernel (tile-start state), kept by tile
// position (the query's offset, or its place in the sorted layout).  With
// interchangeable empty workers (uniform capacity), empty workers are not listed
// one by one: `efeas` says whether an empty worker is feasible (all are alike).
struct QSum {
    uint64_t tkey[TOPK];  // best feasible listed workers: rank keys, descending
    int32_t tw[TOPK];     // their indices (-1 = none)
    uint64_t ntkey;       // best-ranked worker with a near-tie margin
    int32_t ntw;          // its index (-1 = none)
    int32_t ntcnt;        // workers with a near-tie margin
    int32_t nfeas;        // feasible workers (all kinds)
    int32_t ncand;        // feasible workers of the listed kind
    int32_t efeas;        // an empty worker is feasible
    int32_t ex1, w1;      // smallest KV excess (ties: highest index first)
    int32_t ex2, w2;      // second smallest
    int32_t pad;
};

// Device mirror of ald_query_diag_t.
struct Diag {
    int32_t n_feasible;
    int32_t near_tie;
    int64_t kv_peak_chosen;
    int64_t kv_excess_min;
    double ttft_chosen;
    double tdec_chosen;
};

struct State {
    // per worker [NW]
    int64_t* slot_base;
    int32_t* cap;
    int32_t* n;
    int32_t* head;
    int32_t* M;
    int64_t* S1;
    int64_t* S2;
    int32_t* hbs;      // heartbeat stamp of S1/S2
    int32_t* built;
    int32_t* B;
    int64_t* DS;       // 2^gs * sum(c) + gn * sum(r)
    uint64_t* key;     // (2^gs B)^2 + DS^2
    int32_t* peak;     // KV peak without a new query
    double* rhs;       // theta * ((T_dec - c3) - c2 * (B + 1))
    int64_t* SC;       // sum(c)
    int64_t* SR;       // sum(r)
    // Integer forms of the latency checks at the built state, for a query with
    // qD = 2^gs l_in + gn l_pred:  decode (b) holds iff qD <= dq_max, TTFT (c)
    // iff l_in <= lthr (with Scen::mono); a near-tie margin is only possible
    // for qD in [ntd_lo, ntd_hi] or l_in in [ntt_lo, ntt_hi].
    int64_t* dq_max;
    int64_t* ntd_lo;
    int64_t* ntd_hi;
    int32_t* lthr;
    int32_t* ntt_lo;
    int32_t* ntt_hi;
    // Exact near-tie sets where a band spans at most 64 values: bit i of ntd_mask
    // is the decode margin test at qD = ntd_lo + i, bit i of ntt_mask the TTFT
    // margin test at l_in = ntt_lo + i (zero where the band is wider).
    uint64_t* ntd_mask;
    uint64_t* ntt_mask;
    // Constraint (d) (with Scen::use_d): every ongoing request's slack
    // T_dec * g - t_dec grows by T_dec - t_iter at each heartbeat; the worker
    // keeps that running gain in phi (brought up to heartbeat phi_hb) and each
    // request slack - phi in its log entry.  dlim = theta * the smallest slack
    // of the ongoing live requests at the built state (+inf: no limit); the
    // TTFT threshold lthr includes it, and [ntp_lo, ntp_hi] holds every l_in
    // whose prefill time can be within a near tie of dlim.
    double* phi;
    int32_t* phi_hb;
    double* dlim;
    int32_t* ntp_lo;
    int32_t* ntp_hi;
    int32_t* lgn;      // log entries of the worker
    // per slot (the worker's slot range, unordered): the log of its requests
    int32_t* lge;      // e of the request (it has finished once e < tau)
    int32_t* lgw;      // heartbeat window it was placed in (-1: resident at load)
    double* lgs;       // slack - phi
    // per slot
    int32_t* e;
    int32_t* s;
    int4* pms;         // {pme, sm, ss, unused}
    // per worker [NW * LB_MAX] (built workers with B > 0): entry v - 1 = number of
    // live requests with remaining length below v, v = 1 .. LB_MAX
    uint16_t* lbt;
    // per scenario [S]
    const Scen* scen;
    Ctl* ctl;
    Ctl* ctl_host;     // pinned host mirror of ctl, written by the commit kernel
    TileInfo* tinfo;
    int32_t* dlist;    // [S * MAX_DIRTY] workers changed in the last tile (global index)
    int32_t* dcount;   // [S]
    int32_t S;
    int32_t NW;
    int32_t call;      // this launch's placement call: control blocks of another call are not touched
    int32_t* status;   // the last round of an asynchronous call: where the commit kernel writes
                       // the call's outcome (one scenario; null otherwise)
    // tile scratch
    uint64_t* bits_feas;
    uint64_t* bits_nt;
    // Sorted tile layout (one-scenario tiles of at least SORT_MIN_TILE queries;
    // null otherwise): the pair evaluation takes each chunk of EVAL_Q queries in
    // order of l_pred, and the bit words and excess keys are kept by that order.
    // qorig[p] = tile offset of the query at sorted tile position p; qpos is the
    // inverse (both per tile offset, pstride entries).
    int32_t* qorig;
    int32_t* qpos;
    ulonglong2* part;  // per (worker block, query): the two smallest KV-excess keys
    QSum* qsum;
    // queries and outputs
    const int32_t* q_lin;
    const int32_t* q_lpred;
    int32_t* out_worker;
    Diag* out_diag;    // only with S == 1
    int32_t* err_word; // load-time validation
    int32_t* qbad;     // nonzero: a query length of this call is invalid (one-scenario calls; else null)
};

inline __host__ __device__ int32_t tile_end(int32_t start, int32_t Q, int32_t T, int32_t H, int32_t since_hb,
                                            int32_t hb_next) {
    int64_t end = (int64_t)start + T;
    if (end > Q) end = Q;
    if (H > 0) {
        int64_t hb = (int64_t)start + (H - since_hb);
        if (hb < end) end = hb;
    }
    if (hb_next > start && hb_next < end) end = hb_next;
    return (int32_t)end;
}

// host-side launchers (ald_kernels.hip)
hipError_t launch_ingest(const State& st, int32_t W, const int64_t* res_off, const int32_t* lin,
                         const int32_t* lpred, const int32_t* gen, const double* tdec, hipStream_t stream);
// mode 0: every worker whose summaries are stale; 1: only the workers listed by
// the last commit; 2: every worker unconditionally
hipError_t launch_build(const State& st, hipStream_t stream, int mode);
// mode 0: latency checks in fp64; 1: integer thresholds, near-tie margins in
// fp64; 2: integer thresholds and near-tie sets; 3: as 2, with the workers too
// large to stage read through their breakpoint tables in global memory (a
// variant of its own: it holds more registers)
constexpr int EVAL_MODES = 4;
hipError_t launch_eval(const State& st, int32_t blocks, int mode, hipStream_t stream);
// pair-evaluation blocks of the variant launch_eval takes for (mode, ex) that
// one compute unit holds at once, or 0 if the runtime cannot say
int eval_blocks_per_cu(int mode, bool ex);
hipError_t launch_select(const State& st, int32_t blocks, hipStream_t stream);
// use_d: some scenario checks constraint (d)
// cache: the variant that keeps the untouched-worker scan's bit rows and rank
// keys in LDS (scenarios of at most COMMIT_CACHE_W workers)
hipError_t launch_commit(const State& st, int32_t blocks, bool use_d, bool cache, hipStream_t stream);
hipError_t launch_query_stats(const int32_t* lin, const int32_t* lpred, int32_t Q, Ctl* ctl, int32_t S,
                              hipStream_t stream);
// gate: -1, or the asynchronous call that must have finished for this one to start
hipError_t launch_begin(const Ctl& c, const TileInfo& ti, Ctl* ctl, TileInfo* tinfo, int32_t* qbad, int32_t gate,
                        hipStream_t stream);
// status = ALD_OK (an asynchronous call with no queries)
hipError_t launch_status_ok(int32_t* status, hipStream_t stream);
hipError_t launch_summary(const State& st, int32_t W, int32_t* B, int64_t* sc, int64_t* sr, int64_t* peak,
                          hipStream_t stream);
// rejected / first rejected query per scenario, and (min_gpus non-null) the
// scenario with no rejection and the fewest GPUs: {GPUs, scenario} or {-1, -1}
hipError_t launch_sweep_outputs(const State& st, int32_t* rejected, int32_t* first_reject, int64_t* min_gpus,
                                hipStream_t stream);
// status = the outcome of an asynchronous sweep (after its rounds)
hipError_t launch_sweep_status(const State& st, int32_t* status, hipStream_t stream);

}  // namespace ald
