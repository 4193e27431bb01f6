/*
 * libaladdin -- SLO- and KV-aware query placement evaluator for MI355X (gfx950).
 *
 * Implements the request-placement path of Aladdin (Nie, Fonseca, Liu: "Aladdin:
 * Joint Placement and Scaling for SLO-Aware LLM Serving", arXiv 2405.06856):
 * every arriving query is evaluated against every serving worker and placed by
 * the best-fit heuristic (Algorithm 1) in arrival order; the same evaluator runs
 * over many cluster configurations to find the smallest feasible one.
 *
 * Placement rule (per query q = (l_in, l_pred), per worker w):
 *   - constraint (e), KV capacity (Eq. 1 with h = 1, j = 0; footprint vector w of
 *     Sec. 4.2): a request that has generated g tokens holds c = l_in + g tokens
 *     and decodes r = l_pred - g more iterations, holding c + t tokens at future
 *     iteration t <= r.  The worker's demand with q added must stay <= M at
 *     every t; it is evaluated at the request end points only.
 *   - constraint (b), decode SLO (Eq. 3/Eq. 4): with b = batch size + 1 and
 *     D = c + gamma * r per request,
 *       k2 * sum(D) <= theta * ((T_dec - c3) - c2 * b).
 *   - constraint (c), TTFT SLO (Eq. 2 plus a quadratic term): over the requests
 *     placed on w in the current heartbeat plus q,
 *       (c1 + k1 * sum(l_in)) + k1q * sum(l_in^2) <= T_pre.
 *   - Algorithm 1: among workers meeting (b), (c), (e), choose the largest
 *     capacity_norm = ||(B, sum(D))||_2 before placement (compared exactly as an
 *     integer), ties to the lowest worker index; none -> rejected (-1).
 *   - heartbeat: after every H processed queries (or as many as the caller's
 *     clock puts before a query, ald_place_stream_hb) each worker runs one
 *     decode iteration (c += 1, r -= 1, finished requests leave) and the TTFT
 *     sums of constraint (c) restart at zero.
 *   - constraint (d), prefill preemption (only with a decode history, see
 *     ald_load_workers_history): the same prefill time as (c) must also stay
 *     <= theta * min over the worker's ongoing requests of (T_dec * g - t_dec),
 *     g = tokens generated so far, t_dec = decode time so far; each heartbeat's
 *     decode iteration takes (c3 + c2*b) + k2*sum(c) (Eq. 3) and adds one token
 *     and that time to every request in it.  Ongoing = resident at load or placed
 *     in an earlier heartbeat; a worker with none has no such limit.
 *   - split-phase decode workers (Sec. 5): a model with ttft_slo = +INFINITY
 *     checks only (b) and (e).
 *
 * Around the placement: grouped placement (App. A, ald_place_grouped), the
 * sweep with heartbeats (per arrival rate, Eq. 7; ald_sweep_scenarios_hb), and
 * Algorithm 2's re-balancing against output-length prediction errors
 * (ald_rebalance).
 *
 * Conventions
 *   - Every array argument except where marked "host" is a DEVICE pointer to
 *     contiguous memory owned by the caller (e.g. a torch tensor's data_ptr());
 *     the library never frees caller memory.
 *   - The library allocates no device memory.  The caller attaches a device
 *     workspace (ald_set_workspace, e.g. a torch uint8 tensor); the loaded
 *     workers' state lives at its start and every call lays out its own
 *     tables after it.  A call that does not fit returns ALD_ESPACE before
 *     doing any work, and ald_workspace_needed gives the size it needed.  The
 *     only memory the library allocates is one pinned host buffer per handle
 *     (76 bytes per scenario) into which the kernels copy their control blocks.
 *   - All work runs on the stream given to ald_create.  Every call below but
 *     ald_place_stream_async and ald_sweep_scenarios_async returns after that
 *     stream has finished the call's work, so errors are synchronous and
 *     outputs are ready on return; those two validate their arguments, enqueue
 *     their work and return, and report the outcome in a device status word.
 *   - Return value: ALD_OK (0) or a negative ALD_E* code; ald_last_error() gives
 *     a message.  On a validation error nothing is written to the outputs and
 *     the handle's worker state is unchanged.
 *   - A handle is used by one host thread at a time.
 *   - Token counts are integers; latencies are IEEE fp64 evaluated with the
 *     parenthesisation shown above, without fused multiply-add.  Internally the
 *     per-request KV bookkeeping is 32-bit; ALD_EOVERFLOW is returned when a
 *     stream could leave that range (capacities above 2^30 tokens, lengths above
 *     2^24, or a worker state whose demand could pass 2^31).
 */
#ifndef ALADDIN_H
#define ALADDIN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ALD_OK 0
#define ALD_EINVAL (-1)    /* invalid argument or input value */
#define ALD_EHIP (-2)      /* HIP runtime error (launch, copy, allocation) */
#define ALD_ESLOTS (-3)    /* a worker ran out of request slots */
#define ALD_ESTATE (-4)    /* call order: no workers loaded */
#define ALD_EOVERFLOW (-5) /* a value would leave the exactly representable range */
#define ALD_ESPACE (-6)    /* the attached workspace is too small for the call (see ald_workspace_needed) */
#define ALD_EINCOMPLETE (-7) /* an asynchronous placement ran out of rounds (see ald_place_resume) */
#define ALD_EBLOCKED (-8)  /* an asynchronous placement did not run: an earlier one is unfinished */

typedef struct ald_handle* ald_handle_t;

/* Latency / SLO model of one worker type; all fp64 (host struct, copied). */
typedef struct {
    double c1, k1, k1q;        /* prefill: T_p = (c1 + k1*S1) + k1q*S2            (Eq. 2) */
    double c3, c2, k2;         /* decode:  T_d = (c3 + c2*b) + k2*context          (Eq. 3) */
    double ttft_slo;           /* T_pre, seconds                                   (Table 1);
                                  +INFINITY: a decode worker of split-phase serving (Sec. 5),
                                  where only (b) and (e) apply (no TTFT, no (d)) */
    double decode_slo;         /* T_dec, seconds per output token; must exceed c3  (Eq. 4) */
    double theta;              /* prediction-error knob of constraint (b), in (0, 1] */
    int32_t gamma_num;         /* strictness knob gamma = gamma_num / 2^gamma_log2den, */
    int32_t gamma_log2den;     /*   0 <= gamma <= 1, gamma_log2den in [0, 8]           */
} ald_model_t;

/* One cluster configuration of a scaling sweep (host struct). */
typedef struct {
    int32_t n_workers;         /* >= 1 */
    int32_t gpus_per_worker;   /* 1 .. 256; counts the GPUs of the sweep's answer (the latency
                                  model already holds the worker's speed) */
    int64_t kv_capacity;       /* tokens per worker, 1 .. 2^30 */
    ald_model_t model;
} ald_scenario_t;

/* Per-query diagnostics (40 bytes, device array of Q). */
typedef struct {
    int32_t n_feasible;        /* workers meeting (b), (c), (e) (and (d) with a decode
                                  history) for this query */
    int32_t near_tie;          /* 1 if a worker ranked at or above the choice (every worker
                                  when rejected) has a decode, TTFT or (d) margin within 1e-9
                                  relative: fp64 rounding could have decided it */
    int64_t kv_peak_chosen;    /* KV peak of the chosen worker with q added (0 if rejected) */
    int64_t kv_excess_min;     /* min over all workers of (KV peak with q) - capacity */
    double ttft_chosen;        /* prefill time of the chosen worker's batch with q (0 if rejected) */
    double tdec_chosen;        /* (c3 + c2*b) + k2*sum(D) of the chosen worker (0 if rejected) */
} ald_query_diag_t;

/* Create a handle on HIP device `device`, launching on `hip_stream`
 * (a hipStream_t, or NULL for the default stream). */
int ald_create(ald_handle_t* handle, int device, void* hip_stream);

/* Release the handle (the caller's workspace is not touched).  NULL is accepted. */
int ald_destroy(ald_handle_t handle);

/* Attach the caller's device workspace: `workspace` is a device pointer,
 * 256-byte aligned, of `bytes` bytes, kept alive by the caller while the
 * handle uses it (NULL with bytes = 0 detaches).  With workers loaded, their
 * state moves into the new workspace (a copy on the handle's stream, so the
 * old one may be released once the stream has passed this call); the new one
 * must hold it (ALD_ESPACE otherwise) and must not overlap the old state
 * (ALD_EINVAL). */
int ald_set_workspace(ald_handle_t handle, void* workspace, size_t bytes);

/* The workspace size (bytes, including the loaded state) that the last call
 * refused with ALD_ESPACE needed. */
int ald_workspace_needed(ald_handle_t handle, size_t* bytes);

/* Workspace for loading W workers holding n_resident requests in all (model
 * and slots_per_worker as for ald_load_workers; with_history != 0 for
 * ald_load_workers_history) and then placing up to Q queries per
 * ald_place_stream or ald_place_stream_hb call, at the handle's current tile
 * setting.  Grouped placement, moves and Algorithm 2 lay out their own tables
 * after the state; ald_workspace_needed reports what a refused call needed. */
int ald_workspace_size(ald_handle_t handle, int32_t W, int64_t n_resident, const ald_model_t* model,
                       int32_t slots_per_worker, int32_t with_history, int32_t Q, size_t* bytes);

/* Workspace for ald_sweep_scenarios or ald_sweep_scenarios_hb over these S
 * scenarios (host array) and Q queries, beyond the state of loaded workers
 * (the sweep's tables go after it). */
int ald_sweep_workspace_size(ald_handle_t handle, int32_t S, const ald_scenario_t* scen, int32_t Q, size_t* bytes);

/* Queries evaluated per speculative tile (default 4096, 64 .. 1048576).  The
 * result never depends on it; only speed does. */
int ald_set_tile(ald_handle_t handle, int32_t tile_queries);

/* Load W workers with their ongoing requests (Table 1 inputs), replacing any
 * previous state.  Device arrays: kv_capacity[W]; res_offsets[W+1] (CSR: worker
 * i owns residents res_offsets[i] .. res_offsets[i+1]-1, res_offsets[0] = 0);
 * res_l_in, res_l_pred, res_generated [res_offsets[W]] with l_in >= 1,
 * l_pred >= 1, 0 <= generated < l_pred.  `model` is a host pointer.
 * slots_per_worker: request slots kept per worker (0 = derive the bound on the
 * batch size from constraint (b); required when that bound is infinite). */
int ald_load_workers(ald_handle_t handle, int32_t W, const ald_model_t* model,
                     const int64_t* kv_capacity, const int64_t* res_offsets,
                     const int32_t* res_l_in, const int32_t* res_l_pred,
                     const int32_t* res_generated, int32_t slots_per_worker);

/* As ald_load_workers, and every resident's decode time so far in seconds
 * (device array res_t_dec[res_offsets[W]], finite, >= 0), so that constraint
 * (d) of the placement MIP (Sec. 4.2: the new requests' prefill may not exceed
 * the time the ongoing ones have saved against the ATGT limit, scaled by theta)
 * is checked for every later placement.  ALD_EINVAL for a NULL or invalid
 * history.  Costs one fp64 slack base and a window index per request slot. */
int ald_load_workers_history(ald_handle_t handle, int32_t W, const ald_model_t* model,
                             const int64_t* kv_capacity, const int64_t* res_offsets,
                             const int32_t* res_l_in, const int32_t* res_l_pred,
                             const int32_t* res_generated, const double* res_t_dec,
                             int32_t slots_per_worker);

/* Place Q queries (device arrays q_l_in[Q], q_l_pred[Q], values >= 1) in index
 * (arrival) order on the loaded workers, committing every placement: the online
 * best fit of Algorithm 1 under the constraints (b), (c), (d), (e) of the
 * placement problem of Sec. 4.2 (Table 1: each query carries l_in and its
 * predicted l_out; the SLOs are the model's).  Repeated calls continue the same
 * stream.  heartbeat_every = H > 0: a heartbeat after every H processed queries
 * (counted across calls; Sec. 4.2 places requests per heartbeat); 0: no
 * heartbeat in this call.  out_worker[Q] (device): chosen worker or -1 (no
 * worker meets every constraint: the query is rejected and nothing changes).
 * out_diag[Q] (device) or NULL.  ALD_EINVAL (nothing written) for a length
 * outside [1, 2^24]; ALD_ESLOTS when a worker runs out of request slots. */
int ald_place_stream(ald_handle_t handle, int32_t Q, const int32_t* q_l_in, const int32_t* q_l_pred,
                     int32_t heartbeat_every, int32_t* out_worker, ald_query_diag_t* out_diag);

/* ald_place_stream (Algorithm 1 and the constraints of Sec. 4.2, placed in
 * arrival order), stream-asynchronous: the call validates its arguments,
 * enqueues its work on the handle's stream and returns without waiting, so a
 * serving loop can keep placing batches back to back.  Outputs, and *status
 * (a DEVICE int32), are valid once the stream has reached the call.
 *
 * How many tile rounds a call takes depends on the data (a tile is cut where
 * its start-of-tile candidate lists cannot decide a query exactly), and a
 * stream cannot branch on it, so the call enqueues the rounds it needs when no
 * tile is cut plus spare_rounds (>= 0) more; rounds left over after the last
 * query do nothing.  *status is then
 *   ALD_OK           every query was decided (out_worker, out_diag complete);
 *   ALD_EINCOMPLETE  tiles were cut more often than spare_rounds allowed: the
 *                    queries before the stopping point are placed, the rest
 *                    are not yet (their out_worker entries are unwritten);
 *                    ald_place_resume finishes the call;
 *   ALD_EBLOCKED     an earlier asynchronous call on this handle was
 *                    unfinished or failed, so this call did nothing (issue it
 *                    again after ald_place_resume: arrival order is kept);
 *   ALD_EINVAL, ALD_ESLOTS, ALD_EOVERFLOW  as ald_place_stream returns them.
 * Query arrays and outputs must stay valid until the stream has reached the
 * call, or until ald_place_resume has returned if it stopped short.  Every
 * other call on the handle that uses the loaded workers (ald_place_stream,
 * ald_place_stream_hb, ald_place_grouped, ald_move_requests,
 * ald_worker_summary, ald_set_workspace) first waits for the stream and
 * returns ALD_EINCOMPLETE (changing nothing) while an asynchronous call is
 * unfinished, or the error of one that failed.  ald_place_stats is not updated by asynchronous calls.  Returns
 * ALD_EINVAL for a null status or spare_rounds outside [0, 2^20]. */
int ald_place_stream_async(ald_handle_t handle, int32_t Q, const int32_t* q_l_in, const int32_t* q_l_pred,
                           int32_t heartbeat_every, int32_t spare_rounds, int32_t* out_worker,
                           ald_query_diag_t* out_diag, int32_t* status);

/* Wait for the handle's stream and finish the asynchronous placement call
 * that stopped short (ALD_EINCOMPLETE), synchronously, with its own
 * arguments; the calls issued after it (ALD_EBLOCKED) are dropped and must be
 * issued again.  ALD_OK when nothing was unfinished; a device error of the
 * asynchronous calls (ALD_ESLOTS, ...) is returned here as well. */
int ald_place_resume(ald_handle_t handle);

/* As ald_place_stream, with heartbeats driven by the caller's clock instead
 * of a period: hb_before[q] >= 0 (host array [Q]) decode iterations run
 * before query q is placed, each one a heartbeat (one decode iteration on
 * every worker, finished requests leave, the TTFT window restarts).  With
 * arrival times t_q and one decode iteration per T_dec seconds,
 * hb_before[q] = floor(t_q / T_dec) - floor(t_{q-1} / T_dec) (the scheduler
 * places the requests that arrived since its last heartbeat, Sec. 4.2).
 * Counts continue ald_place_stream's stream; ALD_EINVAL for a negative count,
 * ALD_EOVERFLOW when the stream would run more decode iterations than the
 * 32-bit request state holds. */
int ald_place_stream_hb(ald_handle_t handle, int32_t Q, const int32_t* q_l_in, const int32_t* q_l_pred,
                        const int32_t* hb_before, int32_t* out_worker, ald_query_diag_t* out_diag);

/* Move K requests placed in the current heartbeat window (by calls since the
 * last heartbeat) between loaded workers, as if each had been placed on its
 * new worker: Algorithm 2 (Sec. 4.3) re-schedules new requests before they
 * run, and its moves (ald_rebalance) are applied with this call.  Host arrays
 * [K]: the requests' l_in and l_pred, and their workers from and to (global
 * indices, from != to).  A request is found on `from` by its lengths; moves
 * run in order.  The moved requests leave the source's prefill sums of
 * constraint (c) and join the destination's; with a decode history they start
 * at the destination's slack origin.  ALD_EINVAL when a request is not on its
 * worker in the current window, ALD_ESLOTS when a destination has no slot left;
 * then nothing changes.  The placements the caller recorded are the caller's
 * to update. */
int ald_move_requests(ald_handle_t handle, int32_t K, const int32_t* l_in, const int32_t* l_pred,
                      const int32_t* from, const int32_t* to);

/* Grouped placement (App. A, distributed scheduling): the loaded workers are
 * split into G consecutive groups of group_workers[g] workers (host array,
 * each >= 1, summing to W).  A router sends each arriving query to one group,
 * group g receiving the share group_workers[g] / W of the stream (App. A:
 * its arrival rate is N_g / N_w of the total): the deterministic quota method
 * of Balinski and Young, under which every group's count stays strictly
 * within one query of its share after every query, and equal groups take
 * turns (query x to group x mod G).  The router continues across calls while
 * the group sizes stay the same, and restarts with new sizes or a new load.
 * Each group places its own queries on its own workers in arrival order with
 * Algorithm 1, as its own scheduler would.  Heartbeats are the cluster's:
 * after every heartbeat_every processed queries of the whole stream (0 =
 * none), counted across calls as ald_place_stream does.  Device arrays as for
 * ald_place_stream; out_worker gets the global worker index (or -1) and
 * out_diag (or NULL) each query's diagnostics over its group's workers.
 * Grouped and ungrouped calls may alternate on one handle. */
int ald_place_grouped(ald_handle_t handle, int32_t G, const int32_t* group_workers, int32_t Q,
                      const int32_t* q_l_in, const int32_t* q_l_pred, int32_t heartbeat_every,
                      int32_t* out_worker, ald_query_diag_t* out_diag);

/* Scaling sweep (Sec. 4.4: the worker count needed for an arrival rate, found
 * by placing the stream on candidate clusters; Sec. 6.4: the GPUs needed to
 * meet every SLO): S scenarios (host array scen[S]), each starting with empty
 * workers, each placing the same Q queries (device arrays) with Algorithm 1
 * and no heartbeat.  Device outputs: out_rejected[S], out_first_reject[S] (-1
 * if none), if not NULL out_worker[S*Q] (row s = placement of scenario s), and
 * if not NULL out_min_gpus[2] = the answer: the fewest GPUs (n_workers *
 * gpus_per_worker) over scenarios with no rejection and that scenario's index
 * (lowest index on ties), or {-1, -1} when every scenario rejects something.
 * gpus_per_worker lies in [1, 256]; at most 2^24 - 1 scenarios.  The handle's
 * loaded workers are not touched (no ald_load_workers needed). */
int ald_sweep_scenarios(ald_handle_t handle, int32_t S, const ald_scenario_t* scen, int32_t Q,
                        const int32_t* q_l_in, const int32_t* q_l_pred, int32_t* out_rejected,
                        int32_t* out_first_reject, int32_t* out_worker, int64_t* out_min_gpus);

/* As ald_sweep_scenarios, with heartbeats (Sec. 4.2, placement per heartbeat):
 * scenario s runs one decode iteration on all its workers after every
 * heartbeat_every[s] processed queries (host array [S], >= 0; 0 = none), as
 * ald_place_stream does.  With one decode iteration per heartbeat and arrival
 * rate r, a period of r * T_dec queries stands for the stream arriving at r,
 * which gives the smallest cluster per arrival rate (Sec. 4.4, Eq. 7).
 * ALD_EOVERFLOW when a scenario would run more decode iterations than the
 * 32-bit request state holds. */
int ald_sweep_scenarios_hb(ald_handle_t handle, int32_t S, const ald_scenario_t* scen,
                           const int32_t* heartbeat_every, int32_t Q, const int32_t* q_l_in,
                           const int32_t* q_l_pred, int32_t* out_rejected, int32_t* out_first_reject,
                           int32_t* out_worker, int64_t* out_min_gpus);

/* The scaling sweep of Sec. 4.4 (ald_sweep_scenarios, or with heartbeat_every
 * non-NULL ald_sweep_scenarios_hb), stream-asynchronous: the call validates
 * its arguments, enqueues its work and returns without waiting; the host
 * arrays scen and heartbeat_every are read before it returns.  It enqueues
 * the rounds every scenario needs when no tile is cut, plus spare_rounds
 * (>= 0) more.  *status (a DEVICE int32), valid with the outputs once the
 * stream has reached the call, is ALD_OK; ALD_EINCOMPLETE when tiles were cut
 * more often than spare_rounds allowed (the outputs are not valid: run the
 * sweep again, synchronously or with more spare rounds; a sweep changes no
 * handle state, so nothing needs finishing); or the code the synchronous
 * sweep returns for a device error (ALD_EINVAL for a query length outside
 * [1, 2^24]).  The query arrays and outputs must stay valid until the stream
 * has reached the call, and the sweep's tables in the workspace stay in use
 * until then (a later call on the handle is ordered after it on the stream). */
int ald_sweep_scenarios_async(ald_handle_t handle, int32_t S, const ald_scenario_t* scen,
                              const int32_t* heartbeat_every, int32_t Q, const int32_t* q_l_in,
                              const int32_t* q_l_pred, int32_t spare_rounds, int32_t* out_rejected,
                              int32_t* out_first_reject, int32_t* out_worker, int64_t* out_min_gpus,
                              int32_t* status);

/* Algorithm 2 (Sec. 4.3): re-balance the new requests of a heartbeat against
 * the output-length prediction errors of the ongoing ones, for P independent
 * problems (clusters) at once.  Stateless: the loaded workers are not used.
 *
 * Per worker i, from its ongoing requests j:
 *   l_out_j > l_pred_j (decoding past the prediction): l^e_i += l_repred_j, b^e_i += 1
 *   l_real_j < l_pred_j (finished before it):          l^e_i += l_real_j - l_pred_j, b^e_i -= 1
 * The error line of Eq. 4 through (l^e_i, b^e_i) has distance
 * |k2 l^e_i + c2 b^e_i| / sqrt(k2^2 + c2^2) from the origin; divided by k2 it is
 * |c_i| / sqrt(1 + rho^2) with c_i = l^e_i + rho * b^e_i and rho = c2 / k2, the
 * real ratio (not rounded).  Moving new request j (predicted length l_pred_j)
 * from worker x to y moves l_pred_j and one batch slot of error:
 * c_x -= l_pred_j + rho, c_y += l_pred_j + rho.  The moves are greedy: while
 * some (placed request, other worker) pair lowers sum_i |c_i|, the pair that
 * lowers it most is applied (ties: lowest request, then lowest worker); a
 * request may move again after later moves, and unplaced requests (worker
 * -1) stay.  Every comparison is made exactly (each quantity is a + rho * b
 * for integers a, b, and its sign is taken without rounding error).  Every
 * move lowers the objective strictly, so the search ends; as a guard a
 * problem that would take more than 4 * (its new requests) + (its workers)
 * moves stops the call with ALD_EOVERFLOW (outputs then undefined).
 *
 * Host arrays: n_workers[P] (1 .. 4096), models[P] (only c2 and k2 are used:
 * k2 a normal double in (0, 2^900], c2 = 0 or normal in [0, 2^900],
 * c2 / k2 <= 1e9), old_offsets[P+1] and new_offsets[P+1] (CSR over the request
 * arrays, starting at 0; at most 8192 new requests per problem, fewer than
 * 2^30 requests in all).
 * Device arrays: old_worker, old_l_pred, old_l_out (tokens generated so far),
 * old_l_real (real output length, >= old_l_out), old_l_repred (re-predicted
 * output length) [old_offsets[P]]; new_l_pred [new_offsets[P]]; new_worker
 * [new_offsets[P]] in/out.  Worker indices are local to their problem; lengths
 * lie in [1, 2^24] (l_out and l_repred may be 0).
 * Device outputs (each may be NULL): out_le, out_be [sum n_workers] (final
 * errors, problem p's workers after those of problems < p); out_moves[P];
 * out_log[2 * P * log_cap] (problem p's first log_cap moves in order as
 * (request, target) pairs starting at entry 2 * p * log_cap; log_cap >= 0);
 * out_obj[4P] (sum |c_i| before and after, each as the pair (a, b) meaning
 * a + rho * b: entries 4p .. 4p+3 = a_before, b_before, a_after, b_after).
 * ALD_EINVAL for a bad argument or any invalid request; then new_worker is
 * left unchanged. */
int ald_rebalance(ald_handle_t handle, int32_t P, const int32_t* n_workers, const ald_model_t* models,
                  const int64_t* old_offsets, const int32_t* old_worker, const int32_t* old_l_pred,
                  const int32_t* old_l_out, const int32_t* old_l_real, const int32_t* old_l_repred,
                  const int64_t* new_offsets, const int32_t* new_l_pred, int32_t* new_worker,
                  int64_t* out_le, int64_t* out_be, int32_t* out_moves, int32_t log_cap, int32_t* out_log,
                  int64_t* out_obj);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * computation and arguments as ald_rebalance, with every table in a fixed
 * device array of the library (about 1 MB per device, set up by ald_create
 * and held until the process ends) instead of handle memory.  It calls no
 * hipMalloc or hipFree.  out_le and out_be must be given (ALD_EINVAL
 * otherwise); at most 4096 problems and 32767 chunks of ongoing requests (a
 * problem's ongoing requests fill chunks of 1024; ALD_EINVAL beyond).  Every
 * call on one device shares that device's array and leaves its contents
 * behind; calls that overlap on one device (other streams or threads) race. */
int ald_rebalance_noalloc(ald_handle_t handle, int32_t P, const int32_t* n_workers, const ald_model_t* models,
                          const int64_t* old_offsets, const int32_t* old_worker, const int32_t* old_l_pred,
                          const int32_t* old_l_out, const int32_t* old_l_real, const int32_t* old_l_repred,
                          const int64_t* new_offsets, const int32_t* new_l_pred, int32_t* new_worker,
                          int64_t* out_le, int64_t* out_be, int32_t* out_moves, int32_t log_cap, int32_t* out_log,
                          int64_t* out_obj);

/* Current state of every loaded worker (device arrays of W), the quantities of
 * Table 1 that the constraints read: batch size B_i, sum of contexts (input
 * plus generated tokens), sum of remaining lengths (predicted minus generated),
 * and the KV peak over future iterations that constraint (e) compares with the
 * capacity m_i.  Brings every worker to the current decode iteration first. */
int ald_worker_summary(ald_handle_t handle, int32_t* B, int64_t* sum_c, int64_t* sum_r, int64_t* peak);

/* Kernel timing with HIP events on the handle's stream (off by default).
 * kind: 0 = state build, 1 = pair evaluation, 2 = per-query selection,
 * 3 = commit, 4 = re-balancing (both of its kernels).  `kinds` is a bit mask
 * of the kinds to time (bit k = kind k, 31 = all, 0 = off; anything else
 * outside 0..31 is ALD_EINVAL).  Each timed
 * launch records two events, so time only what is needed.  Totals accumulate
 * over calls while enabled; a nonzero mask resets them.  ald_kernel_time
 * gives the total and the launches of one kind so far; with launches of
 * asynchronous calls still timed on the stream it first waits for the stream.
 * A sweep's kernels are timed the same way (the kinds above). */
int ald_set_profiling(ald_handle_t handle, int32_t kinds);
int ald_kernel_time(ald_handle_t handle, int32_t kind, double* total_ms, int64_t* launches);

/* Tile statistics of the handle's last successful placement call
 * (ald_place_stream, ald_place_stream_hb, ald_place_grouped,
 * ald_sweep_scenarios, ald_sweep_scenarios_hb), summed over scenarios, into the
 * host array out[4]: [0] commit rounds run, [1] tiles cut before their end
 * (the candidate lists published at tile start could no longer decide a query
 * exactly, 64 workers had changed, or the stale-scan budget ran out),
 * [2] decisions that scanned the tile-start bit words of the untouched workers
 * instead of cutting, [3] tiles cut on the stale-scan budget.  Placements
 * never depend on these figures; they describe how the arrival-order commit of
 * Algorithm 1 (Sec. 4.2) was split into speculative tiles.  After a failed
 * call the figures are unspecified. */
int ald_place_stats(ald_handle_t handle, int64_t* out);

/* Message for the last error on this handle, or for a code. */
const char* ald_last_error(ald_handle_t handle);
const char* ald_strerror(int code);

#ifdef __cplusplus
}
#endif

#endif /* ALADDIN_H */
