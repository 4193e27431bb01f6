/*
 * Oracle for the SLO- and KV-aware query placement of Aladdin
 * (Nie, Fonseca, Liu: "Aladdin: Joint Placement and Scaling for SLO-Aware LLM
 * Serving", arXiv 2405.06856).
 *
 * TEST INFRASTRUCTURE ONLY.  This is the plain, slow, single-threaded CPU
 * reference that the GPU library is checked against.  Only the test suite, the
 * smoke check and the CPU-baseline leg of the benchmark load it; the product
 * path never does.  It shares no code, header or table with the GPU library.
 *
 * Arithmetic: token counts in int64, latencies in IEEE fp64 with the
 * parenthesisation written below; build with -ffp-contract=off and without
 * fast-math so every fp64 result is one correctly rounded operation.
 *
 * What is computed, per arriving query q = (l_in, l_pred), in arrival order:
 *
 *  KV model, Eq. 1 with h = 1, j = 0: a request with input l_in that has
 *  generated g tokens holds c = l_in + g tokens and will decode r = l_pred - g
 *  more iterations.  Constraint (e) with the footprint vector w of Sec. 4.2
 *  (w = [kv(l_in), kv(l_in+1), ..., kv(l_in+l_pred), 0, ...]) means: at future
 *  iteration t = 0, 1, ... a request holds c + t tokens while t <= r and none
 *  afterwards.  The worker's KV demand is the element-wise sum of those vectors
 *  and must stay <= M at every t.
 *
 *  Decode constraint (b): Eq. 4 bounds the batch's total context by
 *  (T_dec - c3 - c2*b)/k2; with the strictness knob gamma the context of a
 *  request counts as l_in + gamma*l_out, where (reading of Table 1 and the
 *  gamma explanation) l_out is split into tokens already generated and tokens
 *  still to come: D = c + gamma*r.  The check is written multiplied out:
 *      k2 * sum(D)  <=  theta * ((T_dec - c3) - c2*b),   b = batch size.
 *
 *  TTFT constraint (c): the prefill of all requests placed on the worker
 *  during the current heartbeat (plus q) must finish within T_pre:
 *      (c1 + k1*S1) + k1q*S2 <= T_pre,  S1 = sum l_in, S2 = sum l_in^2.
 *  (Eq. 2 is the k1q = 0 case.)
 *
 *  Algorithm 1: sort workers by capacity_norm = ||(B, sum(D))||_2 from large
 *  to small and place q on the first worker meeting (b), (c), (e); the
 *  comparison is done exactly on the integer 2^(2*gs) * capacity_norm^2 with
 *  gamma = gn / 2^gs, ties to the lowest worker index.  With a fixed worker
 *  pool, "open a new bin" is a rejection (worker -1, state unchanged).
 *
 *  Heartbeat: after every H processed queries (H > 0) every worker runs one
 *  decode iteration: c += 1, r -= 1, requests with r < 0 leave, and the
 *  per-heartbeat prefill sums S1, S2 restart at zero.
 *
 *  Constraint (d), evaluated when the caller gives each resident's decode time
 *  so far: prefill preempts the decoding of the ongoing requests, so the
 *  prefill time of the heartbeat's new requests (the same t_p as in (c)) may
 *  not exceed theta times the smallest time an ongoing request has saved
 *  against the ATGT limit:  t_p <= theta * min_j (T_dec * g_j - t_dec_j), with
 *  g_j the tokens generated so far.  Ongoing = residents and requests placed in
 *  earlier heartbeats; a worker with none has no such limit.  At a heartbeat a
 *  worker's decode iteration takes t_iter = (c3 + c2*b) + k2*sum(c) (Eq. 3, b
 *  the batch and sum(c) its total context before the iteration); every request
 *  in it gains one token and t_iter of decode time, so its slack
 *  T_dec*g - t_dec grows by T_dec - t_iter, the same for all of them.  The
 *  worker keeps that running gain as phi and each request its slack minus phi
 *  (s0): slack = s0 + phi.  A request placed in heartbeat window h starts
 *  decoding at the end of h with zero slack, so s0 = -phi at placement (phi
 *  does not change within a window).
 *
 *  Split-phase serving (Sec. 5): a decode worker receives requests whose
 *  prefill ran elsewhere, so only (b) and (e) apply; an infinite TTFT SLO
 *  marks such workers.
 *
 *  Algorithm 2 (ora_rebalance, at the end of this file): per-worker errors of
 *  the output-length predictions and greedy moves of the new requests that
 *  lower the summed distance of the workers' error lines from the origin.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORA_OK 0
#define ORA_EINVAL -1
#define ORA_ENOMEM -2
#define ORA_EOVERFLOW -3
#define ORA_ECHECK -4

typedef struct {
    double c1, k1, k1q;
    double c3, c2, k2;
    double ttft_slo, decode_slo;
    double theta;
    int32_t gamma_num, gamma_log2den;
} ora_model_t;

typedef struct {
    int64_t M;          /* KV capacity in tokens */
    int64_t n, cap;     /* number of requests, allocated length */
    int64_t *c, *r;     /* current context, remaining iterations; sorted by r descending */
    double* s0;         /* per request: slack minus phi (constraint (d)) */
    int64_t* win;       /* per request: heartbeat window it was placed in (-1: resident) */
    int64_t SC, SR;     /* sum of c and sum of r over the requests */
    int64_t S1, S2;     /* prefill sums of requests placed in this heartbeat */
    double phi;         /* running slack gain of the ongoing requests (constraint (d)) */
} worker_t;

typedef struct {
    int rc;
    int feasible, kv_ok, dec_ok, ttft_ok, pre_ok, near_tie;
    int64_t peak;
    double lhs, rhs, ttft, tdec;
    unsigned __int128 key;
} pair_t;

/* ------------------------------------------------------------------ */
/* KV peak: max over t >= 0 of sum over requests alive at t of (c + t).
 * Between two consecutive remaining lengths the alive set is fixed and the sum
 * grows with t, so the maximum sits at one of the request end points t = r_j.
 * The requests are visited in descending r; once every request with r >= t
 * has been added, the running sums give the demand at t.  The optional extra
 * request (cq, rq) joins at its own end point. */
#define DEMAND_AT(t) do { int64_t d_ = sumc + cnt * (t); peak = d_ > peak ? d_ : peak; } while (0)
static int64_t kv_peak(const worker_t* w, int has_q, int64_t cq, int64_t rq)
{
    const int64_t n = w->n;
    const int64_t* c = w->c;
    const int64_t* r = w->r;
    int64_t sumc = 0, cnt = 0, peak = 0;
    int64_t i = 0;
    if (has_q) {
        /* requests that end after q */
        for (; i < n && r[i] > rq; ++i) {
            sumc += c[i]; cnt += 1;
            if (i + 1 == n || r[i + 1] != r[i]) DEMAND_AT(r[i]);
        }
        /* q's end point, together with every request ending at the same time */
        for (; i < n && r[i] == rq; ++i) { sumc += c[i]; cnt += 1; }
        sumc += cq; cnt += 1;
        DEMAND_AT(rq);
    }
    /* requests that end before q */
    for (; i < n; ++i) {
        sumc += c[i]; cnt += 1;
        if (i + 1 == n || r[i + 1] != r[i]) DEMAND_AT(r[i]);
    }
    return peak;
}
#undef DEMAND_AT

static int near(double x, double y)
{
    double m = fmax(fabs(x), fabs(y));
    return fabs(x - y) <= 1e-9 * m;
}

/* One (query, worker) evaluation; returns ORA_EOVERFLOW when an integer
 * quantity leaves the range where its fp64 conversion is exact.  use_d: the
 * decode history is known and (d) is checked; hb: the current heartbeat
 * window. */
static int eval_pair(const worker_t* w, const ora_model_t* m, int64_t lin, int64_t lpred, int use_d, int64_t hb,
                     pair_t* o)
{
    const int gs = m->gamma_log2den;
    const int64_t gn = m->gamma_num;
    const int64_t SC = w->SC, SR = w->SR;
    const int64_t B = w->n;
    const int64_t b = B + 1;

    /* (e) KV capacity */
    o->peak = kv_peak(w, 1, lin, lpred);
    o->kv_ok = o->peak <= w->M;

    /* (b) decode: sum(D) = sum(c) + gamma*sum(r), held exactly as DS * 2^-gs */
    const int64_t DS = SC * ((int64_t)1 << gs) + gn * SR;
    const int64_t DSq = DS + lin * ((int64_t)1 << gs) + gn * lpred;
    if (DSq >= ((int64_t)1 << 53)) return ORA_EOVERFLOW;
    const double sumD = ldexp((double)DSq, -gs);
    o->lhs = m->k2 * sumD;
    o->rhs = m->theta * ((m->decode_slo - m->c3) - m->c2 * (double)b);
    o->dec_ok = o->lhs <= o->rhs;

    /* (c) TTFT of this heartbeat's prefill batch including q.  A decode
     * worker of split-phase serving (Sec. 5) runs no prefill: an infinite
     * T_pre marks it, and then neither (c) nor (d) applies. */
    const int decode_only = isinf(m->ttft_slo);
    const int64_t S1 = w->S1 + lin;
    const int64_t S2 = w->S2 + lin * lin;
    if (S2 >= ((int64_t)1 << 53)) return ORA_EOVERFLOW;
    o->ttft = (m->c1 + m->k1 * (double)S1) + m->k1q * (double)S2;
    o->ttft_ok = decode_only || o->ttft <= m->ttft_slo;

    /* (d) the same prefill time against the ongoing requests' smallest slack */
    o->pre_ok = 1;
    int pre_near = 0;
    if (use_d && !decode_only) {
        int any = 0;
        double smin = 0.0;
        for (int64_t i = 0; i < w->n; ++i) {
            if (w->win[i] >= hb) continue;  /* placed in this heartbeat: not decoding yet */
            const double slack = w->s0[i] + w->phi;
            if (!any || slack < smin) smin = slack;
            any = 1;
        }
        if (any) {
            const double lim = m->theta * smin;
            o->pre_ok = o->ttft <= lim;
            pre_near = near(o->ttft, lim);
        }
    }

    o->feasible = o->kv_ok && o->dec_ok && o->ttft_ok && o->pre_ok;
    o->tdec = (m->c3 + m->c2 * (double)b) + m->k2 * sumD;
    o->near_tie = near(o->lhs, o->rhs) || (!decode_only && near(o->ttft, m->ttft_slo)) || pre_near;

    /* rank key of Algorithm 1, before placement */
    const unsigned __int128 x = (unsigned __int128)(B * ((int64_t)1 << gs));
    const unsigned __int128 y = (unsigned __int128)(DS < 0 ? -DS : DS);
    o->key = x * x + y * y;
    if (o->key >= ((unsigned __int128)1 << 63)) return ORA_EOVERFLOW;
    return ORA_OK;
}

/* (key, -index) comparison: does worker a rank strictly before worker b? */
static int ranks_before(unsigned __int128 ka, int a, unsigned __int128 kb, int b)
{
    if (ka != kb) return ka > kb;
    return a < b;
}

static unsigned __int128* g_sort_keys;
static int cmp_rank(const void* pa, const void* pb)
{
    int a = *(const int*)pa, b = *(const int*)pb;
    if (ranks_before(g_sort_keys[a], a, g_sort_keys[b], b)) return -1;
    if (ranks_before(g_sort_keys[b], b, g_sort_keys[a], a)) return 1;
    return 0;
}

static int add_request(worker_t* w, int64_t c, int64_t r, double s0, int64_t win)
{
    if (w->n == w->cap) {
        int64_t nc = w->cap ? 2 * w->cap : 16;
        int64_t* cc = (int64_t*)realloc(w->c, (size_t)nc * sizeof(int64_t));
        if (!cc) return ORA_ENOMEM;
        w->c = cc;
        int64_t* rr = (int64_t*)realloc(w->r, (size_t)nc * sizeof(int64_t));
        if (!rr) return ORA_ENOMEM;
        w->r = rr;
        double* ss = (double*)realloc(w->s0, (size_t)nc * sizeof(double));
        if (!ss) return ORA_ENOMEM;
        w->s0 = ss;
        int64_t* ww = (int64_t*)realloc(w->win, (size_t)nc * sizeof(int64_t));
        if (!ww) return ORA_ENOMEM;
        w->win = ww;
        w->cap = nc;
    }
    /* keep r descending: insert after every request with r >= the new one */
    int64_t pos = w->n;
    while (pos > 0 && w->r[pos - 1] < r) pos -= 1;
    memmove(w->c + pos + 1, w->c + pos, (size_t)(w->n - pos) * sizeof(int64_t));
    memmove(w->r + pos + 1, w->r + pos, (size_t)(w->n - pos) * sizeof(int64_t));
    memmove(w->s0 + pos + 1, w->s0 + pos, (size_t)(w->n - pos) * sizeof(double));
    memmove(w->win + pos + 1, w->win + pos, (size_t)(w->n - pos) * sizeof(int64_t));
    w->c[pos] = c;
    w->r[pos] = r;
    w->s0[pos] = s0;
    w->win[pos] = win;
    w->n += 1;
    w->SC += c;
    w->SR += r;
    return ORA_OK;
}

static void heartbeat(worker_t* w, const ora_model_t* m)
{
    /* the iteration's time, from the batch before it (constraint (d)'s slack gain) */
    if (w->n > 0) {
        const double t_iter = (m->c3 + m->c2 * (double)w->n) + m->k2 * (double)w->SC;
        w->phi = w->phi + (m->decode_slo - t_iter);
    }
    int64_t keep = 0, SC = 0, SR = 0;
    for (int64_t i = 0; i < w->n; ++i) {
        w->c[i] += 1;
        w->r[i] -= 1;
        if (w->r[i] >= 0) { keep = i + 1; SC += w->c[i]; SR += w->r[i]; }  /* finished ones form the tail */
    }
    w->n = keep;
    w->SC = SC;
    w->SR = SR;
    w->S1 = 0;
    w->S2 = 0;
}

static void free_workers(worker_t* ws, int32_t W)
{
    if (!ws) return;
    for (int32_t i = 0; i < W; ++i) { free(ws[i].c); free(ws[i].r); free(ws[i].s0); free(ws[i].win); }
    free(ws);
}

static int valid_model(const ora_model_t* m)
{
    if (!(isfinite(m->c1) && isfinite(m->k1) && isfinite(m->k1q) && isfinite(m->c3) &&
          isfinite(m->c2) && isfinite(m->k2) && (isfinite(m->ttft_slo) || m->ttft_slo == INFINITY) &&
          isfinite(m->decode_slo) && isfinite(m->theta))) return 0;
    if (m->gamma_log2den < 0 || m->gamma_log2den > 8) return 0;
    if (m->gamma_num < 0 || m->gamma_num > (1 << m->gamma_log2den)) return 0;
    return 1;
}

/*
 * Place a stream of queries.
 *   W workers with capacities M[W]; residents in CSR form (res_off[W+1]) with
 *   input length, predicted output length and tokens generated so far, and
 *   optionally their decode time so far in seconds (res_tdec; NULL: constraint
 *   (d) is not evaluated).
 *   H: heartbeat period in processed queries (0 = none).
 *   no_commit: evaluate every query against the initial state and commit
 *   nothing (used to sample a stream in which no query is ever placed).
 *   check: also run Algorithm 1 literally (sort by rank, first feasible) and
 *   verify after each commit that the worker's new KV peak equals the
 *   evaluated one; returns ORA_ECHECK on any disagreement.
 *   n_threads: threads for the per-worker evaluations of one query (they are
 *   independent; every reduction over workers stays sequential).
 * Outputs (any may be NULL): worker per query (-1 = rejected) and diagnostics;
 * final per-worker batch size, sum(c), sum(r), KV peak, S1, S2.
 */
/* Move the request of query j (placed in the current heartbeat window hb on
 * worker wk[j]) to worker y, as if it had been placed there: it leaves x's
 * request list and prefill sums and joins y's, with y's slack origin for (d). */
static int move_request(worker_t* ws, int32_t W, int32_t* wk, const int64_t* win_of, const int32_t* q_lin,
                        const int32_t* q_lpred, int64_t hb, int32_t j, int32_t y)
{
    const int32_t x = wk[j];
    if (x < 0 || y < 0 || y >= W || x == y || win_of[j] != hb) return ORA_EINVAL;
    worker_t* w = &ws[x];
    const int64_t lin = q_lin[j], lp = q_lpred[j];
    int64_t i = 0;
    while (i < w->n && !(w->c[i] == lin && w->r[i] == lp && w->win[i] == hb)) ++i;
    if (i == w->n) return ORA_EINVAL;
    memmove(w->c + i, w->c + i + 1, (size_t)(w->n - i - 1) * sizeof(int64_t));
    memmove(w->r + i, w->r + i + 1, (size_t)(w->n - i - 1) * sizeof(int64_t));
    memmove(w->s0 + i, w->s0 + i + 1, (size_t)(w->n - i - 1) * sizeof(double));
    memmove(w->win + i, w->win + i + 1, (size_t)(w->n - i - 1) * sizeof(int64_t));
    w->n -= 1;
    w->SC -= lin;
    w->SR -= lp;
    w->S1 -= lin;
    w->S2 -= lin * lin;
    worker_t* v = &ws[y];
    const int rc = add_request(v, lin, lp, -v->phi, hb);
    if (rc) return rc;
    v->S1 += lin;
    v->S2 += lin * lin;
    wk[j] = y;
    return ORA_OK;
}

/*
 * App. A: a router sends each arriving query to one group of workers, group i
 * (N_i workers of N_w) receiving the share N_i / N_w of the stream.  The
 * deterministic round robin used here is the quota method of Balinski and
 * Young: the h-th query (h = 1, 2, ...) goes to the group with the largest
 * N_i / (a_i + 1) among the groups whose count a_i (queries received so far)
 * is still below h * N_i / N_w, ties to the lowest group index.  Every count
 * then stays strictly within one query of its share h * N_i / N_w, and with
 * equal sizes query x goes to group x mod G.  counts[G] carries the router's
 * state from query to query.
 */
static int32_t route_next(int32_t G, const int32_t* N, int64_t Nw, int64_t* counts)
{
    int64_t h = 1;
    for (int32_t i = 0; i < G; ++i) h += counts[i];
    int32_t best = -1;
    for (int32_t i = 0; i < G; ++i) {
        if (!(counts[i] * Nw < h * (int64_t)N[i])) continue;  /* at its upper quota already */
        if (best < 0 || (int64_t)N[i] * (counts[best] + 1) > (int64_t)N[best] * (counts[i] + 1)) best = i;
    }
    counts[best] += 1;
    return best;
}

/* The groups of the first Q queries (out_group[Q]) for group sizes N[G]. */
int ora_route_groups(int32_t G, const int32_t* N, int32_t Q, int32_t* out_group)
{
    if (G < 1 || Q < 0 || !N || !out_group) return ORA_EINVAL;
    int64_t Nw = 0;
    for (int32_t i = 0; i < G; ++i) { if (N[i] < 1) return ORA_EINVAL; Nw += N[i]; }
    int64_t* counts = (int64_t*)calloc((size_t)G, sizeof(int64_t));
    if (!counts) return ORA_ENOMEM;
    for (int32_t q = 0; q < Q; ++q) out_group[q] = route_next(G, N, Nw, counts);
    free(counts);
    return ORA_OK;
}

static int place_impl(int32_t W, const int64_t* M, const int64_t* res_off,
                      const int32_t* res_lin, const int32_t* res_lpred, const int32_t* res_g, const double* res_tdec,
                      const ora_model_t* model, int32_t Q, const int32_t* q_lin, const int32_t* q_lpred,
                      int32_t H, const int32_t* hb_before, int32_t n_moves, const int32_t* mv_at,
                      const int32_t* mv_query, const int32_t* mv_to, int32_t G, const int32_t* gsizes,
                      int32_t no_commit, int32_t check, int32_t n_threads,
                      int32_t* out_worker, int32_t* out_nfeas, int32_t* out_near_tie,
                      int64_t* out_peak_chosen, int64_t* out_excess_min,
                      double* out_ttft_chosen, double* out_tdec_chosen,
                      int64_t* fin_B, int64_t* fin_SC, int64_t* fin_SR, int64_t* fin_peak,
                      int64_t* fin_S1, int64_t* fin_S2)
{
    if (W <= 0 || Q < 0 || H < 0 || !model || !valid_model(model)) return ORA_EINVAL;
    if (hb_before && H != 0) return ORA_EINVAL;
    for (int32_t q = 0; hb_before && q < Q; ++q)
        if (hb_before[q] < 0) return ORA_EINVAL;
    worker_t* ws = (worker_t*)calloc((size_t)W, sizeof(worker_t));
    pair_t* pr = (pair_t*)calloc((size_t)W, sizeof(pair_t));
    int* order = (int*)calloc((size_t)W, sizeof(int));
    unsigned __int128* keys = (unsigned __int128*)calloc((size_t)W, sizeof(unsigned __int128));
    int32_t* wk = NULL;     /* with moves: each query's worker */
    int64_t* win_of = NULL; /* and the window it was placed in */
    int64_t* gcount = NULL; /* grouped: the router's counts */
    int32_t* gfirst = NULL; /* grouped: first worker of each group (G + 1 entries) */
    int64_t Nw = 0;
    int rc = ORA_OK;
    if (!ws || !pr || !order || !keys) { rc = ORA_ENOMEM; goto done; }
    if (gsizes) {
        gcount = (int64_t*)calloc((size_t)G, sizeof(int64_t));
        gfirst = (int32_t*)calloc((size_t)G + 1, sizeof(int32_t));
        if (!gcount || !gfirst) { rc = ORA_ENOMEM; goto done; }
        for (int32_t g = 0; g < G; ++g) { Nw += gsizes[g]; gfirst[g + 1] = gfirst[g] + gsizes[g]; }
    }

    for (int32_t i = 0; i < W; ++i) {
        ws[i].M = M[i];
        for (int64_t k = res_off ? res_off[i] : 0; res_off && k < res_off[i + 1]; ++k) {
            int64_t lin = res_lin[k], lp = res_lpred[k], g = res_g[k];
            if (lin < 1 || lp < 1 || g < 0 || g >= lp) { rc = ORA_EINVAL; goto done; }
            double s0 = 0.0;  /* phi = 0 at load: s0 = the resident's slack */
            if (res_tdec) {
                if (!isfinite(res_tdec[k]) || res_tdec[k] < 0.0) { rc = ORA_EINVAL; goto done; }
                s0 = model->decode_slo * (double)g - res_tdec[k];
            }
            rc = add_request(&ws[i], lin + g, lp - g, s0, -1);
            if (rc) goto done;
        }
    }

    const int use_d = res_tdec != NULL;
    int64_t hb = 0;  /* heartbeat window */
    int32_t since_hb = 0;
    if (n_moves > 0) {  /* moves need each query's worker and placement window */
        wk = (int32_t*)malloc((size_t)(Q > 0 ? Q : 1) * sizeof(int32_t));
        win_of = (int64_t*)malloc((size_t)(Q > 0 ? Q : 1) * sizeof(int64_t));
        if (!wk || !win_of) { rc = ORA_ENOMEM; goto done; }
        for (int32_t q = 0; q < Q; ++q) { wk[q] = -1; win_of[q] = -1; }
    }
    int32_t next_move = 0;
    for (int32_t q = 0; q <= Q; ++q) {
        /* moves scheduled before query q (after the last query when q == Q) */
        while (next_move < n_moves && mv_at[next_move] == q) {
            if (mv_query[next_move] < 0 || mv_query[next_move] >= q) { rc = ORA_EINVAL; goto done; }
            rc = move_request(ws, W, wk, win_of, q_lin, q_lpred, hb, mv_query[next_move], mv_to[next_move]);
            if (rc) goto done;
            if (out_worker) out_worker[mv_query[next_move]] = mv_to[next_move];
            next_move += 1;
        }
        if (q == Q) break;
        const int64_t lin = q_lin[q], lp = q_lpred[q];
        if (lin < 1 || lp < 1) { rc = ORA_EINVAL; goto done; }
        /* heartbeats driven by the caller's clock: hb_before[q] decode
         * iterations (each its own heartbeat) run before query q */
        for (int32_t k = 0; hb_before && !no_commit && k < hb_before[q]; ++k) {
            for (int32_t i = 0; i < W; ++i) heartbeat(&ws[i], model);
            hb += 1;
        }
        /* grouped (App. A): the query's group's workers only */
        int32_t lo = 0, hi = W;
        if (gsizes) {
            const int32_t g = route_next(G, gsizes, Nw, gcount);
            lo = gfirst[g];
            hi = gfirst[g + 1];
        }
        int best = -1;
        int nfeas = 0;
        int64_t excess_min = INT64_MAX;
#ifdef _OPENMP
#pragma omp parallel for num_threads(n_threads > 0 ? n_threads : 1) schedule(static)
#endif
        for (int32_t i = lo; i < hi; ++i) pr[i].rc = eval_pair(&ws[i], model, lin, lp, use_d, hb, &pr[i]);
        for (int32_t i = lo; i < hi; ++i) {
            if (pr[i].rc) { rc = pr[i].rc; goto done; }
            nfeas += pr[i].feasible;
            int64_t ex = pr[i].peak - ws[i].M;
            if (ex < excess_min) excess_min = ex;
            /* exhaustive search: highest (key, -index) among feasible workers */
            if (pr[i].feasible && (best < 0 || ranks_before(pr[i].key, i, pr[best].key, best))) best = i;
        }
        if (check) {
            /* Algorithm 1 as written: sort bins by capacity_norm, first feasible */
            const int32_t n = hi - lo;
            for (int32_t k = 0; k < n; ++k) { order[k] = lo + k; keys[lo + k] = pr[lo + k].key; }
            g_sort_keys = keys;
            qsort(order, (size_t)n, sizeof(int), cmp_rank);
            int first = -1;
            for (int32_t k = 0; k < n; ++k) if (pr[order[k]].feasible) { first = order[k]; break; }
            if (first != best) { rc = ORA_ECHECK; goto done; }
        }
        /* near tie: any worker ranked at or above the choice (all, if rejected)
         * whose decode, TTFT or (d) margin is within 1e-9 relative */
        int nt = 0;
        for (int32_t i = lo; i < hi; ++i) {
            if (!pr[i].near_tie) continue;
            if (best < 0 || i == best || ranks_before(pr[i].key, i, pr[best].key, best)) { nt = 1; break; }
        }
        if (out_worker) out_worker[q] = best;
        if (out_nfeas) out_nfeas[q] = nfeas;
        if (out_near_tie) out_near_tie[q] = nt;
        if (out_excess_min) out_excess_min[q] = excess_min;
        if (out_peak_chosen) out_peak_chosen[q] = best >= 0 ? pr[best].peak : 0;
        if (out_ttft_chosen) out_ttft_chosen[q] = best >= 0 ? pr[best].ttft : 0.0;
        if (out_tdec_chosen) out_tdec_chosen[q] = best >= 0 ? pr[best].tdec : 0.0;

        if (best >= 0 && !no_commit) {
            worker_t* w = &ws[best];
            rc = add_request(w, lin, lp, -w->phi, hb);
            if (wk) { wk[q] = best; win_of[q] = hb; }
            if (rc) goto done;
            w->S1 += lin;
            w->S2 += lin * lin;
            if (check && kv_peak(w, 0, 0, 0) != pr[best].peak) { rc = ORA_ECHECK; goto done; }
        }
        if (H > 0 && !no_commit) {
            since_hb += 1;
            if (since_hb == H) {
                for (int32_t i = 0; i < W; ++i) heartbeat(&ws[i], model);
                since_hb = 0;
                hb += 1;
            }
        }
    }
    for (int32_t i = 0; i < W; ++i) {
        if (fin_B) fin_B[i] = ws[i].n;
        if (fin_SC) fin_SC[i] = ws[i].SC;
        if (fin_SR) fin_SR[i] = ws[i].SR;
        if (fin_peak) fin_peak[i] = kv_peak(&ws[i], 0, 0, 0);
        if (fin_S1) fin_S1[i] = ws[i].S1;
        if (fin_S2) fin_S2[i] = ws[i].S2;
    }
done:
    free_workers(ws, W);
    free(pr);
    free(order);
    free(keys);
    free(wk);
    free(win_of);
    free(gcount);
    free(gfirst);
    return rc;
}

typedef struct {
    int32_t n_workers;
    int32_t gpus_per_worker;
    int64_t kv_capacity;
    ora_model_t model;
} ora_scenario_t;

int ora_place(int32_t W, const int64_t* M, const int64_t* res_off,
              const int32_t* res_lin, const int32_t* res_lpred, const int32_t* res_g, const double* res_tdec,
              const ora_model_t* model, int32_t Q, const int32_t* q_lin, const int32_t* q_lpred,
              int32_t H, int32_t no_commit, int32_t check, int32_t n_threads,
              int32_t* out_worker, int32_t* out_nfeas, int32_t* out_near_tie,
              int64_t* out_peak_chosen, int64_t* out_excess_min,
              double* out_ttft_chosen, double* out_tdec_chosen,
              int64_t* fin_B, int64_t* fin_SC, int64_t* fin_SR, int64_t* fin_peak,
              int64_t* fin_S1, int64_t* fin_S2)
{
    return place_impl(W, M, res_off, res_lin, res_lpred, res_g, res_tdec, model, Q, q_lin, q_lpred, H, NULL,
                      0, NULL, NULL, NULL, 0, NULL, no_commit, check, n_threads, out_worker, out_nfeas, out_near_tie, out_peak_chosen,
                      out_excess_min, out_ttft_chosen, out_tdec_chosen, fin_B, fin_SC, fin_SR, fin_peak, fin_S1,
                      fin_S2);
}

/* As ora_place, with the heartbeats given per query instead of by a period:
 * hb_before[q] >= 0 decode iterations run before query q is placed. */
int ora_place_hb(int32_t W, const int64_t* M, const int64_t* res_off,
                 const int32_t* res_lin, const int32_t* res_lpred, const int32_t* res_g, const double* res_tdec,
                 const ora_model_t* model, int32_t Q, const int32_t* q_lin, const int32_t* q_lpred,
                 const int32_t* hb_before, int32_t check,
                 int32_t* out_worker, int32_t* out_nfeas, int32_t* out_near_tie,
                 int64_t* out_peak_chosen, int64_t* out_excess_min,
                 double* out_ttft_chosen, double* out_tdec_chosen,
                 int64_t* fin_B, int64_t* fin_SC, int64_t* fin_SR, int64_t* fin_peak,
                 int64_t* fin_S1, int64_t* fin_S2)
{
    if (!hb_before && Q > 0) return ORA_EINVAL;
    return place_impl(W, M, res_off, res_lin, res_lpred, res_g, res_tdec, model, Q, q_lin, q_lpred, 0, hb_before,
                      0, NULL, NULL, NULL, 0, NULL, 0, check, 1, out_worker, out_nfeas, out_near_tie, out_peak_chosen, out_excess_min,
                      out_ttft_chosen, out_tdec_chosen, fin_B, fin_SC, fin_SR, fin_peak, fin_S1, fin_S2);
}

/* As ora_place_hb (hb_before may be NULL: no heartbeat), with n_moves moves of
 * placed requests: before query mv_at[k] (mv_at non-decreasing; Q = after the
 * last query), the request of query mv_query[k], placed in the current
 * heartbeat window, moves to worker mv_to[k] as if it had been placed there
 * (out_worker records the move).  ORA_EINVAL for a move of a request that is
 * not in the current window. */
int ora_place_moves(int32_t W, const int64_t* M, const int64_t* res_off,
                    const int32_t* res_lin, const int32_t* res_lpred, const int32_t* res_g, const double* res_tdec,
                    const ora_model_t* model, int32_t Q, const int32_t* q_lin, const int32_t* q_lpred,
                    const int32_t* hb_before, int32_t n_moves, const int32_t* mv_at, const int32_t* mv_query,
                    const int32_t* mv_to, int32_t* out_worker, int32_t* out_nfeas, int32_t* out_near_tie,
                    int64_t* out_peak_chosen, int64_t* out_excess_min,
                    double* out_ttft_chosen, double* out_tdec_chosen,
                    int64_t* fin_B, int64_t* fin_SC, int64_t* fin_SR, int64_t* fin_peak,
                    int64_t* fin_S1, int64_t* fin_S2)
{
    if (n_moves < 0 || (n_moves > 0 && (!mv_at || !mv_query || !mv_to))) return ORA_EINVAL;
    for (int32_t k = 0; k < n_moves; ++k)
        if (mv_at[k] < 0 || mv_at[k] > Q || (k > 0 && mv_at[k] < mv_at[k - 1])) return ORA_EINVAL;
    return place_impl(W, M, res_off, res_lin, res_lpred, res_g, res_tdec, model, Q, q_lin, q_lpred, 0, hb_before,
                      n_moves, mv_at, mv_query, mv_to, 0, NULL, 0, 1, 1, out_worker, out_nfeas, out_near_tie,
                      out_peak_chosen, out_excess_min, out_ttft_chosen, out_tdec_chosen, fin_B, fin_SC, fin_SR,
                      fin_peak, fin_S1, fin_S2);
}

/* Grouped placement (App. A): the W workers form G consecutive groups of
 * gsizes[g] workers; each query goes to the group the router picks
 * (route_next, from the load on) and is placed with Algorithm 1 among that
 * group's workers only, as that group's own scheduler would; the diagnostics
 * are over the group's workers.  Heartbeats are the cluster's: after every H
 * processed queries of the whole stream (H = 0: none), every worker runs one
 * decode iteration. */
int ora_place_grouped(int32_t W, const int64_t* M, const int64_t* res_off,
                      const int32_t* res_lin, const int32_t* res_lpred, const int32_t* res_g, const double* res_tdec,
                      const ora_model_t* model, int32_t G, const int32_t* gsizes, int32_t Q, const int32_t* q_lin,
                      const int32_t* q_lpred, int32_t H, int32_t* out_worker, int32_t* out_nfeas,
                      int32_t* out_near_tie, int64_t* out_peak_chosen, int64_t* out_excess_min,
                      double* out_ttft_chosen, double* out_tdec_chosen,
                      int64_t* fin_B, int64_t* fin_SC, int64_t* fin_SR, int64_t* fin_peak,
                      int64_t* fin_S1, int64_t* fin_S2)
{
    if (G < 1 || !gsizes) return ORA_EINVAL;
    int64_t total = 0;
    for (int32_t g = 0; g < G; ++g) { if (gsizes[g] < 1) return ORA_EINVAL; total += gsizes[g]; }
    if (total != W) return ORA_EINVAL;
    return place_impl(W, M, res_off, res_lin, res_lpred, res_g, res_tdec, model, Q, q_lin, q_lpred, H, NULL,
                      0, NULL, NULL, NULL, G, gsizes, 0, 1, 1, out_worker, out_nfeas, out_near_tie,
                      out_peak_chosen, out_excess_min, out_ttft_chosen, out_tdec_chosen, fin_B, fin_SC, fin_SR,
                      fin_peak, fin_S1, fin_S2);
}

/*
 * Scaling sweep: every scenario starts with empty workers and places the same
 * query stream on its own, with a heartbeat after every H[s] processed queries
 * (H NULL or H[s] = 0: none).  Per scenario: number of rejected queries and
 * the index of the first rejection (-1 if none); optionally the full placement
 * (out_worker[s*Q + q]).
 */
int ora_sweep(int32_t S, const ora_scenario_t* scen, const int32_t* H, int32_t Q, const int32_t* q_lin,
              const int32_t* q_lpred, int32_t n_threads, int32_t* out_rejected,
              int32_t* out_first_reject, int32_t* out_worker)
{
    if (S < 0 || Q < 0) return ORA_EINVAL;
    int rc_all = ORA_OK;
    /* scenarios are independent; each one is placed sequentially */
#ifdef _OPENMP
#pragma omp parallel for num_threads(n_threads > 0 ? n_threads : 1) schedule(dynamic, 1)
#endif
    for (int32_t s = 0; s < S; ++s) {
        const int32_t W = scen[s].n_workers;
        int64_t* M = (int64_t*)malloc((size_t)(W > 0 ? W : 1) * sizeof(int64_t));
        int32_t* tmp = (int32_t*)malloc((size_t)(Q > 0 ? Q : 1) * sizeof(int32_t));
        int rc = (M && tmp) ? ORA_OK : ORA_ENOMEM;
        int32_t* dst = out_worker ? out_worker + (int64_t)s * Q : tmp;
        if (rc == ORA_OK) {
            for (int32_t i = 0; i < W; ++i) M[i] = scen[s].kv_capacity;
            rc = ora_place(W, M, NULL, NULL, NULL, NULL, NULL, &scen[s].model, Q, q_lin, q_lpred, H ? H[s] : 0, 0, 0, 1,
                           dst, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL);
        }
        if (rc == ORA_OK) {
            int32_t rej = 0, first = -1;
            for (int32_t q = 0; q < Q; ++q) if (dst[q] < 0) { if (first < 0) first = q; rej += 1; }
            out_rejected[s] = rej;
            out_first_reject[s] = first;
        } else {
#ifdef _OPENMP
#pragma omp critical
#endif
            rc_all = rc;
        }
        free(M);
        free(tmp);
    }
    return rc_all;
}

/* KV peak of an explicit request list (c, r), exposed for the unit tests. */
int64_t ora_kv_peak(int64_t n, const int64_t* c, const int64_t* r)
{
    worker_t w;
    memset(&w, 0, sizeof w);
    for (int64_t i = 0; i < n; ++i) if (add_request(&w, c[i], r[i], 0.0, -1)) return -1;
    int64_t p = kv_peak(&w, 0, 0, 0);
    free(w.c); free(w.r); free(w.s0); free(w.win);
    return p;
}

/* ------------------------------------------------------------------ */
/*
 * Algorithm 2 (Sec. 4.3): re-balancing new requests against output-length
 * prediction errors.
 *
 * Error of each worker i, from its ongoing requests j (the two tests of the
 * algorithm, applied literally):
 *   l_out_j > l_pred_j (still decoding past its prediction, under-estimate):
 *       l^e_i += l'^pred_j (the re-predicted output length),  b^e_i += 1
 *   l_real_j < l_pred_j (finished before its prediction, over-estimate):
 *       l^e_i += l_real_j - l_pred_j,                          b^e_i -= 1
 * Error line: Eq. 4 bounds k2 * (context) + c2 * (batch); the errors shift a
 * worker's operating point by (l^e, b^e), which moves its decode time by
 * k2 * l^e + c2 * b^e.  The line through that point parallel to Eq. 4's
 * boundary is k2 * l + c2 * b - (k2 * l^e + c2 * b^e) = 0, whose distance from
 * the origin is |k2 * l^e + c2 * b^e| / sqrt(k2^2 + c2^2).  Every worker of a
 * problem shares one model, so the denominator is common and the objective is
 * sum_i |c_i| with c_i = l^e_i + rho * b^e_i, rho = c2 / k2 the real ratio of
 * the two coefficients (not rounded).
 *
 * Exact arithmetic: every quantity the search compares is an integer pair
 * (a, b) standing for a + rho * b, so every comparison is the sign of
 * a * k2 + b * c2 (k2 > 0).  With |a|, |b| < 2^60 and k2, c2 doubles (53-bit
 * significands), each product has at most 113 significant bits and is exact
 * in IEEE binary128 (__float128); the rounded sum of two exact values is zero
 * only when the exact sum is zero and otherwise has its sign.  So rb_sign is
 * the exact sign.
 *
 * Moving a new request j (predicted length l_pred_j) from worker x to worker
 * y moves l_pred_j and one batch slot of error: c_x -= l_pred_j + rho,
 * c_y += l_pred_j + rho.  The search (the paper gives only the objective and
 * the move update): repeatedly apply the single move with the largest
 * decrease of sum |c_i| -- ties to the lowest request index, then the lowest
 * target worker -- while that decrease is positive.  A request may move
 * again after a later move has changed the errors; every applied move lowers
 * the objective strictly, so no assignment repeats and the search ends.  As a
 * guard it stops with ORA_EOVERFLOW after 4 * n_new + W moves (never reached
 * on the workloads).  New requests that were not placed (worker -1) stay.
 *
 * Inputs: W workers; n_old ongoing requests (worker, l_pred, l_out = tokens
 * generated so far, l_real = real output length, with l_out <= l_real, and
 * l_repred = the re-prediction); n_new new requests (l_pred, worker in/out).
 * Outputs (any may be NULL): final l^e, b^e per worker; number of moves; the
 * first log_cap moves in order (request, target); sum |c_i| before and after,
 * each as the pair (a, b) meaning a + rho * b.
 */
typedef struct { int64_t a, b; } rb_pair;  /* a + rho * b */

static int rb_sign(int64_t a, int64_t b, const ora_model_t* m)
{
    /* with b * c2 = 0, or both terms of one sign, the sign needs no arithmetic */
    if (b == 0 || m->c2 == 0.0) return (a > 0) - (a < 0);
    if (a == 0 || (a > 0) == (b > 0)) return b > 0 ? 1 : -1;
    const __float128 x = (__float128)a * (__float128)m->k2;
    const __float128 y = (__float128)b * (__float128)m->c2;
    const __float128 v = x + y;
    return (v > 0) - (v < 0);
}

static rb_pair rb_sub(rb_pair u, rb_pair v) { rb_pair r = {u.a - v.a, u.b - v.b}; return r; }
static rb_pair rb_add(rb_pair u, rb_pair v) { rb_pair r = {u.a + v.a, u.b + v.b}; return r; }
static rb_pair rb_abs(rb_pair u, const ora_model_t* m)
{
    if (rb_sign(u.a, u.b, m) < 0) { u.a = -u.a; u.b = -u.b; }
    return u;
}
static int rb_fits(rb_pair u) { const int64_t L = (int64_t)1 << 60; return u.a > -L && u.a < L && u.b > -L && u.b < L; }

/* Exact sign of a + (c2 / k2) * b, exposed for the unit tests. */
int ora_rb_sign(int64_t a, int64_t b, const ora_model_t* m) { return rb_sign(a, b, m); }

static int rb_model_ok(const ora_model_t* m)
{
    /* k2 > 0 and c2 >= 0 finite, rho = c2 / k2 at most 1e9 */
    return m->k2 > 0.0 && m->c2 >= 0.0 && isfinite(m->k2) && isfinite(m->c2) && m->c2 <= 1e9 * m->k2;
}

int ora_rebalance(int32_t W, const ora_model_t* m,
                  int32_t n_old, const int32_t* old_worker, const int32_t* old_lpred, const int32_t* old_lout,
                  const int32_t* old_lreal, const int32_t* old_lrepred,
                  int32_t n_new, const int32_t* new_lpred, int32_t* new_worker,
                  int64_t* out_le, int64_t* out_be, int32_t* out_moves, int32_t log_cap, int32_t* out_log,
                  int64_t* out_obj_before, int64_t* out_obj_after)
{
    const int32_t LMAX = 1 << 24;
    if (W < 1 || n_old < 0 || n_new < 0 || log_cap < 0 || !m || !new_worker) return ORA_EINVAL;
    if (!rb_model_ok(m)) return ORA_EINVAL;
    for (int32_t j = 0; j < n_old; ++j) {
        if (old_worker[j] < 0 || old_worker[j] >= W) return ORA_EINVAL;
        if (old_lpred[j] < 1 || old_lpred[j] > LMAX || old_lout[j] < 0 || old_lreal[j] < 1 ||
            old_lreal[j] > LMAX || old_lout[j] > old_lreal[j] || old_lrepred[j] < 0 || old_lrepred[j] > LMAX)
            return ORA_EINVAL;
    }
    for (int32_t j = 0; j < n_new; ++j)
        if (new_lpred[j] < 1 || new_lpred[j] > LMAX || new_worker[j] < -1 || new_worker[j] >= W) return ORA_EINVAL;

    rb_pair* c = (rb_pair*)calloc((size_t)W, sizeof(rb_pair));
    if (!c) return ORA_ENOMEM;

    /* the per-worker errors of the ongoing requests: c_i = (l^e_i, b^e_i) */
    for (int32_t j = 0; j < n_old; ++j) {
        const int32_t i = old_worker[j];
        if (old_lout[j] > old_lpred[j]) { c[i].a += old_lrepred[j]; c[i].b += 1; }
        if (old_lreal[j] < old_lpred[j]) { c[i].a += (int64_t)old_lreal[j] - old_lpred[j]; c[i].b -= 1; }
    }
    rb_pair obj = {0, 0};
    for (int32_t i = 0; i < W; ++i) obj = rb_add(obj, rb_abs(c[i], m));
    if (out_obj_before) { out_obj_before[0] = obj.a; out_obj_before[1] = obj.b; }

    /* greedy moves: every (placed request, other worker) pair, in
     * request-then-worker order, keeping the first largest decrease */
    const int64_t max_moves = 4 * (int64_t)n_new + W;
    int32_t moves = 0;
    int rc = ORA_OK;
    rb_pair* absc = (rb_pair*)calloc((size_t)W, sizeof(rb_pair));  /* |c_y| at the current step */
    if (!absc) { free(c); return ORA_ENOMEM; }
    for (;;) {
        rb_pair best = {0, 0};
        int32_t bj = -1, by = -1;
        for (int32_t y = 0; y < W; ++y) absc[y] = rb_abs(c[y], m);
        for (int32_t j = 0; j < n_new; ++j) {
            const int32_t x = new_worker[j];
            if (x < 0) continue;
            const rb_pair d = {new_lpred[j], 1};
            /* decrease of sum |c| = (|c_x| - |c_x - d|) + (|c_y| - |c_y + d|) */
            const rb_pair from_x = rb_sub(absc[x], rb_abs(rb_sub(c[x], d), m));
            for (int32_t y = 0; y < W; ++y) {
                if (y == x) continue;
                const rb_pair gain = rb_add(from_x, rb_sub(absc[y], rb_abs(rb_add(c[y], d), m)));
                const rb_pair diff = rb_sub(gain, best);
                if (!rb_fits(diff)) { rc = ORA_EOVERFLOW; goto done; }
                if (rb_sign(diff.a, diff.b, m) > 0) { best = gain; bj = j; by = y; }
            }
        }
        if (bj < 0) break;
        if (moves >= max_moves) { rc = ORA_EOVERFLOW; goto done; }
        const int32_t x = new_worker[bj];
        const rb_pair d = {new_lpred[bj], 1};
        c[x] = rb_sub(c[x], d);
        c[by] = rb_add(c[by], d);
        new_worker[bj] = by;
        if (out_log && moves < log_cap) { out_log[2 * moves] = bj; out_log[2 * moves + 1] = by; }
        moves += 1;
        obj = rb_sub(obj, best);
    }
    if (out_obj_after) { out_obj_after[0] = obj.a; out_obj_after[1] = obj.b; }
    if (out_moves) *out_moves = moves;
    for (int32_t i = 0; i < W; ++i) {
        if (out_le) out_le[i] = c[i].a;
        if (out_be) out_be[i] = c[i].b;
    }
done:
    free(c);
    free(absc);
    return rc;
}
