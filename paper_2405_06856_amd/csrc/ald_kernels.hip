// HIP kernels of libaladdin for gfx950 (MI355X): wave64, no matrix cores --
// the placement evaluator is integer/fp64 scan-and-reduce work.
//
// Per tile of T consecutive queries (one heartbeat segment at most):
//   k_build   rebuild the breakpoint summaries of workers whose live set moved
//   k_eval    every (query, worker) pair of the tile against the tile-start
//             state: KV peak (constraint (e)), decode (b), TTFT (c), near-tie
//             margins; feasibility / near-tie bits and per-block KV-excess minima
//   k_select  per query: best feasible workers by Algorithm 1's rank, counts,
//             the two smallest KV excesses, the best near-tie worker
//   k_commit  arrival-order commit: one block per scenario walks the tile,
//             re-evaluating only workers changed earlier in the same tile, and
//             cuts the tile when the tile-start lists cannot decide exactly;
//             extra blocks finalize the rejected prefix in parallel.
#include "ald_internal.h"

namespace ald {

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }
__device__ __forceinline__ int wave_id() { return threadIdx.x >> 6; }

struct OpAdd {
    __device__ int64_t operator()(int64_t a, int64_t b) const { return a + b; }
};
struct OpMax {
    __device__ int64_t operator()(int64_t a, int64_t b) const { return a > b ? a : b; }
};
struct OpMin {
    __device__ int64_t operator()(int64_t a, int64_t b) const { return a < b ? a : b; }
};

// Exclusive scan over the threads of the block (prefix: threads before, suffix:
// threads after) of one int64 per thread; *total gets the whole reduction.
// `lds` must hold NT/64 entries.  Contains two block barriers.
template <int NT, bool SUFFIX, typename Op>
__device__ int64_t block_scan_excl(int64_t v, int64_t ident, Op op, int64_t* total, int64_t* lds)
{
    const int lane = lane_id(), wid = wave_id();
    int64_t x = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        int64_t o = SUFFIX ? __shfl_down(x, d, 64) : __shfl_up(x, d, 64);
        bool ok = SUFFIX ? (lane + d < 64) : (lane >= d);
        if (ok) x = op(x, o);
    }
    int64_t ex = SUFFIX ? __shfl_down(x, 1, 64) : __shfl_up(x, 1, 64);
    if (SUFFIX ? lane == 63 : lane == 0) ex = ident;
    if (SUFFIX ? lane == 0 : lane == 63) lds[wid] = x;
    __syncthreads();
    int64_t carry = ident, tot = ident;
#pragma unroll
    for (int j = 0; j < NT / 64; ++j) {
        int64_t t = lds[j];
        tot = op(tot, t);
        if (SUFFIX ? j > wid : j < wid) carry = op(carry, t);
    }
    __syncthreads();
    *total = tot;
    return op(carry, ex);
}

template <int NT, typename Op>
__device__ int64_t block_reduce(int64_t v, int64_t ident, Op op, int64_t* lds)
{
    int64_t tot;
    block_scan_excl<NT, false>(v, ident, op, &tot, lds);
    return tot;
}

// first index in [lo, hi) with a[i] >= x (hi if none)
__device__ __forceinline__ int lower_bound_i32(const int32_t* a, int lo, int hi, int32_t x)
{
    int len = hi - lo;
    while (len > 0) {
        int half = len >> 1;
        int mid = lo + half;
        if (a[mid] < x) {
            lo = mid + 1;
            len = len - half - 1;
        } else {
            len = half;
        }
    }
    return lo;
}

// Algorithm 1 order: does (ka, a) rank strictly before (kb, b)?  An index < 0
// marks an absent entry, which ranks after every present one.
__device__ __forceinline__ bool ranks_before(uint64_t ka, int a, uint64_t kb, int b)
{
    const bool better = (ka > kb) | ((ka == kb) & (a < b));
    return (a >= 0) & ((b < 0) | better);
}

// Insert candidate (ck, cw) into a best-first list of N entries (cw < 0: no-op).
// Written as a compare-exchange chain of selects: no divergent branch touches
// the register-resident list.
template <int N>
__device__ __forceinline__ void topk_insert(uint64_t (&key)[N], int32_t (&idx)[N], uint64_t ck, int32_t cw)
{
#pragma unroll
    for (int k = 0; k < N; ++k) {
        const bool sw = ranks_before(ck, cw, key[k], idx[k]);
        const uint64_t ok = key[k];
        const int32_t ow = idx[k];
        key[k] = sw ? ck : ok;
        idx[k] = sw ? cw : ow;
        ck = sw ? ok : ck;
        cw = sw ? ow : cw;
    }
}

// Keep the two smallest (excess, index) pairs, ordered by excess ascending and
// then index descending.  y < 0: no candidate.
__device__ __forceinline__ void min2_insert(int32_t& ex1, int32_t& w1, int32_t& ex2, int32_t& w2, int32_t x, int32_t y)
{
    const bool present = y >= 0;
    const bool b1 = present & ((w1 < 0) | (x < ex1) | ((x == ex1) & (y > w1)));
    const bool b2 = present & !b1 & ((w2 < 0) | (x < ex2) | ((x == ex2) & (y > w2)));
    ex2 = b1 ? ex1 : (b2 ? x : ex2);
    w2 = b1 ? w1 : (b2 ? y : w2);
    ex1 = b1 ? x : ex1;
    w1 = b1 ? y : w1;
}

__device__ __forceinline__ bool near_tie(double x, double y)
{
    double m = fmax(fabs(x), fabs(y));
    return fabs(x - y) <= 1e-9 * m;
}

// Everything a pair evaluation needs from one worker.
struct View {
    const int32_t* e;
    const int32_t* pme;
    const int32_t* sm;
    const int32_t* ss;
    int32_t head, n, M;
    int64_t DS, S1, S2;
    uint64_t key;
    double rhs;
};

__device__ __forceinline__ View load_view(const State& st, int gw, int32_t hb)
{
    View v;
    const int64_t base = st.slot_base[gw];
    v.e = st.e + base;
    v.pme = st.pme + base;
    v.sm = st.sm + base;
    v.ss = st.ss + base;
    v.head = st.head[gw];
    v.n = st.n[gw];
    v.M = st.M[gw];
    v.DS = st.DS[gw];
    const bool cur = st.hbs[gw] == hb;
    v.S1 = cur ? st.S1[gw] : 0;
    v.S2 = cur ? st.S2[gw] : 0;
    v.key = st.key[gw];
    v.rhs = st.rhs[gw];
    return v;
}

// KV demand peak of the worker with the query (sq = l_in - tau, eq = l_pred + tau) added.
__device__ __forceinline__ int64_t kv_peak_with(const View& v, int32_t sq, int32_t eq)
{
    const int l = lower_bound_i32(v.e, v.head, v.n, eq);
    const int64_t a = (int64_t)v.pme[l] + sq;
    const int64_t b = (int64_t)v.sm[l];
    const int64_t c = (int64_t)v.ss[l] + (int64_t)(v.n - l) * eq + sq + eq;
    int64_t p = a > b ? a : b;
    return p > c ? p : c;
}

struct Latency {
    double lhs, ttft, tdec;
    bool dec_ok, ttft_ok, nt;
};

// Decode constraint (b) and TTFT constraint (c) of one pair.
__device__ __forceinline__ Latency latency(const Scen& sc, const View& v, int32_t lin, int32_t lp, int32_t b)
{
    Latency o;
    const int64_t DSq = v.DS + ((int64_t)lin << sc.gs) + (int64_t)sc.gn * lp;
    const double sumD = ldexp((double)DSq, -sc.gs);
    o.lhs = sc.k2 * sumD;
    o.dec_ok = o.lhs <= v.rhs;
    const int64_t S1 = v.S1 + lin;
    const int64_t S2 = v.S2 + (int64_t)lin * lin;
    o.ttft = (sc.c1 + sc.k1 * (double)S1) + sc.k1q * (double)S2;
    o.ttft_ok = o.ttft <= sc.ttft;
    o.nt = near_tie(o.lhs, v.rhs) || near_tie(o.ttft, sc.ttft);
    o.tdec = (sc.c3 + sc.c2 * (double)b) + sc.k2 * sumD;
    return o;
}

// Scenario owning block `blk` given each scenario's first block (field offset).
template <int32_t Scen::*FIRST>
__device__ __forceinline__ int find_scen(const State& st, int blk)
{
    int lo = 0, hi = st.S - 1;
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if (st.scen[mid].*FIRST <= blk) lo = mid; else hi = mid - 1;
    }
    return lo;
}

__device__ __forceinline__ int find_scen_by_worker(const State& st, int gw)
{
    int lo = 0, hi = st.S - 1;
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if (st.scen[mid].wbase <= gw) lo = mid; else hi = mid - 1;
    }
    return lo;
}

__device__ __forceinline__ void raise_error(int32_t* err, int32_t code)
{
    atomicCAS(err, 0, code);
}

// ---------------------------------------------------------------------------------------------
// Breakpoint summaries of one worker (whole block).  Drops finished requests
// (e < tau), recomputes ss / pme / sm over the live slots and the worker's
// aggregates.  Called with every thread of a BUILD_THREADS block.
__device__ void build_worker(const State& st, const Scen& sc, int gw, int32_t tau, int32_t* err)
{
    constexpr int NT = BUILD_THREADS;
    __shared__ int64_t red[NT / 64];
    const int tid = threadIdx.x;
    const int64_t base = st.slot_base[gw];
    int32_t* e = st.e + base;
    int32_t* s = st.s + base;
    int32_t* ss = st.ss + base;
    int32_t* pme = st.pme + base;
    int32_t* sm = st.sm + base;
    const int n = st.n[gw];
    int head = st.head[gw];

    // finished requests form a prefix of the live range (sorted by e)
    int64_t fin = 0;
    for (int k = head + tid; k < n; k += NT) fin += (e[k] < tau) ? 1 : 0;
    head += (int)block_reduce<NT>(fin, 0, OpAdd(), red);

    const int B = n - head;
    const int CH = (B + NT - 1) / NT;
    const int k0 = head + tid * CH;
    const int k1 = min(n, k0 + CH);

    int64_t ls = 0, le = 0;
    for (int k = k0; k < k1; ++k) { ls += s[k]; le += e[k]; }
    int64_t tot_s, tot_e;
    const int64_t soff = block_scan_excl<NT, true>(ls, 0, OpAdd(), &tot_s, red);
    block_scan_excl<NT, true>(le, 0, OpAdd(), &tot_e, red);

    int64_t run = soff, lmaxP = INT64_MIN, lmaxPe = INT64_MIN;
    for (int k = k1 - 1; k >= k0; --k) {
        run += s[k];
        ss[k] = (int32_t)run;
        const int64_t P = run + (int64_t)(n - k) * e[k];
        lmaxP = P > lmaxP ? P : lmaxP;
        const int64_t Pe = P + e[k];
        lmaxPe = Pe > lmaxPe ? Pe : lmaxPe;
    }
    int64_t totP, totPe;
    const int64_t smoff = block_scan_excl<NT, true>(lmaxP, INT64_MIN, OpMax(), &totP, red);
    const int64_t pmoff = block_scan_excl<NT, false>(lmaxPe, INT64_MIN, OpMax(), &totPe, red);

    int64_t runmax = smoff;
    for (int k = k1 - 1; k >= k0; --k) {
        const int64_t P = (int64_t)ss[k] + (int64_t)(n - k) * e[k];
        runmax = P > runmax ? P : runmax;
        sm[k] = (int32_t)runmax;
    }
    int64_t runpm = pmoff;
    for (int k = k0; k < k1; ++k) {
        pme[k] = runpm == INT64_MIN ? NEG : (int32_t)runpm;
        const int64_t P = (int64_t)ss[k] + (int64_t)(n - k) * e[k];
        const int64_t Pe = P + e[k];
        runpm = Pe > runpm ? Pe : runpm;
    }
    if (tid == 0) {
        ss[n] = 0;
        sm[n] = NEG;
        pme[n] = totPe == INT64_MIN ? NEG : (int32_t)totPe;
        if (B == 0) pme[head] = NEG;
        const int64_t SC = tot_s + (int64_t)B * tau;
        const int64_t SR = tot_e - (int64_t)B * tau;
        const int64_t DS = (SC << sc.gs) + (int64_t)sc.gn * SR;
        const int64_t X = (int64_t)B << sc.gs;
        if (DS >= ((int64_t)1 << 31) || X >= ((int64_t)1 << 31) || DS < 0) raise_error(err, DEV_EOVERFLOW);
        const uint64_t key = (uint64_t)(X * X) + (uint64_t)(DS * DS);
        st.head[gw] = head;
        st.B[gw] = B;
        st.SC[gw] = SC;
        st.SR[gw] = SR;
        st.DS[gw] = DS;
        st.key[gw] = key;
        st.peak[gw] = B > 0 ? (int32_t)totP : 0;
        st.rhs[gw] = sc.theta * ((sc.tdec - sc.c3) - sc.c2 * (double)(B + 1));
    }
    __syncthreads();
}

// ---------------------------------------------------------------------------------------------
// Ingest: validate residents, convert to (e, s) at tau = 0 and sort each worker by e.
constexpr int SORT_MAX = 4096;

__global__ __launch_bounds__(BUILD_THREADS) void k_ingest(State st, const int64_t* res_off,
                                                          const int32_t* lin, const int32_t* lpred,
                                                          const int32_t* gen)
{
    constexpr int NT = BUILD_THREADS;
    __shared__ uint64_t keys[SORT_MAX];
    __shared__ int64_t red[NT / 64];
    const int gw = blockIdx.x;
    const int tid = threadIdx.x;
    const int64_t r0 = res_off[gw];
    const int R = (int)(res_off[gw + 1] - r0);
    const int64_t base = st.slot_base[gw];
    int32_t* e = st.e + base;
    int32_t* s = st.s + base;
    const int32_t LIM = 1 << 24;

    int64_t bad = 0, tot = 0;
    for (int k = tid; k < R; k += NT) {
        const int32_t a = lin[r0 + k], p = lpred[r0 + k], g = gen[r0 + k];
        const bool ok = a >= 1 && p >= 1 && a <= LIM && p <= LIM && g >= 0 && g < p;
        bad += ok ? 0 : 1;
        tot += ok ? ((int64_t)a + p) : 0;  // sum of (c + r), an upper bound of the KV peak
    }
    bad = block_reduce<NT>(bad, 0, OpAdd(), red);
    tot = block_reduce<NT>(tot, 0, OpAdd(), red);
    if (bad) {
        if (tid == 0) raise_error(st.err_word, DEV_EINVAL);
        return;
    }
    if (tot > ((int64_t)1 << 30) || R > st.cap[gw]) {
        if (tid == 0) raise_error(st.err_word, R > st.cap[gw] ? DEV_ESLOTS : DEV_EOVERFLOW);
        return;
    }
    auto make_key = [&](int k) -> uint64_t {
        const int32_t a = lin[r0 + k], p = lpred[r0 + k], g = gen[r0 + k];
        const uint32_t ek = (uint32_t)(p - g);  // r at tau = 0
        const uint32_t sk = (uint32_t)(a + g);  // c at tau = 0
        return ((uint64_t)ek << 32) | sk;
    };
    if (R <= SORT_MAX) {
        int P2 = 1;
        while (P2 < R) P2 <<= 1;
        for (int k = tid; k < P2; k += NT) keys[k] = k < R ? make_key(k) : ~(uint64_t)0;
        __syncthreads();
        for (int size = 2; size <= P2; size <<= 1) {
            for (int stride = size >> 1; stride > 0; stride >>= 1) {
                for (int k = tid; k < P2; k += NT) {
                    const int j = k ^ stride;
                    if (j > k) {
                        const bool up = (k & size) == 0;
                        const uint64_t x = keys[k], y = keys[j];
                        if ((x > y) == up) { keys[k] = y; keys[j] = x; }
                    }
                }
                __syncthreads();
            }
        }
        for (int k = tid; k < R; k += NT) {
            e[k] = (int32_t)(keys[k] >> 32);
            s[k] = (int32_t)(keys[k] & 0xffffffffu);
        }
    } else {
        // rank sort: position = number of keys smaller, ties by input index
        for (int k = tid; k < R; k += NT) {
            const uint64_t x = make_key(k);
            int pos = 0;
            for (int j = 0; j < R; ++j) {
                const uint64_t y = make_key(j);
                pos += (y < x || (y == x && j < k)) ? 1 : 0;
            }
            e[pos] = (int32_t)(x >> 32);
            s[pos] = (int32_t)(x & 0xffffffffu);
        }
    }
    if (tid == 0) {
        st.n[gw] = R;
        st.head[gw] = 0;
        st.built[gw] = 0;
        st.S1[gw] = 0;
        st.S2[gw] = 0;
        st.hbs[gw] = -1;
        st.dirty[gw] = 0;
    }
}

// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(BUILD_THREADS) void k_build(State st, int force)
{
    const int gw = blockIdx.x;
    const int s = find_scen_by_worker(st, gw);
    const Ctl* c = st.ctl + s;
    if (!force) {
        if (c->err || c->start >= c->Q) return;
        if (!c->rebuild && st.built[gw]) return;
    }
    const Scen sc = st.scen[s];
    build_worker(st, sc, gw, c->tau, &st.ctl[s].err);
    if (threadIdx.x == 0) st.built[gw] = 1;
}

// ---------------------------------------------------------------------------------------------
// Pair evaluation: block = (scenario, worker block, 256-query chunk).
__global__ __launch_bounds__(EVAL_THREADS) void k_eval(State st)
{
    const int s = find_scen<&Scen::eval_blk0>(st, blockIdx.x);
    const Scen sc = st.scen[s];
    const Ctl* cp = st.ctl + s;
    const int32_t start = cp->start, Q = cp->Q;
    if (cp->err || start >= Q) return;
    const int32_t end = tile_end(start, Q, cp->T, cp->H, cp->since_hb);
    const int local = blockIdx.x - sc.eval_blk0;
    const int wb = local % sc.nblk;
    const int qc = local / sc.nblk;
    const int q0 = start + qc * EVAL_THREADS;
    if (q0 >= end) return;
    const int32_t tau = cp->tau, hb = cp->hb_index;
    const int qi = q0 + threadIdx.x;
    const bool act = qi < end;
    const int32_t lin = act ? st.q_lin[qi] : 1;
    const int32_t lp = act ? st.q_lpred[qi] : 1;
    const int32_t sq = lin - tau, eq = lp + tau;

    int32_t ex1 = INT32_MAX, w1 = -1, ex2 = INT32_MAX, w2 = -1;
    const int wbeg = wb * sc.wpb;
    const int wend = min(sc.W, wbeg + sc.wpb);
    const int64_t row = sc.bits_off + (int64_t)((q0 - start) >> 6) * sc.W + (threadIdx.x >> 6) * (int64_t)sc.W;
    for (int w = wbeg; w < wend; ++w) {
        const int gw = sc.wbase + w;
        const View v = load_view(st, gw, hb);
        const int64_t peak = kv_peak_with(v, sq, eq);
        const Latency L = latency(sc, v, lin, lp, v.n - v.head + 1);
        const bool kv_ok = peak <= v.M;
        const bool feas = act && kv_ok && L.dec_ok && L.ttft_ok;
        const uint64_t bf = __ballot(feas);
        const uint64_t bn = __ballot(act && L.nt);
        if (lane_id() == 0) {
            st.bits_feas[row + w] = bf;
            st.bits_nt[row + w] = bn;
        }
        min2_insert(ex1, w1, ex2, w2, (int32_t)(peak - v.M), w);
    }
    if (act) st.part[sc.part_off + (int64_t)(qi - start) * sc.nblk + wb] = make_int4(ex1, w1, ex2, w2);
}

// ---------------------------------------------------------------------------------------------
// Per-query selection over all workers of the scenario.
__global__ __launch_bounds__(SEL_THREADS) void k_select(State st)
{
    const int s = find_scen<&Scen::sel_blk0>(st, blockIdx.x);
    const Scen sc = st.scen[s];
    Ctl* cp = st.ctl + s;
    const int32_t start = cp->start, Q = cp->Q;
    const int local = blockIdx.x - sc.sel_blk0;
    const bool done = cp->err || start >= Q;
    const int32_t end = done ? start : tile_end(start, Q, cp->T, cp->H, cp->since_hb);
    const int parity = cp->round & 1;
    if (local == 0 && threadIdx.x == 0) {
        TileInfo* ti = st.tinfo + s;
        ti->start = done ? Q : start;
        ti->end = done ? Q : end;
        ti->parity = parity;
    }
    if (done) return;
    const int q0 = start + local * SEL_THREADS;
    if (q0 >= end) return;
    const int qi = q0 + threadIdx.x;
    const bool act = qi < end;
    const int lane = lane_id();

    uint64_t tkey[TOPK];
    int32_t tw[TOPK];
#pragma unroll
    for (int k = 0; k < TOPK; ++k) { tkey[k] = 0; tw[k] = -1; }
    int32_t nfeas = 0, ntcnt = 0, ntw = -1;
    uint64_t ntkey = 0;
    const int64_t row = sc.bits_off + (int64_t)((qi - start) >> 6) * sc.W;
    for (int w = 0; w < sc.W; ++w) {
        const uint64_t fw = st.bits_feas[row + w];
        const uint64_t nw = st.bits_nt[row + w];
        if ((fw | nw) == 0) continue;  // wave-uniform
        const uint64_t key = st.key[sc.wbase + w];
        const bool f = (fw >> lane) & 1;
        const bool nb = (nw >> lane) & 1;
        nfeas += f ? 1 : 0;
        topk_insert<TOPK>(tkey, tw, key, f ? w : -1);
        ntcnt += nb ? 1 : 0;
        const bool better = nb & ranks_before(key, w, ntkey, ntw);
        ntkey = better ? key : ntkey;
        ntw = better ? w : ntw;
    }
    int32_t ex1 = INT32_MAX, w1 = -1, ex2 = INT32_MAX, w2 = -1;
    const int4* prow = st.part + sc.part_off + (int64_t)(qi - start) * sc.nblk;
    if (act) {
        for (int b = 0; b < sc.nblk; ++b) {
            const int4 p = prow[b];
            min2_insert(ex1, w1, ex2, w2, p.x, p.y);
            min2_insert(ex1, w1, ex2, w2, p.z, p.w);
        }
    }
    if (!act) return;
    QSum q;
#pragma unroll
    for (int k = 0; k < TOPK; ++k) { q.tkey[k] = tkey[k]; q.tw[k] = tw[k]; }
    q.ntkey = ntkey;
    q.ntw = ntw;
    q.ntcnt = ntcnt;
    q.nfeas = nfeas;
    q.ex1 = ex1; q.w1 = w1;
    q.ex2 = ex2; q.w2 = w2;
    q.pad = 0;
    st.qsum[sc.qsum_off + (qi - start)] = q;
    if (nfeas > 0) atomicMin(&st.tinfo[s].first_pc[parity], qi);
}

// ---------------------------------------------------------------------------------------------
// Commit.

struct Resolved {
    int32_t w;        // chosen worker (scenario-local), -1 = rejected
    int32_t abort;    // the tile-start lists cannot decide this query exactly
    Diag d;
};

// Decide query i (and its diagnostics) at the current state, using the
// tile-start summary q for workers untouched in this tile and re-evaluating
// the workers committed to earlier in the tile (dl[0..nd)).
__device__ Resolved resolve(const State& st, const Scen& sc, const QSum& q, int i, int start,
                            int32_t lin, int32_t lp, int32_t tau, int32_t hb, int32_t stamp,
                            const int32_t* dl, int nd, bool want_diag)
{
    Resolved r;
    r.abort = 0;
    r.w = -1;
    const int32_t sq = lin - tau, eq = lp + tau;
    bool have = false;
    uint64_t bk = 0;
    int32_t bw = -1;
    int32_t nf = q.nfeas;
    if (!want_diag && q.nfeas == 0) return r;  // rejected whatever changed in the tile
    const int lim = q.nfeas < TOPK ? q.nfeas : TOPK;
#pragma unroll
    for (int k = 0; k < TOPK; ++k) {
        const int w = q.tw[k];
        const bool clean = (k < lim) && (w >= 0) && (st.dirty[sc.wbase + (w >= 0 ? w : 0)] != stamp);
        const bool take = clean & !have;
        bk = take ? q.tkey[k] : bk;
        bw = take ? w : bw;
        have = have | take;
    }
    if (!have && q.nfeas > TOPK) { r.abort = 1; return r; }
    const int64_t word = sc.bits_off + (int64_t)((i - start) >> 6) * sc.W;
    const int bit = (i - start) & 63;
    int32_t clean_nt = q.ntcnt;
    uint64_t dntk = 0;
    int32_t dntw = -1;
    int64_t chosen_peak = 0;
    bool chosen_peak_known = false;
    for (int j = 0; j < nd; ++j) {
        const int d = dl[j];
        const int gw = sc.wbase + d;
        const bool fs = (st.bits_feas[word + d] >> bit) & 1;
        const bool ns = (st.bits_nt[word + d] >> bit) & 1;
        clean_nt -= ns ? 1 : 0;
        const View v = load_view(st, gw, hb);
        const Latency L = latency(sc, v, lin, lp, v.n - v.head + 1);
        nf -= fs ? 1 : 0;
        bool feas_now = false;
        int64_t peak = 0;
        if (fs && L.dec_ok && L.ttft_ok) {
            peak = kv_peak_with(v, sq, eq);
            feas_now = peak <= v.M;
        }
        nf += feas_now ? 1 : 0;
        const bool better = feas_now & ranks_before(v.key, d, bk, bw);
        bk = better ? v.key : bk;
        bw = better ? d : bw;
        have = have | better;
        chosen_peak = better ? peak : chosen_peak;
        chosen_peak_known = better | (chosen_peak_known & !better);
        const bool ntb = L.nt & ranks_before(v.key, d, dntk, dntw);
        dntk = ntb ? v.key : dntk;
        dntw = ntb ? d : dntw;
    }
    const bool dnt = dntw >= 0;
    r.w = have ? bw : -1;
    if (!want_diag) return r;

    r.d.n_feasible = nf;
    // smallest KV excess over all workers at the current state
    int64_t exmin;
    if (q.w1 >= 0 && st.dirty[sc.wbase + q.w1] == stamp) {
        const View v = load_view(st, sc.wbase + q.w1, hb);
        const int64_t ex_now = kv_peak_with(v, sq, eq) - v.M;
        if (q.w2 < 0) {
            exmin = ex_now;
        } else if (st.dirty[sc.wbase + q.w2] != stamp) {
            exmin = ex_now < q.ex2 ? ex_now : (int64_t)q.ex2;
        } else {
            r.abort = 1;
            return r;
        }
    } else {
        exmin = q.ex1;
    }
    r.d.kv_excess_min = exmin;
    // near tie among workers ranked at or above the choice (all if rejected)
    bool nt = false;
    if (clean_nt > 0) {
        if (q.ntw >= 0 && st.dirty[sc.wbase + q.ntw] != stamp) {
            if (r.w < 0 || !ranks_before(bk, bw, q.ntkey, q.ntw)) nt = true;
        } else if (r.w < 0) {
            nt = true;
        } else {
            r.abort = 1;
            return r;
        }
    }
    if (dnt && (r.w < 0 || !ranks_before(bk, bw, dntk, dntw))) nt = true;
    r.d.near_tie = nt ? 1 : 0;
    if (r.w >= 0) {
        const View v = load_view(st, sc.wbase + r.w, hb);
        const Latency L = latency(sc, v, lin, lp, v.n - v.head + 1);
        r.d.kv_peak_chosen = chosen_peak_known ? chosen_peak : kv_peak_with(v, sq, eq);
        r.d.ttft_chosen = L.ttft;
        r.d.tdec_chosen = L.tdec;
    } else {
        r.d.kv_peak_chosen = 0;
        r.d.ttft_chosen = 0.0;
        r.d.tdec_chosen = 0.0;
    }
    return r;
}

// Insert one request into worker gw (whole block) and rebuild its summaries.
__device__ bool commit_insert(const State& st, const Scen& sc, int gw, int32_t lin, int32_t lp, int32_t tau,
                              int32_t hb, int32_t* err)
{
    constexpr int NT = COMMIT_THREADS;
    __shared__ int64_t red[NT / 64];
    const int tid = threadIdx.x;
    const int64_t base = st.slot_base[gw];
    int32_t* e = st.e + base;
    int32_t* s = st.s + base;
    int32_t* t1 = st.pme + base;  // scratch: summaries are rebuilt right after
    int32_t* t2 = st.sm + base;
    int n = st.n[gw];
    int head = st.head[gw];
    const int cap = st.cap[gw];
    if (n >= cap) {
        if (head == 0) {
            if (tid == 0) raise_error(err, DEV_ESLOTS);
            __syncthreads();
            return false;
        }
        for (int k = head + tid; k < n; k += NT) { t1[k] = e[k]; t2[k] = s[k]; }
        __syncthreads();
        for (int k = head + tid; k < n; k += NT) { e[k - head] = t1[k]; s[k - head] = t2[k]; }
        __syncthreads();
        n -= head;
        head = 0;
    }
    const int32_t eq = lp + tau, sq = lin - tau;
    int64_t le = 0;
    for (int k = head + tid; k < n; k += NT) le += (e[k] <= eq) ? 1 : 0;
    const int u = head + (int)block_reduce<NT>(le, 0, OpAdd(), red);
    for (int k = u + tid; k < n; k += NT) { t1[k] = e[k]; t2[k] = s[k]; }
    __syncthreads();
    for (int k = u + tid; k < n; k += NT) { e[k + 1] = t1[k]; s[k + 1] = t2[k]; }
    if (tid == 0) {
        e[u] = eq;
        s[u] = sq;
        st.n[gw] = n + 1;
        st.head[gw] = head;
        const bool cur = st.hbs[gw] == hb;
        const int64_t S1 = (cur ? st.S1[gw] : 0) + lin;
        const int64_t S2 = (cur ? st.S2[gw] : 0) + (int64_t)lin * lin;
        if (S2 >= ((int64_t)1 << 53)) raise_error(err, DEV_EOVERFLOW);
        st.S1[gw] = S1;
        st.S2[gw] = S2;
        st.hbs[gw] = hb;
    }
    __syncthreads();
    build_worker(st, sc, gw, tau, err);
    return true;
}

__device__ __forceinline__ int block_min_int(int v, int* lds)
{
    // lds: COMMIT_THREADS/64 ints
    for (int d = 32; d > 0; d >>= 1) {
        int o = __shfl_down(v, d, 64);
        v = o < v ? o : v;
    }
    if (lane_id() == 0) lds[wave_id()] = v;
    __syncthreads();
    int m = lds[0];
    for (int j = 1; j < COMMIT_THREADS / 64; ++j) m = lds[j] < m ? lds[j] : m;
    __syncthreads();
    return m;
}

__global__ __launch_bounds__(COMMIT_THREADS) void k_commit(State st)
{
    constexpr int NT = COMMIT_THREADS;
    const int s = find_scen<&Scen::fin_blk0>(st, blockIdx.x);
    const Scen sc = st.scen[s];
    const int part = blockIdx.x - sc.fin_blk0;
    const TileInfo ti = st.tinfo[s];
    Ctl* cp = st.ctl + s;
    const int tid = threadIdx.x;
    __shared__ int mins[NT / 64];
    __shared__ int64_t red[NT / 64];

    if (ti.start >= ti.end) return;
    const int32_t start = ti.start, end = ti.end;
    const int32_t fpc = min(ti.first_pc[ti.parity], end);

    if (part > 0) {
        // queries before the first one with any feasible worker: rejected, and
        // no worker of the tile has changed yet when they are decided
        int64_t cnt = 0;
        for (int i = start + (part - 1) * NT + tid; i < fpc; i += sc.nfin * NT) {
            const QSum& q = st.qsum[sc.qsum_off + (i - start)];
            if (st.out_worker) st.out_worker[sc.out_off + i] = -1;
            if (st.out_diag) {
                Diag d;
                d.n_feasible = 0;
                d.near_tie = q.ntcnt > 0 ? 1 : 0;
                d.kv_peak_chosen = 0;
                d.kv_excess_min = q.ex1;
                d.ttft_chosen = 0.0;
                d.tdec_chosen = 0.0;
                st.out_diag[i] = d;
            }
            ++cnt;
        }
        cnt = block_reduce<NT>(cnt, 0, OpAdd(), red);
        if (tid == 0 && cnt > 0) atomicAdd(&cp->n_rej, (int)cnt);
        if (tid == 0 && part == 1 && fpc > start) atomicMin(&cp->first_rej, start);
        return;
    }

    // ---- sequential block
    const Ctl c = *cp;
    if (c.err) return;
    const int32_t tau = c.tau, hb = c.hb_index;
    const int32_t stamp = c.round + 1;
    __shared__ int32_t dl[MAX_DIRTY];
    __shared__ int nd;
    __shared__ int32_t sh_w, sh_lin, sh_lp;
    if (tid == 0) {
        nd = 0;
        cp->rebuild = 0;
    }
    __syncthreads();
    const bool want_diag = st.out_diag != nullptr;
    int pos = fpc;
    bool cut = false;
    int commits = 0;
    while (pos < end) {
        const int i = pos + tid;
        const bool act = i < end;
        QSum q;
        int32_t lin = 1, lp = 1;
        if (act) {
            q = st.qsum[sc.qsum_off + (i - start)];
            lin = st.q_lin[i];
            lp = st.q_lpred[i];
        } else {
            q.nfeas = 0;
        }
        const int p = block_min_int((act && q.nfeas > 0) ? tid : NT, mins);
        Resolved r;
        r.abort = 0;
        r.w = -1;
        if (act && tid <= p) {
            r = resolve(st, sc, q, i, start, lin, lp, tau, hb, stamp, dl, nd, want_diag);
            if (tid < p) r.w = -1;
        }
        const int ab = block_min_int((act && tid <= p && r.abort) ? tid : NT, mins);
        const int lim = min(p, ab);
        if (act && tid < lim) {
            if (st.out_worker) st.out_worker[sc.out_off + i] = -1;
            if (want_diag) st.out_diag[i] = r.d;
            atomicAdd(&cp->n_rej, 1);
            atomicMin(&cp->first_rej, i);
        }
        if (ab <= p && ab < NT) {
            pos += ab;
            cut = true;
            break;
        }
        if (p >= NT) {
            pos = min(end, pos + NT);
            continue;
        }
        if (tid == p) {
            sh_w = r.w;
            sh_lin = lin;
            sh_lp = lp;
            if (st.out_worker) st.out_worker[sc.out_off + i] = r.w;
            if (want_diag) st.out_diag[i] = r.d;
            if (r.w < 0) {
                atomicAdd(&cp->n_rej, 1);
                atomicMin(&cp->first_rej, i);
            }
        }
        __syncthreads();
        const int w = sh_w;
        pos += p + 1;
        if (w >= 0) {
            const int gw = sc.wbase + w;
            if (!commit_insert(st, sc, gw, sh_lin, sh_lp, tau, hb, &cp->err)) break;
            ++commits;
            if (tid == 0 && st.dirty[gw] != stamp) {
                st.dirty[gw] = stamp;
                dl[nd] = w;
                nd = nd + 1;
            }
            __syncthreads();
            if (nd >= MAX_DIRTY && pos < end) {
                cut = true;
                break;
            }
        }
        __syncthreads();
    }
    if (tid == 0) {
        const int32_t processed = pos - c.start;
        const int32_t since = c.since_hb + processed;
        if (pos == end && c.H > 0 && since >= c.H) {
            cp->tau = c.tau + 1;
            cp->hb_index = c.hb_index + 1;
            cp->since_hb = 0;
            cp->rebuild = 1;
        } else {
            cp->since_hb = since;
        }
        cp->start = pos;
        cp->aborts = c.aborts + (cut ? 1 : 0);
        cp->commits = c.commits + commits;
        cp->round = c.round + 1;
        st.tinfo[s].first_pc[(c.round + 1) & 1] = INT32_MAX;
    }
}

// ---------------------------------------------------------------------------------------------
// Query validation for one call: any length outside [1, 2^24] sets the error
// word of every scenario, which makes every later kernel of the call a no-op.
__global__ __launch_bounds__(256) void k_query_stats(const int32_t* lin, const int32_t* lpred, int32_t Q,
                                                     Ctl* ctl, int32_t S)
{
    __shared__ int64_t red[4];
    int64_t bad = 0;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < Q; i += (int64_t)gridDim.x * blockDim.x) {
        const int32_t a = lin[i], p = lpred[i];
        bad += (a >= 1 && p >= 1 && a <= (1 << 24) && p <= (1 << 24)) ? 0 : 1;
    }
    bad = block_reduce<256>(bad, 0, OpAdd(), red);
    if (threadIdx.x == 0 && bad)
        for (int s = 0; s < S; ++s) atomicCAS(&ctl[s].err, 0, DEV_EINVAL);
}

__global__ void k_summary(State st, int32_t W, int32_t* B, int64_t* sc, int64_t* sr, int64_t* peak)
{
    const int w = blockIdx.x * blockDim.x + threadIdx.x;
    if (w >= W) return;
    B[w] = st.B[w];
    sc[w] = st.SC[w];
    sr[w] = st.SR[w];
    peak[w] = st.peak[w];
}

__global__ void k_sweep_outputs(State st, int32_t* rejected, int32_t* first_reject)
{
    const int s = blockIdx.x * blockDim.x + threadIdx.x;
    if (s >= st.S) return;
    rejected[s] = st.ctl[s].n_rej;
    const int32_t f = st.ctl[s].first_rej;
    first_reject[s] = f == INT32_MAX ? -1 : f;
}

// ---------------------------------------------------------------------------------------------
hipError_t launch_ingest(const State& st, int32_t W, const int64_t* res_off, const int32_t* lin,
                         const int32_t* lpred, const int32_t* gen, hipStream_t stream)
{
    hipLaunchKernelGGL(k_ingest, dim3(W), dim3(BUILD_THREADS), 0, stream, st, res_off, lin, lpred, gen);
    return hipGetLastError();
}

hipError_t launch_build(const State& st, hipStream_t stream, int force)
{
    hipLaunchKernelGGL(k_build, dim3(st.NW), dim3(BUILD_THREADS), 0, stream, st, force);
    return hipGetLastError();
}

hipError_t launch_eval(const State& st, int32_t blocks, hipStream_t stream)
{
    hipLaunchKernelGGL(k_eval, dim3(blocks), dim3(EVAL_THREADS), 0, stream, st);
    return hipGetLastError();
}

hipError_t launch_select(const State& st, int32_t blocks, hipStream_t stream)
{
    hipLaunchKernelGGL(k_select, dim3(blocks), dim3(SEL_THREADS), 0, stream, st);
    return hipGetLastError();
}

hipError_t launch_commit(const State& st, int32_t blocks, hipStream_t stream)
{
    hipLaunchKernelGGL(k_commit, dim3(blocks), dim3(COMMIT_THREADS), 0, stream, st);
    return hipGetLastError();
}

hipError_t launch_query_stats(const int32_t* lin, const int32_t* lpred, int32_t Q, Ctl* ctl, int32_t S,
                              hipStream_t stream)
{
    int blocks = (Q + 255) / 256;
    if (blocks > 256) blocks = 256;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(k_query_stats, dim3(blocks), dim3(256), 0, stream, lin, lpred, Q, ctl, S);
    return hipGetLastError();
}

hipError_t launch_summary(const State& st, int32_t W, int32_t* B, int64_t* sc, int64_t* sr, int64_t* peak,
                          hipStream_t stream)
{
    hipLaunchKernelGGL(k_summary, dim3((W + 255) / 256), dim3(256), 0, stream, st, W, B, sc, sr, peak);
    return hipGetLastError();
}

hipError_t launch_sweep_outputs(const State& st, int32_t* rejected, int32_t* first_reject, hipStream_t stream)
{
    hipLaunchKernelGGL(k_sweep_outputs, dim3((st.S + 255) / 256), dim3(256), 0, stream, st, rejected,
                       first_reject);
    return hipGetLastError();
}

}  // namespace ald
