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

#include <type_traits>

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
    const int4* pms;
    int32_t head, n, M;
    int64_t DS, S1, S2;
    uint64_t key;
    double rhs;
};

// Integer forms of a built worker's latency checks (see State).
struct Thr {
    int64_t dq_max, ntd_lo, ntd_hi;
    int32_t lthr, ntt_lo, ntt_hi;
};

__device__ __forceinline__ Thr load_thr(const State& st, int gw)
{
    Thr t;
    t.dq_max = st.dq_max[gw];
    t.ntd_lo = st.ntd_lo[gw];
    t.ntd_hi = st.ntd_hi[gw];
    t.lthr = st.lthr[gw];
    t.ntt_lo = st.ntt_lo[gw];
    t.ntt_hi = st.ntt_hi[gw];
    return t;
}

__device__ __forceinline__ View load_view(const State& st, int gw, int32_t hb)
{
    View v;
    const int64_t base = st.slot_base[gw];
    v.e = st.e + base;
    v.pms = st.pms + base;
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
    const int4 t = v.pms[l];
    const int64_t a = (int64_t)t.x + sq;
    const int64_t b = (int64_t)t.y;
    const int64_t c = (int64_t)t.z + (int64_t)(v.n - l) * eq + sq + eq;
    int64_t p = a > b ? a : b;
    return p > c ? p : c;
}

struct Latency {
    double lhs, ttft, tdec;
    bool dec_ok, ttft_ok, nt;
};

// Left side of constraint (b) for a worker whose DS with the query added is x
// (sum of D = x * 2^-gs exactly).
__device__ __forceinline__ double dec_lhs(const Scen& sc, int64_t x) { return sc.k2 * ldexp((double)x, -sc.gs); }

// Prefill time of constraint (c) for TTFT sums S1, S2 that include the query.
__device__ __forceinline__ double ttft_of(const Scen& sc, int64_t S1, int64_t S2)
{
    return (sc.c1 + sc.k1 * (double)S1) + sc.k1q * (double)S2;
}

// Decode constraint (b) and TTFT constraint (c) of one pair.
__device__ __forceinline__ Latency latency(const Scen& sc, const View& v, int32_t lin, int32_t lp, int32_t b)
{
    Latency o;
    const int64_t DSq = v.DS + ((int64_t)lin << sc.gs) + (int64_t)sc.gn * lp;
    o.lhs = dec_lhs(sc, DSq);
    o.dec_ok = o.lhs <= v.rhs;
    o.ttft = ttft_of(sc, v.S1 + lin, v.S2 + (int64_t)lin * lin);
    o.ttft_ok = o.ttft <= sc.ttft;
    o.nt = near_tie(o.lhs, v.rhs) || near_tie(o.ttft, sc.ttft);
    o.tdec = (sc.c3 + sc.c2 * (double)b) + o.lhs;
    return o;
}

// Lanes (of the active ones) where p holds.  Takes the predicate as a bool, so
// that a compare result feeds the mask directly.
__device__ __forceinline__ uint64_t ballot(bool p) { return __builtin_amdgcn_ballot_w64(p); }

// Largest x in [lo, hi] for which `pred` holds, where pred holds on a prefix of
// [lo, hi]; lo - 1 if it holds nowhere.  The 64 lanes of the wave test 64
// evenly spaced points per step, so a range of 2^36 takes six steps.  All
// lanes of the wave must call it; all get the result.
template <typename F>
__device__ int64_t wave_last_true(int64_t lo, int64_t hi, F pred)
{
    int64_t a = lo - 1, b = hi;  // the answer lies in [a, b]
    while (a < b) {
        const int64_t step = (b - a + 63) >> 6;
        const int64_t x = a + step * (lane_id() + 1);
        const bool t = x <= b && pred(x);
        const int cnt = __popcll(ballot(t));
        a += step * cnt;
        const int64_t nb = a + step - 1;
        b = nb < b ? nb : b;
    }
    return a;
}

// Half-width of an interval around y that holds every x with near_tie(x, y):
// near_tie gives |x - y| <= 1e-9 max(|x|, |y|) up to rounding, which implies
// |x - y| < 1.0000002e-9 |y|; the extra 25% covers the rounding of y +- width.
__device__ __forceinline__ double tie_band(double y) { return 1.25e-9 * fabs(y); }

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

// ---- cross-lane primitives (readlane and DPP; no LDS permutes)

// Read a lane's value (uniform result).
__device__ __forceinline__ int32_t rdlane(int32_t v, int l) { return __builtin_amdgcn_readlane(v, l); }
__device__ __forceinline__ uint64_t rdlane64(uint64_t v, int l)
{
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l);
    return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ int64_t rdlane64s(int64_t v, int l) { return (int64_t)rdlane64((uint64_t)v, l); }
__device__ __forceinline__ double rdlane_f64(double v, int l)
{
    return __builtin_bit_cast(double, rdlane64(__builtin_bit_cast(uint64_t, v), l));
}

// Inclusive scan over the 64 lanes (lane 0 first) with DPP row shifts and row
// broadcasts; lanes without a source keep the identity.
template <typename Op>
__device__ __forceinline__ int32_t wave_incl_scan(int32_t x, int32_t ident, Op op)
{
    x = op(x, __builtin_amdgcn_update_dpp(ident, x, 0x111, 0xf, 0xf, false));  // row_shr:1
    x = op(x, __builtin_amdgcn_update_dpp(ident, x, 0x112, 0xf, 0xf, false));  // row_shr:2
    x = op(x, __builtin_amdgcn_update_dpp(ident, x, 0x114, 0xf, 0xf, false));  // row_shr:4
    x = op(x, __builtin_amdgcn_update_dpp(ident, x, 0x118, 0xf, 0xf, false));  // row_shr:8
    x = op(x, __builtin_amdgcn_update_dpp(ident, x, 0x142, 0xa, 0xf, false));  // row_bcast:15
    x = op(x, __builtin_amdgcn_update_dpp(ident, x, 0x143, 0xc, 0xf, false));  // row_bcast:31
    return x;
}
struct Add32 {
    __device__ int32_t operator()(int32_t a, int32_t b) const { return a + b; }
};
struct Or32 {
    __device__ uint32_t operator()(uint32_t a, uint32_t b) const { return a | b; }
};
struct Max32 {
    __device__ int32_t operator()(int32_t a, int32_t b) const { return a > b ? a : b; }
};
__device__ __forceinline__ int32_t wave_sum32(int32_t v) { return rdlane(wave_incl_scan(v, 0, Add32()), 63); }
__device__ __forceinline__ int32_t wave_max32(int32_t v) { return rdlane(wave_incl_scan(v, INT32_MIN, Max32()), 63); }
__device__ __forceinline__ uint64_t wave_or64(uint64_t v)
{
    const uint32_t lo = (uint32_t)rdlane((int32_t)wave_incl_scan((int32_t)(uint32_t)v, 0, Or32()), 63);
    const uint32_t hi = (uint32_t)rdlane((int32_t)wave_incl_scan((int32_t)(uint32_t)(v >> 32), 0, Or32()), 63);
    return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ int64_t wave_sum64(int64_t v)
{
#pragma unroll
    for (int d = 32; d > 0; d >>= 1) v += __shfl_xor(v, d, 64);
    return v;
}


// ---------------------------------------------------------------------------------------------
// Breakpoint summaries of one worker (whole block).  Drops finished requests
// (e < tau), recomputes ss / pme / sm over the live slots and the worker's
// aggregates.  Called with every thread of a BUILD_THREADS block.
__device__ void build_worker(const State& st, const Scen& sc, int gw, int32_t tau, int32_t hb, int32_t* err)
{
    constexpr int NT = BUILD_THREADS;
    __shared__ int64_t red[NT / 64];
    const int tid = threadIdx.x;
    const int64_t base = st.slot_base[gw];
    int32_t* e = st.e + base;
    int32_t* s = st.s + base;
    int4* pms = st.pms + base;
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
        pms[k].z = (int32_t)run;
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
        const int64_t P = (int64_t)pms[k].z + (int64_t)(n - k) * e[k];
        runmax = P > runmax ? P : runmax;
        pms[k].y = (int32_t)runmax;
    }
    int64_t runpm = pmoff;
    for (int k = k0; k < k1; ++k) {
        pms[k].x = runpm == INT64_MIN ? PME_NONE : (int32_t)runpm;
        const int64_t P = (int64_t)pms[k].z + (int64_t)(n - k) * e[k];
        const int64_t Pe = P + e[k];
        runpm = Pe > runpm ? Pe : runpm;
    }
    const int64_t SC = tot_s + (int64_t)B * tau;
    const int64_t SR = tot_e - (int64_t)B * tau;
    const int64_t DS = (SC << sc.gs) + (int64_t)sc.gn * SR;
    const double rhs = sc.theta * ((sc.tdec - sc.c3) - sc.c2 * (double)(B + 1));
    if (tid == 0) {
        pms[n] = make_int4(totPe == INT64_MIN ? PME_NONE : (int32_t)totPe, NEG, 0, 0);
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
        st.rhs[gw] = rhs;
    }
    // Breakpoint table: a histogram of the remaining lengths r = e - tau of the
    // live requests (those below LB_MAX), then an exclusive scan, so that entry
    // v - 1 = number of live requests with r < v.
    if (B > 0) {
        __shared__ int32_t hist[LB_MAX];
        for (int v = tid; v < LB_MAX; v += NT) hist[v] = 0;
        __syncthreads();
        for (int k = head + tid; k < n; k += NT) {
            const int32_t r = e[k] - tau;
            if ((uint32_t)r < (uint32_t)LB_MAX) atomicAdd(&hist[r], 1);
        }
        __syncthreads();
        constexpr int CHV = LB_MAX / NT;  // entries per thread
        int32_t loc = 0;
#pragma unroll
        for (int j = 0; j < CHV; ++j) loc += hist[tid * CHV + j];
        int64_t tot;
        int32_t run = (int32_t)block_scan_excl<NT, false>(loc, 0, OpAdd(), &tot, red);
        uint16_t* out = st.lbt + (int64_t)gw * LB_MAX;
#pragma unroll
        for (int j = 0; j < CHV; ++j) {
            run += hist[tid * CHV + j];  // now: requests with r <= tid * CHV + j
            out[tid * CHV + j] = (uint16_t)run;  // entry v - 1 with v = tid * CHV + j + 1
        }
    }
    // Integer forms of the latency checks.  Both left sides are rounded fp64
    // expressions that never decrease as DS + qD (resp. l_in) grows -- each step
    // is an exact conversion, a product with a non-negative constant or a sum,
    // and rounding is monotone -- so each check holds exactly up to a threshold,
    // found by searching with the very expression the pair check evaluates.
    // Queries have qD <= 2^33 and l_in <= 2^24; DS < 2^31.
    constexpr int64_t XMAX = (int64_t)1 << 36;
    constexpr int64_t LMAX = (int64_t)1 << 24;
    const int wv = wave_id();
    const bool l0 = lane_id() == 0;
    // Inside a band of at most 64 values the margin test itself is run once per
    // value (one per lane), giving the exact near-tie set as a bit mask.
    if (wv == 0) {
        const int64_t x = wave_last_true(0, XMAX, [&](int64_t v) { return dec_lhs(sc, v) <= rhs; });
        if (l0) st.dq_max[gw] = x - DS;
    } else if (wv == 1) {
        const double band = tie_band(rhs);
        const double lo = rhs - band, hi = rhs + band;
        const int64_t xl = wave_last_true(0, XMAX, [&](int64_t v) { return dec_lhs(sc, v) < lo; }) + 1;
        const int64_t xh = wave_last_true(0, XMAX, [&](int64_t v) { return dec_lhs(sc, v) <= hi; });
        const int64_t width = xh - xl + 1;
        const uint64_t mask = ballot(lane_id() < width && near_tie(dec_lhs(sc, xl + lane_id()), rhs));
        if (l0) {
            st.ntd_lo[gw] = xl - DS;
            st.ntd_hi[gw] = xh - DS;
            st.ntd_mask[gw] = width <= 64 ? mask : 0;
            if (width > 64 && sc.ntint) raise_error(err, DEV_EOVERFLOW);
        }
    } else if (wv <= 3) {
        const bool cur = st.hbs[gw] == hb;
        const int64_t S1 = cur ? st.S1[gw] : 0;
        const int64_t S2 = cur ? st.S2[gw] : 0;
        auto tt = [&](int64_t l) { return ttft_of(sc, S1 + l, S2 + l * l); };
        if (wv == 2) {
            const int64_t l = wave_last_true(1, LMAX, [&](int64_t v) { return tt(v) <= sc.ttft; });
            if (l0) st.lthr[gw] = (int32_t)l;
        } else {
            const double band = tie_band(sc.ttft);
            const double lo = sc.ttft - band, hi = sc.ttft + band;
            const int64_t ll = wave_last_true(1, LMAX, [&](int64_t v) { return tt(v) < lo; }) + 1;
            const int64_t lh = wave_last_true(1, LMAX, [&](int64_t v) { return tt(v) <= hi; });
            const int64_t width = lh - ll + 1;
            const uint64_t mask = ballot(lane_id() < width && near_tie(tt(ll + lane_id()), sc.ttft));
            if (l0) {
                st.ntt_lo[gw] = (int32_t)ll;
                st.ntt_hi[gw] = (int32_t)lh;
                st.ntt_mask[gw] = width <= 64 ? mask : 0;
                if (width > 64 && sc.ntint) raise_error(err, DEV_EOVERFLOW);
            }
        }
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
    }
}

// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(BUILD_THREADS) void k_build(State st, int mode)
{
    int gw, s;
    if (mode == 1) {
        s = blockIdx.x / MAX_DIRTY;
        const int j = blockIdx.x % MAX_DIRTY;
        if (s >= st.S || j >= st.dcount[s]) return;
        gw = st.dlist[s * MAX_DIRTY + j];
        if (st.built[gw]) return;
    } else {
        gw = blockIdx.x;
        s = find_scen_by_worker(st, gw);
    }
    const Ctl* c = st.ctl + s;
    if (mode == 0) {
        if (c->err || c->start >= c->Q) return;
        if (!c->rebuild && st.built[gw]) return;
    }
    const Scen sc = st.scen[s];
    build_worker(st, sc, gw, c->tau, c->hb_index, &st.ctl[s].err);
    if (threadIdx.x == 0) st.built[gw] = 1;
}

// ---------------------------------------------------------------------------------------------
// What the pair evaluation needs of one worker, gathered into LDS once per
// block so that the evaluation loop reads no per-worker global data.
struct WInfo {
    int64_t base;  // first live slot
    int64_t DS, S1, S2;
    double rhs;
    int64_t dq_max, ntd_lo, ntd_hi;
    uint64_t ntd_mask, ntt_mask;
    int32_t head, n, M, lthr, ntt_lo, ntt_hi;
    int32_t nt_any;  // some query of the block's chunk may have a near-tie margin with this worker
};

__device__ __forceinline__ View winfo_view(const State& st, const WInfo& wi)
{
    View v;
    v.e = st.e + (wi.base - wi.head);
    v.pms = st.pms + (wi.base - wi.head);
    v.head = wi.head;
    v.n = wi.n;
    v.M = wi.M;
    v.DS = wi.DS;
    v.S1 = wi.S1;
    v.S2 = wi.S2;
    v.key = 0;
    v.rhs = wi.rhs;
    return v;
}

// Block-wide reductions of one int64 per thread (all threads get the result).
template <int NT, typename Op>
__device__ __forceinline__ int64_t block_all(int64_t v, int64_t ident, Op op, int64_t* lds)
{
#pragma unroll
    for (int d = 32; d > 0; d >>= 1) v = op(v, __shfl_xor(v, d, 64));
    if (lane_id() == 0) lds[wave_id()] = v;
    __syncthreads();
    int64_t r = ident;
#pragma unroll
    for (int j = 0; j < NT / 64; ++j) r = op(r, lds[j]);
    __syncthreads();
    return r;
}

// Two smallest KV excesses of a query as packed keys: excess (offset to
// unsigned) in the high word, the complement of the worker index in the low
// word -- smaller key = smaller excess, then higher index (the order the
// commit's tie rule expects).  ~0 marks an empty entry.
__device__ __forceinline__ uint64_t ex_key(int32_t ex, int32_t w)
{
    return ((uint64_t)((uint32_t)ex ^ 0x80000000u) << 32) | (uint32_t)~(uint32_t)w;
}
__device__ __forceinline__ void ex_unpack(uint64_t k, int32_t& ex, int32_t& w)
{
    ex = k == ~0ull ? INT32_MAX : (int32_t)((uint32_t)(k >> 32) ^ 0x80000000u);
    w = k == ~0ull ? -1 : (int32_t)~(uint32_t)k;
}

// Word `acc` with lane J's value replaced by the wave-uniform `v`
// (v_writelane_b32 on each half, the lane an inline constant, J < 16).  The s_nop
// gives an SGPR that a VALU instruction wrote just before (a compare's lane
// mask) its wait states before v_writelane reads it: the compiler does not
// look inside the asm for that hazard, and without the wait the lanes took
// stale words.
template <int J>
__device__ __forceinline__ uint64_t put_lane_c(uint64_t acc, uint64_t v)
{
    uint32_t lo = (uint32_t)acc, hi = (uint32_t)(acc >> 32);
    asm("s_nop 4\n\tv_writelane_b32 %0, %2, %4\n\tv_writelane_b32 %1, %3, %4"
        : "+v"(lo), "+v"(hi)
        : "s"((uint32_t)v), "s"((uint32_t)(v >> 32)), "n"(J));
    return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ uint64_t put_lane(uint64_t acc, uint64_t v, int j)
{
    switch (j) {
    case 0: return put_lane_c<0>(acc, v);
    case 1: return put_lane_c<1>(acc, v);
    case 2: return put_lane_c<2>(acc, v);
    case 3: return put_lane_c<3>(acc, v);
    case 4: return put_lane_c<4>(acc, v);
    case 5: return put_lane_c<5>(acc, v);
    case 6: return put_lane_c<6>(acc, v);
    case 7: return put_lane_c<7>(acc, v);
    case 8: return put_lane_c<8>(acc, v);
    case 9: return put_lane_c<9>(acc, v);
    case 10: return put_lane_c<10>(acc, v);
    case 11: return put_lane_c<11>(acc, v);
    case 12: return put_lane_c<12>(acc, v);
    case 13: return put_lane_c<13>(acc, v);
    case 14: return put_lane_c<14>(acc, v);
    default: return put_lane_c<15>(acc, v);
    }
}

// Keep a query's two smallest KV excesses as (excess, worker) pairs, smaller
// excess first, then the higher index; e1 = INT32_MAX, w1 = -1 when empty
// (every excess is below INT32_MAX).  IN_ORDER: w is above every index seen so
// far, so an equal excess replaces.
template <bool IN_ORDER>
__device__ __forceinline__ void keep_two(int32_t ex, int32_t w, int32_t& e1, int32_t& w1, int32_t& e2, int32_t& w2)
{
    const bool b1 = IN_ORDER ? ex <= e1 : ((ex < e1) | ((ex == e1) & (w > w1)));
    const bool b2 = IN_ORDER ? ex <= e2 : ((ex < e2) | ((ex == e2) & (w > w2)));
    e2 = b1 ? e1 : (b2 ? ex : e2);
    w2 = b1 ? w1 : (b2 ? w : w2);
    e1 = b1 ? ex : e1;
    w1 = b1 ? w : w1;
}

// One thread's share of a staged worker: slots tid + j * EVAL_THREADS of the
// summaries (clamped to slot B, which exists) and LBV entries of its table.
constexpr int PF_N = (STAGE_MAX + EVAL_THREADS - 1) / EVAL_THREADS;
constexpr int LBV = LB_MAX / EVAL_THREADS;  // table entries per thread (8 or 4)
static_assert(LBV == 8 || LBV == 4, "one 16- or 8-byte table load per thread");
using LBVec = std::conditional_t<LBV == 8, uint4, uint2>;
struct Prefetch {
    int4 p[PF_N];
    LBVec lb;  // LBV entries of the worker's breakpoint table (zeros for an empty worker)
};

__device__ __forceinline__ Prefetch prefetch_worker(const State& st, const WInfo& x, int gw, int tid)
{
    Prefetch f;
    const int B = x.n - x.head;
#pragma unroll
    for (int j = 0; j < PF_N; ++j) f.p[j] = st.pms[x.base + min(tid + j * EVAL_THREADS, B)];
    f.lb = LBVec{};
    if (B > 0) f.lb = reinterpret_cast<const LBVec*>(st.lbt + (int64_t)gw * LB_MAX)[tid];
    return f;
}

// Write one thread's share of a staged worker into LDS: the summaries of
// slots 0 .. B and the table entries below L (the chunk's largest l_pred).
__device__ __forceinline__ void stage_put(uint16_t* LBs, int4* Ss, const Prefetch& pf, int tid, int B, int L)
{
#pragma unroll
    for (int j = 0; j < PF_N; ++j)
        if (tid + j * EVAL_THREADS <= B) Ss[tid + j * EVAL_THREADS] = pf.p[j];
    if (LBV * tid < L) reinterpret_cast<LBVec*>(LBs)[tid] = pf.lb;
}

// First worker at or after j (block-local index) that is evaluated from LDS.
__device__ __forceinline__ int next_staged(const WInfo* Wi, int nw, bool use_lb, int j)
{
    if (!use_lb) return nw;
    while (j < nw && Wi[j].n - Wi[j].head >= STAGE_MAX) ++j;
    return j;
}

// Ranges of a chunk's query figures, for skipping near-tie work per worker.
struct QRange {
    int64_t qdmin, qdmax, lnmin, lnmax;
};

// Evaluate this thread's queries against one worker and store the wave's bit
// words (lane j < 2 EVAL_QPT stores word j).  STAGED: breakpoint slot from the block's
// table and summaries in LDS; else binary search over global memory.  MODE as
// for launch_eval.
template <int MODE, bool EX, bool STAGED>
__device__ __forceinline__ void eval_worker(const State& st, const Scen& sc, const WInfo& wi, int w, int32_t tau,
                                            const int32_t (&lin)[EVAL_QPT], const int32_t (&lp)[EVAL_QPT],
                                            const bool (&act)[EVAL_QPT], const uint64_t (&am)[EVAL_QPT],
                                            int32_t (&e1)[EVAL_QPT],
                                            int32_t (&w1)[EVAL_QPT], int32_t (&e2)[EVAL_QPT],
                                            int32_t (&w2)[EVAL_QPT], const uint16_t* LBs, const int4* Ss,
                                            uint64_t* bdst)
{
    constexpr bool MONO = MODE >= 1;
    const int lane = lane_id();
    const int B = wi.n - wi.head;
    const View v = winfo_view(st, wi);
    // KV peaks first: the table reads of all queries, then their summary reads,
    // so that the LDS latencies overlap
    int32_t peak[EVAL_QPT];
    if (STAGED) {
        int l[EVAL_QPT];
        int4 t[EVAL_QPT];
#pragma unroll
        for (int m = 0; m < EVAL_QPT; ++m) l[m] = LBs[lp[m] - 1];  // live requests ending before the query
#pragma unroll
        for (int m = 0; m < EVAL_QPT; ++m) t[m] = Ss[l[m]];
#pragma unroll
        for (int m = 0; m < EVAL_QPT; ++m) {
            // every candidate below is a KV demand with the query added, so it
            // lies under the worker's peak (<= 2^30) plus l_in + l_pred: 32-bit
            // wrap-around arithmetic gives it exactly
            const uint32_t sq = (uint32_t)(lin[m] - tau), eq = (uint32_t)(lp[m] + tau);
            const int32_t a = (int32_t)((uint32_t)t[m].x + sq);
            const int32_t c = (int32_t)((uint32_t)t[m].z + (uint32_t)(B - l[m]) * eq + sq + eq);
            const int32_t p = a > t[m].y ? a : t[m].y;
            peak[m] = p > c ? p : c;
        }
    } else {
#pragma unroll
        for (int m = 0; m < EVAL_QPT; ++m) peak[m] = (int32_t)kv_peak_with(v, lin[m] - tau, lp[m] + tau);
    }
    uint64_t bits = 0;  // lane j < 2 EVAL_QPT: the word it stores
    if (MONO) {
        // feasibility from the integer thresholds (the worker's figures read
        // once; no short-circuit, so no branch per query)
        const int32_t M = wi.M, lthr = wi.lthr;
        const int64_t dq_max = wi.dq_max;
#pragma unroll
        for (int m = 0; m < EVAL_QPT; ++m) {
            const int64_t qD = ((int64_t)lin[m] << sc.gs) + (int64_t)sc.gn * lp[m];
            // one ballot per compare: each compare's lane mask is its ballot
            const uint64_t bf = am[m] & ballot(peak[m] <= M) & ballot(qD <= dq_max) & ballot(lin[m] <= lthr);
            bits = put_lane(bits, bf, m);
            if (EX) keep_two<STAGED>(peak[m] - M, w, e1[m], w1[m], e2[m], w2[m]);
        }
        // near-tie words (lanes EVAL_QPT .. 2 EVAL_QPT - 1) stay zero here: near_tie_words fills
        // them in for the workers with nt_any
    } else {
#pragma unroll
        for (int m = 0; m < EVAL_QPT; ++m) {
            const Latency Lt = latency(sc, v, lin[m], lp[m], B + 1);
            const uint64_t bf = ballot(act[m] && peak[m] <= wi.M && Lt.dec_ok && Lt.ttft_ok);
            const uint64_t bn = ballot(act[m] && Lt.nt);
            bits = put_lane(bits, bf, m);
            bits = put_lane(bits, bn, m + EVAL_QPT);
            if (EX) keep_two<STAGED>(peak[m] - wi.M, w, e1[m], w1[m], e2[m], w2[m]);
        }
    }
    if (lane < 2 * EVAL_QPT) bdst[w] = bits;
}

// Near-tie words of one worker (lanes EVAL_QPT .. 2 EVAL_QPT - 1 store the
// wave's words for its queries m = lane - EVAL_QPT), with the integer thresholds (MODE >= 1): from the
// worker's exact near-tie sets (MODE 2) or by the fp64 margin tests of the
// queries inside a tie band (MODE 1).  Independent of the KV peak, so it runs
// after the staged loop, apart from its registers.
template <int MODE>
__device__ __forceinline__ void near_tie_words(const State& st, const Scen& sc, const WInfo& wi, int w,
                                               const int32_t (&lin)[EVAL_QPT], const int32_t (&lp)[EVAL_QPT],
                                               const bool (&act)[EVAL_QPT], uint64_t* bdst)
{
    const int lane = lane_id();
    const View v = winfo_view(st, wi);
    const int B = wi.n - wi.head;
    uint64_t bits = 0;
#pragma unroll
    for (int m = 0; m < EVAL_QPT; ++m) {
        const int64_t qD = ((int64_t)lin[m] << sc.gs) + (int64_t)sc.gn * lp[m];
        bool nt;
        if (MODE == 2) {
            const uint64_t dd = (uint64_t)(qD - wi.ntd_lo);
            const uint32_t dl = (uint32_t)(lin[m] - wi.ntt_lo);
            nt = (dd < 64 && ((wi.ntd_mask >> dd) & 1)) || (dl < 64 && ((wi.ntt_mask >> dl) & 1));
        } else {
            const bool maybe = (qD >= wi.ntd_lo && qD <= wi.ntd_hi) || (lin[m] >= wi.ntt_lo && lin[m] <= wi.ntt_hi);
            nt = maybe && latency(sc, v, lin[m], lp[m], B + 1).nt;
        }
        const uint64_t bn = ballot(act[m] && nt);
        bits = put_lane(bits, bn, m + EVAL_QPT);
    }
    if (lane >= EVAL_QPT && lane < 2 * EVAL_QPT) bdst[w] = bits;
}

// Pair evaluation: block = (scenario, worker block, chunk of EVAL_Q queries).
// Thread t holds queries t, t + 256, t + 512, t + 768 of the chunk.  For each
// worker of the block, its summaries and breakpoint table (built with the
// summaries) are staged in LDS; a query's breakpoint slot is then one table
// read, l = LB[l_pred - 1], and the summaries of slot l give the KV peak with the
// query added.  The next worker's data travels in registers while the current
// one is evaluated.  Workers with B >= STAGE_MAX, or chunks with an l_pred above
// LB_MAX, take the binary search over global memory instead.  MODE: how the
// latency checks are taken (launch_eval); EX: the two smallest KV excesses are
// tracked (diagnostics).
template <int MODE, bool EX>
__global__ __launch_bounds__(EVAL_THREADS) __attribute__((amdgpu_waves_per_eu(4))) void k_eval(State st)
{
    constexpr int NT = EVAL_THREADS;
    constexpr int QPT = EVAL_QPT;
    static_assert(2 * QPT <= 16, "lane words by put_lane");
    __shared__ uint16_t LBs[LB_MAX];               // the worker's breakpoint table
    __shared__ int4 Ss[PF_N * NT];                 // pms of live slot k, k = 0..B
    __shared__ WInfo Wi[EVAL_WPB_MAX];
    __shared__ int64_t red[NT / 64];

    const int s = find_scen<&Scen::eval_blk0>(st, blockIdx.x);
    const Scen sc = st.scen[s];
    const Ctl* cp = st.ctl + s;
    const int32_t start = cp->start, Q = cp->Q;
    if (st.qbad != nullptr && start == 0) {
        // first round of a one-scenario call: check every query length of the
        // call before the first commit can run (grid-stride over all queries)
        bool bad = false;
        for (int64_t i = (int64_t)blockIdx.x * EVAL_THREADS + threadIdx.x; i < Q; i += (int64_t)gridDim.x * EVAL_THREADS) {
            const int32_t a = st.q_lin[i], p = st.q_lpred[i];
            bad = bad || !(a >= 1 && p >= 1 && a <= (1 << 24) && p <= (1 << 24));
        }
        if (ballot(bad) != 0 && lane_id() == 0) atomicOr(st.qbad, 1);
    }
    if (cp->err || start >= Q) return;
    const int32_t end = tile_end(start, Q, cp->T, cp->H, cp->since_hb);
    const int local = blockIdx.x - sc.eval_blk0;
    const int wb = local % sc.nblk;
    const int qc = local / sc.nblk;
    const int q0 = start + qc * EVAL_Q;
    if (q0 >= end) return;
    const int32_t tau = cp->tau, hb = cp->hb_index;
    const int tid = threadIdx.x;
    const int lane = lane_id();

    int32_t lin[QPT], lp[QPT];
    bool act[QPT];
    int32_t e1[QPT], w1[QPT], e2[QPT], w2[QPT];  // two smallest KV excesses per query
    int64_t lpmax = 0, qdmin = INT64_MAX, qdmax = INT64_MIN, lnmin = INT64_MAX, lnmax = INT64_MIN;
#pragma unroll
    for (int m = 0; m < QPT; ++m) {
        const int qi = q0 + m * NT + tid;
        act[m] = qi < end;
        lin[m] = act[m] ? st.q_lin[qi] : 1;
        lp[m] = act[m] ? st.q_lpred[qi] : 1;
        e1[m] = e2[m] = INT32_MAX;
        w1[m] = w2[m] = -1;
        const int64_t qD = ((int64_t)lin[m] << sc.gs) + (int64_t)sc.gn * lp[m];
        if (act[m]) {
            lpmax = lp[m] > lpmax ? lp[m] : lpmax;
            qdmin = qD < qdmin ? qD : qdmin;
            qdmax = qD > qdmax ? qD : qdmax;
            lnmin = lin[m] < lnmin ? lin[m] : lnmin;
            lnmax = lin[m] > lnmax ? lin[m] : lnmax;
        }
    }
    uint64_t am[QPT];  // the wave's lanes holding a query m
#pragma unroll
    for (int m = 0; m < QPT; ++m) am[m] = ballot(act[m]);
    lpmax = block_all<NT>(lpmax, 0, OpMax(), red);
    QRange qr;
    qr.qdmin = block_all<NT>(qdmin, INT64_MAX, OpMin(), red);
    qr.qdmax = block_all<NT>(qdmax, INT64_MIN, OpMax(), red);
    qr.lnmin = block_all<NT>(lnmin, INT64_MAX, OpMin(), red);
    qr.lnmax = block_all<NT>(lnmax, INT64_MIN, OpMax(), red);
    const int L = (int)lpmax;  // table covers v = 0 .. L
    const bool use_lb = L <= LB_MAX;

    const int wbeg = wb * sc.wpb;
    const int nw = min(sc.W, wbeg + sc.wpb) - wbeg;
    if (tid < nw) {
        const int gw = sc.wbase + wbeg + tid;
        WInfo x;
        x.head = st.head[gw];
        x.n = st.n[gw];
        x.base = st.slot_base[gw] + x.head;
        x.M = st.M[gw];
        x.DS = st.DS[gw];
        const bool cur = st.hbs[gw] == hb;
        x.S1 = cur ? st.S1[gw] : 0;
        x.S2 = cur ? st.S2[gw] : 0;
        x.rhs = st.rhs[gw];
        x.dq_max = st.dq_max[gw];
        x.ntd_lo = st.ntd_lo[gw];
        x.ntd_hi = st.ntd_hi[gw];
        x.lthr = st.lthr[gw];
        x.ntt_lo = st.ntt_lo[gw];
        x.ntt_hi = st.ntt_hi[gw];
        x.ntd_mask = st.ntd_mask[gw];
        x.ntt_mask = st.ntt_mask[gw];
        // a near-tie margin needs some query of the chunk inside a tie band
        x.nt_any = MODE == 0 || (qr.qdmax >= x.ntd_lo && qr.qdmin <= x.ntd_hi) ||
                   (qr.lnmax >= x.ntt_lo && qr.lnmin <= x.ntt_hi);
        Wi[tid] = x;
    }
    __syncthreads();

    // The next worker's e column and summaries travel in registers while the
    // current one is evaluated.  Plain loads of clamped (in-range) slots, masked
    // only where they are used, so nothing waits for them before then.
    Prefetch pf;
    // bit word of (query group, worker) for lane j < 2 QPT of each wave:
    // feasibility (j < QPT) or near-tie (j >= QPT) of the wave's queries m = j % QPT
    const int64_t brow = sc.bits_off + (int64_t)(((q0 - start) >> 6) + wave_id() + (lane % QPT) * (NT / 64)) * sc.W;
    uint64_t* const bdst = (lane < QPT ? st.bits_feas : st.bits_nt) + brow;

    int cur = next_staged(Wi, nw, use_lb, 0);
    if (cur < nw) pf = prefetch_worker(st, Wi[cur], sc.wbase + wbeg + cur, tid);
    while (cur < nw) {
        __syncthreads();  // the previous worker's readers of LBs / Ss are done
        stage_put(LBs, Ss, pf, tid, Wi[cur].n - Wi[cur].head, L);
        __syncthreads();
        const int nxt = next_staged(Wi, nw, use_lb, cur + 1);
        if (nxt < nw) pf = prefetch_worker(st, Wi[nxt], sc.wbase + wbeg + nxt, tid);
        eval_worker<MODE, EX, true>(st, sc, Wi[cur], wbeg + cur, tau, lin, lp, act, am, e1, w1, e2, w2, LBs, Ss, bdst);
        cur = nxt;
    }
    // workers too large to stage: binary search over global memory
    for (int j0 = 0; j0 < nw; ++j0) {
        const WInfo wi = Wi[j0];
        if (use_lb && wi.n - wi.head < STAGE_MAX) continue;
        eval_worker<MODE, EX, false>(st, sc, wi, wbeg + j0, tau, lin, lp, act, am, e1, w1, e2, w2, LBs, Ss, bdst);
    }
    if (MODE >= 1 && EX) {  // near-tie margins feed only the diagnostics
        for (int j0 = 0; j0 < nw; ++j0)
            if (Wi[j0].nt_any) near_tie_words<MODE>(st, sc, Wi[j0], wbeg + j0, lin, lp, act, bdst);
    }
    if (!EX) return;
#pragma unroll
    for (int m = 0; m < QPT; ++m) {
        const int qi = q0 + m * NT + tid;
        const uint64_t k1 = w1[m] < 0 ? ~0ull : ex_key(e1[m], w1[m]);
        const uint64_t k2 = w2[m] < 0 ? ~0ull : ex_key(e2[m], w2[m]);
        if (act[m]) st.part[sc.part_off + (int64_t)wb * sc.pstride + (qi - start)] = make_ulonglong2(k1, k2);
    }
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
    // waves of the block: sel_g of them per 64-query group, each scanning its
    // share of the workers
    constexpr int NWV = SEL_THREADS / 64;
    const int G = sc.sel_g;
    const int wv = wave_id();
    const int group = local * (NWV / G) + wv / G;  // 64-query group of this wave
    const int slice = wv % G;                       // its share of the workers
    const int q0 = start + group * 64;
    const bool live = q0 < end;                     // wave-uniform
    const int lane = lane_id();
    const int qi = q0 + lane;
    const bool act = live && qi < end;

    uint64_t tkey[TOPK];
    int32_t tw[TOPK];
#pragma unroll
    for (int k = 0; k < TOPK; ++k) { tkey[k] = 0; tw[k] = -1; }
    int32_t nfeas = 0, ntcnt = 0, ntw = -1, ncand = 0;
    bool efeas = false;
    uint64_t ntkey = 0;
    // the group's 64 queries share one bit word per worker; 64 workers' words
    // are read at once and only workers with a set bit are visited
    const int64_t row = sc.bits_off + (int64_t)group * sc.W;
    const int span = ((sc.W + G * 64 - 1) / (G * 64)) * 64;  // workers per wave, whole batches
    const int wlo = live ? min(sc.W, slice * span) : 0;
    const int whi = live ? min(sc.W, wlo + span) : 0;
    // Without diagnostics only the choice matters: near-tie words are not
    // read, and the interchangeable empty workers of a uniform-capacity
    // scenario are taken 64 at a time (an OR of their words); nfeas then only
    // says whether some worker is feasible.
    const bool diag = st.out_diag != nullptr;
    const bool bulk_empty = !diag && sc.uniform_M;
    constexpr int UB = 8;  // 64-worker batches whose words are loaded together
    for (int g0 = wlo; g0 < whi; g0 += 64 * UB) {
        uint64_t fls[UB], nls[UB];
#pragma unroll
        for (int u = 0; u < UB; ++u) {
            const int wl = g0 + u * 64 + lane;
            const bool in = wl < whi;
            fls[u] = in ? st.bits_feas[row + wl] : 0;
            nls[u] = (in && diag) ? st.bits_nt[row + wl] : 0;
        }
#pragma unroll
        for (int u = 0; u < UB; ++u) {
            const int wb0 = g0 + u * 64;
            const uint64_t fl = fls[u], nl = nls[u];
            uint64_t mask = ballot((fl | nl) != 0);
            if (!mask) continue;
            const int wl = wb0 + lane;
            const uint64_t kl = wl < whi ? st.key[sc.wbase + wl] : 0;
            if (bulk_empty) {
                const uint64_t em = mask & ballot(kl == 0);
                if (em) {
                    const uint64_t any = wave_or64(((em >> lane) & 1) ? fl : 0);
                    efeas = efeas | (((any >> lane) & 1) != 0);
                    mask &= ~em;
                }
            }
            while (mask) {
                const int j = __ffsll((unsigned long long)mask) - 1;
                mask &= mask - 1;
                const uint64_t fw = rdlane64(fl, j);
                const uint64_t nw = rdlane64(nl, j);
                const uint64_t key = rdlane64(kl, j);
                const int w = wb0 + j;
                const bool f = (fw >> lane) & 1;
                const bool nb = (nw >> lane) & 1;
                nfeas += f ? 1 : 0;
                // an empty worker has rank key 0; with uniform capacity all empty
                // workers are alike and stand in one class
                const bool cls = sc.uniform_M && key == 0;
                efeas = efeas | (cls & f);
                ncand += (f & !cls) ? 1 : 0;
                topk_insert<TOPK>(tkey, tw, key, (f && !cls) ? w : -1);
                ntcnt += nb ? 1 : 0;
                const bool better = nb & ranks_before(key, w, ntkey, ntw);
                ntkey = better ? key : ntkey;
                ntw = better ? w : ntw;
            }
        }
    }
    // merge the group's partial results into its first wave (lists by rank,
    // counts summed)
    struct Part {
        uint64_t tkey[TOPK];
        int32_t tw[TOPK];
        uint64_t ntkey;
        int32_t ntw, nfeas, ncand, ntcnt, efeas, pad;
    };
    __shared__ Part parts[NWV][64];
    if (G > 1) {
        if (slice > 0) {
            Part& pt = parts[wv][lane];
#pragma unroll
            for (int k = 0; k < TOPK; ++k) { pt.tkey[k] = tkey[k]; pt.tw[k] = tw[k]; }
            pt.ntkey = ntkey;
            pt.ntw = ntw;
            pt.nfeas = nfeas;
            pt.ncand = ncand;
            pt.ntcnt = ntcnt;
            pt.efeas = efeas ? 1 : 0;
        }
        __syncthreads();
        if (slice > 0) return;
        for (int v = wv + 1; v < wv + G; ++v) {
            const Part& pt = parts[v][lane];
#pragma unroll
            for (int k = 0; k < TOPK; ++k) topk_insert<TOPK>(tkey, tw, pt.tkey[k], pt.tw[k]);
            const bool better = ranks_before(pt.ntkey, pt.ntw, ntkey, ntw);
            ntkey = better ? pt.ntkey : ntkey;
            ntw = better ? pt.ntw : ntw;
            nfeas += pt.nfeas;
            ncand += pt.ncand;
            ntcnt += pt.ntcnt;
            efeas = efeas | (pt.efeas != 0);
        }
    }
    if (!live) return;
    int32_t ex1 = INT32_MAX, w1 = -1, ex2 = INT32_MAX, w2 = -1;
    // the two smallest KV excesses feed only the diagnostics: merge the worker
    // blocks' two smallest keys (new first = smaller first; new second =
    // min(larger first, smaller second))
    if (act && st.out_diag) {
        const ulonglong2* prow = st.part + sc.part_off + (qi - start);
        uint64_t a1 = ~0ull, a2 = ~0ull;
#pragma unroll 8
        for (int b = 0; b < sc.nblk; ++b) {
            const ulonglong2 p = prow[(int64_t)b * sc.pstride];
            const uint64_t lo = p.x < a1 ? p.x : a1;
            const uint64_t hi = p.x < a1 ? a1 : p.x;
            const uint64_t s2 = p.y < a2 ? p.y : a2;
            a1 = lo;
            a2 = hi < s2 ? hi : s2;
        }
        ex_unpack(a1, ex1, w1);
        ex_unpack(a2, ex2, w2);
    }
    if (!act) return;
    QSum q;
#pragma unroll
    for (int k = 0; k < TOPK; ++k) { q.tkey[k] = tkey[k]; q.tw[k] = tw[k]; }
    q.ntkey = ntkey;
    q.ntw = ntw;
    q.ntcnt = ntcnt;
    q.nfeas = bulk_empty ? ncand + (efeas ? 1 : 0) : nfeas;  // bulk: > 0 exactly when some worker is feasible
    q.ncand = ncand;
    q.efeas = efeas ? 1 : 0;
    q.ex1 = ex1; q.w1 = w1;
    q.ex2 = ex2; q.w2 = w2;
    q.pad = 0;
    st.qsum[sc.qsum_off + (qi - start)] = q;
    if (q.nfeas > 0) {
        atomicMin(&st.tinfo[s].first_pc[parity], qi);
    } else if (st.qbad == nullptr || *st.qbad == 0) {
        // no feasible worker at tile start: rejected whatever the tile commits
        // before it.  These tile-start diagnostics are exact for the queries
        // before the tile's first commit; the commit overwrites every query
        // from its first feasible one on.
        if (st.out_worker) st.out_worker[sc.out_off + qi] = -1;
        if (st.out_diag) {
            Diag d;
            d.n_feasible = 0;
            d.near_tie = ntcnt > 0 ? 1 : 0;
            d.kv_peak_chosen = 0;
            d.kv_excess_min = ex1;
            d.ttft_chosen = 0.0;
            d.tdec_chosen = 0.0;
            st.out_diag[qi] = d;
        }
    }
}

// ---------------------------------------------------------------------------------------------
// Commit.  One wave per scenario walks the tile in arrival order.  Workers
// committed to earlier in the tile ("dirty") are re-evaluated from their live
// aggregates, kept in LDS; the worker last committed to keeps its live request
// columns in LDS.  A commit updates the columns in LDS, writes them through to
// HBM and only marks the worker's summaries stale: the build kernel of the next
// round rebuilds them.  Columns this wave wrote are read back only with
// device-coherent loads after a release fence.

constexpr int DBITS_W = 2048;  // dirty bitmap words in LDS: scenarios of up to 65536 workers

// Lane holding the best (key, index) by Algorithm 1's order among lanes with
// `valid`, or -1.  A scalar walk over the (few) candidate lanes.
__device__ __forceinline__ int wave_best_lane(uint64_t key, int32_t w, bool valid)
{
    uint64_t m = ballot(valid);
    int best = -1;
    uint64_t bk = 0;
    int32_t bw = -1;
    while (m) {
        const int l = __ffsll((unsigned long long)m) - 1;
        m &= m - 1;
        const uint64_t k = rdlane64(key, l);
        const int32_t ww = rdlane(w, l);
        if (ranks_before(k, ww, bk, bw)) {
            best = l;
            bk = k;
            bw = ww;
        }
    }
    return best;
}

// Column element: plain LDS read, or a device-coherent global read of data
// that this wave may have written earlier in the launch.
template <bool GLOBAL>
__device__ __forceinline__ int32_t col(const int32_t* p, int k)
{
    if (GLOBAL) return __hip_atomic_load(p + k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return p[k];
}

// KV demand peak with the query added, from a worker's live columns e, s
// (B entries sorted by e).  All lanes take part; all get the result, and the
// worker's peak without the query in *p0.  Lane l takes chunk 63 - l, so a
// prefix over lanes is a suffix over slots.  Every value here is a KV demand
// below 2^31 (the worker's peak is at most 2^30, the query adds l_in + l_pred).
template <bool GLOBAL>
__device__ int64_t wave_kv_peak(const int32_t* e, const int32_t* s, int B, int32_t sq, int32_t eq, int32_t* p0)
{
    const int lane = lane_id();
    const int CH = (B + 63) >> 6;
    const int c = 63 - lane;
    const int k0 = min(B, c * CH);
    const int k1 = min(B, k0 + CH);
    int32_t ls = 0;
    for (int k = k0; k < k1; ++k) ls += col<GLOBAL>(s, k);
    int64_t run = (int64_t)(wave_incl_scan(ls, 0, Add32()) - ls);  // slots after this chunk
    int32_t best = INT32_MIN, best0 = 0, ssge = 0, cge = 0;
    for (int k = k1 - 1; k >= k0; --k) {
        const int32_t ek = col<GLOBAL>(e, k), sk = col<GLOBAL>(s, k);
        run += sk;  // sum of s over slots >= k
        const int64_t P = run + (int64_t)(B - k) * ek;
        const bool before = ek < eq;  // the query is still alive at this end point
        const int32_t val = (int32_t)(before ? P + sq + ek : P);
        best = val > best ? val : best;
        best0 = (int32_t)P > best0 ? (int32_t)P : best0;
        ssge += before ? 0 : sk;
        cge += before ? 0 : 1;
    }
    *p0 = wave_max32(best0);
    const int64_t bmax = wave_max32(best);
    const int64_t own = (int64_t)wave_sum32(ssge) + (int64_t)wave_sum32(cge) * eq + sq + eq;
    return bmax > own ? bmax : own;
}

// The same, evaluated by one lane alone.
template <bool GLOBAL>
__device__ int64_t lane_kv_peak(const int32_t* e, const int32_t* s, int B, int32_t sq, int32_t eq)
{
    int64_t run = 0, best = INT64_MIN, ssge = 0, cge = 0;
    for (int k = B - 1; k >= 0; --k) {
        const int32_t ek = col<GLOBAL>(e, k), sk = col<GLOBAL>(s, k);
        run += sk;
        const int64_t P = run + (int64_t)(B - k) * ek;
        const bool before = ek < eq;
        const int64_t val = before ? P + sq + ek : P;
        best = val > best ? val : best;
        ssge += before ? 0 : sk;
        cge += before ? 0 : 1;
    }
    const int64_t own = ssge + cge * eq + sq + eq;
    return best > own ? best : own;
}

// Orders LDS traffic between the lanes of the (single-wave) commit block
// without waiting for outstanding global memory operations.
__device__ __forceinline__ void wave_sync() { __builtin_amdgcn_wave_barrier(); }

// A worker committed to earlier in the tile.  The commit wave holds the j-th
// such worker in lane j's registers.
struct DAgg {
    int32_t w;       // scenario-local index, -1 = none
    int32_t B, n, head, M, hbs;
    int32_t empty0;  // it was empty when the tile started
    int32_t cap;
    int32_t pub;     // upper bound of its KV peak without a new query (exact after a scan)
    int32_t pad;
    int64_t base;    // first slot
    int64_t DS, S1, S2, SC, SR;
    uint64_t key;
    double rhs;
};

// Bit words of the tile-start feasibility / near-tie masks that cover one
// 64-query window, cached per dirty worker (one worker per lane).
struct WinBits {
    uint64_t f0, f1, n0, n1;
};

__device__ __forceinline__ WinBits load_win_bits(const State& st, const Scen& sc, int w, int start, int w0, int end)
{
    WinBits b;
    const int64_t g0 = (w0 - start) >> 6;
    const int64_t row0 = sc.bits_off + g0 * sc.W + w;
    b.f0 = st.bits_feas[row0];
    b.n0 = st.bits_nt[row0];
    const bool two = (int64_t)(end - start) > (g0 + 1) * 64;
    b.f1 = two ? st.bits_feas[row0 + sc.W] : 0;
    b.n1 = two ? st.bits_nt[row0 + sc.W] : 0;
    return b;
}

// bit of query i (tile offset) in a cached window
__device__ __forceinline__ bool win_bit(uint64_t lo, uint64_t hi, int start, int w0, int i)
{
    const int g = ((i - start) >> 6) - ((w0 - start) >> 6);
    const uint64_t word = g == 0 ? lo : hi;
    return (word >> ((i - start) & 63)) & 1;
}

__device__ __forceinline__ View dagg_view(const DAgg& a, int32_t hb)
{
    View v;
    v.e = nullptr;
    v.pms = nullptr;
    v.head = a.head;
    v.n = a.n;
    v.M = a.M;
    v.DS = a.DS;
    const bool cur = a.hbs == hb;
    v.S1 = cur ? a.S1 : 0;
    v.S2 = cur ? a.S2 : 0;
    v.key = a.key;
    v.rhs = a.rhs;
    return v;
}

// Per-launch commit state held in LDS.  dag[] mirrors the lanes' DAgg for the
// per-lane diagnostics of rejected queries (diagnostics only); dw[] and dbits
// say which workers are dirty.
struct CommitLDS {
    DAgg dag[MAX_DIRTY];
    int32_t dw[MAX_DIRTY];
    uint32_t dbits[DBITS_W];
    int32_t he[HOT];
    int32_t hs[HOT];
};

// Is worker w (scenario-local) dirty in this tile?  (any lane, any w)
__device__ __forceinline__ bool dirty_w(const CommitLDS& L, int W, int nd, int w)
{
    if (W <= DBITS_W * 32) return (L.dbits[w >> 5] >> (w & 31)) & 1u;
    bool d = false;
    for (int j = 0; j < nd; ++j) d = d | (L.dw[j] == w);
    return d;
}

// Lane holding dirty worker w (wave-uniform w; -1 if w is not dirty).
__device__ __forceinline__ int dirty_lane(const DAgg& a, int w)
{
    const uint64_t m = ballot(a.w == w && w >= 0);
    return m ? __ffsll((unsigned long long)m) - 1 : -1;
}

// Lowest-index worker at or after `from` that is empty and untouched in this
// tile (wave-cooperative; -1 if none).  Empty workers have rank key 0.
__device__ int next_empty_worker(const State& st, const Scen& sc, const CommitLDS& L, int nd, int from)
{
    for (int base = from; base < sc.W; base += 64) {
        const int w = base + lane_id();
        const bool emp = w < sc.W && st.key[sc.wbase + w] == 0 && !dirty_w(L, sc.W, nd, w);
        const uint64_t m = ballot(emp);
        if (m) return base + __ffsll((unsigned long long)m) - 1;
    }
    return -1;
}

struct QView {  // the committing query's summary, broadcast to the whole wave
    uint64_t tkey[TOPK];
    int32_t tw[TOPK];
    uint64_t ntkey;
    int32_t ntw, ntcnt, nfeas, ncand, efeas, ex1, w1, ex2, w2;
};

__device__ __forceinline__ QView broadcast_q(const QSum& q, int p)
{
    QView v;
#pragma unroll
    for (int k = 0; k < TOPK; ++k) {
        v.tkey[k] = rdlane64(q.tkey[k], p);
        v.tw[k] = rdlane(q.tw[k], p);
    }
    v.ntkey = rdlane64(q.ntkey, p);
    v.ntw = rdlane(q.ntw, p);
    v.ntcnt = rdlane(q.ntcnt, p);
    v.nfeas = rdlane(q.nfeas, p);
    v.ncand = rdlane(q.ncand, p);
    v.efeas = rdlane(q.efeas, p);
    v.ex1 = rdlane(q.ex1, p);
    v.w1 = rdlane(q.w1, p);
    v.ex2 = rdlane(q.ex2, p);
    v.w2 = rdlane(q.w2, p);
    return v;
}

// Diagnostics of a query with no feasible worker at tile start (so none now),
// decided by its own lane (diagnostics only: reads the LDS mirror of the dirty
// workers).
__device__ Diag reject_diag(const State& st, const Scen& sc, const QSum& q, int i, int start, int w0, int32_t lin,
                            int32_t lp, int32_t tau, int32_t hb, const CommitLDS& L, int nd, int hot,
                            const WinBits& wb, int* abort)
{
    Diag d;
    d.n_feasible = 0;
    d.kv_peak_chosen = 0;
    d.ttft_chosen = 0.0;
    d.tdec_chosen = 0.0;
    d.kv_excess_min = 0;
    d.near_tie = 0;
    *abort = 0;
    const int32_t sq = lin - tau, eq = lp + tau;
    int64_t exmin = q.ex1;
    if (q.w1 >= 0 && dirty_w(L, sc.W, nd, q.w1)) {
        if (q.w2 >= 0 && dirty_w(L, sc.W, nd, q.w2)) {
            *abort = 1;
            return d;
        }
        int j = 0;
        while (j < nd && L.dw[j] != q.w1) ++j;
        const DAgg& a = L.dag[j];
        const int64_t base = a.base + a.head;
        const int64_t pk = (j == hot) ? lane_kv_peak<false>(L.he, L.hs, a.B, sq, eq)
                                      : lane_kv_peak<true>(st.e + base, st.s + base, a.B, sq, eq);
        const int64_t ex_now = pk - a.M;
        exmin = q.w2 < 0 ? ex_now : (ex_now < q.ex2 ? ex_now : (int64_t)q.ex2);
    }
    d.kv_excess_min = exmin;
    // near tie over every worker (the query is rejected)
    int clean_nt = q.ntcnt;
    bool nt = false;
    for (int j = 0; j < nd; ++j) {
        const DAgg& a = L.dag[j];
        const uint64_t n0 = rdlane64(wb.n0, j), n1 = rdlane64(wb.n1, j);
        clean_nt -= win_bit(n0, n1, start, w0, i) ? 1 : 0;
        nt = nt | latency(sc, dagg_view(a, hb), lin, lp, a.B + 1).nt;
    }
    nt = nt | (clean_nt > 0);
    d.near_tie = nt ? 1 : 0;
    return d;
}

struct Decision {
    int32_t w;      // chosen worker, -1 = rejected
    int32_t lane;   // dirty lane holding w, -1 when w was untouched in the tile
    int32_t abort;  // the tile-start lists cannot decide this query exactly
    Diag d;
};

// Exact KV scans a decision ran, per lane.
struct Scan {
    bool done;   // this lane's worker was scanned for the query
    int32_t pk;  // its KV peak with the query
    int32_t p0;  // its KV peak without
};

// Number of entries of the sorted a[0, n) that are <= x.
__device__ __forceinline__ int upper_bound_i32(const int32_t* a, int n, int32_t x)
{
    int lo = 0, len = n;
    while (len > 0) {
        const int half = len >> 1;
        const bool right = a[lo + half] <= x;
        lo = right ? lo + half + 1 : lo;
        len = right ? len - half - 1 : half;
    }
    return lo;
}

// Insert (x, y) into the sorted LDS columns he/hs[0, B), after every entry
// with he <= x (whole wave; the columns must have room for B + 1 entries).
__device__ __forceinline__ void lds_sorted_insert(CommitLDS& L, int B, int32_t x, int32_t y)
{
    const int lane = lane_id();
    int u = 0;
    for (int k0 = 0; k0 < B; k0 += COMMIT_THREADS)
        u += __popcll(ballot(k0 + lane < B && L.he[k0 + lane] <= x));
    // shift [u, B) up by one, highest block first (each pass reads before it writes)
    for (int top = B; top > u; top -= COMMIT_THREADS) {
        const int k = top - COMMIT_THREADS + lane;
        const bool mv = k >= u && k < top;
        int32_t ve = 0, vs = 0;
        if (mv) {
            ve = L.he[k];
            vs = L.hs[k];
        }
        wave_sync();
        if (mv) {
            L.he[k + 1] = ve;
            L.hs[k + 1] = vs;
        }
        wave_sync();
    }
    if (lane == 0) {
        L.he[u] = x;
        L.hs[u] = y;
    }
    wave_sync();
}

// The hot worker's LDS columns are a sorted prefix [0, Bs) and, without
// diagnostics, an unsorted tail [Bs, Bs + m) of requests committed since it
// became hot, in commit order.  Sort the tail into the prefix (in commit order,
// so equal end points keep the order a sorted insert would give them).
__device__ __noinline__ int lds_merge_tail(CommitLDS& L, int Bs, int m)
{
    for (int t = 0; t < m; ++t) {
        const int32_t x = L.he[Bs + t], y = L.hs[Bs + t];  // read before the insert may move it
        lds_sorted_insert(L, Bs + t, x, y);
    }
    return Bs + m;
}

// KV peak with the query for dirty lane bl (whole wave): the hot worker's
// columns from LDS (its tail sorted in first), the others from HBM.
__device__ __forceinline__ int64_t dirty_kv_peak(const State& st, CommitLDS& L, const DAgg& a, int bl, int hot,
                                                 int& hotBs, int& hotm, int32_t sq, int32_t eq, int32_t* p0)
{
    const int32_t cB = rdlane(a.B, bl);
    if (bl == hot) {
        if (hotm > 0) {
            hotBs = lds_merge_tail(L, hotBs, hotm);
            hotm = 0;
        }
        return wave_kv_peak<false>(L.he, L.hs, cB, sq, eq, p0);
    }
    const int64_t base = rdlane64s(a.base, bl) + rdlane(a.head, bl);
    return wave_kv_peak<true>(st.e + base, st.s + base, cB, sq, eq, p0);
}

// Decide one query with the whole wave.  `a` is this lane's dirty worker.
__device__ Decision decide(const State& st, const Scen& sc, const QView& q, int i, int start, int w0, int32_t lin,
                           int32_t lp, int32_t tau, int32_t hb, CommitLDS& L, int nd, int hot, int& hotBs,
                           int& hotm, int next_empty, bool want_diag, const WinBits& wb, const DAgg& a, Scan& sn)
{
    Decision r;
    r.w = -1;
    r.lane = -1;
    r.abort = 0;
    r.d.n_feasible = 0;
    r.d.near_tie = 0;
    r.d.kv_peak_chosen = 0;
    r.d.kv_excess_min = 0;
    r.d.ttft_chosen = 0.0;
    r.d.tdec_chosen = 0.0;
    sn.done = false;
    sn.pk = sn.p0 = 0;
    const int lane = lane_id();
    const int32_t sq = lin - tau, eq = lp + tau;
    // best untouched candidate from the tile-start list
    bool have = false;
    uint64_t bk = 0;
    int32_t bw = -1;
    const int lim = q.ncand < TOPK ? q.ncand : TOPK;
#pragma unroll
    for (int k = 0; k < TOPK; ++k) {
        const int w = q.tw[k];
        const bool listed = (k < lim) && (w >= 0);
        const bool clean = listed && dirty_lane(a, w) < 0;
        const bool take = clean & !have;
        bk = take ? q.tkey[k] : bk;
        bw = take ? w : bw;
        have = have | take;
    }
    if (!have && q.ncand > TOPK) {
        r.abort = 1;
        return r;
    }
    if (!have && sc.uniform_M && q.efeas && next_empty >= 0) {
        have = true;
        bk = 0;
        bw = next_empty;
    }
    // workers changed earlier in the tile: one per lane
    const bool valid = lane < nd;
    bool fs = false, ns = false;
    Latency Lt;
    Lt.dec_ok = Lt.ttft_ok = Lt.nt = false;
    Lt.lhs = Lt.ttft = Lt.tdec = 0.0;
    if (valid) {
        fs = (sc.uniform_M && a.empty0) ? (q.efeas != 0) : win_bit(wb.f0, wb.f1, start, w0, i);
        ns = win_bit(wb.n0, wb.n1, start, w0, i);
        Lt = latency(sc, dagg_view(a, hb), lin, lp, a.B + 1);
    }
    const bool unknown = valid && fs && Lt.dec_ok && Lt.ttft_ok;  // KV check still needed

    if (!want_diag) {
        // best-ranked first, stop at the first feasible one; a worker whose peak
        // bound plus the query's own demand fits needs no scan (the query adds at
        // most l_in + l_pred to the demand at any iteration)
        bool cand = unknown && ranks_before(a.key, a.w, bk, bw);
        const bool sure = cand && (int64_t)a.pub + lin + lp <= (int64_t)a.M;
        for (;;) {
            const int bl = wave_best_lane(a.key, a.w, cand);
            if (bl < 0) break;
            if ((ballot(sure) >> bl) & 1) {
                r.w = rdlane(a.w, bl);
                r.lane = bl;
                return r;
            }
            int32_t p0;
            const int64_t pk = dirty_kv_peak(st, L, a, bl, hot, hotBs, hotm, sq, eq, &p0);
            if (lane == bl) {
                sn.done = true;
                sn.pk = (int32_t)pk;
                sn.p0 = p0;
                cand = false;
            }
            if (pk <= rdlane(a.M, bl)) {
                r.w = rdlane(a.w, bl);
                r.lane = bl;
                return r;
            }
        }
        r.w = have ? bw : -1;
        return r;
    }

    // ---- with diagnostics: every dirty candidate is scanned
    bool cand = unknown;
    bool feas_now = false;
    for (;;) {
        const int bl = wave_best_lane(a.key, a.w, cand);
        if (bl < 0) break;
        int32_t p0;
        const int64_t pk = dirty_kv_peak(st, L, a, bl, hot, hotBs, hotm, sq, eq, &p0);
        const bool ok = pk <= rdlane(a.M, bl);
        if (lane == bl) {
            cand = false;
            feas_now = ok;
            sn.done = true;
            sn.pk = (int32_t)pk;
            sn.p0 = p0;
        }
    }
    const bool fdirty = valid && feas_now;
    {
        const int bl = wave_best_lane(a.key, a.w, fdirty);
        if (bl >= 0) {
            const uint64_t dk = rdlane64(a.key, bl);
            const int32_t dw = rdlane(a.w, bl);
            if (!have || ranks_before(dk, dw, bk, bw)) {
                have = true;
                bk = dk;
                bw = dw;
                r.lane = bl;
            }
        }
    }
    r.w = have ? bw : -1;
    r.d.n_feasible = q.nfeas - __popcll(ballot(valid && fs)) + __popcll(ballot(fdirty));
    // smallest KV excess
    int64_t exmin = q.ex1;
    const int j1 = dirty_lane(a, q.w1);
    if (q.w1 >= 0 && j1 >= 0) {
        if (q.w2 >= 0 && dirty_lane(a, q.w2) >= 0) {
            r.abort = 1;
            return r;
        }
        int32_t p0;
        const int64_t pk = dirty_kv_peak(st, L, a, j1, hot, hotBs, hotm, sq, eq, &p0);
        const int64_t ex_now = pk - rdlane(a.M, j1);
        exmin = q.w2 < 0 ? ex_now : (ex_now < q.ex2 ? ex_now : (int64_t)q.ex2);
    }
    r.d.kv_excess_min = exmin;
    // near tie among workers ranked at or above the choice (all when rejected)
    const int clean_nt = q.ntcnt - __popcll(ballot(valid && ns));
    bool nt = false;
    if (clean_nt > 0) {
        if (q.ntw >= 0 && dirty_lane(a, q.ntw) < 0) {
            nt = r.w < 0 || !ranks_before(bk, bw, q.ntkey, q.ntw);
        } else if (r.w < 0) {
            nt = true;
        } else {
            r.abort = 1;
            return r;
        }
    }
    const bool dnt = valid && Lt.nt && (r.w < 0 || !ranks_before(bk, bw, a.key, a.w));
    nt = nt | (ballot(dnt) != 0);
    r.d.near_tie = nt ? 1 : 0;
    // the chosen worker's figures
    if (r.w >= 0) {
        if (r.lane >= 0) {
            r.d.kv_peak_chosen = rdlane(sn.pk, r.lane);
            r.d.ttft_chosen = rdlane_f64(Lt.ttft, r.lane);
            r.d.tdec_chosen = rdlane_f64(Lt.tdec, r.lane);
        } else {
            // untouched in this tile: its summaries are current
            const View v = load_view(st, sc.wbase + r.w, hb);
            const Latency Lc = latency(sc, v, lin, lp, v.n - v.head + 1);
            r.d.kv_peak_chosen = kv_peak_with(v, sq, eq);
            r.d.ttft_chosen = Lc.ttft;
            r.d.tdec_chosen = Lc.tdec;
        }
    }
    return r;
}

// Write the hot worker's LDS columns back to its slot range in sorted order
// (from slot 0 when the range would run past the worker's last slot) and
// point its aggregates at them.  A prefix entry moves up by the number of tail
// entries ending strictly before it; a tail entry lands after every prefix
// entry ending no later and after earlier tail entries ending no later.  Whole
// wave.
__device__ void writeback_hot(const State& st, CommitLDS& L, DAgg& a, int hot, int Bs, int m, bool mirror)
{
    const int lane = lane_id();
    const int B = Bs + m;
    const int cap = rdlane(a.cap, hot);
    const int head0 = rdlane(a.head, hot);
    const int head = head0 + B <= cap ? head0 : 0;
    int32_t* ge = st.e + rdlane64s(a.base, hot) + head;
    int32_t* gs = st.s + rdlane64s(a.base, hot) + head;
    for (int k0 = 0; k0 < Bs; k0 += COMMIT_THREADS) {
        const int k = k0 + lane;
        const bool in = k < Bs;
        const int32_t x = in ? L.he[k] : 0, y = in ? L.hs[k] : 0;
        int cnt = 0;
        for (int t0 = 0; t0 < m; t0 += COMMIT_THREADS) {
            const int32_t tv = t0 + lane < m ? L.he[Bs + t0 + lane] : INT32_MAX;
            const int lim = min(COMMIT_THREADS, m - t0);
            for (int jj = 0; jj < lim; ++jj) cnt += rdlane(tv, jj) < x ? 1 : 0;
        }
        if (in) {
            ge[k + cnt] = x;
            gs[k + cnt] = y;
        }
    }
    for (int t0 = 0; t0 < m; t0 += COMMIT_THREADS) {
        const int t = t0 + lane;
        const bool in = t < m;
        const int32_t x = in ? L.he[Bs + t] : 0, y = in ? L.hs[Bs + t] : 0;
        int pos = upper_bound_i32(L.he, Bs, x);
        for (int u0 = 0; u0 < m; u0 += COMMIT_THREADS) {
            const int32_t tv = u0 + lane < m ? L.he[Bs + u0 + lane] : INT32_MAX;
            const int lim = min(COMMIT_THREADS, m - u0);
            for (int jj = 0; jj < lim; ++jj) {
                const int32_t v = rdlane(tv, jj);
                pos += (v < x || (v == x && u0 + jj < t)) ? 1 : 0;
            }
        }
        if (in) {
            ge[pos] = x;
            gs[pos] = y;
        }
    }
    if (lane == hot) {
        a.head = head;
        a.n = head + B;
        if (mirror) L.dag[hot] = a;
    }
}

template <bool DIAG>
__global__ __launch_bounds__(COMMIT_THREADS) void k_commit(State st)
{
    constexpr int NT = COMMIT_THREADS;
    const int s = find_scen<&Scen::fin_blk0>(st, blockIdx.x);
    const Scen sc = st.scen[s];
    const int part = blockIdx.x - sc.fin_blk0;  // 0: one block per scenario
    const TileInfo ti = st.tinfo[s];
    Ctl* cp = st.ctl + s;
    const int lane = threadIdx.x;
    // the control block as the host will read it (after the stream synchronises)
    auto publish = [&]() {
        if (st.ctl_host != nullptr && part == 0 && lane == 0) st.ctl_host[s] = *cp;
    };
    if (st.qbad != nullptr && *st.qbad) {  // an invalid query length: nothing is written
        if (part == 0 && lane == 0) cp->err = DEV_EINVAL;
        publish();
        return;
    }
    if (ti.start >= ti.end) {
        publish();
        return;
    }
    const int32_t start = ti.start, end = ti.end;
    const int32_t fpc = min(st.tinfo[s].first_pc[ti.parity & 1], end);  // (no local copy indexed at run time)

    // ---- the sequential wave
    const Ctl c = *cp;
    if (c.err) {
        publish();
        return;
    }
    const int32_t tau = c.tau, hb = c.hb_index;
    __shared__ CommitLDS L;
    if (sc.W <= DBITS_W * 32)
        for (int k = lane; k < (sc.W + 31) / 32; k += NT) L.dbits[k] = 0u;
    if (lane == 0) cp->rebuild = 0;
    wave_sync();
    constexpr bool want_diag = DIAG;  // st.out_diag != nullptr
    int nd = 0;    // dirty workers (wave-uniform); lane j < nd holds the j-th in `a`
    DAgg a;
    a.w = -1;
    a.B = a.n = a.head = a.M = a.hbs = a.empty0 = a.cap = a.pub = a.pad = 0;
    a.base = 0;
    a.DS = a.S1 = a.S2 = a.SC = a.SR = 0;
    a.key = 0;
    a.rhs = 0.0;
    // The hot worker's sorted live columns are in L.he / L.hs and its HBM copy
    // is stale until it is written back (when another worker becomes hot, and at
    // the end); every other dirty worker's columns are current in HBM and are
    // read with device-coherent loads after the write-back's release fence.
    int hot = -1;
    int hotBs = 0, hotm = 0;  // the hot worker's sorted prefix and unsorted tail in L.he / L.hs
    // lowest-index empty untouched worker, looked up only when a decision can
    // use it (-2 = not looked up yet; the search resumes at next_from)
    int next_empty = sc.uniform_M ? -2 : -1;
    int next_from = 0;
    int pos = fpc;
    bool cut = false, err = false;
    int commits = 0;
    int nrej = fpc - start;  // the rejected prefix (its outputs come from the selection kernel)
    int firstrej = fpc > start ? start : INT32_MAX;
    WinBits wb;
    wb.f0 = wb.f1 = wb.n0 = wb.n1 = 0;
    while (pos < end && !cut) {
        // one window of 64 queries; `cur` is the first undecided lane
        const int w0 = pos;
        const int i = w0 + lane;
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
        if (lane < nd) wb = load_win_bits(st, sc, a.w, start, w0, end);
        const uint64_t potm = ballot(act && q.nfeas > 0);
        int cur = 0;
        while (cur < NT && w0 + cur < end) {
            const uint64_t pm = potm & (~0ull << cur);
            const int p = pm ? __ffsll((unsigned long long)pm) - 1 : NT;
            // lanes cur..p-1: rejected whatever happened earlier in the tile
            Diag dr;
            int ab = 0;
            const bool mine = act && lane >= cur && lane < p;
            if (want_diag && mine) dr = reject_diag(st, sc, q, i, start, w0, lin, lp, tau, hb, L, nd, hot, wb, &ab);
            const uint64_t am = ballot(mine && ab);
            const int abl = am ? __ffsll((unsigned long long)am) - 1 : NT;
            const int lim = min(p, abl);
            if (act && lane >= cur && lane < lim) {
                if (st.out_worker) st.out_worker[sc.out_off + i] = -1;
                if (want_diag) st.out_diag[i] = dr;
            }
            const uint64_t rm = ballot(act && lane >= cur && lane < lim);
            nrej += __popcll(rm);
            if (rm && firstrej == INT32_MAX) firstrej = w0 + __ffsll((unsigned long long)rm) - 1;
            if (abl < p) {
                pos = w0 + abl;
                cut = true;
                break;
            }
            if (p >= NT) {
                cur = NT;
                break;
            }
            // the query of lane p, decided by the whole wave
            const int ip = w0 + p;
            const QView qv = broadcast_q(q, p);
            const int32_t plin = rdlane(lin, p), plp = rdlane(lp, p);
            if (next_empty == -2 && qv.efeas) next_empty = next_empty_worker(st, sc, L, nd, next_from);
            Scan sn;
            const Decision dc = decide(st, sc, qv, ip, start, w0, plin, plp, tau, hb, L, nd, hot, hotBs, hotm,
                                       next_empty, want_diag, wb, a, sn);
            if (dc.abort) {
                pos = ip;
                cut = true;
                break;
            }
            if (lane == 0) {
                if (st.out_worker) st.out_worker[sc.out_off + ip] = dc.w;
                if (want_diag) st.out_diag[ip] = dc.d;
            }
            cur = p + 1;
            // a scanned worker that does not take the query keeps its exact peak
            if (sn.done && lane != dc.lane) a.pub = sn.p0;
            if (dc.w < 0) {
                nrej += 1;
                if (firstrej == INT32_MAX) firstrej = ip;
                continue;
            }

            // ---- commit the query to worker w
            const int w = dc.w;
            int j = dc.lane;
            if (j < 0) {  // first commit to w in this tile: its tile-start state is in HBM
                j = nd;
                const int gw = sc.wbase + w;
                if (lane == j) {
                    a.w = w;
                    a.n = st.n[gw];
                    a.head = st.head[gw];
                    a.B = st.B[gw];
                    a.M = st.M[gw];
                    a.hbs = st.hbs[gw];
                    a.empty0 = a.B == 0 ? 1 : 0;
                    a.cap = st.cap[gw];
                    a.pub = a.B == 0 ? 0 : st.peak[gw];
                    a.base = st.slot_base[gw];
                    a.DS = st.DS[gw];
                    a.S1 = st.S1[gw];
                    a.S2 = st.S2[gw];
                    a.SC = st.SC[gw];
                    a.SR = st.SR[gw];
                    a.key = st.key[gw];
                    a.rhs = st.rhs[gw];
                    wb = load_win_bits(st, sc, w, start, w0, end);
                }
                if (lane == 0) {
                    L.dw[j] = w;
                    if (sc.W <= DBITS_W * 32) L.dbits[w >> 5] |= 1u << (w & 31);
                }
                nd += 1;
            }
            const int B0 = rdlane(a.B, j);
            if (B0 + 1 > rdlane(a.cap, j)) {  // no slot left for one more live request
                if (lane == 0) raise_error(&cp->err, DEV_ESLOTS);
                err = true;
                cut = true;
                pos = ip + 1;
                break;
            }
            if (hot != j) {
                if (hot >= 0) {
                    writeback_hot(st, L, a, hot, hotBs, hotm, want_diag);
                    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
                }
                const int64_t gb = rdlane64s(a.base, j) + rdlane(a.head, j);
                for (int k = lane; k < B0; k += NT) {
                    L.he[k] = col<true>(st.e + gb, k);
                    L.hs[k] = col<true>(st.s + gb, k);
                }
                hot = j;
                hotBs = B0;
                hotm = 0;
            }
            wave_sync();
            const int32_t eq = plp + tau, sq = plin - tau;
            if (want_diag) {
                // the per-lane diagnostics of rejected queries read sorted columns
                lds_sorted_insert(L, B0, eq, sq);
                hotBs = B0 + 1;
            } else {
                if (lane == 0) {
                    L.he[B0] = eq;
                    L.hs[B0] = sq;
                }
                hotm += 1;
                wave_sync();
            }
            // aggregates of lane j
            if (lane == j) {
                const int B1 = B0 + 1;
                a.B = B1;
                a.SC += plin;
                a.SR += plp;
                a.DS += ((int64_t)plin << sc.gs) + (int64_t)sc.gn * plp;
                const int64_t X = (int64_t)B1 << sc.gs;
                if (a.DS >= ((int64_t)1 << 31) || X >= ((int64_t)1 << 31)) raise_error(&cp->err, DEV_EOVERFLOW);
                a.key = (uint64_t)(X * X) + (uint64_t)(a.DS * a.DS);
                a.rhs = sc.theta * ((sc.tdec - sc.c3) - sc.c2 * (double)(B1 + 1));
                const bool curhb = a.hbs == hb;
                a.S1 = (curhb ? a.S1 : 0) + plin;
                a.S2 = (curhb ? a.S2 : 0) + (int64_t)plin * plin;
                a.hbs = hb;
                if (a.S2 >= ((int64_t)1 << 53)) raise_error(&cp->err, DEV_EOVERFLOW);
                // exact peak when this decision scanned the worker, else a bound
                a.pub = sn.done ? sn.pk : (int32_t)((int64_t)a.pub + plin + plp);
                if (want_diag) L.dag[j] = a;
            }
            wave_sync();
            ++commits;
            if (w == next_empty) {
                next_empty = -2;
                next_from = w + 1;
            }
            if (nd >= MAX_DIRTY && w0 + cur < end) {
                pos = w0 + cur;
                cut = true;
                break;
            }
        }
        if (err) break;
        if (!cut) pos = min(end, w0 + NT);
    }
    // write back the hot worker's columns and every dirty worker's aggregates;
    // list the workers whose summaries the next round must rebuild
    if (hot >= 0) writeback_hot(st, L, a, hot, hotBs, hotm, false);
    if (lane < nd) {
        const int gw = sc.wbase + a.w;
        st.n[gw] = a.n;
        st.head[gw] = a.head;
        st.B[gw] = a.B;
        st.SC[gw] = a.SC;
        st.SR[gw] = a.SR;
        st.DS[gw] = a.DS;
        st.key[gw] = a.key;
        st.rhs[gw] = a.rhs;
        st.S1[gw] = a.S1;
        st.S2[gw] = a.S2;
        st.hbs[gw] = a.hbs;
        st.built[gw] = 0;
        st.dlist[s * MAX_DIRTY + lane] = gw;
    }
    if (lane == 0) {
        if (nrej) atomicAdd(&cp->n_rej, nrej);
        if (firstrej != INT32_MAX) atomicMin(&cp->first_rej, firstrej);
        st.dcount[s] = nd;
        cp->ndirty = nd;
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
    publish();
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

// Start of an ald_place_stream call (one scenario): the control block, the
// tile record and a cleared query-error word (the first round's pair
// evaluation checks the query lengths).
__global__ void k_begin(Ctl c, TileInfo ti, Ctl* ctl, TileInfo* tinfo, int32_t* qbad)
{
    *ctl = c;
    *tinfo = ti;
    *qbad = 0;
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

hipError_t launch_build(const State& st, hipStream_t stream, int mode)
{
    const int blocks = mode == 1 ? st.S * MAX_DIRTY : st.NW;
    hipLaunchKernelGGL(k_build, dim3(blocks), dim3(BUILD_THREADS), 0, stream, st, mode);
    return hipGetLastError();
}

hipError_t launch_eval(const State& st, int32_t blocks, int mode, hipStream_t stream)
{
    const bool ex = st.out_diag != nullptr;
    const dim3 g(blocks), b(EVAL_THREADS);
    if (mode == 2) {
        if (ex) hipLaunchKernelGGL((k_eval<2, true>), g, b, 0, stream, st);
        else hipLaunchKernelGGL((k_eval<2, false>), g, b, 0, stream, st);
    } else if (mode == 1) {
        if (ex) hipLaunchKernelGGL((k_eval<1, true>), g, b, 0, stream, st);
        else hipLaunchKernelGGL((k_eval<1, false>), g, b, 0, stream, st);
    } else {
        if (ex) hipLaunchKernelGGL((k_eval<0, true>), g, b, 0, stream, st);
        else hipLaunchKernelGGL((k_eval<0, false>), g, b, 0, stream, st);
    }
    return hipGetLastError();
}

hipError_t launch_select(const State& st, int32_t blocks, hipStream_t stream)
{
    hipLaunchKernelGGL(k_select, dim3(blocks), dim3(SEL_THREADS), 0, stream, st);
    return hipGetLastError();
}

hipError_t launch_commit(const State& st, int32_t blocks, hipStream_t stream)
{
    if (st.out_diag != nullptr)
        hipLaunchKernelGGL(k_commit<true>, dim3(blocks), dim3(COMMIT_THREADS), 0, stream, st);
    else
        hipLaunchKernelGGL(k_commit<false>, dim3(blocks), dim3(COMMIT_THREADS), 0, stream, st);
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

hipError_t launch_begin(const Ctl& c, const TileInfo& ti, Ctl* ctl, TileInfo* tinfo, int32_t* qbad,
                        hipStream_t stream)
{
    hipLaunchKernelGGL(k_begin, dim3(1), dim3(1), 0, stream, c, ti, ctl, tinfo, qbad);
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
