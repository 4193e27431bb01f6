// Device primitives shared by the kernels of libaladdin: block and wave scans
// and reductions, cross-lane reads, the order of Algorithm 1, and the pair
// checks of constraints (b), (c), (d) and (e) on one worker's view.
#pragma once

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

// An int64 that orders like the double it encodes (finite values and +inf).
__device__ __forceinline__ int64_t ord_of(double x)
{
    const int64_t b = __builtin_bit_cast(int64_t, x);
    return b >= 0 ? b : (b ^ INT64_MAX);
}
__device__ __forceinline__ double double_of(int64_t k)
{
    return __builtin_bit_cast(double, k >= 0 ? k : (k ^ INT64_MAX));
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
    double dlim;  // constraint (d)'s limit on the prefill time (+inf: none)
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
    v.dlim = st.dlim[gw];
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
    // (c) and (d) bound the same prefill time
    const bool has_d = v.dlim != INFINITY;
    o.ttft_ok = o.ttft <= sc.ttft && (!has_d || o.ttft <= v.dlim);
    o.nt = near_tie(o.lhs, v.rhs) || (sc.ttft != INFINITY && near_tie(o.ttft, sc.ttft)) ||
           (has_d && near_tie(o.ttft, v.dlim));
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
struct Min32 {
    __device__ int32_t operator()(int32_t a, int32_t b) const { return a < b ? a : b; }
};
__device__ __forceinline__ int32_t wave_sum32(int32_t v) { return rdlane(wave_incl_scan(v, 0, Add32()), 63); }
__device__ __forceinline__ int32_t wave_min32(int32_t v) { return rdlane(wave_incl_scan(v, INT32_MAX, Min32()), 63); }
// Largest 64-bit unsigned value over the 64 lanes: the same scan on both
// halves of the word, the comparison on the whole word.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t ident, uint64_t x)
{
    const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)ident, (int)(uint32_t)x, CTRL, ROW_MASK,
                                                              0xf, false);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)(ident >> 32), (int)(uint32_t)(x >> 32),
                                                              CTRL, ROW_MASK, 0xf, false);
    return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t x)
{
    auto mx = [](uint64_t a, uint64_t b) { return a > b ? a : b; };
    x = mx(x, dpp_u64<0x111, 0xf>(0, x));  // row_shr:1
    x = mx(x, dpp_u64<0x112, 0xf>(0, x));  // row_shr:2
    x = mx(x, dpp_u64<0x114, 0xf>(0, x));  // row_shr:4
    x = mx(x, dpp_u64<0x118, 0xf>(0, x));  // row_shr:8
    x = mx(x, dpp_u64<0x142, 0xa>(0, x));  // row_bcast:15
    x = mx(x, dpp_u64<0x143, 0xc>(0, x));  // row_bcast:31
    return rdlane64(x, 63);
}
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

}  // namespace ald
