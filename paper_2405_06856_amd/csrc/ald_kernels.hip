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
//             extra blocks finalize the rejected prefix in parallel
//             (ald_commit.h; launched from ald_commit.hip and ald_commit_d.hip).
#include "ald_device.h"

#include <type_traits>

namespace ald {

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

    // Constraint (d): bring the worker's slack gain phi up to the current
    // heartbeat.  Each heartbeat since the last update ran one decode iteration
    // over the requests live at its start (e >= that iteration's tau; nothing
    // is placed between heartbeats without a build), taking Eq. 3's time.
    double phi = 0.0;
    if (sc.use_d) {
        phi = st.phi[gw];
        const int pending = hb - st.phi_hb[gw];
        if (pending < 0) {
            if (tid == 0) raise_error(err, DEV_EINVAL);
        } else {
            for (int p = 0; p < pending; ++p) {
                const int32_t tk = tau - pending + p;
                int64_t cnt = 0, ssum = 0;
                for (int k = head + tid; k < n; k += NT) {
                    const bool in = e[k] >= tk;
                    cnt += in ? 1 : 0;
                    ssum += in ? s[k] : 0;
                }
                cnt = block_reduce<NT>(cnt, 0, OpAdd(), red);
                ssum = block_reduce<NT>(ssum, 0, OpAdd(), red);
                if (cnt == 0) break;  // the live set only shrinks: no later iteration runs a batch
                const int64_t ctx = ssum + cnt * (int64_t)tk;  // sum of the contexts c = s + tau
                const double t_iter = (sc.c3 + sc.c2 * (double)cnt) + sc.k2 * (double)ctx;
                phi = phi + (sc.tdec - t_iter);
            }
            if (tid == 0) {
                st.phi[gw] = phi;
                st.phi_hb[gw] = hb;
            }
        }
    }

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
        pms[k].w = n - k;
        const int64_t P = (int64_t)pms[k].z + (int64_t)(n - k) * e[k];
        const int64_t Pe = P + e[k];
        runpm = Pe > runpm ? Pe : runpm;
    }
    // Constraint (d)'s limit: drop finished requests from the worker's log and
    // take theta * the smallest slack of the ongoing ones (placed before this
    // heartbeat).  In place, 256 entries at a time: every entry of a chunk is
    // read before any kept one is written, and kept entries only move down.
    double dl = INFINITY;
    if (sc.use_d) {
        int32_t* lge = st.lge + base;
        int32_t* lgw = st.lgw + base;
        double* lgs = st.lgs + base;
        const int L0 = st.lgn[gw];
        int wpos = 0;
        double mn = INFINITY;
        for (int c0 = 0; c0 < L0; c0 += NT) {
            const int k = c0 + tid;
            const bool in = k < L0;
            const int32_t ek = in ? lge[k] : 0, wk = in ? lgw[k] : 0;
            const double sk = in ? lgs[k] : 0.0;
            const bool keep = in && ek >= tau;
            if (keep && wk < hb) mn = fmin(mn, sk);
            int64_t kept;
            const int pos = (int)block_scan_excl<NT, false>(keep ? 1 : 0, 0, OpAdd(), &kept, red);
            if (keep) {
                lge[wpos + pos] = ek;
                lgw[wpos + pos] = wk;
                lgs[wpos + pos] = sk;
            }
            wpos += (int)kept;
            __syncthreads();
        }
        mn = double_of(block_reduce<NT>(ord_of(mn), ord_of(INFINITY), OpMin(), red));
        if (mn != INFINITY) dl = sc.theta * (mn + phi);
        if (tid == 0) st.lgn[gw] = wpos;
    }
    if (tid == 0) st.dlim[gw] = dl;

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
    // Breakpoint table (workers with 0 < B < LB_SLOTS): a histogram of the
    // remaining lengths r = e - tau of the live requests (those below LB_MAX),
    // then an exclusive scan, so that entry v - 1 = the byte offset, from the
    // first live slot's summaries, of the first live slot with r >= v (16
    // bytes per slot before it).
    if (B > 0 && B < LB_SLOTS) {
        __shared__ int32_t hist[LB_MAX];
        for (int v = tid; v < LB_MAX; v += NT) hist[v] = 0;
        __syncthreads();
        for (int k = head + tid; k < n; k += NT) {
            const int32_t r = e[k] - tau;
            if ((uint32_t)r < (uint32_t)LB_MAX) atomicAdd(&hist[r], 1);
        }
        __syncthreads();
        static_assert((LB_SLOTS - 1) * sizeof(int4) <= 0xFFFF && STAGE_MAX <= LB_SLOTS,
                      "byte offsets of the slots fit 16 bits; every staged worker has a table");
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
            out[tid * CHV + j] = (uint16_t)(run * (int32_t)sizeof(int4));  // entry v - 1, v = tid * CHV + j + 1
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
            // (c) and (d) bound the same prefill time
            const int64_t l = wave_last_true(1, LMAX, [&](int64_t v) { const double t = tt(v); return t <= sc.ttft && t <= dl; });
            if (l0) st.lthr[gw] = (int32_t)l;
        } else {
            // the TTFT band (empty on a decode worker, whose T_pre is +inf)
            int64_t ll = 1, lh = 0;
            if (sc.ttft != INFINITY) {
                const double band = tie_band(sc.ttft);
                const double lo = sc.ttft - band, hi = sc.ttft + band;
                ll = wave_last_true(1, LMAX, [&](int64_t v) { return tt(v) < lo; }) + 1;
                lh = wave_last_true(1, LMAX, [&](int64_t v) { return tt(v) <= hi; });
            }
            const int64_t width = lh - ll + 1;
            const uint64_t mask = ballot(lane_id() < width && near_tie(tt(ll + lane_id()), sc.ttft));
            if (l0) {
                st.ntt_lo[gw] = (int32_t)ll;
                st.ntt_hi[gw] = (int32_t)lh;
                st.ntt_mask[gw] = width <= 64 ? mask : 0;
                if (width > 64 && sc.ntint) raise_error(err, DEV_EOVERFLOW);
            }
            // the band of (d)'s limit (empty without one)
            int64_t pl = 1, ph = 0;
            if (dl != INFINITY) {
                const double pband = tie_band(dl);
                const double plo = dl - pband, phi_ = dl + pband;
                pl = wave_last_true(1, LMAX, [&](int64_t v) { return tt(v) < plo; }) + 1;
                ph = wave_last_true(1, LMAX, [&](int64_t v) { return tt(v) <= phi_; });
            }
            if (l0) {
                st.ntp_lo[gw] = (int32_t)pl;
                st.ntp_hi[gw] = (int32_t)ph;
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
                                                          const int32_t* gen, const double* tdec)
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
        const bool ok = a >= 1 && p >= 1 && a <= LIM && p <= LIM && g >= 0 && g < p &&
                        (tdec == nullptr || (isfinite(tdec[r0 + k]) && tdec[r0 + k] >= 0.0));
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
    // constraint (d)'s log exists only where (d) is checked (a decode worker's
    // model ignores the decode history, and its log arrays hold no slots)
    const bool keep_log = tdec != nullptr && st.scen[0].use_d;
    if (keep_log) {
        // the log, in input order: phi = 0 at load, so each resident's entry
        // holds its slack T_dec * g - t_dec
        const Scen& sc = st.scen[0];
        for (int k = tid; k < R; k += NT) {
            const int32_t p = lpred[r0 + k], g = gen[r0 + k];
            st.lge[base + k] = p - g;  // e at tau = 0
            st.lgw[base + k] = -1;
            st.lgs[base + k] = sc.tdec * (double)g - tdec[r0 + k];
        }
    }
    if (tid == 0) {
        st.n[gw] = R;
        st.head[gw] = 0;
        st.built[gw] = 0;
        st.S1[gw] = 0;
        st.S2[gw] = 0;
        st.hbs[gw] = -1;
        st.lgn[gw] = keep_log ? R : 0;
    }
}

// ---------------------------------------------------------------------------------------------
// One worker's rebuild decision and build (all threads of the block).
__device__ __forceinline__ void build_one(const State& st, int mode, int gw, int s)
{
    const Ctl* c = st.ctl + s;
    if (mode != 2 && c->call != st.call) return;  // another call's control block
    if (mode == 0) {
        if (c->err || c->start >= c->Q) return;
        if (st.built[gw]) {
            if (!c->rebuild) return;
            // A worker that held no live request at its last build and has taken
            // none since (a placement clears `built`), with no prefill sum, has
            // the same summaries and thresholds at any tau: only the slack clock
            // of constraint (d) moves on (its gain is zero without a batch).
            if (st.B[gw] == 0 && st.S1[gw] == 0) {
                if (threadIdx.x == 0 && st.scen[s].use_d) st.phi_hb[gw] = c->hb_index;
                return;
            }
        }
    }
    const Scen sc = st.scen[s];
    build_worker(st, sc, gw, c->tau, c->hb_index, &st.ctl[s].err);
    if (threadIdx.x == 0) st.built[gw] = 1;
}

// mode 1: the workers the last commit round listed; modes 0 and 2: every
// worker (one block each).
__global__ __launch_bounds__(BUILD_THREADS) void k_build(State st, int mode)
{
    if (mode == 1) {
        const int s = blockIdx.x / MAX_DIRTY;
        const int j = blockIdx.x % MAX_DIRTY;
        if (s >= st.S || j >= st.dcount[s]) return;
        const int gw = st.dlist[s * MAX_DIRTY + j];
        if (st.built[gw]) return;
        build_one(st, mode, gw, s);
        return;
    }
    build_one(st, mode, blockIdx.x, find_scen_by_worker(st, blockIdx.x));
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
    int32_t head, n, M, lthr;  // (one 16-byte read)
    int32_t dq32;    // dq_max - the block's smallest qD, clamped to [-1, 2^31 - 1]
    int32_t nt_any;  // some query of the block's chunk may have a near-tie margin with this worker
    int32_t ntt_lo, ntt_hi, ntp_lo, ntp_hi;
    double dlim;
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
    v.dlim = wi.dlim;
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

// LLVM's writelane intrinsic (v_writelane_b32): the value of lane `lane` of
// `old` replaced by the wave-uniform `v`.  Through the intrinsic the compiler
// sees the instruction and inserts whatever wait states its operands need.
__device__ int ald_writelane(int v, int lane, int old) __asm("llvm.amdgcn.writelane.i32");
// v_mul_u32_u24: the product of the low 24 bits of each operand (full rate)
__device__ uint32_t ald_mul_u24(uint32_t a, uint32_t b) __asm("llvm.amdgcn.mul.u24");

// Word `acc` with lane J's value replaced by the wave-uniform `v` (one
// v_writelane_b32 per half, the lane an inline constant, J < 16).
template <int J>
__device__ __forceinline__ uint64_t put_lane_c(uint64_t acc, uint64_t v)
{
    const uint32_t lo = (uint32_t)ald_writelane((int)(uint32_t)v, J, (int)(uint32_t)acc);
    const uint32_t hi = (uint32_t)ald_writelane((int)(uint32_t)(v >> 32), J, (int)(uint32_t)(acc >> 32));
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
// for launch_eval.  STAGED requires every l_pred + tau of the block below 2^24
// (the count-times-end product takes the full-rate 24-bit multiply).  TAB: an
// unstaged worker with a table is read through it from global memory for the
// queries the table covers (l_pred <= LB_MAX), by a binary search for the rest.
template <int MODE, bool EX, bool STAGED, bool TAB>
__device__ __forceinline__ void eval_worker(const State& st, const Scen& sc, const WInfo& wi, int w, int32_t tau,
                                            const int32_t (&lin)[EVAL_QPT], const int32_t (&lp)[EVAL_QPT],
                                            const bool (&act)[EVAL_QPT], const uint64_t (&am)[EVAL_QPT],
                                            const int32_t (&qd)[EVAL_QPT], int32_t (&e1)[EVAL_QPT],
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
        int ofs[EVAL_QPT];
        int4 t[EVAL_QPT];
#pragma unroll
        for (int m = 0; m < EVAL_QPT; ++m) ofs[m] = LBs[lp[m] - 1];  // byte offset of the first slot ending at or after the query
#pragma unroll
        for (int m = 0; m < EVAL_QPT; ++m) t[m] = *reinterpret_cast<const int4*>(reinterpret_cast<const char*>(Ss) + ofs[m]);
#pragma unroll
        for (int m = 0; m < EVAL_QPT; ++m) {
            // every candidate below is a KV demand with the query added, so it
            // lies under the worker's peak (<= 2^30) plus l_in + l_pred: 32-bit
            // wrap-around arithmetic gives it exactly (t.w = live slots from
            // the breakpoint on, below STAGE_MAX)
            const uint32_t sq = (uint32_t)(lin[m] - tau), eq = (uint32_t)(lp[m] + tau);
            const uint32_t ne = ald_mul_u24((uint32_t)t[m].w, eq);
            const int32_t a = (int32_t)((uint32_t)t[m].x + sq);
            const int32_t c = (int32_t)((uint32_t)t[m].z + ne + sq + eq);
            const int32_t p = a > t[m].y ? a : t[m].y;
            peak[m] = p > c ? p : c;
        }
    } else if (TAB && B < LB_SLOTS) {
        // two dependent reads per query, table entry then summaries (32-bit
        // wrap-around arithmetic as above, with a full 32-bit multiply); a
        // query past the table's range searches
        const uint16_t* tb = st.lbt + (int64_t)(sc.wbase + w) * LB_MAX;
        int kq[EVAL_QPT];
#pragma unroll
        for (int m = 0; m < EVAL_QPT; ++m) kq[m] = (B > 0 && lp[m] <= LB_MAX) ? tb[lp[m] - 1] / (int)sizeof(int4) : 0;
        int4 t[EVAL_QPT];
#pragma unroll
        for (int m = 0; m < EVAL_QPT; ++m) t[m] = v.pms[v.head + kq[m]];
#pragma unroll
        for (int m = 0; m < EVAL_QPT; ++m) {
            const uint32_t sq = (uint32_t)(lin[m] - tau), eq = (uint32_t)(lp[m] + tau);
            const int32_t a = (int32_t)((uint32_t)t[m].x + sq);
            const int32_t c = (int32_t)((uint32_t)t[m].z + (uint32_t)t[m].w * eq + sq + eq);
            const int32_t p = a > t[m].y ? a : t[m].y;
            peak[m] = p > c ? p : c;
            if (lp[m] > LB_MAX) peak[m] = (int32_t)kv_peak_with(v, lin[m] - tau, lp[m] + tau);
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
#pragma unroll
        for (int m = 0; m < EVAL_QPT; ++m) {
            // constraint (b) as qD <= dq_max: staged, relative to the block's
            // smallest qD in 32 bits (the block's qD span is below 2^31)
            const bool bok = STAGED ? qd[m] <= wi.dq32
                                    : ((int64_t)lin[m] << sc.gs) + (int64_t)sc.gn * lp[m] <= wi.dq_max;
            // one ballot per compare: each compare's lane mask is its ballot
            const uint64_t bf = am[m] & ballot(peak[m] <= M) & ballot(bok) & ballot(lin[m] <= lthr);
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
            const bool maybe = (qD >= wi.ntd_lo && qD <= wi.ntd_hi) || (lin[m] >= wi.ntt_lo && lin[m] <= wi.ntt_hi) ||
                               (lin[m] >= wi.ntp_lo && lin[m] <= wi.ntp_hi);
            nt = maybe && latency(sc, v, lin[m], lp[m], B + 1).nt;
        }
        const uint64_t bn = ballot(act[m] && nt);
        bits = put_lane(bits, bn, m + EVAL_QPT);
    }
    if (lane >= EVAL_QPT && lane < 2 * EVAL_QPT) bdst[w] = bits;
}

// Sorted layout (a one-scenario tile with State::qorig): the order in which
// the block evaluates its chunk of EVAL_Q queries, by l_pred in buckets of 8
// (the last bucket also takes every l_pred above 2032), ties by arrival, the
// chunk's missing queries (offsets >= nact) last, so that the lanes of a wave
// read neighbouring breakpoint entries and summaries.  Every worker block of
// the chunk computes the same order.  A stable counting sort: the lanes of a
// wave with the same bucket find each other by eight ballots (one per key
// bit); a histogram per (segment of 64 offsets, bucket) and one scan over the
// buckets give each query its position.  On return o[m] is the chunk offset
// of the query at position m * NT + tid (its lengths are then read again:
// passing them through LDS, or holding them through the sort, measured
// slower); the chunk's first worker block writes the tile's permutation
// (qorig, qpos).  `sh`: 10 KB of scratch (histogram, then the permutation);
// `red` that of block_scan_excl.
template <int QPT>
__device__ __forceinline__ void sort_chunk(const State& st, const Scen& sc, int start, int q0, int nact, bool writer,
                                           int (&o)[QPT], uint16_t* sh, int64_t* red)
{
    constexpr int NT = EVAL_THREADS;
    constexpr int NB = 256;                 // buckets (one per thread for the scan)
    constexpr int NS = QPT * (NT / 64);     // segments of 64 offsets: segment m * 4 + wave
    static_assert(NT == NB, "one bucket per thread");
    uint16_t* H = sh;                       // [NS][NB] counts, then positions
    uint16_t* perm = sh + NS * NB;          // sorted position -> chunk offset
    const int tid = threadIdx.x, lane = lane_id(), wv = wave_id();
    const uint64_t below = (1ull << lane) - 1;
    for (int k = tid; k < NS * NB / 4; k += NT) reinterpret_cast<uint64_t*>(H)[k] = 0;
    int key[QPT];
#pragma unroll
    for (int m = 0; m < QPT; ++m) {
        const int off = m * NT + tid;
        const bool in = off < nact;
        const int32_t l = in ? st.q_lpred[q_at(sc, q0 + off)] : 1;
        // (an invalid length, which fails the call, still gets a bucket)
        key[m] = in ? min(max(l - 1, 0) >> 3, NB - 2) : NB - 1;
    }
    __syncthreads();
    int rank[QPT];
#pragma unroll
    for (int m = 0; m < QPT; ++m) {
        uint64_t peers = ~0ull;
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            const bool kb = (key[m] >> b) & 1;
            const uint64_t bb = ballot(kb);
            peers &= kb ? bb : ~bb;
        }
        rank[m] = __popcll(peers & below);
        if (rank[m] == 0) H[(m * (NT / 64) + wv) * NB + key[m]] = (uint16_t)__popcll(peers);
    }
    __syncthreads();
    int64_t cnt = 0;
    for (int sg = 0; sg < NS; ++sg) cnt += H[sg * NB + tid];
    int64_t all;
    int64_t at = block_scan_excl<NT, false>(cnt, 0, OpAdd(), &all, red);
    for (int sg = 0; sg < NS; ++sg) {
        const int n = H[sg * NB + tid];
        H[sg * NB + tid] = (uint16_t)at;
        at += n;
    }
    __syncthreads();
#pragma unroll
    for (int m = 0; m < QPT; ++m) perm[H[(m * (NT / 64) + wv) * NB + key[m]] + rank[m]] = (uint16_t)(m * NT + tid);
    __syncthreads();
    const int t0 = q0 - start;  // the chunk's first tile offset
#pragma unroll
    for (int m = 0; m < QPT; ++m) {
        const int p = m * NT + tid;
        const int off = perm[p];
        o[m] = off;
        if (writer && p < nact) {
            st.qorig[t0 + p] = t0 + off;
            st.qpos[t0 + off] = t0 + p;
        }
    }
    __syncthreads();  // the scratch is the staging area of the evaluation
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
// tracked (diagnostics); TAB: unstaged workers are read through their tables.
template <int MODE, bool EX, bool TAB = false>
__global__ __launch_bounds__(EVAL_THREADS) __attribute__((amdgpu_waves_per_eu(4))) void k_eval(State st)
{
    constexpr int NT = EVAL_THREADS;
    constexpr int QPT = EVAL_QPT;
    static_assert(2 * QPT <= 16, "lane words by put_lane");
    __shared__ uint16_t LBs[LB_MAX];               // the worker's breakpoint table
    __shared__ int4 Ss[PF_N * NT];                 // pms of live slot k, k = 0..B
    __shared__ WInfo Wi[EVAL_WPB_MAX];
    __shared__ int64_t red[NT / 64];
    static_assert(sizeof(Ss) >= 10 * 1024, "the sort's scratch");

    const int s = find_scen<&Scen::eval_blk0>(st, blockIdx.x);
    const Scen sc = st.scen[s];
    const Ctl* cp = st.ctl + s;
    const int32_t start = cp->start, Q = cp->Q;
    const bool mine = cp->call == st.call;
    if (st.qbad != nullptr && start == 0 && mine) {
        // first round of a one-scenario call: check every query length of the
        // call before the first commit can run (grid-stride over all queries)
        bool bad = false;
        for (int64_t i = (int64_t)blockIdx.x * EVAL_THREADS + threadIdx.x; i < Q; i += (int64_t)gridDim.x * EVAL_THREADS) {
            const int32_t a = st.q_lin[i], p = st.q_lpred[i];
            bad = bad || !(a >= 1 && p >= 1 && a <= (1 << 24) && p <= (1 << 24));
        }
        if (ballot(bad) != 0 && lane_id() == 0) atomicOr(st.qbad, 1);
    }
    if (cp->err || start >= Q || !mine) return;
    const int32_t end = tile_end(start, Q, cp->T, cp->H, cp->since_hb, cp->hb_next);
    const int local = blockIdx.x - sc.eval_blk0;
    const int wb = local % sc.nblk;
    const int qc = local / sc.nblk;
    const int q0 = start + qc * EVAL_Q;
    if (q0 >= end) return;
    const int32_t tau = cp->tau, hb = cp->hb_index;
    const int tid = threadIdx.x;
    const int lane = lane_id();

    // Thread tid evaluates chunk positions m * NT + tid: the chunk's queries in
    // arrival order, or (sorted layout) in order of l_pred.  o[m] = the chunk
    // offset of the query at position m * NT + tid.
    // Thread tid evaluates chunk positions m * NT + tid: the queries in
    // arrival order, or (sorted layout) in order of l_pred
    int o[QPT];  // chunk offset of the query at position m * NT + tid
#pragma unroll
    for (int m = 0; m < QPT; ++m) o[m] = m * NT + tid;
    if (st.qorig != nullptr)
        sort_chunk<QPT>(st, sc, start, q0, min(EVAL_Q, end - q0), wb == 0, o, reinterpret_cast<uint16_t*>(Ss), red);
    int32_t lin[QPT], lp[QPT];
    bool act[QPT];
    int32_t e1[QPT], w1[QPT], e2[QPT], w2[QPT];  // two smallest KV excesses per query
    int64_t lpmax = 0, qdmin = INT64_MAX, qdmax = INT64_MIN, lnmin = INT64_MAX, lnmax = INT64_MIN;
#pragma unroll
    for (int m = 0; m < QPT; ++m) {
        act[m] = q0 + m * NT + tid < end;
        lin[m] = act[m] ? st.q_lin[q_at(sc, q0 + o[m])] : 1;
        lp[m] = act[m] ? st.q_lpred[q_at(sc, q0 + o[m])] : 1;
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
    // staging needs the table to cover every l_pred of the block, every
    // eq = l_pred + tau (idle lanes: 1 + tau) below 2^24 for the 24-bit
    // multiply, and the block's qD within a 2^31 span
    const bool use_lb = L <= LB_MAX && (int64_t)max(L, 1) + tau < ((int64_t)1 << 24) &&
                        qr.qdmax - qr.qdmin < ((int64_t)1 << 31);
    int32_t qd[QPT];  // qD - the block's smallest (idle lanes: anything; masked)
#pragma unroll
    for (int m = 0; m < QPT; ++m)
        qd[m] = (int32_t)(((int64_t)lin[m] << sc.gs) + (int64_t)sc.gn * lp[m] - qr.qdmin);

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
        const int64_t dqr = x.dq_max - qr.qdmin;
        x.dq32 = dqr < 0 ? -1 : (dqr > INT32_MAX ? INT32_MAX : (int32_t)dqr);
        x.ntd_lo = st.ntd_lo[gw];
        x.ntd_hi = st.ntd_hi[gw];
        x.lthr = st.lthr[gw];
        x.ntt_lo = st.ntt_lo[gw];
        x.ntt_hi = st.ntt_hi[gw];
        x.ntd_mask = st.ntd_mask[gw];
        x.ntt_mask = st.ntt_mask[gw];
        // constraint (d) never runs with the integer near-tie sets (mode 2)
        x.dlim = MODE == 2 ? INFINITY : st.dlim[gw];
        x.ntp_lo = MODE == 2 ? 1 : st.ntp_lo[gw];
        x.ntp_hi = MODE == 2 ? 0 : st.ntp_hi[gw];
        // a near-tie margin needs some query of the chunk inside a tie band
        x.nt_any = MODE == 0 || (qr.qdmax >= x.ntd_lo && qr.qdmin <= x.ntd_hi) ||
                   (qr.lnmax >= x.ntt_lo && qr.lnmin <= x.ntt_hi) || (qr.lnmax >= x.ntp_lo && qr.lnmin <= x.ntp_hi);
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
        eval_worker<MODE, EX, true, false>(st, sc, Wi[cur], wbeg + cur, tau, lin, lp, act, am, qd, e1, w1, e2, w2,
                                           LBs, Ss, bdst);
        cur = nxt;
    }
    // workers too large to stage: binary search over global memory
    for (int j0 = 0; j0 < nw; ++j0) {
        const WInfo wi = Wi[j0];
        if (use_lb && wi.n - wi.head < STAGE_MAX) continue;
        eval_worker<MODE, EX, false, TAB>(st, sc, wi, wbeg + j0, tau, lin, lp, act, am, qd, e1, w1, e2, w2, LBs, Ss,
                                          bdst);
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
    if (cp->call != st.call) return;  // another call's control block (its tile record too)
    const bool done = cp->err || start >= Q;
    const int32_t end = done ? start : tile_end(start, Q, cp->T, cp->H, cp->since_hb, cp->hb_next);
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
    // the group's words hold tile positions q0 - start + lane: the queries in
    // arrival order, or (sorted layout) the query qorig of each position
    const int slot = q0 - start + lane;
    const bool act = live && q0 + lane < end;
    const int qi = (act && st.qorig != nullptr) ? start + st.qorig[slot] : q0 + lane;

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
    // the two smallest KV excesses feed only the diagnostics: each wave of
    // the group merges its share of the worker blocks' two smallest keys (new
    // first = smaller first; new second = min(larger first, smaller second))
    uint64_t a1 = ~0ull, a2 = ~0ull;
    auto merge = [&](ulonglong2 p) {
        const uint64_t lo = p.x < a1 ? p.x : a1;
        const uint64_t hi = p.x < a1 ? a1 : p.x;
        const uint64_t s2 = p.y < a2 ? p.y : a2;
        a1 = lo;
        a2 = hi < s2 ? hi : s2;
    };
    if (act && st.out_diag) {
        const ulonglong2* prow = st.part + sc.part_off + slot;
        if (sc.nblk > 64 * G) {  // many worker blocks (short tiles over many workers): more reads in flight
#pragma unroll 16
            for (int b = slice; b < sc.nblk; b += G) merge(prow[(int64_t)b * sc.pstride]);
        } else {
#pragma unroll 8
            for (int b = slice; b < sc.nblk; b += G) merge(prow[(int64_t)b * sc.pstride]);
        }
    }
    // merge the group's partial results into its first wave (lists by rank,
    // counts summed, excess keys as above)
    struct Part {
        uint64_t tkey[TOPK];
        int32_t tw[TOPK];
        uint64_t ntkey, a1, a2;
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
            pt.a1 = a1;
            pt.a2 = a2;
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
            const uint64_t lo = pt.a1 < a1 ? pt.a1 : a1;
            const uint64_t hi = pt.a1 < a1 ? a1 : pt.a1;
            const uint64_t s2 = pt.a2 < a2 ? pt.a2 : a2;
            a1 = lo;
            a2 = hi < s2 ? hi : s2;
        }
    }
    if (!live) return;
    int32_t ex1 = INT32_MAX, w1 = -1, ex2 = INT32_MAX, w2 = -1;
    if (act && st.out_diag) {
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
    st.qsum[sc.qsum_off + slot] = q;  // by tile position, as the bit words
    if (q.nfeas > 0) {
        atomicMin(&st.tinfo[s].first_pc[parity], qi);
    } else if (st.qbad == nullptr || *st.qbad == 0) {
        // no feasible worker at tile start: rejected whatever the tile commits
        // before it.  These tile-start diagnostics are exact for the queries
        // before the tile's first commit; the commit overwrites every query
        // from its first feasible one on.
        if (st.out_worker) st.out_worker[sc.out_off + q_at(sc, qi)] = -1;
        if (st.out_diag) {
            Diag d;
            d.n_feasible = 0;
            d.near_tie = ntcnt > 0 ? 1 : 0;
            d.kv_peak_chosen = 0;
            d.kv_excess_min = ex1;
            d.ttft_chosen = 0.0;
            d.tdec_chosen = 0.0;
            st.out_diag[q_at(sc, qi)] = d;
        }
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

// Start of an ald_place_stream call (one scenario): the control block, the
// tile record and a cleared query-error word (the first round's pair
// evaluation checks the query lengths).  With gate >= 0 the call follows
// asynchronous call `gate` and starts only if that call finished without an
// error; otherwise the control block stays that call's, and every kernel of
// this call finds it foreign and does nothing.
__global__ void k_begin(Ctl c, TileInfo ti, Ctl* ctl, TileInfo* tinfo, int32_t* qbad, int32_t gate)
{
    if (gate >= 0) {
        const Ctl o = *ctl;
        if (o.call != gate || o.err || o.start < o.Q) return;
    }
    *ctl = c;
    *tinfo = ti;
    *qbad = 0;
}

// The outcome of an asynchronous call with no queries.
__global__ void k_status_ok(int32_t* status) { *status = ALD_OK; }

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

// The sweep's answer (Sec. 4.4, Sec. 6.4: the fewest GPUs that serve the
// stream with no violation): among scenarios with no rejection, the smallest
// n_workers * GPUs per worker, ties to the lowest scenario index.  One block;
// the (GPUs, index) pairs are ordered as one int64 key.
__global__ __launch_bounds__(256) void k_sweep_best(State st, int64_t* min_gpus)
{
    __shared__ int64_t red[4];
    int64_t best = INT64_MAX;
    for (int s = threadIdx.x; s < st.S; s += 256) {
        const Scen sc = st.scen[s];
        if (st.ctl[s].n_rej != 0 || st.ctl[s].err != 0) continue;
        // GPUs < 2^38 and s < 2^24 (checked on the host): the key fits in 62 bits
        const int64_t key = ((int64_t)sc.W * sc.gpw << 24) + s;
        best = key < best ? key : best;
    }
    best = block_reduce<256>(best, INT64_MAX, OpMin(), red);
    if (threadIdx.x == 0) {
        min_gpus[0] = best == INT64_MAX ? -1 : best >> 24;
        min_gpus[1] = best == INT64_MAX ? -1 : (best & ((1 << 24) - 1));
    }
}

// The outcome of an asynchronous sweep: the first scenario (by index) with a
// device error gives the code, as the synchronous sweep returns it; else
// ALD_EINCOMPLETE if a scenario has queries left, else ALD_OK.  One block.
__global__ __launch_bounds__(256) void k_sweep_status(State st, int32_t* status)
{
    __shared__ int64_t red[4];
    int64_t first_err = INT32_MAX, left = 0;
    for (int s = threadIdx.x; s < st.S; s += 256) {
        const Ctl c = st.ctl[s];
        if (c.err != 0 && s < first_err) first_err = s;
        left |= c.start < c.Q ? 1 : 0;
    }
    first_err = block_reduce<256>(first_err, (int64_t)INT32_MAX, OpMin(), red);
    left = block_reduce<256>(left, (int64_t)0, OpMax(), red);
    if (threadIdx.x == 0)
        *status = first_err != INT32_MAX ? ctl_status(st.ctl[first_err]) : (left ? ALD_EINCOMPLETE : ALD_OK);
}

// ---------------------------------------------------------------------------------------------
hipError_t launch_ingest(const State& st, int32_t W, const int64_t* res_off, const int32_t* lin,
                         const int32_t* lpred, const int32_t* gen, const double* tdec, hipStream_t stream)
{
    hipLaunchKernelGGL(k_ingest, dim3(W), dim3(BUILD_THREADS), 0, stream, st, res_off, lin, lpred, gen, tdec);
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
    if (mode == 3) {
        if (ex) hipLaunchKernelGGL((k_eval<2, true, true>), g, b, 0, stream, st);
        else hipLaunchKernelGGL((k_eval<2, false, true>), g, b, 0, stream, st);
    } else if (mode == 2) {
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

int eval_blocks_per_cu(int mode, bool ex)
{
    const void* f = mode == 3 ? (ex ? (const void*)k_eval<2, true, true> : (const void*)k_eval<2, false, true>)
                  : mode == 2 ? (ex ? (const void*)k_eval<2, true> : (const void*)k_eval<2, false>)
                  : mode == 1 ? (ex ? (const void*)k_eval<1, true> : (const void*)k_eval<1, false>)
                              : (ex ? (const void*)k_eval<0, true> : (const void*)k_eval<0, false>);
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, f, EVAL_THREADS, 0) != hipSuccess) return 0;
    return n;
}

hipError_t launch_select(const State& st, int32_t blocks, hipStream_t stream)
{
    hipLaunchKernelGGL(k_select, dim3(blocks), dim3(SEL_THREADS), 0, stream, st);
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

hipError_t launch_begin(const Ctl& c, const TileInfo& ti, Ctl* ctl, TileInfo* tinfo, int32_t* qbad, int32_t gate,
                        hipStream_t stream)
{
    hipLaunchKernelGGL(k_begin, dim3(1), dim3(1), 0, stream, c, ti, ctl, tinfo, qbad, gate);
    return hipGetLastError();
}

hipError_t launch_status_ok(int32_t* status, hipStream_t stream)
{
    hipLaunchKernelGGL(k_status_ok, dim3(1), dim3(1), 0, stream, status);
    return hipGetLastError();
}

hipError_t launch_summary(const State& st, int32_t W, int32_t* B, int64_t* sc, int64_t* sr, int64_t* peak,
                          hipStream_t stream)
{
    hipLaunchKernelGGL(k_summary, dim3((W + 255) / 256), dim3(256), 0, stream, st, W, B, sc, sr, peak);
    return hipGetLastError();
}

hipError_t launch_sweep_outputs(const State& st, int32_t* rejected, int32_t* first_reject, int64_t* min_gpus,
                                hipStream_t stream)
{
    hipLaunchKernelGGL(k_sweep_outputs, dim3((st.S + 255) / 256), dim3(256), 0, stream, st, rejected,
                       first_reject);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || min_gpus == nullptr) return e;
    hipLaunchKernelGGL(k_sweep_best, dim3(1), dim3(256), 0, stream, st, min_gpus);
    return hipGetLastError();
}

hipError_t launch_sweep_status(const State& st, int32_t* status, hipStream_t stream)
{
    hipLaunchKernelGGL(k_sweep_status, dim3(1), dim3(256), 0, stream, st, status);
    return hipGetLastError();
}

}  // namespace ald
