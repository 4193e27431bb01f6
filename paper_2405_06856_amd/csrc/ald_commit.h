// The arrival-order commit kernel (template over diagnostics and constraint
// (d)).  Its instantiations are split over two translation units, so that the
// variants without decode history are compiled as they are without the others
// beside them.
#pragma once

#include "ald_device.h"

namespace ald {

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
    int32_t lgn;     // entries in its constraint-(d) log
    int64_t base;    // first slot
    int64_t DS, S1, S2, SC, SR;
    uint64_t key;
    double rhs;
    double dlim;     // constraint (d)'s limit, fixed within a heartbeat (no ongoing request joins or leaves)
    double phi;      // its slack gain: a request placed now logs slack - phi = -phi
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

// Sorted tile layout: the window cache of the dirty workers dw[0 .. cnt)
// (lane jb + k gets worker dw[k]'s words), in the arrival order that
// load_win_bits gives in the arrival layout.  The wave gathers them: lane i
// reads, for each worker, the word holding query w0 + i at its sorted tile
// position tp, and the two ballots are that worker's bits for the window.
// Eight workers' loads go out together.
__device__ __forceinline__ void gather_win_bits(const State& st, const Scen& sc, const int32_t* dw, int jb, int cnt,
                                                int start, int w0, bool act, int tp, WinBits& wb)
{
    const int lane = lane_id();
    const int64_t row = sc.bits_off + (int64_t)(tp >> 6) * sc.W;
    const int bit = tp & 63, s = (w0 - start) & 63;
    for (int j0 = 0; j0 < cnt; j0 += 8) {
        uint64_t f[8], n[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const bool ok = act && j0 + u < cnt;
            const int w = dw[min(j0 + u, cnt - 1)];
            f[u] = ok ? st.bits_feas[row + w] : 0;
            n[u] = ok ? st.bits_nt[row + w] : 0;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const uint64_t fb = ballot((f[u] >> bit) & 1), nb = ballot((n[u] >> bit) & 1);
            if (j0 + u < cnt && lane == jb + j0 + u) {
                wb.f0 = fb << s;
                wb.n0 = nb << s;
                wb.f1 = s ? fb >> (64 - s) : 0;
                wb.n1 = s ? nb >> (64 - s) : 0;
            }
        }
    }
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
    v.dlim = a.dlim;
    return v;
}

// Per-launch commit state held in LDS.  dag[] mirrors the lanes' DAgg for the
// per-lane diagnostics of rejected queries (diagnostics only); dw[] and dbits
// say which workers are dirty.
// The kernel variant with the LDS copies (CACHE), for scenarios of up to CW
// workers, also keeps for the untouched-worker scan the tile-start rank keys
// (read at the tile's first scan) and the last bit row of each kind that a
// scan read: a later scan of the same 64-query window reads LDS only.
constexpr int CW = COMMIT_CACHE_W;
struct CommitLDS {
    DAgg dag[MAX_DIRTY];
    int32_t dw[MAX_DIRTY];
    uint32_t dbits[DBITS_W];
    int32_t he[HOT];
    int32_t hs[HOT];
    uint64_t ckey[CW];     // tile-start rank keys (valid once kok)
    uint64_t crow[2][CW];  // bit rows: [0] feasibility, [1] near tie
    int64_t ctag[2];       // offset of the row held in crow[k] (-1: none)
    int32_t kok;
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
__device__ __forceinline__ int next_empty_worker(const State& st, const Scen& sc, const CommitLDS& L, int nd, int from)
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
__device__ __forceinline__ Diag reject_diag(const State& st, const Scen& sc, const QSum& q, int i, int start, int w0, int32_t lin,
                            int32_t lp, int32_t tau, int32_t hb, const CommitLDS& L, int nd, int hot,
                            const WinBits& wb, int* abort, int* scanned)
{
    Diag d;
    d.n_feasible = 0;
    d.kv_peak_chosen = 0;
    d.ttft_chosen = 0.0;
    d.tdec_chosen = 0.0;
    d.kv_excess_min = 0;
    d.near_tie = 0;
    *abort = 0;
    *scanned = 0;
    const int32_t sq = lin - tau, eq = lp + tau;
    int64_t exmin = q.ex1;
    if (q.w1 >= 0 && dirty_w(L, sc.W, nd, q.w1)) {
        if (q.w2 >= 0 && dirty_w(L, sc.W, nd, q.w2)) {
            *abort = 1;
            return d;
        }
        *scanned = 1;
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
    int32_t stale;  // exact scans of workers that turned out infeasible
    int32_t fallback;  // the untouched workers' bit words were scanned
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

// Algorithm 1's best worker among the workers untouched in this tile whose
// tile-start bit for query i is set in `words` (feasibility or near tie): for
// them the tile-start results are still exact.  With `listed`, only workers of
// the kind the selection lists (with interchangeable empty workers, the
// non-empty ones).  The whole wave scans the scenario's bit words and rank
// keys, from the LDS copies (kind 0: feasibility, 1: near tie) in the CACHE
// variant, else from global memory sixteen batches of 64 workers per round
// trip; every lane gets (key, worker), worker -1 when there is none.
struct KeyW {
    uint64_t k;
    int32_t w;
};
template <bool CACHE>
__device__ __forceinline__ KeyW best_untouched(const uint64_t* words, const uint64_t* keys, CommitLDS* L, int W,
                                            int nd, int64_t row0, int bit, bool listed, bool uniform_M, bool dpp,
                                            int kind)
{
    const int lane = lane_id();
    uint64_t k = 0;
    int32_t w = -1;
    static_assert(CW <= DBITS_W * 32, "the LDS scan reads the dirty bitmap");
    if (CACHE) {  // (the launch checked W <= CW)
        // the row (and, at the tile's first scan, the keys) into LDS, sixteen
        // batches per round trip
        const bool need_row = L->ctag[kind] != row0, need_keys = L->kok == 0;  // wave-uniform
        if (need_row || need_keys) {
            const uint64_t* row = words + row0;
            for (int b0 = 0; b0 < W; b0 += 64 * 16) {
                uint64_t wd[16], kd[16];
#pragma unroll
                for (int u = 0; u < 16; ++u) {
                    const int ww = b0 + u * 64 + lane;
                    wd[u] = (need_row && ww < W) ? row[ww] : 0;
                    kd[u] = (need_keys && ww < W) ? keys[ww] : 0;
                }
#pragma unroll
                for (int u = 0; u < 16; ++u) {
                    const int ww = b0 + u * 64 + lane;
                    if (ww < W) {
                        if (need_row) L->crow[kind][ww] = wd[u];
                        if (need_keys) L->ckey[ww] = kd[u];
                    }
                }
            }
            wave_sync();
            if (lane == 0) {
                L->ctag[kind] = row0;
                L->kok = 1;
            }
            wave_sync();
        }
        // each lane its own workers lane + 64 j in increasing index (a later
        // one replaces only with a larger key), eight per round of LDS reads
        // (slots up to CW exist; those at or past W are masked)
        const bool skip_empty = listed && uniform_M;
        const int nb = (W + 63) / 64;
        for (int j0 = 0; j0 < nb; j0 += 8) {
            uint64_t wd[8], kd[8];
            uint32_t db[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int ww = min((j0 + u) * 64 + lane, CW - 1);
                wd[u] = L->crow[kind][ww];
                kd[u] = L->ckey[ww];
                db[u] = L->dbits[ww >> 5];
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int ww = (j0 + u) * 64 + lane;
                const bool ok = ww < W && ((wd[u] >> bit) & 1) && !((db[u] >> (ww & 31)) & 1u) &&
                                !(skip_empty && kd[u] == 0);
                const bool take = ok && (w < 0 || kd[u] > k);
                k = take ? kd[u] : k;
                w = take ? ww : w;
            }
        }
    } else {
        const uint64_t* row = words + row0;
        for (int b0 = 0; b0 < W; b0 += 64 * 16) {
            // the words and the rank keys of the batch in one round trip
            uint64_t wd[16], kd[16];
#pragma unroll
            for (int u = 0; u < 16; ++u) {
                const int ww = b0 + u * 64 + lane;
                wd[u] = ww < W ? row[ww] : 0;
                kd[u] = ww < W ? keys[ww] : 0;
            }
#pragma unroll
            for (int u = 0; u < 16; ++u) {
                const int ww = b0 + u * 64 + lane;
                bool ok = (wd[u] >> bit) & 1;
                if (!ballot(ok)) continue;
                ok = ok && !dirty_w(*L, W, nd, ww);
                const uint64_t kk = ok ? kd[u] : 0;
                ok = ok && !(listed && uniform_M && kk == 0);
                const bool take = ok && ranks_before(kk, ww, k, w);
                k = take ? kk : k;
                w = take ? ww : w;
            }
        }
    }
    // the best over the lanes (the largest key, then the lowest index), by
    // DPP scans or by a shuffle butterfly: the same result; which form leaves
    // the caller more scalar registers depends on the kernel variant (`dpp`)
    if (dpp) {
        const bool valid = w >= 0;
        const uint64_t kmax = wave_max_u64(valid ? k : 0);
        const bool top = valid && k == kmax;
        const int32_t wmin = wave_min32(top ? w : INT32_MAX);
        return ballot(top) ? KeyW{kmax, wmin} : KeyW{0, -1};
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const uint64_t ok2 = __shfl_xor(k, off, 64);
        const int32_t ow = __shfl_xor(w, off, 64);
        const bool take = ranks_before(ok2, ow, k, w);
        k = take ? ok2 : k;
        w = take ? ow : w;
    }
    return KeyW{k, w};
}

// Decide one query with the whole wave.  `a` is this lane's dirty worker.
template <bool CACHE>
__device__ __forceinline__ Decision decide(const State& st, const Scen& sc, const QView& q, int i, int start, int w0, int32_t lin,
                           int32_t lp, int32_t tau, int32_t hb, CommitLDS& L, int nd, int hot, int& hotBs,
                           int& hotm, int next_empty, bool want_diag, const WinBits& wb, const DAgg& a, Scan& sn)
{
    Decision r;
    r.w = -1;
    r.lane = -1;
    r.abort = 0;
    r.stale = 0;
    r.fallback = 0;
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
    if (!have && q.ncand > TOPK) {  // every listed candidate was committed to: the best untouched one
        const int tp = st.qpos != nullptr ? st.qpos[i - start] : i - start;  // the query's bit position
        const KeyW c = best_untouched<CACHE>(st.bits_feas, st.key + sc.wbase, &L, sc.W, nd,
                                      sc.bits_off + (int64_t)(tp >> 6) * sc.W, tp & 63, true,
                                      sc.uniform_M != 0, !want_diag, 0);
        have = c.w >= 0;
        bk = have ? c.k : bk;
        bw = have ? c.w : bw;
        r.fallback = 1;
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
            r.stale += 1;
        }
        r.w = have ? bw : -1;
        return r;
    }

    // ---- with diagnostics: the feasibility of every dirty candidate; a worker
    // whose peak bound plus the query's own demand fits needs no scan
    const bool sure = unknown && (int64_t)a.pub + lin + lp <= (int64_t)a.M;
    bool cand = unknown && !sure;
    bool feas_now = sure;
    for (;;) {
        const int bl = wave_best_lane(a.key, a.w, cand);
        if (bl < 0) break;
        int32_t p0;
        const int64_t pk = dirty_kv_peak(st, L, a, bl, hot, hotBs, hotm, sq, eq, &p0);
        const bool ok = pk <= rdlane(a.M, bl);
        r.stale += ok ? 0 : 1;
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
    const int j2 = q.w2 >= 0 ? dirty_lane(a, q.w2) : -1;
    if (q.w1 >= 0 && j1 >= 0 && j2 >= 0) {  // both dirty: the tile-start lists cannot decide
        r.abort = 1;
        return r;
    } else if (q.w1 >= 0 && j1 >= 0) {
        int32_t p0;
        const int64_t pk = dirty_kv_peak(st, L, a, j1, hot, hotBs, hotm, sq, eq, &p0);
        r.stale += 1;
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
        } else {  // the best near-tie worker was committed to: the best untouched one with a near tie
            const int tp = st.qpos != nullptr ? st.qpos[i - start] : i - start;
            const KeyW c = best_untouched<CACHE>(st.bits_nt, st.key + sc.wbase, &L, sc.W, nd,
                                          sc.bits_off + (int64_t)(tp >> 6) * sc.W, tp & 63, false,
                                          sc.uniform_M != 0, !want_diag, 1);
            nt = c.w >= 0 && !ranks_before(bk, bw, c.k, c.w);
            r.fallback = 1;
        }
    }
    const bool dnt = valid && Lt.nt && (r.w < 0 || !ranks_before(bk, bw, a.key, a.w));
    nt = nt | (ballot(dnt) != 0);
    r.d.near_tie = nt ? 1 : 0;
    // the chosen worker's figures
    if (r.w >= 0) {
        if (r.lane >= 0) {
            if (!((ballot(sn.done) >> r.lane) & 1)) {  // chosen on its bound: its exact peak now
                int32_t p0;
                const int64_t pk = dirty_kv_peak(st, L, a, r.lane, hot, hotBs, hotm, sq, eq, &p0);
                if (lane == r.lane) {
                    sn.done = true;
                    sn.pk = (int32_t)pk;
                    sn.p0 = p0;
                }
            }
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
__device__ __forceinline__ void writeback_hot(const State& st, CommitLDS& L, DAgg& a, int hot, int Bs, int m, bool mirror)
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

template <bool DIAG, bool USE_D, bool CACHE>
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
        if (part != 0 || lane != 0) return;
        if (st.ctl_host != nullptr) st.ctl_host[s] = *cp;
        if (st.status != nullptr) *st.status = ctl_status(*cp);
    };
    if (cp->call != st.call) {  // another call's control block: this call was blocked
        if (st.status != nullptr && part == 0 && lane == 0) *st.status = ALD_EBLOCKED;
        return;
    }
    if (st.qbad != nullptr && *st.qbad) {  // an invalid query length: nothing is written
        if (part == 0 && lane == 0) cp->err = DEV_EINVAL;
        publish();
        return;
    }
    if (ti.start >= ti.end) {
        publish();
        return;
    }
    if (CACHE && sc.W > CW) {  // the LDS copies hold CW workers (the host never launches this)
        if (part == 0 && lane == 0) cp->err = DEV_EINVAL;
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
    if (lane == 0) {
        cp->rebuild = 0;
        if (CACHE) {
            L.ctag[0] = L.ctag[1] = -1;
            L.kok = 0;
        }
    }
    wave_sync();
    constexpr bool want_diag = DIAG;  // st.out_diag != nullptr
    int nd = 0;    // dirty workers (wave-uniform); lane j < nd holds the j-th in `a`
    DAgg a;
    a.w = -1;
    a.B = a.n = a.head = a.M = a.hbs = a.empty0 = a.cap = a.pub = a.lgn = 0;
    a.base = 0;
    a.DS = a.S1 = a.S2 = a.SC = a.SR = 0;
    a.key = 0;
    a.rhs = 0.0;
    a.dlim = INFINITY;
    a.phi = 0.0;
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
    // Exact scans forced by tile-start lists gone stale.  Past a budget a fresh
    // tile (rebuilt summaries, re-evaluated pairs) is the cheaper way on, and
    // the tile is cut before the next decision.
    int stale = 0, fallbacks = 0;
    bool stale_cut = false;
    while (pos < end && !cut) {
        // one window of 64 queries; `cur` is the first undecided lane
        const int w0 = pos;
        const int i = w0 + lane;
        const bool act = i < end;
        // the tile position of this lane's query: its own offset, or in the
        // sorted layout where the pair evaluation put it (the selection's
        // summaries and the bit words are kept by position)
        const int tp = (st.qpos != nullptr && act) ? st.qpos[i - start] : i - start;
        QSum q;
        int32_t lin = 1, lp = 1;
        if (act) {
            q = st.qsum[sc.qsum_off + tp];
            lin = st.q_lin[q_at(sc, i)];
            lp = st.q_lpred[q_at(sc, i)];
        } else {
            q.nfeas = 0;
        }
        // the window's bit words of the dirty workers
        if (st.qpos != nullptr)
            gather_win_bits(st, sc, L.dw, 0, nd, start, w0, act, tp, wb);
        else if (lane < nd)
            wb = load_win_bits(st, sc, a.w, start, w0, end);
        const uint64_t potm = ballot(act && q.nfeas > 0);
        int cur = 0;
        while (cur < NT && w0 + cur < end) {
            const uint64_t pm = potm & (~0ull << cur);
            const int p = pm ? __ffsll((unsigned long long)pm) - 1 : NT;
            // lanes cur..p-1: rejected whatever happened earlier in the tile
            Diag dr;
            int ab = 0, scn = 0;
            const bool mine = act && lane >= cur && lane < p;
            if (want_diag && mine)
                dr = reject_diag(st, sc, q, i, start, w0, lin, lp, tau, hb, L, nd, hot, wb, &ab, &scn);
            stale += ballot(mine && scn) ? 1 : 0;
            const uint64_t am = ballot(mine && ab);
            const int abl = am ? __ffsll((unsigned long long)am) - 1 : NT;
            const int lim = min(p, abl);
            if (act && lane >= cur && lane < lim) {
                if (st.out_worker) st.out_worker[sc.out_off + q_at(sc, i)] = -1;
                if (want_diag) st.out_diag[q_at(sc, i)] = dr;
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
            if (stale >= STALE_CUT) {
                pos = ip;
                cut = true;
                stale_cut = true;
                break;
            }
            const QView qv = broadcast_q(q, p);
            const int32_t plin = rdlane(lin, p), plp = rdlane(lp, p);
            if (next_empty == -2 && qv.efeas) next_empty = next_empty_worker(st, sc, L, nd, next_from);
            Scan sn;
            const Decision dc = decide<CACHE>(st, sc, qv, ip, start, w0, plin, plp, tau, hb, L, nd, hot, hotBs, hotm,
                                       next_empty, want_diag, wb, a, sn);
            if (dc.abort) {
                pos = ip;
                cut = true;
                break;
            }
            stale += dc.stale;
            fallbacks += dc.fallback;
            if (lane == 0) {
                if (st.out_worker) st.out_worker[sc.out_off + q_at(sc, ip)] = dc.w < 0 ? dc.w : dc.w + sc.out_add;
                if (want_diag) st.out_diag[q_at(sc, ip)] = dc.d;
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
                    if (USE_D) {
                        a.dlim = st.dlim[gw];
                        a.phi = st.phi[gw];
                        a.lgn = st.lgn[gw];
                    }
                    a.base = st.slot_base[gw];
                    a.DS = st.DS[gw];
                    a.S1 = st.S1[gw];
                    a.S2 = st.S2[gw];
                    a.SC = st.SC[gw];
                    a.SR = st.SR[gw];
                    a.key = st.key[gw];
                    a.rhs = st.rhs[gw];
                    if (st.qpos == nullptr) wb = load_win_bits(st, sc, w, start, w0, end);
                }
                if (lane == 0) {
                    L.dw[j] = w;
                    if (sc.W <= DBITS_W * 32) L.dbits[w >> 5] |= 1u << (w & 31);
                }
                if (st.qpos != nullptr) {
                    wave_sync();  // L.dw[j] written
                    gather_win_bits(st, sc, L.dw + j, j, 1, start, w0, act, tp, wb);
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
                if (USE_D) {
                    // the new request decodes from the end of this heartbeat with zero slack
                    const int64_t p = a.base + a.lgn;
                    st.lge[p] = eq;
                    st.lgw[p] = hb;
                    st.lgs[p] = -a.phi;
                    a.lgn += 1;
                }
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
        if (USE_D) st.lgn[gw] = a.lgn;
        st.built[gw] = 0;
        st.dlist[s * MAX_DIRTY + lane] = gw;
    }
    // per-query heartbeats: the tile ended at a query that heartbeats precede;
    // they run now, and the whole wave finds the next such query
    const bool hb_here = sc.hb != nullptr && pos == end && pos == c.hb_next && pos < c.Q;
    int32_t hb_n = 0, hb_after = c.Q;
    if (hb_here) {
        hb_n = sc.hb[pos];
        for (int32_t b = pos + 1; b < c.Q; b += NT) {
            const uint64_t m = ballot(b + lane < c.Q && sc.hb[b + lane] > 0);
            if (m) {
                hb_after = b + __ffsll((unsigned long long)m) - 1;
                break;
            }
        }
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
        } else if (hb_here) {  // hb_n decode iterations, each its own heartbeat
            cp->tau = c.tau + hb_n;
            cp->hb_index = c.hb_index + hb_n;
            cp->since_hb = 0;
            cp->rebuild = 1;
            cp->hb_next = hb_after;
        } else {
            cp->since_hb = since;
        }
        cp->start = pos;
        cp->aborts = c.aborts + (cut ? 1 : 0);
        cp->fallbacks = c.fallbacks + fallbacks;
        cp->stale_cuts = c.stale_cuts + (stale_cut ? 1 : 0);
        cp->commits = c.commits + commits;
        cp->round = c.round + 1;
        st.tinfo[s].first_pc[(c.round + 1) & 1] = INT32_MAX;
    }
    publish();
}

// The other variants, each pair in a unit of its own (so that the register
// allocation of one does not depend on the others): with the LDS copies of
// the scan; checking constraint (d); both.
hipError_t launch_commit_c(const State& st, int32_t blocks, hipStream_t stream);
hipError_t launch_commit_d(const State& st, int32_t blocks, bool cache, hipStream_t stream);
hipError_t launch_commit_dc(const State& st, int32_t blocks, hipStream_t stream);

}  // namespace ald
