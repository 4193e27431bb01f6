// Host side of libaladdin: argument validation, the layout of the caller's
// workspace, and the round loop that drives the tile pipeline (build -> eval ->
// select -> commit) on the caller's HIP stream.  Every entry point but
// ald_place_stream_async returns after its stream work is done.
//
// Device memory: the library allocates none.  The caller attaches a workspace
// (ald_set_workspace); the loaded workers' state occupies its start
// (state_bytes), and every call lays out its own tables in the rest.  A call
// that does not fit is refused with ALD_ESPACE before any device work, and
// ald_workspace_needed gives the size it needed.
#include "../../include/aladdin.h"
#include "ald_internal.h"
#include "ald_rebalance.h"
#include "ald_move.h"

#include <algorithm>
#include <cfloat>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <string>
#include <type_traits>
#include <vector>

using namespace ald;

namespace {

struct Arena {
    char* mem = nullptr;  // every worker, slot and control array, carved from the workspace
    size_t mem_bytes = 0;
    State st{};
    std::vector<Scen> hscen;
    std::vector<int32_t> hW;  // workers per scenario
    int32_t S = 0, NW = 0;
    int32_t T = 0;            // tile the scratch is laid out for
    int32_t target = 0;       // and the evaluation grid it aimed at
    int32_t eval_blocks = 0, sel_blocks = 0, commit_blocks = 0;
    char* scratch = nullptr;  // where the tile scratch was laid out (in the call part of the workspace)
    Scen* dscen = nullptr;
    int eval_mode = 2;    // how the pair evaluation takes the latency checks (launch_eval)
    bool use_d = false;   // some scenario checks constraint (d)
    // the commit keeps its untouched-worker scan's rows and keys in LDS: one
    // scenario of at most COMMIT_CACHE_W workers whose tiles heartbeats cut
    // (short tiles whose queries commit, so that scans repeat within a window)
    bool commit_cache = false;
    Ctl* hctl = nullptr;  // pinned host copy of the control blocks
    int32_t hctl_n = 0;
    // per scenario: the host copy of its per-query heartbeats during a call
    // (empty: no scenario has any)
    std::vector<const int32_t*> hb_host;

    ~Arena()
    {
        if (hctl) (void)hipHostFree(hctl);
    }
};

struct Events {
    hipEvent_t a, b;
    int kind;
};

// Where the stream of the loaded workers stands (what the next call starts from).
struct Pos {
    int32_t tau, hb_index, since_hb;
    bool rebuild;
    int64_t qcount;
};

// An asynchronous placement call, kept until the host has seen how it ended:
// the arguments a resumption needs, and the stream position before the call
// and after it (heartbeats fall at the same queries whatever tiles are cut,
// so the position after a finished call is known when it is issued).
struct AsyncCall {
    int32_t call;
    State st;         // its kernels' arguments (queries, outputs)
    int32_t T, wave;  // its tile and evaluation grid target
    bool moves;       // heartbeats move tau within the call
    Pos before, after;
};

}  // namespace

struct ald_handle {
    int device = 0;
    hipStream_t stream = nullptr;
    std::string err;
    int32_t tile = 4096;
    // pair-evaluation blocks the device holds at once per evaluation variant
    // [mode][diagnostics] (compute units x blocks per unit): a placement's
    // evaluation grid is sized to one such wave of blocks, since a partial
    // second wave leaves most of the chip idle
    int32_t eval_wave[EVAL_MODES][2] = {};
    Arena* main = nullptr;
    Arena* sweep = nullptr;  // the arena of the last sweep (in the call part of the workspace)
    int32_t W = 0;
    ald_model_t model{};
    int32_t max_cap = 0;
    // stream position carried across ald_place_stream calls
    int32_t tau = 0, hb_index = 0, since_hb = 0, round = 0;
    bool rebuild_pending = false;  // the last call ended with a heartbeat: every worker is stale
    bool dirty_pending = false;    // the last commit round left workers with stale summaries
    bool check_all = false;        // stale workers are not listed (after grouped placement): check every one
    int64_t qcount = 0;            // queries processed since the load (routes grouped placement)
    int32_t call_seq = 0;          // placement calls issued (the id in their control blocks)
    std::vector<AsyncCall> issued; // asynchronous calls whose end the host has not seen yet
    int64_t stats[4] = {0, 0, 0, 0};  // the last placement call: rounds, cuts, fallbacks, stale cuts
    Arena* grouped = nullptr;      // scenario view of the loaded workers for grouped placement
    // App. A's router: the group sizes it routes for and the queries each group
    // received since the load (or since the sizes changed)
    std::vector<int32_t> route_sizes;
    std::vector<int64_t> route_counts;
    // the caller's workspace: the loaded state in [ws, ws + state_bytes), each
    // call's own tables after it
    char* ws = nullptr;
    size_t ws_bytes = 0;
    size_t state_bytes = 0;
    size_t need = 0;  // bytes the last call refused with ALD_ESPACE needed
    int32_t prof = 0;  // kernel kinds timed (bit k = kind k)
    std::vector<Events> pending;
    std::vector<Events> pool;
    double tot_ms[5] = {0, 0, 0, 0, 0};
    int64_t launches[5] = {0, 0, 0, 0, 0};
};

namespace {

int fail(ald_handle* h, int code, const std::string& msg)
{
    if (h) h->err = msg;
    return code;
}

#define HIPCHK(h, call)                                                                   \
    do {                                                                                  \
        hipError_t e_ = (call);                                                           \
        if (e_ != hipSuccess)                                                             \
            return fail((h), ALD_EHIP, std::string(#call) + ": " + hipGetErrorString(e_)); \
    } while (0)

// Finite coefficients; the TTFT SLO may also be +inf (a decode worker of
// split-phase serving: no prefill runs there, so (c) and (d) do not apply).
bool finite_model(const ald_model_t& m)
{
    const double v[] = {m.c1, m.k1, m.k1q, m.c3, m.c2, m.k2, m.decode_slo, m.theta};
    for (double x : v)
        if (!std::isfinite(x)) return false;
    return std::isfinite(m.ttft_slo) || m.ttft_slo == INFINITY;
}

// Reasons a model is unusable, or empty.
std::string check_model(const ald_model_t& m)
{
    if (!finite_model(m)) return "model coefficients must be finite";
    if (!(m.k2 > 0.0)) return "k2 must be > 0";
    if (!(m.c2 >= 0.0)) return "c2 must be >= 0";
    if (!(m.decode_slo > m.c3)) return "decode_slo must exceed c3 (Eq. 4)";
    if (!(m.theta > 0.0 && m.theta <= 1.0)) return "theta must lie in (0, 1]";
    if (m.gamma_log2den < 0 || m.gamma_log2den > 8) return "gamma_log2den must lie in [0, 8]";
    if (m.gamma_num < 0 || m.gamma_num > (1 << m.gamma_log2den)) return "gamma must lie in [0, 1]";
    return "";
}

// Largest batch size b for which constraint (b) can still hold: a feasible
// placement needs theta*((T_dec - c3) - c2*b) >= k2*sum(D) > 0.  Evaluated with
// the same fp64 expression as the kernels.  -1 = unbounded (c2 == 0).
int64_t batch_bound(const ald_model_t& m)
{
    if (m.c2 == 0.0) return -1;
    auto ok = [&](int64_t b) { return m.theta * ((m.decode_slo - m.c3) - m.c2 * (double)b) > 0.0; };
    if (!ok(1)) return 0;
    int64_t lo = 1, hi = (int64_t)1 << 31;
    while (lo < hi) {
        int64_t mid = lo + (hi - lo + 1) / 2;
        if (ok(mid)) lo = mid; else hi = mid - 1;
    }
    return lo;
}

// Whether every near-tie band of a scenario spans at most 64 integer values,
// for workers of up to `capmax` live requests.  Decode: the band around
// rhs = theta ((T_dec - c3) - c2 (B + 1)) is under 3e-9 |rhs| wide including
// rounding, while the left side grows by k2 2^-gs per unit of qD.  TTFT: the
// band around T_pre is under 3e-9 T_pre wide plus the rounding of two TTFT
// values (under 2e-15 (|c1| + T_pre)), while the TTFT grows by at least
// k1 + k1q per unit of l_in.  Three values of slack on each side.
bool nt_integer(const Scen& s, int32_t capmax)
{
    if (!s.mono) return false;
    const double rmax = s.theta * (std::fabs(s.tdec - s.c3) + std::fabs(s.c2) * ((double)capmax + 1.0)) * (1.0 + 1e-12);
    const double wd = 3e-9 * rmax / std::ldexp(s.k2, -s.gs) + 3.0;
    const double tstep = s.k1 + s.k1q;
    if (!(tstep > 0.0)) return false;
    if (s.ttft == INFINITY) return wd <= 64.0;  // no TTFT band
    const double wt = (3e-9 * std::fabs(s.ttft) + 2e-15 * (std::fabs(s.c1) + std::fabs(s.ttft))) / tstep + 3.0;
    return wd <= 64.0 && wt <= 64.0;
}

Scen make_scen(const ald_model_t& m)
{
    Scen s{};
    s.c1 = m.c1; s.k1 = m.k1; s.k1q = m.k1q;
    s.c3 = m.c3; s.c2 = m.c2; s.k2 = m.k2;
    s.ttft = m.ttft_slo; s.tdec = m.decode_slo; s.theta = m.theta;
    s.gn = m.gamma_num; s.gs = m.gamma_log2den;
    s.mono = (m.k1 >= 0.0 && m.k1q >= 0.0) ? 1 : 0;
    return s;
}

// Hands out 256-byte aligned pieces of one buffer; with a null base it only
// adds up the size.
struct Carver {
    char* base;
    size_t off = 0;
    template <typename T>
    void take(T** p, size_t count)
    {
        if (count == 0) count = 1;
        off = (off + 255) & ~(size_t)255;
        *p = base ? (T*)(base + off) : nullptr;
        off += count * sizeof(T);
    }
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Worker and slot arrays for S scenarios, laid out at `at` (in the caller's
// workspace).  caps[w] = request slots of worker w.  With `at` null only the
// size is computed (*bytes).
int make_arena(ald_handle* h, Arena* a, const std::vector<Scen>& scen, const std::vector<int32_t>& W,
               const std::vector<int32_t>& caps, const std::vector<int32_t>& Ms, char* at, size_t* bytes)
{
    a->S = (int32_t)scen.size();
    a->hscen = scen;
    a->hW = W;
    int64_t NW = 0;
    for (int32_t w : W) NW += w;
    a->NW = (int32_t)NW;
    std::vector<int64_t> base(NW);
    int64_t slots = 0;
    for (int64_t i = 0; i < NW; ++i) {
        base[i] = slots;
        slots += (int64_t)caps[i] + 1;
    }
    int32_t wb = 0;
    for (int s = 0; s < a->S; ++s) {
        a->hscen[s].W = W[s];
        a->hscen[s].wbase = wb;
        wb += W[s];
    }
    State& st = a->st;
    Ctl* ctl = nullptr;
    TileInfo* ti = nullptr;
    int32_t* qbad = nullptr;
    size_t worker_bytes = 0;
    bool use_d = false;  // constraint (d)'s per-request log is only kept where it is checked
    for (const Scen& x : scen) use_d = use_d || x.use_d;
    const int64_t log_slots = use_d ? slots : 1;
    auto carve = [&](Carver& c) {
        c.take(&st.slot_base, NW); c.take(&st.cap, NW); c.take(&st.n, NW); c.take(&st.head, NW);
        c.take(&st.M, NW); c.take(&st.S1, NW); c.take(&st.S2, NW); c.take(&st.hbs, NW);
        c.take(&st.built, NW); c.take(&st.B, NW); c.take(&st.DS, NW); c.take(&st.key, NW);
        c.take(&st.peak, NW); c.take(&st.rhs, NW); c.take(&st.SC, NW); c.take(&st.SR, NW);
        c.take(&st.dq_max, NW); c.take(&st.ntd_lo, NW); c.take(&st.ntd_hi, NW);
        c.take(&st.lthr, NW); c.take(&st.ntt_lo, NW); c.take(&st.ntt_hi, NW);
        c.take(&st.ntd_mask, NW); c.take(&st.ntt_mask, NW);
        c.take(&st.phi, NW); c.take(&st.phi_hb, NW); c.take(&st.dlim, NW); c.take(&st.ntp_lo, NW);
        c.take(&st.ntp_hi, NW); c.take(&st.lgn, NW);
        worker_bytes = c.off;
        c.take(&st.e, slots); c.take(&st.s, slots); c.take(&st.pms, slots);
        c.take(&st.lge, log_slots); c.take(&st.lgw, log_slots); c.take(&st.lgs, log_slots);
        c.take(&st.lbt, (size_t)NW * LB_MAX);
        c.take(&st.dlist, (size_t)a->S * MAX_DIRTY); c.take(&st.dcount, a->S);
        c.take(&ctl, a->S); c.take(&ti, a->S); c.take(&a->dscen, a->S); c.take(&qbad, 1);
    };
    Carver sizing{nullptr};
    carve(sizing);
    *bytes = align256(sizing.off);
    if (!at) return ALD_OK;
    a->mem = at;
    a->mem_bytes = *bytes;
    Carver placing{at};
    carve(placing);
    st.ctl = ctl;
    st.tinfo = ti;
    st.scen = a->dscen;
    st.qbad = a->S == 1 ? qbad : nullptr;  // the sweep checks its queries up front instead
    st.S = a->S;
    st.NW = a->NW;
    // every per-worker array starts at zero, then slot bases, slot counts and capacities
    HIPCHK(h, hipMemsetAsync(a->mem, 0, worker_bytes, h->stream));
    HIPCHK(h, hipMemcpyAsync(st.slot_base, base.data(), NW * sizeof(int64_t), hipMemcpyHostToDevice, h->stream));
    HIPCHK(h, hipMemcpyAsync(st.cap, caps.data(), NW * sizeof(int32_t), hipMemcpyHostToDevice, h->stream));
    HIPCHK(h, hipMemcpyAsync(st.M, Ms.data(), NW * sizeof(int32_t), hipMemcpyHostToDevice, h->stream));
    HIPCHK(h, hipMemsetAsync(st.dcount, 0, a->S * sizeof(int32_t), h->stream));
    HIPCHK(h, hipMemsetAsync(qbad, 0, sizeof(int32_t), h->stream));
    bool mono = true, ntint = true;
    int64_t wfirst = 0;
    for (int s = 0; s < a->S; ++s) {
        int32_t capmax = 0;
        for (int32_t i = 0; i < W[s]; ++i) capmax = std::max(capmax, caps[wfirst + i]);
        wfirst += W[s];
        // constraint (d)'s limit depends on the decode history, so its near-tie
        // band has no bound from the coefficients
        a->hscen[s].ntint = (nt_integer(a->hscen[s], capmax) && !a->hscen[s].use_d) ? 1 : 0;
        mono = mono && a->hscen[s].mono;
        ntint = ntint && a->hscen[s].ntint;
    }
    a->eval_mode = ntint ? 2 : (mono ? 1 : 0);
    a->use_d = use_d;
    // empty workers of a scenario are interchangeable when they share one capacity
    int64_t w0 = 0;
    for (int s = 0; s < a->S; ++s) {
        bool uni = true;
        for (int32_t i = 1; i < W[s]; ++i) uni = uni && Ms[w0 + i] == Ms[w0];
        a->hscen[s].uniform_M = uni ? 1 : 0;
        w0 += W[s];
    }
    return ALD_OK;
}

// Lay out the tile scratch for tile length T at `base` (in the call part of
// the workspace) and fill in the grid geometry; with base null only the
// geometry and the size (*bytes) are computed.
int layout_scratch(ald_handle* h, Arena* a, int32_t T, int32_t target_blocks, char* base, size_t* bytes)
{
    // evaluation: blocks of EVAL_Q queries x wpb workers; selection: blocks of
    // SEL_THREADS queries; bit words: one per 64 queries and worker
    const int32_t echunks = (T + EVAL_Q - 1) / EVAL_Q;
    const int32_t schunks = (T + SEL_THREADS - 1) / SEL_THREADS;
    const int64_t groups = (int64_t)echunks * (EVAL_Q / 64);
    int64_t NWtot = 0;
    for (int s = 0; s < a->S; ++s) NWtot += a->hW[s];
    int32_t Wmax = 1;
    for (int s = 0; s < a->S; ++s) Wmax = std::max(Wmax, a->hW[s]);
    int32_t wpb = (int32_t)std::max<int64_t>(1, (NWtot * echunks + target_blocks - 1) / target_blocks);
    // at most 512 worker blocks per scenario: the selection merges one excess
    // entry per worker block and query (for short tiles over many workers the
    // evaluation's extra blocks outweigh the longer merge up to about there)
    wpb = std::max(wpb, (Wmax + 511) / 512);
    wpb = std::min(wpb, EVAL_WPB_MAX);
    int64_t bits = 0, part = 0, qs = 0;
    int32_t eb = 0, sb = 0, cb = 0;
    std::vector<Scen> hs = a->hscen;  // the arena changes only when the layout is placed
    for (int s = 0; s < a->S; ++s) {
        Scen& sc = hs[s];
        sc.wpb = std::min(wpb, std::max(1, sc.W));
        sc.nblk = (sc.W + sc.wpb - 1) / sc.wpb;
        sc.eval_blk0 = eb;
        eb += sc.nblk * echunks;
        sc.sel_blk0 = sb;
        // waves per 64-query group: more for wide scenarios, whose per-query
        // scan over workers is long
        sc.sel_g = sc.W >= 2048 ? 4 : (sc.W >= 1024 ? 2 : 1);
        const int32_t qgroups = (T + 63) / 64;
        const int32_t per_blk = (SEL_THREADS / 64) / sc.sel_g;
        sb += (qgroups + per_blk - 1) / per_blk;
        sc.fin_blk0 = cb;
        cb += 1;
        sc.bits_off = bits;
        bits += groups * sc.W;
        sc.part_off = part;
        sc.pstride = (int64_t)echunks * EVAL_Q;
        part += sc.pstride * sc.nblk;
        sc.qsum_off = qs;
        qs += (int64_t)schunks * SEL_THREADS;
    }
    // one-scenario tiles this long are evaluated in l_pred order: the tile's
    // permutation and its inverse
    const bool sorted = a->S == 1 && T >= SORT_MIN_TILE;
    const size_t perm_bytes = sorted ? align256((size_t)echunks * EVAL_Q * sizeof(int32_t)) : 0;
    *bytes = align256((size_t)bits * 16 + (size_t)part * sizeof(ulonglong2) + (size_t)qs * sizeof(QSum) + 1024) +
             2 * perm_bytes;
    if (!base) return ALD_OK;
    a->hscen = hs;
    a->eval_blocks = eb;
    a->sel_blocks = sb;
    a->commit_blocks = cb;
    a->T = T;
    a->target = target_blocks;
    a->scratch = base;
    char* p = base;
    a->st.bits_feas = (uint64_t*)p;
    p += (size_t)bits * 8;
    a->st.bits_nt = (uint64_t*)p;
    p += (size_t)bits * 8;
    p = (char*)(((uintptr_t)p + 255) & ~(uintptr_t)255);
    a->st.part = (ulonglong2*)p;
    p += (size_t)part * sizeof(ulonglong2);
    p = (char*)(((uintptr_t)p + 255) & ~(uintptr_t)255);
    a->st.qsum = (QSum*)p;
    p += (size_t)qs * sizeof(QSum);
    p = (char*)(((uintptr_t)p + 255) & ~(uintptr_t)255);
    a->st.qorig = sorted ? (int32_t*)p : nullptr;
    a->st.qpos = sorted ? (int32_t*)(p + perm_bytes) : nullptr;

    HIPCHK(h, hipMemcpyAsync(a->dscen, a->hscen.data(), a->S * sizeof(Scen), hipMemcpyHostToDevice, h->stream));
    return ALD_OK;
}

hipError_t prof_begin(ald_handle* h, int kind, Events* ev)
{
    ev->kind = -1;
    if (!((h->prof >> kind) & 1)) return hipSuccess;
    if (h->pool.empty()) {
        Events e;
        // timing only: no system-scope fence when the events are recorded
        hipError_t r = hipEventCreateWithFlags(&e.a, hipEventDisableSystemFence);
        if (r != hipSuccess) return r;
        r = hipEventCreateWithFlags(&e.b, hipEventDisableSystemFence);
        if (r != hipSuccess) return r;
        h->pool.push_back(e);
    }
    *ev = h->pool.back();
    h->pool.pop_back();
    ev->kind = kind;
    return hipEventRecord(ev->a, h->stream);
}

hipError_t prof_end(ald_handle* h, Events* ev)
{
    if (ev->kind < 0) return hipSuccess;
    h->pending.push_back(*ev);
    return hipEventRecord(ev->b, h->stream);
}

// After a stream sync: fold recorded event pairs into the totals.
void prof_collect(ald_handle* h)
{
    for (Events& e : h->pending) {
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, e.a, e.b) == hipSuccess) {
            h->tot_ms[e.kind] += ms;
            h->launches[e.kind] += 1;
        }
        h->pool.push_back(e);
    }
    h->pending.clear();
}

#define LAUNCH(h, kind, expr)                         \
    do {                                              \
        Events ev_;                                   \
        HIPCHK(h, prof_begin(h, kind, &ev_));         \
        HIPCHK(h, (expr));                            \
        HIPCHK(h, prof_end(h, &ev_));                 \
    } while (0)

// Refuse a call that needs more workspace than is attached (before any device work).
int need_space(ald_handle* h, size_t need)
{
    h->need = need;
    return fail(h, ALD_ESPACE, "the call needs a workspace of " + std::to_string(need) + " bytes (" +
                                   std::to_string(h->ws_bytes) + " attached)");
}

// Move every pointer of the arena that points into [from, from + n) by d bytes.
void relocate(Arena* a, const char* from, size_t n, ptrdiff_t d)
{
    auto mv = [&](auto*& p) {
        const char* c = (const char*)p;
        if (p != nullptr && c >= from && c < from + n) p = (std::remove_reference_t<decltype(p)>)(c + d);
    };
    State& st = a->st;
    mv(st.slot_base); mv(st.cap); mv(st.n); mv(st.head); mv(st.M); mv(st.S1); mv(st.S2); mv(st.hbs);
    mv(st.built); mv(st.B); mv(st.DS); mv(st.key); mv(st.peak); mv(st.rhs); mv(st.SC); mv(st.SR);
    mv(st.dq_max); mv(st.ntd_lo); mv(st.ntd_hi); mv(st.lthr); mv(st.ntt_lo); mv(st.ntt_hi);
    mv(st.ntd_mask); mv(st.ntt_mask); mv(st.phi); mv(st.phi_hb); mv(st.dlim); mv(st.ntp_lo); mv(st.ntp_hi);
    mv(st.lgn); mv(st.lge); mv(st.lgw); mv(st.lgs); mv(st.e); mv(st.s); mv(st.pms); mv(st.lbt);
    mv(st.scen); mv(st.ctl); mv(st.tinfo); mv(st.dlist); mv(st.dcount); mv(st.qbad);
    mv(a->dscen);
    a->mem += d;
}

int map_dev_error(ald_handle* h, int32_t code)
{
    switch (code) {
    case DEV_ESLOTS: return fail(h, ALD_ESLOTS, "a worker ran out of request slots (raise slots_per_worker)");
    case DEV_EOVERFLOW: return fail(h, ALD_EOVERFLOW, "a worker's state left the exactly representable range");
    case DEV_EINVAL: return fail(h, ALD_EINVAL, "query lengths must lie in [1, 2^24]");
    default: return fail(h, ALD_EHIP, "device error " + std::to_string(code));
    }
}

// First query after `from` that heartbeats precede (Q if none).
int32_t next_hb(const int32_t* hb, int32_t from, int32_t Q)
{
    int32_t j = from + 1;
    while (j < Q && hb[j] == 0) ++j;
    return j;
}

// Rounds needed to finish every scenario from its control state, if no tile
// is cut (hbs[s]: scenario s's per-query heartbeats, or null; hbs may be empty).
int64_t rounds_needed(const std::vector<Ctl>& c, const std::vector<const int32_t*>& hbs)
{
    int64_t most = 0;
    for (size_t s = 0; s < c.size(); ++s) {
        const Ctl& x = c[s];
        const int32_t* hb = s < hbs.size() ? hbs[s] : nullptr;
        if (x.err) continue;
        int64_t r = 0;
        int32_t pos = x.start, since = x.since_hb, nxt = x.hb_next;
        while (pos < x.Q) {
            int32_t end = tile_end(pos, x.Q, x.T, x.H, since, nxt);
            if (end <= pos) return -1;  // a tile that cannot advance (never set up so)
            since += end - pos;
            if (x.H > 0 && since >= x.H) since = 0;
            if (hb && end == nxt && end < x.Q) {
                since = 0;
                nxt = next_hb(hb, end, x.Q);
            }
            pos = end;
            ++r;
        }
        most = std::max(most, r);
    }
    return most;
}

// Drive the tile pipeline until every scenario has consumed its queries.
// `hc` holds the control blocks as last written to the device; on return it
// holds their final device values.  The first round's build runs in
// `first_mode` (-1: skipped, nothing is stale); later rounds check every worker
// when a heartbeat can have moved tau, else only the ones the previous commit
// round listed.
// The pinned host mirror the commit kernel copies the control blocks into.
int ensure_hctl(ald_handle* h, Arena* a)
{
    if (a->hctl_n < a->S) {
        if (a->hctl) HIPCHK(h, hipHostFree(a->hctl));
        a->hctl = nullptr;
        a->hctl_n = 0;
        HIPCHK(h, hipHostMalloc((void**)&a->hctl, a->S * sizeof(Ctl), hipHostMallocDefault));
        a->hctl_n = a->S;
    }
    HIPCHK(h, hipHostGetDevicePointer((void**)&a->st.ctl_host, a->hctl, 0));
    return ALD_OK;
}

// One round of the tile pipeline on every scenario of the arena.
int launch_round(ald_handle* h, Arena* a, int mode)
{
    if (mode >= 0) LAUNCH(h, 0, launch_build(a->st, h->stream, mode));
    LAUNCH(h, 1, launch_eval(a->st, a->eval_blocks, a->eval_mode, h->stream));
    LAUNCH(h, 2, launch_select(a->st, a->sel_blocks, h->stream));
    LAUNCH(h, 3, launch_commit(a->st, a->commit_blocks, a->use_d, a->commit_cache, h->stream));
    return ALD_OK;
}

int run_rounds(ald_handle* h, Arena* a, bool build_every_round, int first_mode, std::vector<Ctl>& hc)
{
    std::fill(h->stats, h->stats + 4, 0);
    std::vector<Ctl> c0(hc);
    int rc = ensure_hctl(h, a);
    if (rc != ALD_OK) return rc;
    bool first = true;
    for (;;) {
        int64_t need = rounds_needed(hc, a->hb_host);
        if (need < 0) return fail(h, ALD_EHIP, "internal error: a tile of no queries");
        if (need == 0) break;
        for (int64_t r = 0; r < need; ++r) {
            rc = launch_round(h, a, first ? first_mode : (build_every_round ? 0 : 1));
            if (rc != ALD_OK) return rc;
            first = false;
        }
        // every commit launch wrote its scenarios' control blocks to the pinned mirror
        HIPCHK(h, hipStreamSynchronize(h->stream));
        std::copy(a->hctl, a->hctl + a->S, hc.begin());
        prof_collect(h);
        for (const Ctl& x : hc)
            if (x.err) return map_dev_error(h, x.err);
    }
    for (size_t i = 0; i < hc.size(); ++i) {
        h->stats[0] += hc[i].round - c0[i].round;
        h->stats[1] += hc[i].aborts - c0[i].aborts;
        h->stats[2] += hc[i].fallbacks - c0[i].fallbacks;
        h->stats[3] += hc[i].stale_cuts - c0[i].stale_cuts;
    }
    return ALD_OK;
}

// The stream position after a call that starts from control block `c` and
// finishes: tiles end at heartbeats whatever tiles are cut, so the position
// follows from the tile sequence without cuts (as the commit kernel updates it).
Pos project(Ctl c, const int32_t* hb, int64_t qcount)
{
    while (c.start < c.Q) {
        const int32_t end = tile_end(c.start, c.Q, c.T, c.H, c.since_hb, c.hb_next);
        const int32_t since = c.since_hb + (end - c.start);
        c.rebuild = 0;
        if (c.H > 0 && since >= c.H) {
            c.tau += 1;
            c.hb_index += 1;
            c.since_hb = 0;
            c.rebuild = 1;
        } else if (hb && end == c.hb_next && end < c.Q) {
            c.tau += hb[end];
            c.hb_index += hb[end];
            c.since_hb = 0;
            c.rebuild = 1;
            c.hb_next = next_hb(hb, end, c.Q);
        } else {
            c.since_hb = since;
        }
        c.start = end;
    }
    return Pos{c.tau, c.hb_index, c.since_hb, c.rebuild != 0, qcount + c.Q};
}

void set_pos(ald_handle* h, const Pos& p)
{
    h->tau = p.tau;
    h->hb_index = p.hb_index;
    h->since_hb = p.since_hb;
    h->rebuild_pending = p.rebuild;
    h->qcount = p.qcount;
}

bool same_pos(const Ctl& c, const Pos& p)
{
    return c.tau == p.tau && c.hb_index == p.hb_index && c.since_hb == p.since_hb && (c.rebuild != 0) == p.rebuild;
}

// Read how the asynchronous placement calls issued since the host last looked
// have ended.  All finished: the position they projected is confirmed.  One
// stopped short of its queries (every later one was blocked on the device and
// did nothing): with `resume` its remaining rounds run now and the blocked
// calls are forgotten (their callers issue them again), else ALD_EINCOMPLETE.
// A device error is returned as the synchronous call would have returned it.
int settle(ald_handle* h, bool resume)
{
    if (h->issued.empty()) return ALD_OK;
    Arena* a = h->main;
    Ctl c{};
    HIPCHK(h, hipMemcpyAsync(&c, a->st.ctl, sizeof(Ctl), hipMemcpyDeviceToHost, h->stream));
    HIPCHK(h, hipStreamSynchronize(h->stream));
    prof_collect(h);
    size_t k = 0;
    while (k < h->issued.size() && h->issued[k].call != c.call) ++k;
    if (k == h->issued.size()) {
        h->issued.clear();
        return fail(h, ALD_EHIP, "internal error: the control block belongs to no issued call");
    }
    const AsyncCall x = h->issued[k];
    const bool last = k + 1 == h->issued.size();
    if (c.err) {
        h->issued.clear();
        set_pos(h, x.before);
        return map_dev_error(h, c.err);
    }
    if (c.start < c.Q && !resume)
        return fail(h, ALD_EINCOMPLETE, "an asynchronous placement stopped at query " + std::to_string(c.start) +
                                            " of " + std::to_string(c.Q) + ": ald_place_resume finishes it");
    h->issued.clear();
    if (c.start < c.Q) {
        // lay the tile scratch out for the call again (a blocked call may have
        // changed it), then run its remaining rounds with its own arguments
        a->hscen[0].hb = nullptr;
        size_t sb = 0;
        int rc = layout_scratch(h, a, x.T, x.wave, h->ws + h->state_bytes, &sb);
        if (rc != ALD_OK) return rc;
        a->st.q_lin = x.st.q_lin;
        a->st.q_lpred = x.st.q_lpred;
        a->st.out_worker = x.st.out_worker;
        a->st.out_diag = x.st.out_diag;
        a->st.call = x.call;
        a->commit_cache = x.moves && a->S == 1 && a->hW[0] <= COMMIT_CACHE_W;
        std::vector<Ctl> hc(1, c);
        rc = run_rounds(h, a, x.moves, x.moves ? 0 : 1, hc);
        if (rc != ALD_OK) {
            set_pos(h, x.before);
            return rc;
        }
        c = hc[0];
    } else if (!last) {
        set_pos(h, x.before);
        return fail(h, ALD_EHIP, "internal error: a call after a finished one did not start");
    }
    if (c.start < c.Q || !same_pos(c, x.after)) {
        set_pos(h, x.before);
        return fail(h, ALD_EHIP, "internal error: the stream position differs from the one projected");
    }
    set_pos(h, x.after);
    h->round = c.round;
    h->dirty_pending = c.ndirty > 0;
    h->check_all = false;
    return ALD_OK;
}

}  // namespace

extern "C" {

const char* ald_strerror(int code)
{
    switch (code) {
    case ALD_OK: return "ok";
    case ALD_EINVAL: return "invalid argument";
    case ALD_EHIP: return "HIP runtime error";
    case ALD_ESLOTS: return "worker request slots exhausted";
    case ALD_ESTATE: return "no workers loaded";
    case ALD_EOVERFLOW: return "value outside the exactly representable range";
    case ALD_ESPACE: return "workspace too small";
    case ALD_EINCOMPLETE: return "asynchronous placement unfinished";
    case ALD_EBLOCKED: return "asynchronous placement blocked by an unfinished one";
    default: return "unknown error";
    }
}

const char* ald_last_error(ald_handle_t h) { return h ? h->err.c_str() : "null handle"; }

int ald_create(ald_handle_t* out, int device, void* hip_stream)
{
    if (!out) return ALD_EINVAL;
    *out = nullptr;
    int count = 0;
    if (hipGetDeviceCount(&count) != hipSuccess || count <= 0) return ALD_EHIP;
    if (device < 0 || device >= count) return ALD_EINVAL;
    if (hipSetDevice(device) != hipSuccess) return ALD_EHIP;
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess || cus <= 0)
        return ALD_EHIP;
    int32_t wave[EVAL_MODES][2];
    for (int m = 0; m < EVAL_MODES; ++m)
        for (int x = 0; x < 2; ++x) {
            const int per_cu = eval_blocks_per_cu(m, x == 1);
            if (per_cu <= 0) return ALD_EHIP;
            wave[m][x] = cus * per_cu;
        }
    // the allocation-free entry point's fixed device array, once per device
    if (rb_static_init(device) != hipSuccess) return ALD_EHIP;
    ald_handle* h = new ald_handle();
    h->device = device;
    h->stream = (hipStream_t)hip_stream;
    std::copy(&wave[0][0], &wave[0][0] + 2 * EVAL_MODES, &h->eval_wave[0][0]);
    *out = h;
    return ALD_OK;
}

int ald_set_workspace(ald_handle_t h, void* workspace, size_t bytes)
{
    if (!h) return ALD_EINVAL;
    HIPCHK(h, hipSetDevice(h->device));
    if (bytes > 0 && !workspace) return fail(h, ALD_EINVAL, "null workspace");
    if (h->main) {
        if (int rc0 = settle(h, false)) return rc0;
    }
    if (((uintptr_t)workspace & 255) != 0) return fail(h, ALD_EINVAL, "the workspace must be 256-byte aligned");
    char* ws = bytes > 0 ? (char*)workspace : nullptr;
    if (h->main) {
        if (bytes < h->state_bytes) {
            h->need = h->state_bytes;
            return fail(h, ALD_ESPACE, "the loaded workers' state needs " + std::to_string(h->state_bytes) + " bytes");
        }
        if (ws != h->ws) {
            if (ws < h->ws + h->state_bytes && h->ws < ws + h->state_bytes)
                return fail(h, ALD_EINVAL, "the new workspace overlaps the loaded state");
            // the state moves with its pointers; the call part is laid out again by the next call
            HIPCHK(h, hipMemcpyAsync(ws, h->ws, h->state_bytes, hipMemcpyDeviceToDevice, h->stream));
            relocate(h->main, h->ws, h->state_bytes, ws - h->ws);
            h->main->scratch = nullptr;
            h->main->T = 0;
            HIPCHK(h, hipMemcpyAsync(h->main->dscen, h->main->hscen.data(), h->main->S * sizeof(Scen),
                                     hipMemcpyHostToDevice, h->stream));
        }
    }
    // the arenas of grouped placement and of the sweep lived in the call part
    delete h->grouped;
    h->grouped = nullptr;
    delete h->sweep;
    h->sweep = nullptr;
    h->ws = ws;
    h->ws_bytes = bytes;
    return ALD_OK;
}

int ald_workspace_needed(ald_handle_t h, size_t* bytes)
{
    if (!h || !bytes) return ALD_EINVAL;
    *bytes = h->need;
    return ALD_OK;
}

int ald_destroy(ald_handle_t h)
{
    if (!h) return ALD_OK;
    (void)hipSetDevice(h->device);
    (void)hipStreamSynchronize(h->stream);
    delete h->grouped;
    delete h->main;
    delete h->sweep;
    for (Events& e : h->pool) { (void)hipEventDestroy(e.a); (void)hipEventDestroy(e.b); }
    for (Events& e : h->pending) { (void)hipEventDestroy(e.a); (void)hipEventDestroy(e.b); }
    delete h;
    return ALD_OK;
}

int ald_set_tile(ald_handle_t h, int32_t tile_queries)
{
    if (!h) return ALD_EINVAL;
    if (tile_queries < 64 || tile_queries > (1 << 20)) return fail(h, ALD_EINVAL, "tile must lie in [64, 2^20]");
    h->tile = tile_queries;
    return ALD_OK;
}

int ald_set_profiling(ald_handle_t h, int32_t kinds)
{
    if (!h) return ALD_EINVAL;
    if (kinds < 0 || kinds > 31) return fail(h, ALD_EINVAL, "kinds must be a mask of bits 0..4");
    h->prof = kinds;
    if (h->prof) {
        for (int k = 0; k < 5; ++k) { h->tot_ms[k] = 0; h->launches[k] = 0; }
    }
    return ALD_OK;
}

int ald_place_stats(ald_handle_t h, int64_t* out)
{
    if (!h || !out) return ALD_EINVAL;
    std::copy(h->stats, h->stats + 4, out);
    return ALD_OK;
}

int ald_kernel_time(ald_handle_t h, int32_t kind, double* total_ms, int64_t* launches)
{
    if (!h || kind < 0 || kind > 4) return ALD_EINVAL;
    if (!h->pending.empty()) {  // launches of asynchronous calls
        HIPCHK(h, hipSetDevice(h->device));
        HIPCHK(h, hipStreamSynchronize(h->stream));
        prof_collect(h);
    }
    if (total_ms) *total_ms = h->tot_ms[kind];
    if (launches) *launches = h->launches[kind];
    return ALD_OK;
}

namespace {
int load_workers(ald_handle_t h, int32_t W, const ald_model_t* model, const int64_t* kv_capacity,
                 const int64_t* res_offsets, const int32_t* res_l_in, const int32_t* res_l_pred,
                 const int32_t* res_generated, int32_t slots_per_worker, const double* res_t_dec)
{
    if (!h) return ALD_EINVAL;
    HIPCHK(h, hipSetDevice(h->device));
    if (W <= 0) return fail(h, ALD_EINVAL, "W must be >= 1");
    if (!model || !kv_capacity || !res_offsets) return fail(h, ALD_EINVAL, "null argument");
    if (slots_per_worker < 0) return fail(h, ALD_EINVAL, "slots_per_worker must be >= 0");
    std::string why = check_model(*model);
    if (!why.empty()) return fail(h, ALD_EINVAL, why);
    std::vector<int64_t> off(W + 1), cap64(W);
    HIPCHK(h, hipMemcpyAsync(off.data(), res_offsets, (W + 1) * sizeof(int64_t), hipMemcpyDeviceToHost, h->stream));
    HIPCHK(h, hipMemcpyAsync(cap64.data(), kv_capacity, W * sizeof(int64_t), hipMemcpyDeviceToHost, h->stream));
    HIPCHK(h, hipStreamSynchronize(h->stream));
    if (off[0] != 0) return fail(h, ALD_EINVAL, "res_offsets[0] must be 0");
    for (int i = 0; i < W; ++i) {
        if (off[i + 1] < off[i]) return fail(h, ALD_EINVAL, "res_offsets must be non-decreasing");
        if (cap64[i] < 1) return fail(h, ALD_EINVAL, "kv_capacity must be >= 1");
        if (cap64[i] > ((int64_t)1 << 30)) return fail(h, ALD_EOVERFLOW, "kv_capacity above 2^30 tokens");
    }
    if (off[W] > 0 && (!res_l_in || !res_l_pred || !res_generated)) return fail(h, ALD_EINVAL, "null resident array");
    int64_t bound = slots_per_worker > 0 ? slots_per_worker : batch_bound(*model);
    if (bound < 0) return fail(h, ALD_EINVAL, "c2 == 0 leaves the batch size unbounded: pass slots_per_worker");
    std::vector<int32_t> caps(W), Ms(W);
    int64_t total = 0;
    int32_t maxcap = 0;
    for (int i = 0; i < W; ++i) {
        const int64_t R = off[i + 1] - off[i];
        const int64_t c = std::max<int64_t>(R, bound) + 1;
        if (c > HOT) return fail(h, ALD_EINVAL, "more than " + std::to_string(HOT - 1) + " request slots per worker");
        caps[i] = (int32_t)c;
        Ms[i] = (int32_t)cap64[i];
        total += c + 1;
        maxcap = std::max(maxcap, (int32_t)c);
    }
    if (total * 24 > ((int64_t)64 << 30)) return fail(h, ALD_EINVAL, "worker state would exceed 64 GiB");

    Arena* a = new Arena();
    std::vector<Scen> sc(1, make_scen(*model));
    sc[0].use_d = (res_t_dec != nullptr && model->ttft_slo != INFINITY) ? 1 : 0;
    // the state at the start of the workspace, then the load's error word and
    // a first tile layout
    size_t sb = 0, lb = 0;
    int rc = make_arena(h, a, sc, std::vector<int32_t>(1, W), caps, Ms, nullptr, &sb);
    if (rc == ALD_OK) rc = layout_scratch(h, a, 256, 4096, nullptr, &lb);
    if (rc != ALD_OK) { delete a; return rc; }
    if (sb + 256 + lb > h->ws_bytes) { delete a; return need_space(h, sb + 256 + lb); }
    // from here the previous workers are gone (with any asynchronous call on them)
    prof_collect(h);
    h->issued.clear();
    delete h->grouped;
    h->grouped = nullptr;
    delete h->main;
    h->main = nullptr;
    h->state_bytes = 0;
    rc = make_arena(h, a, sc, std::vector<int32_t>(1, W), caps, Ms, h->ws, &sb);
    // workers loaded with more requests than the evaluation stages: the variant
    // that reads them through their tables (any choice gives the same results)
    int64_t maxres = 0;
    for (int i = 0; i < W; ++i) maxres = std::max<int64_t>(maxres, off[i + 1] - off[i]);
    if (rc == ALD_OK && a->eval_mode == 2 && maxres >= STAGE_MAX) a->eval_mode = 3;
    if (rc == ALD_OK) rc = layout_scratch(h, a, 256, 4096, h->ws + sb + 256, &lb);
    if (rc != ALD_OK) { delete a; return rc; }
    int32_t* err_word = (int32_t*)(h->ws + sb);
    a->st.err_word = err_word;
    HIPCHK(h, hipMemsetAsync(err_word, 0, sizeof(int32_t), h->stream));
    HIPCHK(h, launch_ingest(a->st, W, res_offsets, res_l_in, res_l_pred, res_generated, res_t_dec, h->stream));
    int32_t dev_err = 0;
    HIPCHK(h, hipMemcpyAsync(&dev_err, err_word, sizeof(int32_t), hipMemcpyDeviceToHost, h->stream));
    HIPCHK(h, hipStreamSynchronize(h->stream));
    if (dev_err) {
        delete a;
        if (dev_err == DEV_EINVAL)
            return fail(h, ALD_EINVAL, "resident lengths must satisfy 1 <= l_in, l_pred <= 2^24 and 0 <= generated < l_pred "
                                       "(and decode times be finite and >= 0)");
        if (dev_err == DEV_EOVERFLOW) return fail(h, ALD_EOVERFLOW, "a worker's residents exceed 2^30 tokens of future KV demand");
        return map_dev_error(h, dev_err);
    }
    // build the breakpoint summaries once (one pass of the build kernel)
    Ctl c{};
    c.Q = 1;
    c.T = 1;
    c.rebuild = 1;
    c.first_rej = INT32_MAX;
    HIPCHK(h, hipMemcpyAsync(a->st.ctl, &c, sizeof(Ctl), hipMemcpyHostToDevice, h->stream));
    HIPCHK(h, launch_build(a->st, h->stream, 0));
    HIPCHK(h, hipMemcpyAsync(&c, a->st.ctl, sizeof(Ctl), hipMemcpyDeviceToHost, h->stream));
    HIPCHK(h, hipStreamSynchronize(h->stream));
    if (c.err) { delete a; return map_dev_error(h, c.err); }
    h->main = a;
    h->state_bytes = sb;
    h->W = W;
    h->model = *model;
    h->max_cap = maxcap;
    h->tau = h->hb_index = h->since_hb = h->round = 0;
    h->rebuild_pending = h->dirty_pending = h->check_all = false;
    h->qcount = 0;
    h->route_sizes.clear();
    h->route_counts.clear();
    return ALD_OK;
}
}  // namespace

int ald_load_workers(ald_handle_t h, int32_t W, const ald_model_t* model, const int64_t* kv_capacity,
                     const int64_t* res_offsets, const int32_t* res_l_in, const int32_t* res_l_pred,
                     const int32_t* res_generated, int32_t slots_per_worker)
{
    return load_workers(h, W, model, kv_capacity, res_offsets, res_l_in, res_l_pred, res_generated,
                        slots_per_worker, nullptr);
}

int ald_load_workers_history(ald_handle_t h, int32_t W, const ald_model_t* model, const int64_t* kv_capacity,
                             const int64_t* res_offsets, const int32_t* res_l_in, const int32_t* res_l_pred,
                             const int32_t* res_generated, const double* res_t_dec, int32_t slots_per_worker)
{
    if (!res_t_dec) return fail(h, ALD_EINVAL, "null decode history");
    return load_workers(h, W, model, kv_capacity, res_offsets, res_l_in, res_l_pred, res_generated,
                        slots_per_worker, res_t_dec);
}

}  // extern "C"

namespace {

// Forgets the per-query heartbeats of a call when it ends, however it ends.
struct HbScope {
    Arena* a;
    ~HbScope() { a->hb_host.clear(); }
};

// One stream call: heartbeats every H processed queries, or hb_before[q]
// (host array) decode iterations before query q.  With `status` (a device
// word) the call is asynchronous: it enqueues the rounds the call needs if no
// tile is cut, plus `spare` more, and the status kernel writes its outcome.
int place_stream(ald_handle_t h, int32_t Q, const int32_t* q_l_in, const int32_t* q_l_pred, int32_t heartbeat_every,
                 const int32_t* hb_before, int32_t* out_worker, ald_query_diag_t* out_diag,
                 int32_t* status = nullptr, int32_t spare = 0)
{
    if (!h) return ALD_EINVAL;
    HIPCHK(h, hipSetDevice(h->device));
    if (!h->main) return fail(h, ALD_ESTATE, "ald_load_workers has not been called");
    if (Q < 0 || heartbeat_every < 0) return fail(h, ALD_EINVAL, "Q and heartbeat_every must be >= 0");
    const bool async = status != nullptr;
    if (async && (spare < 0 || spare > (1 << 20))) return fail(h, ALD_EINVAL, "spare_rounds must lie in [0, 2^20]");
    int rc = async ? ALD_OK : settle(h, false);
    if (rc != ALD_OK) return rc;
    if (Q == 0) {
        if (async) HIPCHK(h, launch_status_ok(status, h->stream));
        return ALD_OK;
    }
    if (!q_l_in || !q_l_pred || !out_worker) return fail(h, ALD_EINVAL, "null argument");
    const int32_t H = heartbeat_every;
    int32_t tau = h->tau, hb = h->hb_index, since = h->since_hb;
    bool rebuild = h->rebuild_pending;
    if (H > 0 && since >= H) {  // a heartbeat already due from an earlier, longer period
        tau += 1;
        hb += 1;
        since = 0;
        rebuild = true;
    }
    int64_t iters = H > 0 ? (int64_t)Q / H + 2 : 0;
    if (hb_before) {
        int64_t tot = 0;
        for (int32_t q = 0; q < Q; ++q) {
            if (hb_before[q] < 0) return fail(h, ALD_EINVAL, "hb_before must be >= 0");
            tot += hb_before[q];
        }
        if (hb_before[0] > 0) {  // the heartbeats before the first query run first
            tau += hb_before[0];
            hb += hb_before[0];
            since = 0;
            rebuild = true;
            tot -= hb_before[0];
        }
        iters = tot + 2;
    }
    const int64_t tau_final = (int64_t)tau + iters;
    if (tau_final >= ((int64_t)1 << 27) || (int64_t)h->max_cap * tau_final >= ((int64_t)1 << 27))
        return fail(h, ALD_EOVERFLOW, "too many heartbeats for the 32-bit request state");
    Arena* a = h->main;
    int32_t T = std::min(h->tile, Q);
    if (H > 0) T = std::min(T, H);
    const int32_t wave = h->eval_wave[a->eval_mode][out_diag ? 1 : 0];
    // the call part of the workspace: the tile scratch, then the per-query heartbeats
    char* const call = h->ws + h->state_bytes;
    size_t scratch_bytes = 0;
    rc = layout_scratch(h, a, T, wave, nullptr, &scratch_bytes);
    if (rc != ALD_OK) return rc;
    const size_t need = h->state_bytes + scratch_bytes + (hb_before ? align256((size_t)Q * sizeof(int32_t)) : 0);
    if (need > h->ws_bytes) return need_space(h, need);
    HbScope hb_scope{a};
    int32_t* hb_dev = (int32_t*)(call + scratch_bytes);
    if (hb_before) {
        HIPCHK(h, hipMemcpyAsync(hb_dev, hb_before, (size_t)Q * sizeof(int32_t), hipMemcpyHostToDevice, h->stream));
        a->hb_host.assign(1, hb_before);
    }
    const int32_t* want_hb = hb_before ? hb_dev : nullptr;
    if (T != a->T || wave != a->target || a->scratch != call) {
        a->hscen[0].hb = want_hb;
        rc = layout_scratch(h, a, T, wave, call, &scratch_bytes);  // also copies the scenario table
        if (rc != ALD_OK) return rc;
    } else if (a->hscen[0].hb != want_hb) {
        a->hscen[0].hb = want_hb;
        HIPCHK(h, hipMemcpyAsync(a->dscen, a->hscen.data(), sizeof(Scen), hipMemcpyHostToDevice, h->stream));
    }
    Ctl c{};
    c.start = 0;
    c.Q = Q;
    c.T = T;
    c.H = H;
    c.since_hb = since;
    c.tau = tau;
    c.hb_index = hb;
    c.rebuild = rebuild ? 1 : 0;
    c.first_rej = INT32_MAX;
    c.round = h->round;
    c.hb_next = hb_before ? next_hb(hb_before, 0, Q) : 0;
    h->call_seq = h->call_seq == INT32_MAX ? 1 : h->call_seq + 1;
    c.call = h->call_seq;
    // an asynchronous call after another one starts only if that one finished
    const int32_t gate = (async && !h->issued.empty()) ? h->issued.back().call : -1;
    TileInfo ti{};
    ti.first_pc[0] = ti.first_pc[1] = INT32_MAX;
    HIPCHK(h, launch_begin(c, ti, a->st.ctl, a->st.tinfo, a->st.qbad, gate, h->stream));
    a->st.q_lin = q_l_in;
    a->st.q_lpred = q_l_pred;
    a->st.out_worker = out_worker;
    a->st.out_diag = (Diag*)out_diag;
    a->st.call = c.call;
    std::vector<Ctl> hc(1, c);
    // first build: every worker after a heartbeat, the last commit round's
    // workers if it changed any (unknown after an asynchronous call), else nothing
    const bool moves = H > 0 || hb_before != nullptr;  // heartbeats can move tau within the call
    a->commit_cache = moves && a->S == 1 && a->hW[0] <= COMMIT_CACHE_W;
    const bool dirty = h->dirty_pending || !h->issued.empty();
    const int first_mode = (rebuild || moves || h->check_all) ? 0 : (dirty ? 1 : -1);
    if (async) {
        rc = ensure_hctl(h, a);
        if (rc != ALD_OK) return rc;
        const int64_t need = rounds_needed(hc, a->hb_host);
        if (need < 1) return fail(h, ALD_EHIP, "internal error: a tile of no queries");
        // the last round's commit kernel writes the call's outcome
        for (int64_t r = 0; r < need + spare; ++r) {
            a->st.status = r + 1 == need + spare ? status : nullptr;
            rc = launch_round(h, a, r == 0 ? first_mode : (moves ? 0 : 1));
            a->st.status = nullptr;
            if (rc != ALD_OK) return rc;
        }
        AsyncCall x;
        x.call = c.call;
        x.st = a->st;
        x.T = T;
        x.wave = wave;
        x.moves = moves;
        x.before = Pos{h->tau, h->hb_index, h->since_hb, h->rebuild_pending, h->qcount};
        x.after = project(c, nullptr, h->qcount);
        h->issued.push_back(x);
        set_pos(h, x.after);
        h->check_all = false;
        return ALD_OK;
    }
    rc = run_rounds(h, a, moves, first_mode, hc);
    if (rc != ALD_OK) return rc;
    c = hc[0];
    h->qcount += Q;
    h->check_all = false;
    h->tau = c.tau;
    h->hb_index = c.hb_index;
    h->since_hb = c.since_hb;
    h->round = c.round;
    h->rebuild_pending = c.rebuild != 0;
    h->dirty_pending = c.ndirty > 0;
    return ALD_OK;
}

}  // namespace

extern "C" {

int ald_place_stream(ald_handle_t h, int32_t Q, const int32_t* q_l_in, const int32_t* q_l_pred,
                     int32_t heartbeat_every, int32_t* out_worker, ald_query_diag_t* out_diag)
{
    return place_stream(h, Q, q_l_in, q_l_pred, heartbeat_every, nullptr, out_worker, out_diag);
}

int ald_place_stream_async(ald_handle_t h, int32_t Q, const int32_t* q_l_in, const int32_t* q_l_pred,
                           int32_t heartbeat_every, int32_t spare_rounds, int32_t* out_worker,
                           ald_query_diag_t* out_diag, int32_t* status)
{
    if (h && !status) return fail(h, ALD_EINVAL, "null status");
    return place_stream(h, Q, q_l_in, q_l_pred, heartbeat_every, nullptr, out_worker, out_diag, status,
                        spare_rounds);
}

int ald_place_resume(ald_handle_t h)
{
    if (!h) return ALD_EINVAL;
    HIPCHK(h, hipSetDevice(h->device));
    if (!h->main) return fail(h, ALD_ESTATE, "ald_load_workers has not been called");
    return settle(h, true);
}

int ald_move_requests(ald_handle_t h, int32_t K, const int32_t* l_in, const int32_t* l_pred, const int32_t* from,
                      const int32_t* to)
{
    if (!h) return ALD_EINVAL;
    HIPCHK(h, hipSetDevice(h->device));
    if (!h->main) return fail(h, ALD_ESTATE, "ald_load_workers has not been called");
    if (int rc0 = settle(h, false)) return rc0;
    if (K < 0) return fail(h, ALD_EINVAL, "K must be >= 0");
    if (K == 0) return ALD_OK;
    if (!l_in || !l_pred || !from || !to) return fail(h, ALD_EINVAL, "null argument");
    const int32_t LMAX = 1 << 24;
    // per worker: the requests it gives up, then the ones it takes
    std::vector<std::vector<int32_t>> rm(h->W), in(h->W);
    for (int32_t k = 0; k < K; ++k) {
        if (from[k] < 0 || from[k] >= h->W || to[k] < 0 || to[k] >= h->W || from[k] == to[k])
            return fail(h, ALD_EINVAL, "move " + std::to_string(k) + ": workers out of range or equal");
        if (l_in[k] < 1 || l_in[k] > LMAX || l_pred[k] < 1 || l_pred[k] > LMAX)
            return fail(h, ALD_EINVAL, "move " + std::to_string(k) + ": lengths must lie in [1, 2^24]");
        rm[from[k]].push_back(k);
        in[to[k]].push_back(k);
    }
    std::vector<MoveWorker> mw;
    std::vector<int32_t> lin, lp;
    for (int32_t w = 0; w < h->W; ++w) {
        if (rm[w].empty() && in[w].empty()) continue;
        MoveWorker x{};
        x.gw = w;
        x.rm0 = (int32_t)lin.size();
        for (int32_t k : rm[w]) { lin.push_back(l_in[k]); lp.push_back(l_pred[k]); }
        x.rm1 = x.in0 = (int32_t)lin.size();
        for (int32_t k : in[w]) { lin.push_back(l_in[k]); lp.push_back(l_pred[k]); }
        x.in1 = (int32_t)lin.size();
        mw.push_back(x);
    }
    auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
    const size_t b_mw = up(mw.size() * sizeof(MoveWorker)), b_q = up(lin.size() * sizeof(int32_t));
    // the call part of the workspace: the error word, then the tables
    const size_t need = h->state_bytes + 256 + b_mw + 2 * b_q;
    if (need > h->ws_bytes) return need_space(h, need);
    int32_t* err_word = (int32_t*)(h->ws + h->state_bytes);
    char* base = h->ws + h->state_bytes + 256;
    MoveArgs a{};
    a.mw = (const MoveWorker*)base;
    a.nw = (int32_t)mw.size();
    a.tau = h->tau;
    a.hb = h->hb_index;
    a.lin = (const int32_t*)(base + b_mw);
    a.lpred = (const int32_t*)(base + b_mw + b_q);
    a.err = err_word;
    HIPCHK(h, hipMemcpyAsync(base, mw.data(), mw.size() * sizeof(MoveWorker), hipMemcpyHostToDevice, h->stream));
    HIPCHK(h, hipMemcpyAsync(base + b_mw, lin.data(), lin.size() * sizeof(int32_t), hipMemcpyHostToDevice, h->stream));
    HIPCHK(h, hipMemcpyAsync(base + b_mw + b_q, lp.data(), lp.size() * sizeof(int32_t), hipMemcpyHostToDevice,
                             h->stream));
    HIPCHK(h, hipMemsetAsync(err_word, 0, sizeof(int32_t), h->stream));
    a.apply = 0;  // check every worker first: a move that cannot be applied changes nothing
    HIPCHK(h, launch_move(h->main->st, a, h->stream));
    a.apply = 1;
    HIPCHK(h, launch_move(h->main->st, a, h->stream));
    int32_t dev_err = 0;
    HIPCHK(h, hipMemcpyAsync(&dev_err, err_word, sizeof(int32_t), hipMemcpyDeviceToHost, h->stream));
    HIPCHK(h, hipStreamSynchronize(h->stream));
    if (dev_err == DEV_ESLOTS) return fail(h, ALD_ESLOTS, "a worker has no request slot left for a moved request");
    if (dev_err != 0)
        return fail(h, ALD_EINVAL, "a moved request is not on its worker in the current heartbeat window");
    h->check_all = true;  // the changed workers are rebuilt by the next call
    return ALD_OK;
}

int ald_place_stream_hb(ald_handle_t h, int32_t Q, const int32_t* q_l_in, const int32_t* q_l_pred,
                        const int32_t* hb_before, int32_t* out_worker, ald_query_diag_t* out_diag)
{
    if (h && Q > 0 && !hb_before) return fail(h, ALD_EINVAL, "null hb_before");
    return place_stream(h, Q, q_l_in, q_l_pred, 0, Q > 0 ? hb_before : nullptr, out_worker, out_diag);
}

}  // extern "C"

namespace {

// App. A's router: the group of each of the next Q queries, continuing the
// counts.  The quota method of Balinski and Young: the h-th query goes to the
// group with the largest N_i / (a_i + 1) among the groups whose count a_i is
// still below h * N_i / N_w (ties to the lowest index), which keeps every
// count strictly within one query of its share h * N_i / N_w.  The candidates
// come off a heap in order of N_i / (a_i + 1); groups at their quota are set
// aside for the step.
void route_groups(const std::vector<int32_t>& N, std::vector<int64_t>& counts, int32_t Q, std::vector<int32_t>& out)
{
    const int32_t G = (int32_t)N.size();
    int64_t Nw = 0, h = 0;
    for (int32_t i = 0; i < G; ++i) {
        Nw += N[i];
        h += counts[i];
    }
    // does i come before j: larger N / (a + 1), then the lower index
    auto before = [&](int32_t i, int32_t j) {
        const int64_t l = (int64_t)N[i] * (counts[j] + 1), r = (int64_t)N[j] * (counts[i] + 1);
        return l != r ? l > r : i < j;
    };
    auto heap_less = [&](int32_t i, int32_t j) { return before(j, i); };  // max-heap on `before`
    std::vector<int32_t> heap(G), aside;
    for (int32_t i = 0; i < G; ++i) heap[i] = i;
    std::make_heap(heap.begin(), heap.end(), heap_less);
    out.resize(Q);
    for (int32_t q = 0; q < Q; ++q) {
        h += 1;
        int32_t pick = -1;
        while (!heap.empty()) {
            std::pop_heap(heap.begin(), heap.end(), heap_less);
            const int32_t i = heap.back();
            heap.pop_back();
            if (counts[i] * Nw < h * (int64_t)N[i]) {
                pick = i;
                break;
            }
            aside.push_back(i);
        }
        // some group is always below its quota: the counts add up to h - 1 < h
        counts[pick] += 1;
        out[q] = pick;
        heap.push_back(pick);
        std::push_heap(heap.begin(), heap.end(), heap_less);
        for (int32_t i : aside) {
            heap.push_back(i);
            std::push_heap(heap.begin(), heap.end(), heap_less);
        }
        aside.clear();
    }
}

// A scenario view of the loaded workers, one scenario per group: the worker
// arrays are the loaded arena's, the control and scratch arrays its own, laid
// out at `base` (with base null only the size, *bytes, is computed).
int grouped_view(ald_handle* h, int32_t G, const int32_t* sizes, char* base, size_t* bytes)
{
    Arena* m = h->main;
    if (!h->grouped) h->grouped = new Arena();
    Arena& a = *h->grouped;
    a.S = G;
    a.NW = m->NW;
    a.hW.assign(sizes, sizes + G);
    a.hscen.assign(G, m->hscen[0]);
    int32_t wb = 0;
    for (int32_t g = 0; g < G; ++g) {
        a.hscen[g].W = sizes[g];
        a.hscen[g].wbase = wb;
        a.hscen[g].qmap = nullptr;
        a.hscen[g].hb = nullptr;
        wb += sizes[g];
    }
    a.eval_mode = m->eval_mode;
    a.use_d = m->use_d;
    a.st = m->st;  // worker and slot arrays
    a.st.call = 0;  // as in its own control blocks
    Carver c{nullptr};
    Ctl* ctl = nullptr;
    TileInfo* ti = nullptr;
    int32_t* dlist = nullptr;
    int32_t* dcount = nullptr;
    Scen* dscen = nullptr;
    auto carve = [&](Carver& k) {
        k.take(&ctl, G); k.take(&ti, G); k.take(&dscen, G); k.take(&dlist, (size_t)G * MAX_DIRTY); k.take(&dcount, G);
    };
    carve(c);
    *bytes = align256(c.off);
    if (!base) return ALD_OK;
    a.mem = base;
    a.mem_bytes = *bytes;
    Carver k{base};
    carve(k);
    a.dscen = dscen;
    a.st.scen = dscen;
    a.st.ctl = ctl;
    a.st.tinfo = ti;
    a.st.dlist = dlist;
    a.st.dcount = dcount;
    a.st.qbad = nullptr;  // the queries are checked up front
    a.st.S = G;
    HIPCHK(h, hipMemsetAsync(dcount, 0, G * sizeof(int32_t), h->stream));
    a.T = 0;  // lay the scratch out again
    return ALD_OK;
}

}  // namespace

extern "C" {

int ald_place_grouped(ald_handle_t h, int32_t G, const int32_t* group_workers, int32_t Q, const int32_t* q_l_in,
                      const int32_t* q_l_pred, int32_t heartbeat_every, int32_t* out_worker,
                      ald_query_diag_t* out_diag)
{
    if (!h) return ALD_EINVAL;
    HIPCHK(h, hipSetDevice(h->device));
    if (!h->main) return fail(h, ALD_ESTATE, "ald_load_workers has not been called");
    if (int rc0 = settle(h, false)) return rc0;
    if (G < 1 || !group_workers) return fail(h, ALD_EINVAL, "G must be >= 1 with a size per group");
    int64_t wsum = 0;
    for (int32_t g = 0; g < G; ++g) {
        if (group_workers[g] < 1) return fail(h, ALD_EINVAL, "every group needs a worker");
        wsum += group_workers[g];
    }
    if (wsum != h->W) return fail(h, ALD_EINVAL, "the group sizes must add up to the loaded worker count");
    const int32_t H = heartbeat_every;
    if (Q < 0 || H < 0) return fail(h, ALD_EINVAL, "Q and heartbeat_every must be >= 0");
    if (Q == 0) return ALD_OK;
    if (!q_l_in || !q_l_pred || !out_worker) return fail(h, ALD_EINVAL, "null argument");
    int32_t tau = h->tau, hb = h->hb_index, since = h->since_hb;
    bool rebuild = h->rebuild_pending;
    if (H > 0 && since >= H) {  // a heartbeat already due from an earlier, longer period
        tau += 1;
        hb += 1;
        since = 0;
        rebuild = true;
    }
    // the cluster's heartbeats: one after every H processed queries of the
    // stream; hb_upto(k) of them come before the call's query k
    auto hb_upto = [&](int64_t k) -> int64_t { return H > 0 ? ((int64_t)since + k) / H : 0; };
    const int64_t fired = hb_upto(Q);
    const int64_t tau_final = (int64_t)tau + fired + 2;
    if (tau_final >= ((int64_t)1 << 27) || (int64_t)h->max_cap * tau_final >= ((int64_t)1 << 27))
        return fail(h, ALD_EOVERFLOW, "too many heartbeats for the 32-bit request state");
    // route: each query to a group (the router's counts continue across calls
    // while the group sizes stay the same)
    const std::vector<int32_t> sizes(group_workers, group_workers + G);
    std::vector<int64_t> counts = h->route_sizes == sizes ? h->route_counts : std::vector<int64_t>(G, 0);
    std::vector<int32_t> grp;
    route_groups(sizes, counts, Q, grp);
    // per group, in arrival order: its queries' positions in the call (qmap)
    // and the cluster heartbeats that come before each of them since its
    // previous query of the call (hbq)
    std::vector<int32_t> off(G + 1, 0);
    for (int32_t q = 0; q < Q; ++q) off[grp[q] + 1] += 1;
    for (int32_t g = 0; g < G; ++g) off[g + 1] += off[g];
    std::vector<int32_t> tab(2 * (size_t)Q);  // qmap, then hbq
    int32_t* qmap = tab.data();
    int32_t* hbq = tab.data() + Q;
    {
        std::vector<int32_t> fill(off.begin(), off.end() - 1);
        std::vector<int64_t> last(G, 0);
        for (int32_t q = 0; q < Q; ++q) {
            const int32_t g = grp[q];
            const int64_t u = hb_upto(q);
            qmap[fill[g]] = q;
            hbq[fill[g]] = (int32_t)(u - last[g]);
            last[g] = u;
            fill[g] += 1;
        }
    }
    // the call part of the workspace: the groups' control arrays, the query
    // maps and heartbeat counts, then the tile scratch
    int32_t qmax = 1;
    for (int32_t g = 0; g < G; ++g) qmax = std::max(qmax, off[g + 1] - off[g]);
    const int32_t T = std::min(h->tile, qmax);
    const int32_t wave = h->eval_wave[h->main->eval_mode][out_diag ? 1 : 0];
    size_t vb = 0, sbytes = 0;
    int rc = grouped_view(h, G, group_workers, nullptr, &vb);
    if (rc == ALD_OK) rc = layout_scratch(h, h->grouped, T, wave, nullptr, &sbytes);
    if (rc != ALD_OK) return rc;
    const size_t tb = align256(2 * (size_t)Q * sizeof(int32_t));
    const size_t need = h->state_bytes + vb + tb + sbytes;
    if (need > h->ws_bytes) return need_space(h, need);
    char* const call = h->ws + h->state_bytes;
    rc = grouped_view(h, G, group_workers, call, &vb);
    if (rc != ALD_OK) return rc;
    int32_t* const dtab = (int32_t*)(call + vb);
    Arena& a = *h->grouped;
    HbScope hb_scope{&a};
    HIPCHK(h, hipMemcpyAsync(dtab, tab.data(), 2 * (size_t)Q * sizeof(int32_t), hipMemcpyHostToDevice, h->stream));
    std::vector<Ctl> c(G);
    if (H > 0) a.hb_host.resize(G);
    for (int32_t g = 0; g < G; ++g) {
        Scen& sc = a.hscen[g];
        const int32_t n = off[g + 1] - off[g];
        sc.qmap = dtab + off[g];
        sc.hb = H > 0 ? dtab + Q + off[g] : nullptr;
        sc.out_off = 0;
        sc.out_add = sc.wbase;
        Ctl& x = c[g];
        x = Ctl{};
        x.Q = n;
        x.tau = tau;
        x.hb_index = hb;
        x.rebuild = rebuild ? 1 : 0;
        x.first_rej = INT32_MAX;
        if (H > 0 && n > 0) {
            const int32_t* hg = hbq + off[g];
            a.hb_host[g] = hg;
            if (hg[0] > 0) {  // the heartbeats before the group's first query run first
                x.tau += hg[0];
                x.hb_index += hg[0];
                x.rebuild = 1;
            }
            x.hb_next = next_hb(hg, 0, n);
        }
    }
    for (Ctl& x : c) x.T = T;
    rc = layout_scratch(h, &a, T, wave, call + vb + tb, &sbytes);  // also copies the scenario table
    if (rc != ALD_OK) return rc;
    std::vector<TileInfo> ti(G);
    for (auto& t : ti) { t = TileInfo{}; t.first_pc[0] = t.first_pc[1] = INT32_MAX; }
    HIPCHK(h, hipMemcpyAsync(a.st.ctl, c.data(), G * sizeof(Ctl), hipMemcpyHostToDevice, h->stream));
    HIPCHK(h, hipMemcpyAsync(a.st.tinfo, ti.data(), G * sizeof(TileInfo), hipMemcpyHostToDevice, h->stream));
    a.st.q_lin = q_l_in;
    a.st.q_lpred = q_l_pred;
    a.st.out_worker = out_worker;
    a.st.out_diag = (Diag*)out_diag;
    a.st.err_word = nullptr;
    HIPCHK(h, launch_query_stats(q_l_in, q_l_pred, Q, a.st.ctl, G, h->stream));
    rc = run_rounds(h, &a, H > 0, 0, c);
    if (rc != ALD_OK) return rc;
    // the stream's clock after the call; heartbeats after a group's last query
    // reach its workers through the rebuild at the start of the next call
    h->tau = tau + (int32_t)fired;
    h->hb_index = hb + (int32_t)fired;
    h->since_hb = H > 0 ? (int32_t)(((int64_t)since + Q) % H) : since + Q;
    h->qcount += Q;
    h->route_sizes = sizes;
    h->route_counts = counts;
    h->rebuild_pending = rebuild || fired > 0;
    h->dirty_pending = false;
    h->check_all = true;
    return ALD_OK;
}

}  // extern "C"

namespace {

// rho = c2 / k2 split into exact integer significands and exponents.
RbRho rb_rho(double k2, double c2)
{
    RbRho r{};
    r.k2 = k2;
    r.c2 = c2;
    r.rho_d = c2 / k2;
    // rho <= 1e9: R fits easily; c2 - R k2 is a multiple of the smaller of the
    // two significands' units, so the single rounding of the fma keeps its sign
    r.R = (int64_t)std::nearbyint(r.rho_d);
    const double rem = std::fma(-(double)r.R, k2, c2);
    r.fs = rem > 0.0 ? 1 : (rem < 0.0 ? -1 : 0);
    // |rho - R| <= |rho_d - R| + |rho - rho_d|, the latter at most 2^-53 rho_d
    r.f_up = (std::fabs(r.rho_d - (double)r.R) + std::ldexp(r.rho_d, -52)) * (1.0 + std::ldexp(1.0, -50));
    int ek = 0, ec = 0;
    const double fk = std::frexp(k2, &ek);
    r.mk = (uint64_t)std::ldexp(fk, 53);
    ek -= 53;
    if (c2 != 0.0) {
        const double fc = std::frexp(c2, &ec);
        r.mc = (uint64_t)std::ldexp(fc, 53);
        ec -= 53;
    }
    r.sh = ek - ec;
    return r;
}

// Algorithm 2 over P problems.  noalloc: the tables live in the library's
// fixed device array (rb_static_ptr) and the caller passes the error arrays;
// otherwise they live in the call part of the caller's workspace.
int rebalance_impl(ald_handle_t h, int32_t P, const int32_t* n_workers, const ald_model_t* models,
                  const int64_t* old_offsets, const int32_t* old_worker, const int32_t* old_l_pred,
                  const int32_t* old_l_out, const int32_t* old_l_real, const int32_t* old_l_repred,
                  const int64_t* new_offsets, const int32_t* new_l_pred, int32_t* new_worker,
                  int64_t* out_le, int64_t* out_be, int32_t* out_moves, int32_t log_cap, int32_t* out_log,
                  int64_t* out_obj,
                   bool noalloc)
{
    if (!h) return ALD_EINVAL;
    HIPCHK(h, hipSetDevice(h->device));
    if (P < 1) return fail(h, ALD_EINVAL, "P must be >= 1");
    if (!n_workers || !models || !old_offsets || !new_offsets) return fail(h, ALD_EINVAL, "null argument");
    if (old_offsets[0] != 0 || new_offsets[0] != 0) return fail(h, ALD_EINVAL, "offsets must start at 0");
    std::vector<RbProblem> prob(P);
    std::vector<RbChunk> chunks;
    int64_t wtot = 0;
    int32_t wmax = 1, jmax = 0;
    for (int32_t p = 0; p < P; ++p) {
        const std::string tag = "problem " + std::to_string(p) + ": ";
        if (n_workers[p] < 1 || n_workers[p] > RB_WMAX)
            return fail(h, ALD_EINVAL, tag + "n_workers must lie in [1, " + std::to_string(RB_WMAX) + "]");
        const int64_t o0 = old_offsets[p], o1 = old_offsets[p + 1], n0 = new_offsets[p], n1 = new_offsets[p + 1];
        if (o1 < o0 || n1 < n0) return fail(h, ALD_EINVAL, tag + "offsets must not decrease");
        if (n1 - n0 > RB_JMAX) return fail(h, ALD_EINVAL, tag + "more than " + std::to_string(RB_JMAX) + " new requests");
        const ald_model_t& m = models[p];
        const double big = std::ldexp(1.0, 900);
        const bool k2_ok = std::isfinite(m.k2) && m.k2 >= DBL_MIN && m.k2 <= big;
        const bool c2_ok = std::isfinite(m.c2) && (m.c2 == 0.0 || (m.c2 >= DBL_MIN && m.c2 <= big));
        if (!k2_ok || !c2_ok || !(m.c2 <= 1e9 * m.k2))
            return fail(h, ALD_EINVAL, tag + "needs normal k2 > 0 and c2 >= 0 (at most 2^900) with c2 / k2 <= 1e9");
        prob[p] = RbProblem{o0, o1, n0, wtot, rb_rho(m.k2, m.c2), n_workers[p], (int32_t)(n1 - n0)};
        for (int64_t b = o0; b < o1; b += RB_CHUNK) chunks.push_back(RbChunk{b, std::min(o1, b + RB_CHUNK), p, 0});
        wtot += n_workers[p];
        wmax = std::max(wmax, n_workers[p]);
        jmax = std::max(jmax, (int32_t)(n1 - n0));
    }
    const int64_t n_old = old_offsets[P], n_new = new_offsets[P];
    if (n_old >= ((int64_t)1 << 30) || n_new >= ((int64_t)1 << 30)) return fail(h, ALD_EINVAL, "too many requests");
    if (log_cap < 0 || (out_log != nullptr && (int64_t)P * log_cap > ((int64_t)1 << 30)))
        return fail(h, ALD_EINVAL, "log_cap must be >= 0 with P * log_cap <= 2^30");
    if ((n_old > 0 && (!old_worker || !old_l_pred || !old_l_out || !old_l_real || !old_l_repred)) ||
        (n_new > 0 && (!new_l_pred || !new_worker)))
        return fail(h, ALD_EINVAL, "null request array");
    if (chunks.size() + (size_t)P > (size_t)INT32_MAX) return fail(h, ALD_EINVAL, "too many blocks");
    // device tables (and error arrays when the caller passes none)
    const bool own_err = out_le == nullptr || out_be == nullptr;
    auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
    const size_t b_prob = up(P * sizeof(RbProblem)), b_chunk = up((chunks.size() + 1) * sizeof(RbChunk));
    const size_t b_err = own_err ? up(wtot * sizeof(int64_t)) : 0;
    const size_t need = b_prob + b_chunk + 2 * b_err;
    char* base = nullptr;
    int32_t* err_word = nullptr;
    if (noalloc) {
        if (own_err) return fail(h, ALD_EINVAL, "the allocation-free call needs out_le and out_be");
        if (P > RB_STATIC_P || chunks.size() + 1 > (size_t)RB_STATIC_CHUNKS)
            return fail(h, ALD_EINVAL, "the allocation-free call takes at most " + std::to_string(RB_STATIC_P) +
                                           " problems and " + std::to_string(RB_STATIC_CHUNKS - 1) +
                                           " chunks of ongoing requests (a problem's requests fill chunks of " +
                                           std::to_string(RB_CHUNK) + ")");
        char* mem = (char*)rb_static_ptr(h->device);
        if (mem == nullptr) return fail(h, ALD_EHIP, "the fixed device array was not set up for this device");
        base = mem;
        err_word = (int32_t*)(mem + RB_STATIC_TABLES);
    } else {
        // the call part of the workspace: the error word, then the tables
        const size_t total = h->state_bytes + 256 + need;
        if (total > h->ws_bytes) return need_space(h, total);
        err_word = (int32_t*)(h->ws + h->state_bytes);
        base = h->ws + h->state_bytes + 256;
    }
    RbArgs a{};
    a.prob = (const RbProblem*)base;
    a.chunk = (const RbChunk*)(base + b_prob);
    a.nchunk = (int32_t)chunks.size();
    a.P = P;
    a.old_worker = old_worker;
    a.old_lpred = old_l_pred;
    a.old_lout = old_l_out;
    a.old_lreal = old_l_real;
    a.old_lrepred = old_l_repred;
    a.new_lpred = new_l_pred;
    a.new_worker = new_worker;
    a.le = own_err ? (int64_t*)(base + b_prob + b_chunk) : out_le;
    a.be = own_err ? (int64_t*)(base + b_prob + b_chunk + b_err) : out_be;
    a.moves = out_moves;
    a.log = out_log;
    a.log_cap = log_cap;
    a.obj = out_obj;
    a.err = err_word;
    a.wmax = wmax;
    a.jmax = jmax;
    {
        int lds_max = 0;
        HIPCHK(h, hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, h->device));
        if (rb_moves_lds(wmax, jmax) + 512 > (size_t)lds_max)  // and the kernel's own small arrays
            return fail(h, ALD_EINVAL, "the largest problem's workers and new requests need " +
                                           std::to_string(rb_moves_lds(wmax, jmax)) + " bytes of LDS, more than the " +
                                           std::to_string(lds_max) + " of a workgroup");
    }
    HIPCHK(h, hipMemcpyAsync(base, prob.data(), P * sizeof(RbProblem), hipMemcpyHostToDevice, h->stream));
    if (!chunks.empty())
        HIPCHK(h, hipMemcpyAsync(base + b_prob, chunks.data(), chunks.size() * sizeof(RbChunk),
                                 hipMemcpyHostToDevice, h->stream));
    HIPCHK(h, hipMemsetAsync(a.le, 0, wtot * sizeof(int64_t), h->stream));
    HIPCHK(h, hipMemsetAsync(a.be, 0, wtot * sizeof(int64_t), h->stream));
    HIPCHK(h, hipMemsetAsync(err_word, 0, sizeof(int32_t), h->stream));
    LAUNCH(h, 4, launch_rebalance(a, h->stream));
    int32_t dev_err = 0;
    HIPCHK(h, hipMemcpyAsync(&dev_err, err_word, sizeof(int32_t), hipMemcpyDeviceToHost, h->stream));
    HIPCHK(h, hipStreamSynchronize(h->stream));
    prof_collect(h);
    if (dev_err == DEV_EOVERFLOW)
        return fail(h, ALD_EOVERFLOW, "a problem's moves did not settle within 4 * (new requests) + (workers) steps");
    if (dev_err != 0) return fail(h, ALD_EINVAL, "invalid request (worker index out of range, length outside "
                                                 "[1, 2^24], or more tokens generated than the real length)");
    return ALD_OK;
}


}  // namespace

namespace {

// The sweep, with a heartbeat period per scenario (H null: none).
// With `status` (a device word) the sweep is asynchronous: it enqueues the
// rounds every scenario needs if no tile is cut, plus `spare` more, and a
// status kernel writes the outcome.
int sweep(ald_handle_t h, int32_t S, const ald_scenario_t* scen, const int32_t* H, int32_t Q, const int32_t* q_l_in,
          const int32_t* q_l_pred, int32_t* out_rejected, int32_t* out_first_reject, int32_t* out_worker,
          int64_t* out_min_gpus, size_t* size_only = nullptr, int32_t* status = nullptr, int32_t spare = 0)
{
    if (!h) return ALD_EINVAL;
    HIPCHK(h, hipSetDevice(h->device));
    if (S <= 0 || Q < 0) return fail(h, ALD_EINVAL, "S must be >= 1 and Q >= 0");
    if (status && (spare < 0 || spare > (1 << 20))) return fail(h, ALD_EINVAL, "spare_rounds must lie in [0, 2^20]");
    if (S >= (1 << 24)) return fail(h, ALD_EINVAL, "at most 2^24 - 1 scenarios");
    if (!scen) return fail(h, ALD_EINVAL, "null argument");
    if (!size_only && (!out_rejected || !out_first_reject)) return fail(h, ALD_EINVAL, "null argument");
    if (!size_only && Q > 0 && (!q_l_in || !q_l_pred)) return fail(h, ALD_EINVAL, "null query array");
    bool any_hb = false;
    for (int32_t s = 0; s < S && H; ++s) {
        if (H[s] < 0) return fail(h, ALD_EINVAL, "heartbeat_every must be >= 0");
        any_hb = any_hb || H[s] > 0;
    }
    std::vector<Scen> sc(S);
    std::vector<int32_t> W(S), caps, Ms;
    int64_t NW = 0, slots = 0;
    for (int s = 0; s < S; ++s) {
        if (scen[s].n_workers < 1) return fail(h, ALD_EINVAL, "scenario with no workers");
        if (scen[s].gpus_per_worker < 1 || scen[s].gpus_per_worker > 256)
            return fail(h, ALD_EINVAL, "gpus_per_worker must lie in [1, 256]");
        if (scen[s].kv_capacity < 1) return fail(h, ALD_EINVAL, "kv_capacity must be >= 1");
        if (scen[s].kv_capacity > ((int64_t)1 << 30)) return fail(h, ALD_EOVERFLOW, "kv_capacity above 2^30 tokens");
        std::string why = check_model(scen[s].model);
        if (!why.empty()) return fail(h, ALD_EINVAL, "scenario " + std::to_string(s) + ": " + why);
        NW += scen[s].n_workers;
        int64_t b = batch_bound(scen[s].model);
        int64_t cap = (b < 0 ? (int64_t)Q : std::min<int64_t>(Q, b)) + 1;
        if (cap > HOT)
            return fail(h, ALD_EINVAL, "scenario " + std::to_string(s) + " admits more than " + std::to_string(HOT - 1) +
                                           " requests per worker");
        if (H && H[s] > 0) {  // the 32-bit request state counts decode iterations (as in ald_place_stream)
            const int64_t tau_final = (int64_t)Q / H[s] + 2;
            if (tau_final >= ((int64_t)1 << 27) || cap * tau_final >= ((int64_t)1 << 27))
                return fail(h, ALD_EOVERFLOW, "scenario " + std::to_string(s) + ": too many heartbeats for the "
                                                                                  "32-bit request state");
        }
        slots += scen[s].n_workers * (cap + 1);
    }
    if (NW > (1 << 30)) return fail(h, ALD_EINVAL, "too many workers");
    if (slots * 24 + NW * (int64_t)LB_MAX * 2 > ((int64_t)128 << 30)) return fail(h, ALD_EINVAL, "sweep state would exceed 128 GiB");
    for (int s = 0; s < S; ++s) {
        sc[s] = make_scen(scen[s].model);
        sc[s].gpw = scen[s].gpus_per_worker;
        W[s] = scen[s].n_workers;
        int64_t b = batch_bound(scen[s].model);
        int32_t cap = (int32_t)((b < 0 ? (int64_t)Q : std::min<int64_t>(Q, b)) + 1);
        for (int i = 0; i < W[s]; ++i) {
            caps.push_back(cap);
            Ms.push_back((int32_t)scen[s].kv_capacity);
        }
    }
    // the call part of the workspace: every scenario's workers, then the tile scratch
    if (!h->sweep) h->sweep = new Arena();
    Arena& a = *h->sweep;
    const int32_t T = std::max(1, std::min(h->tile, Q));
    size_t ab = 0, sbytes = 0;
    int rc = make_arena(h, &a, sc, W, caps, Ms, nullptr, &ab);
    if (rc == ALD_OK) rc = layout_scratch(h, &a, T, 16384, nullptr, &sbytes);
    if (rc != ALD_OK) return rc;
    const size_t need = h->state_bytes + ab + sbytes;
    if (size_only) {
        *size_only = ab + sbytes;
        return ALD_OK;
    }
    if (need > h->ws_bytes) return need_space(h, need);
    char* const call = h->ws + h->state_bytes;
    rc = make_arena(h, &a, sc, W, caps, Ms, call, &ab);
    if (rc == ALD_OK) rc = layout_scratch(h, &a, T, 16384, call + ab, &sbytes);
    if (rc != ALD_OK) return rc;
    std::vector<Ctl> c(S);
    for (int s = 0; s < S; ++s) {
        c[s] = Ctl{};
        c[s].Q = Q;
        c[s].T = T;
        c[s].H = H ? H[s] : 0;
        c[s].rebuild = 1;
        c[s].first_rej = INT32_MAX;
    }
    std::vector<TileInfo> ti(S);
    for (auto& t : ti) { t = TileInfo{}; t.first_pc[0] = t.first_pc[1] = INT32_MAX; }
    HIPCHK(h, hipMemcpyAsync(a.st.ctl, c.data(), S * sizeof(Ctl), hipMemcpyHostToDevice, h->stream));
    HIPCHK(h, hipMemcpyAsync(a.st.tinfo, ti.data(), S * sizeof(TileInfo), hipMemcpyHostToDevice, h->stream));
    a.st.q_lin = q_l_in;
    a.st.q_lpred = q_l_pred;
    a.st.out_worker = out_worker;
    a.st.out_diag = nullptr;
    a.st.err_word = nullptr;
    a.st.qbad = nullptr;  // (also with one scenario) the queries are checked below, before the rounds
    for (int s = 0; s < S; ++s) a.hscen[s].out_off = (int64_t)s * Q;
    HIPCHK(h, hipMemcpyAsync(a.dscen, a.hscen.data(), S * sizeof(Scen), hipMemcpyHostToDevice, h->stream));
    if (Q > 0) {
        HIPCHK(h, launch_query_stats(q_l_in, q_l_pred, Q, a.st.ctl, S, h->stream));
        if (status) {
            rc = ensure_hctl(h, &a);
            if (rc != ALD_OK) return rc;
            const int64_t need = rounds_needed(c, a.hb_host);
            if (need < 1) return fail(h, ALD_EHIP, "internal error: a tile of no queries");
            for (int64_t r = 0; r < need + spare; ++r) {
                rc = launch_round(h, &a, r == 0 ? 0 : (any_hb ? 0 : 1));
                if (rc != ALD_OK) return rc;
            }
        } else {
            rc = run_rounds(h, &a, any_hb, 0, c);
            if (rc != ALD_OK) return rc;
        }
    }
    HIPCHK(h, launch_sweep_outputs(a.st, out_rejected, out_first_reject, out_min_gpus, h->stream));
    if (status) {
        HIPCHK(h, launch_sweep_status(a.st, status, h->stream));
        return ALD_OK;
    }
    HIPCHK(h, hipStreamSynchronize(h->stream));
    return ALD_OK;
}

}  // namespace

extern "C" {

int ald_sweep_scenarios(ald_handle_t h, int32_t S, const ald_scenario_t* scen, int32_t Q, const int32_t* q_l_in,
                        const int32_t* q_l_pred, int32_t* out_rejected, int32_t* out_first_reject,
                        int32_t* out_worker, int64_t* out_min_gpus)
{
    return sweep(h, S, scen, nullptr, Q, q_l_in, q_l_pred, out_rejected, out_first_reject, out_worker, out_min_gpus);
}

int ald_sweep_scenarios_async(ald_handle_t h, int32_t S, const ald_scenario_t* scen, const int32_t* heartbeat_every,
                              int32_t Q, const int32_t* q_l_in, const int32_t* q_l_pred, int32_t spare_rounds,
                              int32_t* out_rejected, int32_t* out_first_reject, int32_t* out_worker,
                              int64_t* out_min_gpus, int32_t* status)
{
    if (h && !status) return fail(h, ALD_EINVAL, "null status");
    return sweep(h, S, scen, heartbeat_every, Q, q_l_in, q_l_pred, out_rejected, out_first_reject, out_worker,
                 out_min_gpus, nullptr, status, spare_rounds);
}

int ald_sweep_workspace_size(ald_handle_t h, int32_t S, const ald_scenario_t* scen, int32_t Q, size_t* bytes)
{
    if (!h || !bytes) return ALD_EINVAL;
    return sweep(h, S, scen, nullptr, Q, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, bytes);
}

int ald_workspace_size(ald_handle_t h, int32_t W, int64_t n_resident, const ald_model_t* model,
                       int32_t slots_per_worker, int32_t with_history, int32_t Q, size_t* bytes)
{
    if (!h || !bytes || !model) return ALD_EINVAL;
    if (W <= 0 || n_resident < 0 || slots_per_worker < 0 || Q < 0) return fail(h, ALD_EINVAL, "bad size");
    std::string why = check_model(*model);
    if (!why.empty()) return fail(h, ALD_EINVAL, why);
    int64_t bound = slots_per_worker > 0 ? slots_per_worker : batch_bound(*model);
    if (bound < 0) return fail(h, ALD_EINVAL, "c2 == 0 leaves the batch size unbounded: pass slots_per_worker");
    // the state's size depends on the total of the workers' slot ranges, at
    // most n_resident + W (bound + 2), which these slot counts add up to
    std::vector<int32_t> caps(W, (int32_t)std::min<int64_t>(bound + 1, INT32_MAX)), Ms(W, 1);
    const int64_t extra = std::min<int64_t>(n_resident, INT32_MAX - caps[0]);
    caps[0] += (int32_t)extra;
    Arena a;
    std::vector<Scen> sc(1, make_scen(*model));
    sc[0].use_d = (with_history && model->ttft_slo != INFINITY) ? 1 : 0;
    size_t sb = 0, lb = 0, most = 0;
    int rc = make_arena(h, &a, sc, std::vector<int32_t>(1, W), caps, Ms, nullptr, &sb);
    if (rc == ALD_OK) rc = layout_scratch(h, &a, 256, 4096, nullptr, &lb);
    if (rc != ALD_OK) return rc;
    most = 256 + lb;
    // a placement call of up to Q queries, for any evaluation variant the
    // model can take, with per-query heartbeats
    const int32_t T = std::max(1, std::min(h->tile, Q));
    for (int m = 0; m < EVAL_MODES; ++m)
        for (int x = 0; x < 2; ++x) {
            size_t tb = 0;
            rc = layout_scratch(h, &a, T, h->eval_wave[m][x], nullptr, &tb);
            if (rc != ALD_OK) return rc;
            most = std::max(most, tb + align256((size_t)Q * sizeof(int32_t)));
        }
    *bytes = sb + most;
    return ALD_OK;
}

int ald_sweep_scenarios_hb(ald_handle_t h, int32_t S, const ald_scenario_t* scen, const int32_t* heartbeat_every,
                           int32_t Q, const int32_t* q_l_in, const int32_t* q_l_pred, int32_t* out_rejected,
                           int32_t* out_first_reject, int32_t* out_worker, int64_t* out_min_gpus)
{
    if (h && !heartbeat_every) return fail(h, ALD_EINVAL, "null heartbeat_every");
    return sweep(h, S, scen, heartbeat_every, Q, q_l_in, q_l_pred, out_rejected, out_first_reject, out_worker,
                 out_min_gpus);
}

int ald_rebalance(ald_handle_t h, int32_t P, const int32_t* n_workers, const ald_model_t* models,
                  const int64_t* old_offsets, const int32_t* old_worker, const int32_t* old_l_pred,
                  const int32_t* old_l_out, const int32_t* old_l_real, const int32_t* old_l_repred,
                  const int64_t* new_offsets, const int32_t* new_l_pred, int32_t* new_worker,
                  int64_t* out_le, int64_t* out_be, int32_t* out_moves, int32_t log_cap, int32_t* out_log,
                  int64_t* out_obj)
{
    return rebalance_impl(h, P, n_workers, models, old_offsets, old_worker, old_l_pred, old_l_out, old_l_real,
                          old_l_repred, new_offsets, new_l_pred, new_worker, out_le, out_be, out_moves, log_cap,
                          out_log, out_obj, false);
}

int ald_rebalance_noalloc(ald_handle_t h, int32_t P, const int32_t* n_workers, const ald_model_t* models,
                          const int64_t* old_offsets, const int32_t* old_worker, const int32_t* old_l_pred,
                          const int32_t* old_l_out, const int32_t* old_l_real, const int32_t* old_l_repred,
                          const int64_t* new_offsets, const int32_t* new_l_pred, int32_t* new_worker,
                          int64_t* out_le, int64_t* out_be, int32_t* out_moves, int32_t log_cap, int32_t* out_log,
                  int64_t* out_obj)
{
    return rebalance_impl(h, P, n_workers, models, old_offsets, old_worker, old_l_pred, old_l_out, old_l_real,
                          old_l_repred, new_offsets, new_l_pred, new_worker, out_le, out_be, out_moves, log_cap,
                          out_log, out_obj, true);
}

int ald_worker_summary(ald_handle_t h, int32_t* B, int64_t* sum_c, int64_t* sum_r, int64_t* peak)
{
    if (!h) return ALD_EINVAL;
    HIPCHK(h, hipSetDevice(h->device));
    if (!h->main) return fail(h, ALD_ESTATE, "ald_load_workers has not been called");
    if (int rc0 = settle(h, false)) return rc0;
    if (!B || !sum_c || !sum_r || !peak) return fail(h, ALD_EINVAL, "null argument");
    // bring every worker's summaries to the current decode iteration first
    HIPCHK(h, launch_build(h->main->st, h->stream, 2));
    HIPCHK(h, launch_summary(h->main->st, h->W, B, sum_c, sum_r, peak, h->stream));
    HIPCHK(h, hipStreamSynchronize(h->stream));
    h->rebuild_pending = false;
    h->dirty_pending = false;
    return ALD_OK;
}

}  // extern "C"
