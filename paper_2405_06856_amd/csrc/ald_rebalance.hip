// Algorithm 2 (Sec. 4.3): re-balance a heartbeat's new requests against the
// output-length prediction errors of the ongoing ones.
//
// k_rb_errors  per chunk of ongoing requests: the two tests of the algorithm
//              (generated past the prediction: +re-prediction, +1 batch;
//              finished before it: +(real - predicted), -1 batch), summed per
//              worker across each wave's lanes and added to the problem's error
//              arrays; extra blocks validate each problem's new requests.
// k_rb_moves   one block per problem: c_i = l^e_i + rho * b^e_i (the error
//              line of Eq. 4 divided by k2, rho = c2 / k2 the real ratio) held
//              as the integer pair (l^e_i, b^e_i) in LDS, then greedy moves: of
//              every (placed request j, other worker y) pair, the one that
//              lowers sum |c| most (ties to the lowest j, then y) while that
//              decrease is positive -- found per step from the smallest c and
//              one gain per request.  Gains are ranked with fp64 stand-ins of
//              proven error; whatever lies within that error of the top is
//              compared exactly as the sign of a + rho * b for integer a, b
//              (rb_sign), so the choices are exact.
#include "ald_device.h"
#include "ald_rebalance.h"

#include <mutex>

namespace ald {

// The allocation-free entry point's tables and error word (see rb_static_init).
static __device__ __align__(256) unsigned char scratch[RB_STATIC_BYTES];

namespace {
constexpr int RB_STATIC_DEVICES = 64;
std::mutex g_static_mu;
void* g_static_ptr[RB_STATIC_DEVICES] = {};
}  // namespace

hipError_t rb_static_init(int device)
{
    if (device < 0 || device >= RB_STATIC_DEVICES) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_static_mu);
    if (g_static_ptr[device] != nullptr) return hipSuccess;
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    if (cur != device) return hipErrorInvalidDevice;  // the caller makes `device` current
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_static_ptr[device] = p;
    return hipSuccess;
}

void* rb_static_ptr(int device)
{
    if (device < 0 || device >= RB_STATIC_DEVICES) return nullptr;
    std::lock_guard<std::mutex> lk(g_static_mu);
    return g_static_ptr[device];
}

__global__ __launch_bounds__(RB_ETHREADS) void k_rb_errors(RbArgs a)
{
    const int tid = threadIdx.x, lane = lane_id();
    if ((int)blockIdx.x >= a.nchunk) {  // the new requests of one problem
        const RbProblem pr = a.prob[blockIdx.x - a.nchunk];
        bool bad = false;
        for (int j = tid; j < pr.n_new; j += RB_ETHREADS) {
            const int32_t l = a.new_lpred[pr.new0 + j], w = a.new_worker[pr.new0 + j];
            bad = bad || l < 1 || l > RB_LEN_MAX || w < -1 || w >= pr.W;
        }
        if (bad) raise_error(a.err, DEV_EINVAL);
        return;
    }
    const RbChunk ch = a.chunk[blockIdx.x];
    const RbProblem pr = a.prob[ch.p];
    bool bad = false;
    // coalesced: a wave takes 64 consecutive requests per step
    for (int64_t k0 = ch.begin + (int64_t)wave_id() * 64; k0 < ch.end; k0 += RB_ETHREADS) {
        const int64_t k = k0 + lane;
        int32_t x = -1;
        int64_t dl = 0, db = 0;
        if (k < ch.end) {
            const int32_t w = a.old_worker[k], lp = a.old_lpred[k], lo = a.old_lout[k];
            const int32_t lr = a.old_lreal[k], rp = a.old_lrepred[k];
            const bool ok = w >= 0 && w < pr.W && lp >= 1 && lp <= RB_LEN_MAX && lo >= 0 && lr >= 1 &&
                            lr <= RB_LEN_MAX && lo <= lr && rp >= 0 && rp <= RB_LEN_MAX;
            bad = bad || !ok;
            // with lo <= lr the two cases exclude each other
            if (ok && lo > lp) {  // under-estimated: still decoding past the prediction
                dl = rp;
                db = 1;
                x = w;
            } else if (ok && lr < lp) {  // over-estimated: finished before the prediction
                dl = (int64_t)lr - lp;
                db = -1;
                x = w;
            }
        }
        // one sum per distinct worker among the lanes (requests usually come
        // grouped by worker, so one or two), added by its first lane
        uint64_t act = ballot(x >= 0);
        while (act) {
            const int lead = __ffsll((unsigned long long)act) - 1;
            const int32_t xk = rdlane(x, lead);
            const bool mine = x == xk;
            // |dl| <= 2^24 and |db| <= 1 per lane: the wave's sums fit 32 bits
            const int64_t sl = wave_sum32(mine ? (int32_t)dl : 0), sb = wave_sum32(mine ? (int32_t)db : 0);
            if (lane == lead) {
                atomicAdd((unsigned long long*)&a.le[pr.wbase + xk], (unsigned long long)sl);
                atomicAdd((unsigned long long*)&a.be[pr.wbase + xk], (unsigned long long)sb);
            }
            act &= ~ballot(mine);
        }
    }
    if (bad) raise_error(a.err, DEV_EINVAL);
}

// ---------------------------------------------------------------------------------------------
// Exact sign of a + rho * b, i.e. of a * k2 + b * c2 (k2 > 0), for |a|, |b| < 2^62.
// Equal signs decide at once.  Otherwise fp64 decides when the computed sum
// is far from zero: each product carries a relative error of at most 2u
// (u = 2^-53: the conversion of the integer and the product) and the sum one
// more u, so |v - exact| < 4u (|x| + |y|), and |v| > 2^-50 (|x| + |y|) (computed)
// leaves the sign of v exact (no underflow: |x| >= k2 >= 2^-1022 and the
// coefficients are at most 2^900, checked on the host).  Else |a| k2 is
// compared with |b| c2 in 128-bit integers: |a| mk 2^sh against |b| mc (or the
// shift on the other side), first by bit length, and when the lengths agree
// the shifted product has at most 115 bits.
struct RbPair {
    int64_t a, b;  // a + rho * b
};
__device__ __forceinline__ RbPair rp_add(RbPair u, RbPair v) { return RbPair{u.a + v.a, u.b + v.b}; }
__device__ __forceinline__ RbPair rp_sub(RbPair u, RbPair v) { return RbPair{u.a - v.a, u.b - v.b}; }

__device__ __forceinline__ int bitlen128(unsigned __int128 v)
{
    const uint64_t hi = (uint64_t)(v >> 64), lo = (uint64_t)v;
    return hi ? 128 - __builtin_clzll(hi) : (lo ? 64 - __builtin_clzll(lo) : 0);
}

__device__ __noinline__ int rb_sign_exact(int64_t a, int64_t b, const RbRho& r)
{
    const int sa = a > 0 ? 1 : -1, sb = b > 0 ? 1 : -1;
    const unsigned __int128 p1 = (unsigned __int128)(uint64_t)(a > 0 ? a : -a) * r.mk;
    const unsigned __int128 p2 = (unsigned __int128)(uint64_t)(b > 0 ? b : -b) * r.mc;
    const int s1 = r.sh > 0 ? r.sh : 0, s2 = r.sh < 0 ? -r.sh : 0;
    const int l1 = bitlen128(p1) + s1, l2 = bitlen128(p2) + s2;
    int cmp;
    if (l1 != l2) {
        cmp = l1 > l2 ? 1 : -1;
    } else {
        const unsigned __int128 q1 = p1 << s1, q2 = p2 << s2;
        cmp = (q1 > q2) - (q1 < q2);
    }
    return cmp > 0 ? sa : (cmp < 0 ? sb : 0);
}

// When fp64 cannot decide, a + rho b = (a + R b) + (rho - R) b: a zero first
// term leaves the sign of (rho - R) b, and a first term of at least 1 in size
// decides alone while |(rho - R) b| < 1/2.  Only what is left takes the
// 128-bit comparison.
__device__ __forceinline__ int rb_sign(int64_t a, int64_t b, const RbRho& r)
{
    const int sa = (a > 0) - (a < 0), sb = (b > 0) - (b < 0);
    if (sb == 0 || r.mc == 0) return sa;
    if (sa == 0 || sa == sb) return sb;
    const double x = (double)a * r.k2, y = (double)b * r.c2;
    const double v = x + y, t = fabs(x) + fabs(y);
    if (fabs(v) > 0x1p-50 * t) return v > 0.0 ? 1 : -1;
    const __int128 A = (__int128)a + (__int128)r.R * b;
    if (A == 0) return r.fs * sb;
    if (fabs((double)b) * r.f_up < 0.5) return A > 0 ? 1 : -1;
    return rb_sign_exact(a, b, r);
}
__device__ __forceinline__ int rp_sign(RbPair u, const RbRho& r) { return rb_sign(u.a, u.b, r); }
__device__ __forceinline__ RbPair rp_abs(RbPair u, const RbRho& r)
{
    return rp_sign(u, r) < 0 ? RbPair{-u.a, -u.b} : u;
}

// Better candidate: larger gain, then the lower request index (a request's
// best target is unique, so the index order is the (request, worker) order).
__device__ __forceinline__ bool rb_better(RbPair g, int32_t o, RbPair bg, int32_t bo, const RbRho& r)
{
    if (o == INT32_MAX) return false;
    if (bo == INT32_MAX) return true;
    const int s = rp_sign(rp_sub(g, bg), r);
    return s > 0 || (s == 0 && o < bo);
}

// Smaller c, then the lower worker index (INT32_MAX: none).
__device__ __forceinline__ bool rb_lower(RbPair c, int32_t y, RbPair bc, int32_t by, const RbRho& r)
{
    if (y == INT32_MAX) return false;
    if (by == INT32_MAX) return true;
    const int s = rp_sign(rp_sub(c, bc), r);
    return s < 0 || (s == 0 && y < by);
}

__device__ __forceinline__ RbPair shfl_pair(RbPair v, int off)
{
    return RbPair{__shfl_xor(v.a, off, 64), __shfl_xor(v.b, off, 64)};
}

// ---------------------------------------------------------------------------------------------
// fp64 stand-ins.  For integers a, b (|a| < 2^56, |b| < 2^31) and rho_d =
// fl(c2 / k2), fl(fl(a) + fl(rho_d * b)) lies within 3.1 u T of a + rho * b,
// with T = |a| + rho |b| and u = 2^-53 (the conversion of a, the rounding of
// rho_d and of the product, and the sum).  S below bounds T over every value
// the kernel compares, and each decision taken in fp64 keeps a margin of
// tol = 2^-46 S (128 u S) against that error; whatever falls inside the margin
// is decided with exact pairs.
__device__ __forceinline__ double rb_approx(int64_t a, int64_t b, double rho_d)
{
    return (double)a + rho_d * (double)b;
}
__device__ __forceinline__ double rb_mag(int64_t a, int64_t b, double rho_d)
{
    return fabs((double)a) + rho_d * fabs((double)b);
}
// Wave-wide max / min of a double and min of an int: an inclusive scan with
// DPP row shifts and row broadcasts (as wave_incl_scan), read from lane 63.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ double dpp_f64(double ident, double x)
{
    const uint64_t ui = __builtin_bit_cast(uint64_t, ident), ux = __builtin_bit_cast(uint64_t, x);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)ui, (int)(uint32_t)ux, CTRL, ROW_MASK,
                                                              0xf, false);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)(ui >> 32), (int)(uint32_t)(ux >> 32),
                                                              CTRL, ROW_MASK, 0xf, false);
    return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}
template <bool MAX>
__device__ __forceinline__ double wave_ext_f64(double x)
{
    constexpr double id = MAX ? -INFINITY : INFINITY;
    auto op = [](double u, double v) { return MAX ? fmax(u, v) : fmin(u, v); };
    x = op(x, dpp_f64<0x111, 0xf>(id, x));  // row_shr:1
    x = op(x, dpp_f64<0x112, 0xf>(id, x));  // row_shr:2
    x = op(x, dpp_f64<0x114, 0xf>(id, x));  // row_shr:4
    x = op(x, dpp_f64<0x118, 0xf>(id, x));  // row_shr:8
    x = op(x, dpp_f64<0x142, 0xa>(id, x));  // row_bcast:15
    x = op(x, dpp_f64<0x143, 0xc>(id, x));  // row_bcast:31
    return rdlane_f64(x, 63);
}
__device__ __forceinline__ double wave_max_f64(double v) { return wave_ext_f64<true>(v); }
__device__ __forceinline__ double wave_min_f64(double v) { return wave_ext_f64<false>(v); }
__device__ __forceinline__ int32_t wave_min_i32(int32_t v) { return wave_min32(v); }

// sum |c| over the problem's workers (whole wave; every lane gets it)
__device__ RbPair rb_objective(const int64_t* cle, const int32_t* cbe, int W, const RbRho& rho)
{
    RbPair s{0, 0};
    for (int y = lane_id(); y < W; y += 64) s = rp_add(s, rp_abs(RbPair{cle[y], cbe[y]}, rho));
    return RbPair{wave_sum64(s.a), wave_sum64(s.b)};
}

// Half the decrease of sum |c| when a request of d = (l, 1) moves from a worker
// with c_x > 0 to one with c_min < 0:
// (|c_x| - |c_x - d| + |c_min| - |c_min + d|) / 2 = min(d, c_x) - max(0, d + c_min).
__device__ __forceinline__ double rb_half_gain(double dd, double cxd, double cmd)
{
    return fmin(dd, cxd) - fmax(0.0, dd + cmd);
}
// The same half decrease as an exact pair; the two signs it branches on are
// read off the stand-ins when they clear the margin (their error is below
// 9 u S), else taken exactly.
// With M = -c_min, the half decrease is min(d, c_x) - max(0, d - M) <= M,
// with equality exactly when M <= d <= c_x: such a request (`plateau`) holds
// the largest decrease of all.
struct RbHalfGain {
    RbPair g;
    bool plateau;
};
__device__ __forceinline__ RbHalfGain rb_half_gain_exact(RbPair cx, double cxd, RbPair cm, double cmd, int64_t l,
                                                         double dd, double tol, const RbRho& rho)
{
    const RbPair d{l, 1};
    const double t1 = dd - cxd, t2 = dd + cmd;
    const int s1 = t1 < -tol ? -1 : (t1 > tol ? 1 : rp_sign(rp_sub(d, cx), rho));  // sign of d - c_x
    const int s2 = t2 < -tol ? -1 : (t2 > tol ? 1 : rp_sign(rp_add(d, cm), rho));  // sign of d - M
    const RbPair mn = s1 <= 0 ? d : cx;
    return RbHalfGain{s2 > 0 ? rp_sub(mn, rp_add(d, cm)) : mn, s1 <= 0 && s2 >= 0};
}

// Wave-wide choice among lanes that hold an exact candidate (o != INT32_MAX),
// by the strict order `better`; `key` is the candidate's fp64 stand-in,
// larger for better ones.  A few candidates are taken in turn with uniform
// operands.  Otherwise the lane with the largest key (lowest index on equal
// keys) is the champion, every lane compares itself with it exactly, and the
// search goes on among those that beat it: the champion improves every round,
// and ties (equal pairs) and near ties settle in one or two.
template <typename Better>
__device__ __forceinline__ void rb_pick(RbPair& v, int32_t& o, double key, Better better)
{
    uint64_t m = ballot(o != INT32_MAX);
    if (m == 0) return;
    if (__popcll(m) <= 4) {
        int l = __ffsll((unsigned long long)m) - 1;
        RbPair bv{rdlane64s(v.a, l), rdlane64s(v.b, l)};
        int32_t bo = rdlane(o, l);
        m &= m - 1;
        while (m) {
            l = __ffsll((unsigned long long)m) - 1;
            const RbPair cv{rdlane64s(v.a, l), rdlane64s(v.b, l)};
            const int32_t co = rdlane(o, l);
            if (better(cv, co, bv, bo)) {
                bv = cv;
                bo = co;
            }
            m &= m - 1;
        }
        v = bv;
        o = bo;
        return;
    }
    bool in = o != INT32_MAX;
    for (;;) {
        const double kmax = wave_max_f64(in ? key : -INFINITY);
        const int32_t omin = wave_min_i32(in && key == kmax ? o : INT32_MAX);
        const int l = __ffsll((unsigned long long)ballot(in && key == kmax && o == omin)) - 1;
        const RbPair cv{rdlane64s(v.a, l), rdlane64s(v.b, l)};
        const int32_t co = rdlane(o, l);
        in = in && better(v, o, cv, co);
        if (!ballot(in)) {
            v = cv;
            o = co;
            return;
        }
    }
}

// One block of RB_WAVES waves per problem.  LDS (sized by the launch for its
// largest problem): c_y as the exact pair (cle, cbe), the fp64 stand-in of
// every positive c_y, the receivers list, and each new request's length and
// current worker.  A step:
// every wave finds c_min (the same result in each), takes the gains of its
// share of the requests and its best candidate; the waves' results meet in
// LDS; wave 0 finds the receiver and applies the move.  Three block barriers
// per step.
template <int JT>  // new requests per lane: at least jmax / (64 RB_WAVES)
__global__ __launch_bounds__(64 * RB_WAVES) void k_rb_moves(RbArgs a)
{
    extern __shared__ __align__(16) unsigned char rb_lds[];
    __shared__ double x_g[RB_WAVES];              // each wave's largest stand-in gain
    __shared__ int64_t x_a[RB_WAVES], x_b[RB_WAVES];  // each wave's best exact gain
    __shared__ int32_t x_j[RB_WAVES];             // and its request
    __shared__ int32_t x_p[RB_WAVES];             // each wave's lowest request on the plateau
    __shared__ double s_S;                        // bound on |a| + rho |b| over the values compared
    __shared__ int32_t s_nneg;                    // receivers listed
    __shared__ int32_t s_err;
    // invalid input somewhere: nothing changes (one read for the whole block,
    // as another block may raise the word meanwhile)
    if (threadIdx.x == 0) s_err = *a.err;
    __syncthreads();
    if (s_err != 0) return;
    const int p = blockIdx.x;
    const RbProblem pr = a.prob[p];
    const RbRho rho = pr.rho;
    const double rho_d = rho.rho_d;
    const int lane = lane_id(), wv = wave_id();
    const int W = pr.W, n = pr.n_new;
    const int Wm = a.wmax, Jm = a.jmax;
    int64_t* cle = (int64_t*)rb_lds;
    double* cdp = (double*)(cle + Wm);  // [Wm + 1] stand-in of c where c > 0 (the sources), else -inf;
                                        // slot W: unplaced
    int32_t* cbe = (int32_t*)(cdp + Wm + 1);
    int32_t* jl = cbe + Wm;
    int16_t* jx = (int16_t*)(jl + Jm);  // current worker of each new request (W: unplaced)
    int16_t* neg = jx + Jm;    // the workers with c < 0, in no particular order
    int16_t* pos = neg + Wm;   // index of a worker in neg (-1: not there)
    const int64_t max_moves = 4 * (int64_t)n + W;  // a guard; every move lowers sum |c| strictly
    const uint64_t below = (1ull << lane) - 1;
    auto lower = [&](RbPair u, int32_t uy, RbPair v, int32_t vy) { return rb_lower(u, uy, v, vy, rho); };
    auto better = [&](RbPair u, int32_t uj, RbPair v, int32_t vj) { return rb_better(u, uj, v, vj, rho); };

    RbPair obj0{0, 0};
    if (wv == 0) {
        double S = 0.0;
        int nneg = 0;
        for (int y0 = 0; y0 < W; y0 += 64) {
            const int y = y0 + lane;
            const bool in = y < W;
            const int64_t le = in ? a.le[pr.wbase + y] : 0;
            const int32_t be = in ? (int32_t)a.be[pr.wbase + y] : 0;
            const int sg = in ? rb_sign(le, be, rho) : 0;
            const uint64_t nm = ballot(in && sg < 0);
            const int at = nneg + __popcll(nm & below);
            if (in) {
                cle[y] = le;
                cbe[y] = be;
                cdp[y] = sg > 0 ? rb_approx(le, be, rho_d) : -INFINITY;
                pos[y] = (int16_t)(sg < 0 ? at : -1);
                if (sg < 0) neg[at] = (int16_t)y;
                S = fmax(S, rb_mag(le, be, rho_d));
            }
            nneg += __popcll(nm);
        }
        if (lane == 0) cdp[W] = -INFINITY;
        for (int j = lane; j < n; j += 64) {
            const int32_t w = a.new_worker[pr.new0 + j];
            jx[j] = (int16_t)(w < 0 ? W : w);
            const int32_t l = a.new_lpred[pr.new0 + j];
            jl[j] = l;
            S = fmax(S, (double)l + rho_d);
        }
        S = wave_max_f64(S) * (1.0 + 0x1p-40);
        __builtin_amdgcn_wave_barrier();
        obj0 = rb_objective(cle, cbe, W, rho);
        if (lane == 0) {
            s_S = S;
            s_nneg = nneg;
        }
    }
    __syncthreads();

    // A move of j from x to y lowers sum |c| by A + G with A = |c_x| - |c_x - d|
    // and G = |c_y| - |c_y + d| (d = l_pred_j + rho > 0).  G = -d when c_y >= 0
    // and A <= d always, so only workers with c_y < 0 can take a move that
    // gains, and only requests on workers with c_x > 0 (else A = -d <= -G);
    // source and target then differ by sign.  Over c < 0, G = d for c <= -d
    // and -2c - d above, never increasing in c: the largest G of any target is
    // G(c_min), reached by the lowest-index worker with c <= -d when
    // c_min <= -d, and otherwise only by the workers at c_min (the lowest index
    // of them).  So each step needs c_min, one gain per request and, for the
    // winning request, one scan of the receivers: the same choice as trying
    // every (request, worker) pair.
    int32_t moves = 0;
    for (;;) {
        const int nneg = s_nneg;
        const double S = s_S;
        if (nneg == 0) break;  // no move gains
        const double tol = S * 0x1p-46;
        // ---- c_min and the lowest worker index at it (every wave alike)
        double m1 = INFINITY, m2 = INFINITY;
        int32_t y1 = INT32_MAX;
        RbPair p1{0, 0};
        for (int k = lane; k < nneg; k += 64) {
            const int32_t y = neg[k];
            const RbPair v{cle[y], cbe[y]};
            const double vd = rb_approx(v.a, v.b, rho_d);
            if (vd < m1) {
                m2 = m1;
                m1 = vd;
                y1 = y;
                p1 = v;
            } else {
                m2 = fmin(m2, vd);
            }
        }
        const double cthr = wave_min_f64(m1) + 2.0 * tol;
        RbPair cm{0, 0};
        int32_t ci = INT32_MAX;
        if (m2 <= cthr) {  // several near the minimum in this lane: all of them exactly
            for (int k = lane; k < nneg; k += 64) {
                const int32_t y = neg[k];
                const RbPair v{cle[y], cbe[y]};
                if (rb_approx(v.a, v.b, rho_d) > cthr) continue;
                if (lower(v, y, cm, ci)) {
                    cm = v;
                    ci = y;
                }
            }
        } else if (m1 <= cthr) {
            cm = p1;
            ci = y1;
        }
        rb_pick(cm, ci, -rb_approx(cm.a, cm.b, rho_d), lower);
        const double cmd = rb_approx(cm.a, cm.b, rho_d);

        // ---- this wave's share of the requests, j = jw + t * 64 * RB_WAVES:
        // their stand-in gains stay in registers (a request that cannot move
        // has gain -inf)
        const int jw = wv * 64 + lane;
        const int tn = n > wv * 64 ? (n - wv * 64 + 64 * RB_WAVES - 1) / (64 * RB_WAVES) : 0;  // wave-uniform
        double gq[JT], cq[JT];  // stand-in gain and c_x of each request
        int32_t xq[JT], lq[JT];  // its worker and length
        double gl = -INFINITY;
#pragma unroll
        for (int t = 0; t < JT; ++t) {
            const int j = jw + t * 64 * RB_WAVES;
            const bool in = t < tn && j < n;
            xq[t] = in ? jx[j] : W;
            lq[t] = in ? jl[j] : 1;
        }
#pragma unroll
        for (int t = 0; t < JT; ++t) {
            cq[t] = cdp[xq[t]];
            gq[t] = rb_half_gain((double)lq[t] + rho_d, cq[t], cmd);
            gl = fmax(gl, gq[t]);
        }
        {
            const double gw = wave_max_f64(gl);
            if (lane == 0) x_g[wv] = gw;
        }
        __syncthreads();
        double gmax = x_g[0];
#pragma unroll
        for (int w = 1; w < RB_WAVES; ++w) gmax = fmax(gmax, x_g[w]);
        if (!(gmax + tol > 0.0)) break;  // every exact gain is <= 0 (or nothing can move)
        // every request whose stand-in lies within twice the margin of the top
        // may hold the largest exact gain: those of this lane, exactly, in
        // increasing j (ties are common: equal lengths give equal gains)
        const double gthr = gmax - 2.0 * tol;
        RbPair bg{0, 0};
        int32_t bj = INT32_MAX, pj = INT32_MAX;  // best candidate; lowest request on the plateau
        int64_t ca[JT];
        int32_t cb[JT];
#pragma unroll
        for (int t = 0; t < JT; ++t) {  // the exact c_x of every candidate, loads issued together
            const bool nr = gq[t] >= gthr;
            ca[t] = nr ? cle[xq[t]] : 0;
            cb[t] = nr ? cbe[xq[t]] : 0;
        }
#pragma unroll
        for (int t = 0; t < JT; ++t) {
            if (gq[t] >= gthr) {
                const int j = jw + t * 64 * RB_WAVES;
                const int32_t l = lq[t];
                const RbHalfGain h =
                    rb_half_gain_exact(RbPair{ca[t], cb[t]}, cq[t], cm, cmd, l, (double)l + rho_d, tol, rho);
                pj = (h.plateau && j < pj) ? j : pj;
                if (!h.plateau && better(h.g, j, bg, bj)) {
                    bg = h.g;
                    bj = j;
                }
            }
        }
        // a plateau request anywhere settles the step (the lowest such index);
        // otherwise the best candidate of each wave, then of the block
        const int32_t pw = wave_min_i32(pj);
        if (pw == INT32_MAX) rb_pick(bg, bj, rb_approx(bg.a, bg.b, rho_d), better);
        if (lane == 0) {
            x_a[wv] = bg.a;
            x_b[wv] = bg.b;
            x_j[wv] = bj;
            x_p[wv] = pw;
        }
        __syncthreads();
        int32_t pb = x_p[0];
#pragma unroll
        for (int w = 1; w < RB_WAVES; ++w) pb = min(pb, x_p[w]);
        if (pb != INT32_MAX) {
            bg = RbPair{-cm.a, -cm.b};
            bj = pb;
        } else {
            bg = RbPair{x_a[0], x_b[0]};
            bj = x_j[0];
#pragma unroll
            for (int w = 1; w < RB_WAVES; ++w) {
                const RbPair g{x_a[w], x_b[w]};
                const int32_t j = x_j[w];
                if (better(g, j, bg, bj)) {
                    bg = g;
                    bj = j;
                }
            }
        }
        if (bj == INT32_MAX || rp_sign(bg, rho) <= 0) break;  // no move lowers the objective
        if (moves >= max_moves) {
            if (threadIdx.x == 0) raise_error(a.err, DEV_EOVERFLOW);
            break;
        }

        if (wv == 0) {
            // ---- the receiver: the workers at c_min, or the lowest-index one with c <= -d
            const RbPair d{(int64_t)jl[bj], 1};
            const double dd = (double)d.a + rho_d;
            const int x = jx[bj];  // (its loads go out before the receiver's)
            const RbPair cx = rp_sub(RbPair{cle[x], cbe[x]}, d);
            int32_t y = ci;
            // on the plateau d >= M, so no worker but those at c_min has c <= -d
            if (pb == INT32_MAX && rp_sign(rp_add(cm, d), rho) <= 0) {
                int32_t lo = INT32_MAX;
                for (int k = lane; k < nneg; k += 64) {
                    const int32_t w = neg[k];
                    if (w >= lo) continue;
                    const double sd = rb_approx(cle[w], cbe[w], rho_d) + dd;
                    const bool takes = sd <= -tol ||
                                       (sd < tol && rp_sign(rp_add(RbPair{cle[w], cbe[w]}, d), rho) <= 0);
                    if (takes) lo = w;
                }
                y = wave_min_i32(lo);
            }
            // ---- apply (every lane computes the same values; lane 0 writes them)
            const RbPair cy = rp_add(RbPair{cle[y], cbe[y]}, d);
            // signs from the stand-ins where they clear the margin
            const double vx = rb_approx(cx.a, cx.b, rho_d), vy = rb_approx(cy.a, cy.b, rho_d);
            const int sx = vx > tol ? 1 : (vx < -tol ? -1 : rp_sign(cx, rho));
            const int sy = vy > tol ? 1 : (vy < -tol ? -1 : rp_sign(cy, rho));
            const double S1 = fmax(S, fmax(rb_mag(cx.a, cx.b, rho_d), rb_mag(cy.a, cy.b, rho_d)) * (1.0 + 0x1p-40));
            const int at_y = pos[y], last = nneg - 1, wl = neg[last];
            __builtin_amdgcn_wave_barrier();
            if (lane == 0) {
                cle[x] = cx.a;
                cbe[x] = (int32_t)cx.b;
                cdp[x] = sx > 0 ? vx : -INFINITY;
                cle[y] = cy.a;
                cbe[y] = (int32_t)cy.b;
                cdp[y] = sy > 0 ? vy : -INFINITY;
                jx[bj] = (int16_t)y;
                if (a.log != nullptr && moves < a.log_cap) {
                    a.log[2 * ((int64_t)p * a.log_cap + moves)] = bj;
                    a.log[2 * ((int64_t)p * a.log_cap + moves) + 1] = y;
                }
                // y (c_y was < 0, listed) leaves when c_y >= 0: the last entry
                // takes its place; x (c_x was > 0) joins when c_x < 0, appended
                int nn = nneg;
                if (sy >= 0) {
                    neg[at_y] = (int16_t)wl;
                    pos[wl] = (int16_t)at_y;
                    pos[y] = -1;
                    nn -= 1;
                }
                if (sx < 0) {
                    pos[x] = (int16_t)nn;
                    neg[nn] = (int16_t)x;
                    nn += 1;
                }
                s_nneg = nn;
                s_S = S1;
            }
        }
        moves += 1;
        __syncthreads();  // the move is applied before the next step reads the state
    }
    if (wv != 0) return;
    // final errors and workers
    for (int y = lane; y < W; y += 64) {
        a.le[pr.wbase + y] = cle[y];
        a.be[pr.wbase + y] = cbe[y];
    }
    for (int j = lane; j < n; j += 64) {
        const int x = jx[j];
        a.new_worker[pr.new0 + j] = x == W ? -1 : x;
    }
    const RbPair obj1 = rb_objective(cle, cbe, W, rho);
    if (lane == 0) {
        if (a.moves != nullptr) a.moves[p] = moves;
        if (a.obj != nullptr) {
            a.obj[4 * p] = obj0.a;
            a.obj[4 * p + 1] = obj0.b;
            a.obj[4 * p + 2] = obj1.a;
            a.obj[4 * p + 3] = obj1.b;
        }
    }
}

size_t rb_moves_lds(int32_t wmax, int32_t jmax)
{
    return (size_t)wmax * (8 + 8 + 4 + 2 + 2) + 8 + (size_t)jmax * (4 + 2);
}

hipError_t launch_rebalance(const RbArgs& a, hipStream_t stream)
{
    hipLaunchKernelGGL(k_rb_errors, dim3(a.nchunk + a.P), dim3(RB_ETHREADS), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const size_t lds = rb_moves_lds(a.wmax, a.jmax);
    const int per_lane = (a.jmax + 64 * RB_WAVES - 1) / (64 * RB_WAVES);
    static_assert(RB_JMAX <= 32 * 64 * RB_WAVES, "the widest variant covers RB_JMAX");
    if (per_lane <= 4)
        hipLaunchKernelGGL(k_rb_moves<4>, dim3(a.P), dim3(64 * RB_WAVES), lds, stream, a);
    else if (per_lane <= 8)
        hipLaunchKernelGGL(k_rb_moves<8>, dim3(a.P), dim3(64 * RB_WAVES), lds, stream, a);
    else if (per_lane <= 16)
        hipLaunchKernelGGL(k_rb_moves<16>, dim3(a.P), dim3(64 * RB_WAVES), lds, stream, a);
    else
        hipLaunchKernelGGL(k_rb_moves<32>, dim3(a.P), dim3(64 * RB_WAVES), lds, stream, a);
    return hipGetLastError();
}

}  // namespace ald
