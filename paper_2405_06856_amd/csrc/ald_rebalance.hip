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
//              one gain per request.  Every comparison is the sign of
//              a + rho * b for integer a, b, taken exactly (rb_sign), so the
//              choices are exact.
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
            const int64_t sl = wave_sum64(mine ? dl : 0), sb = wave_sum64(mine ? db : 0);
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

__device__ __forceinline__ int rb_sign(int64_t a, int64_t b, const RbRho& r)
{
    const int sa = (a > 0) - (a < 0), sb = (b > 0) - (b < 0);
    if (sb == 0 || r.mc == 0) return sa;
    if (sa == 0 || sa == sb) return sb;
    const double x = (double)a * r.k2, y = (double)b * r.c2;
    const double v = x + y, t = fabs(x) + fabs(y);
    if (fabs(v) > 0x1p-50 * t) return v > 0.0 ? 1 : -1;
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

// sum |c| over the problem's workers (block-wide; every thread gets it)
__device__ RbPair rb_objective(const int64_t* cle, const int32_t* cbe, int W, const RbRho& rho, int64_t* red)
{
    RbPair s{0, 0};
    for (int y = threadIdx.x; y < W; y += RB_THREADS) s = rp_add(s, rp_abs(RbPair{cle[y], cbe[y]}, rho));
    const int64_t oa = block_reduce<RB_THREADS>(s.a, 0, OpAdd(), red);
    const int64_t ob = block_reduce<RB_THREADS>(s.b, 0, OpAdd(), red);
    return RbPair{oa, ob};
}

__global__ __launch_bounds__(RB_THREADS) void k_rb_moves(RbArgs a)
{
    constexpr int NWAVE = RB_THREADS / 64;
    constexpr int JPT = RB_JMAX / RB_THREADS;  // new requests per thread
    __shared__ int64_t cle[RB_WMAX];   // c_y = (cle[y], cbe[y])
    __shared__ int32_t cbe[RB_WMAX];
    __shared__ int32_t jl[RB_JMAX];    // predicted length of new request j
    __shared__ int16_t jx[RB_JMAX];    // current worker of new request j (-1: unplaced)
    __shared__ int16_t neg[RB_WMAX];   // the workers with c < 0, in no particular order
    __shared__ int16_t pos[RB_WMAX];   // index of a worker in neg (-1: not there)
    __shared__ uint8_t cpos[RB_WMAX];  // c_y > 0
    __shared__ int64_t wga[NWAVE], wgb[NWAVE];
    __shared__ int32_t wo[NWAVE];
    __shared__ int64_t red[NWAVE];
    __shared__ int32_t s_nneg;
    if (*a.err != 0) return;  // invalid input somewhere: nothing changes
    const int p = blockIdx.x;
    const RbProblem pr = a.prob[p];
    const RbRho rho = pr.rho;
    const int tid = threadIdx.x, lane = lane_id(), wv = wave_id();
    const int W = pr.W, n = pr.n_new;
    const int64_t max_moves = 4 * (int64_t)n + W;  // a guard; every move lowers sum |c| strictly

    if (tid == 0) s_nneg = 0;
    __syncthreads();
    for (int y = tid; y < W; y += RB_THREADS) {
        const int64_t le = a.le[pr.wbase + y];
        const int32_t be = (int32_t)a.be[pr.wbase + y];
        cle[y] = le;
        cbe[y] = be;
        const int sg = rb_sign(le, be, rho);
        int32_t at = -1;
        if (sg < 0) {
            at = atomicAdd(&s_nneg, 1);
            neg[at] = (int16_t)y;
        }
        pos[y] = (int16_t)at;
        cpos[y] = sg > 0 ? 1 : 0;
    }
    for (int j = tid; j < n; j += RB_THREADS) {
        jx[j] = (int16_t)a.new_worker[pr.new0 + j];
        jl[j] = a.new_lpred[pr.new0 + j];
    }
    __syncthreads();
    const RbPair obj0 = rb_objective(cle, cbe, W, rho, red);  // ends with a barrier

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
        if (nneg == 0) break;  // no move gains
        // c_min and the lowest worker index at it, in every wave
        RbPair cm{0, 0};
        int32_t ci = INT32_MAX;
        for (int k = lane; k < nneg; k += 64) {
            const int32_t y = neg[k];
            const RbPair v{cle[y], cbe[y]};
            if (rb_lower(v, y, cm, ci, rho)) {
                cm = v;
                ci = y;
            }
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
            const RbPair ov = shfl_pair(cm, off);
            const int32_t oy = __shfl_xor(ci, off, 64);
            if (rb_lower(ov, oy, cm, ci, rho)) {
                cm = ov;
                ci = oy;
            }
        }
        // each thread's requests, in increasing j: the first largest gain
        RbPair bg{0, 0};
        int32_t bj = INT32_MAX;
#pragma unroll
        for (int u = 0; u < JPT; ++u) {
            const int j = tid + u * RB_THREADS;
            if (j >= n) break;
            const int x = jx[j];
            if (x < 0 || !cpos[x]) continue;
            const RbPair cx{cle[x], cbe[x]};
            const RbPair d{(int64_t)jl[j], 1};
            // (|c_x| - |c_x - d|) + (|c_min| - |c_min + d|), c_x > 0 > c_min
            const RbPair g = rp_add(rp_sub(cx, rp_abs(rp_sub(cx, d), rho)),
                                    rp_sub(RbPair{-cm.a, -cm.b}, rp_abs(rp_add(cm, d), rho)));
            if (rp_sign(rp_sub(g, bg), rho) > 0) {  // strictly: only positive gains, earlier j on ties
                bg = g;
                bj = j;
            }
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
            const RbPair og = shfl_pair(bg, off);
            const int32_t oj = __shfl_xor(bj, off, 64);
            if (rb_better(og, oj, bg, bj, rho)) {
                bg = og;
                bj = oj;
            }
        }
        if (lane == 0) {
            wga[wv] = bg.a;
            wgb[wv] = bg.b;
            wo[wv] = bj;
        }
        __syncthreads();
        // every wave finds the block's best from the per-wave ones
        RbPair g = lane < NWAVE ? RbPair{wga[lane], wgb[lane]} : RbPair{0, 0};
        int32_t jb = lane < NWAVE ? wo[lane] : INT32_MAX;
#pragma unroll
        for (int off = NWAVE / 2; off > 0; off >>= 1) {
            const RbPair og = shfl_pair(g, off);
            const int32_t oj = __shfl_xor(jb, off, 64);
            if (rb_better(og, oj, g, jb, rho)) {
                g = og;
                jb = oj;
            }
        }
        jb = rdlane(jb, 0);
        if (jb == INT32_MAX) break;  // no move lowers the objective
        if (moves >= max_moves) {
            if (tid == 0) raise_error(a.err, DEV_EOVERFLOW);
            break;
        }
        if (wv == 0) {
            const RbPair d{(int64_t)jl[jb], 1};
            int32_t y = ci;
            if (rp_sign(rp_add(cm, d), rho) <= 0) {  // the lowest-index receiver at or below -d
                int32_t lo = INT32_MAX;
                for (int k = lane; k < nneg; k += 64) {
                    const int32_t w = neg[k];
                    if (w < lo && rp_sign(rp_add(RbPair{cle[w], cbe[w]}, d), rho) <= 0) lo = w;
                }
#pragma unroll
                for (int off = 32; off > 0; off >>= 1) {
                    const int32_t o = __shfl_xor(lo, off, 64);
                    lo = o < lo ? o : lo;
                }
                y = rdlane(lo, 0);
            }
            if (lane == 0) {
                const int x = jx[jb];
                const RbPair cx = rp_sub(RbPair{cle[x], cbe[x]}, d);
                const RbPair cy = rp_add(RbPair{cle[y], cbe[y]}, d);
                cle[x] = cx.a;
                cbe[x] = (int32_t)cx.b;
                cle[y] = cy.a;
                cbe[y] = (int32_t)cy.b;
                const int sx = rp_sign(cx, rho), sy = rp_sign(cy, rho);
                cpos[x] = sx > 0 ? 1 : 0;
                cpos[y] = sy > 0 ? 1 : 0;
                if (sx < 0) {  // x (c_x was > 0) joins the receivers
                    pos[x] = (int16_t)s_nneg;
                    neg[s_nneg] = (int16_t)x;
                    s_nneg += 1;
                }
                if (sy >= 0) {  // y (c_y was < 0, listed) leaves: the last entry takes its place
                    const int at = pos[y], last = s_nneg - 1, wl = neg[last];
                    neg[at] = (int16_t)wl;
                    pos[wl] = (int16_t)at;
                    pos[y] = -1;
                    s_nneg = last;
                }
                jx[jb] = (int16_t)y;
                if (a.log != nullptr && moves < a.log_cap) {
                    a.log[2 * ((int64_t)p * a.log_cap + moves)] = jb;
                    a.log[2 * ((int64_t)p * a.log_cap + moves) + 1] = y;
                }
            }
        }
        moves += 1;
        __syncthreads();  // the move is applied before the next step reads the lists
    }
    // final errors and workers
    for (int y = tid; y < W; y += RB_THREADS) {
        a.le[pr.wbase + y] = cle[y];
        a.be[pr.wbase + y] = cbe[y];
    }
    for (int j = tid; j < n; j += RB_THREADS) a.new_worker[pr.new0 + j] = jx[j];
    const RbPair obj1 = rb_objective(cle, cbe, W, rho, red);
    if (tid == 0) {
        if (a.moves != nullptr) a.moves[p] = moves;
        if (a.obj != nullptr) {
            a.obj[4 * p] = obj0.a;
            a.obj[4 * p + 1] = obj0.b;
            a.obj[4 * p + 2] = obj1.a;
            a.obj[4 * p + 3] = obj1.b;
        }
    }
}

hipError_t launch_rebalance(const RbArgs& a, hipStream_t stream)
{
    hipLaunchKernelGGL(k_rb_errors, dim3(a.nchunk + a.P), dim3(RB_ETHREADS), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_rb_moves, dim3(a.P), dim3(RB_THREADS), 0, stream, a);
    return hipGetLastError();
}

}  // namespace ald
