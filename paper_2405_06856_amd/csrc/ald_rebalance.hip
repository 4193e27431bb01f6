// Algorithm 2 (Sec. 4.3): re-balance a heartbeat's new requests against the
// output-length prediction errors of the ongoing ones.
//
// k_rb_errors  per chunk of ongoing requests: the two tests of the algorithm
//              (generated past the prediction: +re-prediction, +1 batch;
//              finished before it: +(real - predicted), -1 batch), summed per
//              worker across each wave's lanes and added to the problem's error
//              arrays; extra blocks validate each problem's new requests.
// k_rb_moves   one block per problem: c_i = l^e_i + rho * b^e_i (the error
//              line of Eq. 4 divided by k2, rho = c2 / k2 in whole tokens) in
//              LDS, then greedy moves: of every (unmoved placed request j,
//              other worker y) pair, the one that lowers sum |c| most (ties to
//              the lowest j, then y) while that decrease is positive -- found
//              per step from the smallest c and one gain per request.  All
//              int64: the choices are exact.
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

__device__ __forceinline__ int64_t abs64(int64_t v) { return v < 0 ? -v : v; }

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

// Better candidate: larger gain, then the lower (request, worker) order.
__device__ __forceinline__ bool rb_better(int64_t g, int32_t o, int64_t bg, int32_t bo)
{
    return g > bg || (g == bg && o < bo);
}

__global__ __launch_bounds__(RB_THREADS) void k_rb_moves(RbArgs a)
{
    constexpr int NWAVE = RB_THREADS / 64;
    constexpr int JPT = RB_JMAX / RB_THREADS;  // new requests per thread
    __shared__ int64_t c[RB_WMAX];
    __shared__ int64_t negc[RB_WMAX];  // c of the workers listed in neg
    __shared__ int32_t jl[RB_JMAX];    // predicted length of new request j
    // worker of new request j: >= 0 movable, -1 unplaced, -2 - x moved away from x
    __shared__ int16_t jx[RB_JMAX];
    __shared__ int16_t jy[RB_JMAX];    // where a moved request went
    __shared__ int16_t neg[RB_WMAX];   // the workers with c < 0, in no particular order
    __shared__ int16_t pos[RB_WMAX];   // index of a worker in neg (-1: not there)
    __shared__ int64_t wg[NWAVE];
    __shared__ int32_t wo[NWAVE];
    __shared__ int64_t red[NWAVE];
    __shared__ int32_t s_nneg;
    if (*a.err != 0) return;  // invalid input somewhere: nothing changes
    const int p = blockIdx.x;
    const RbProblem pr = a.prob[p];
    const int tid = threadIdx.x, lane = lane_id(), wv = wave_id();
    const int W = pr.W, n = pr.n_new;
    const int64_t rho = pr.rho;

    if (tid == 0) s_nneg = 0;
    __syncthreads();
    int64_t sabs = 0;
    for (int y = tid; y < W; y += RB_THREADS) {
        const int64_t v = a.le[pr.wbase + y] + rho * a.be[pr.wbase + y];
        c[y] = v;
        sabs += abs64(v);
        int32_t at = -1;
        if (v < 0) {
            at = atomicAdd(&s_nneg, 1);
            neg[at] = (int16_t)y;
            negc[at] = v;
        }
        pos[y] = (int16_t)at;
    }
    for (int j = tid; j < n; j += RB_THREADS) {
        jx[j] = (int16_t)a.new_worker[pr.new0 + j];
        jl[j] = a.new_lpred[pr.new0 + j];
    }
    const int64_t obj0 = block_reduce<RB_THREADS>(sabs, 0, OpAdd(), red);  // ends with a barrier
    int64_t obj = obj0;

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
        if (nneg == 0) break;  // no move gains (uniform)
        // c_min and the lowest worker index at it, in every wave
        int64_t cm = INT64_MAX;
        int32_t ci = INT32_MAX;
        for (int k = lane; k < nneg; k += 64) {
            const int64_t v = negc[k];
            const int32_t y = neg[k];
            if (v < cm || (v == cm && y < ci)) {
                cm = v;
                ci = y;
            }
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
            const int64_t ov = __shfl_xor(cm, off, 64);
            const int32_t oy = __shfl_xor(ci, off, 64);
            if (ov < cm || (ov == cm && oy < ci)) {
                cm = ov;
                ci = oy;
            }
        }
        // each thread's requests, in increasing j: the first largest gain
        int64_t bg = 0;
        int32_t bj = INT32_MAX;
#pragma unroll
        for (int u = 0; u < JPT; ++u) {
            const int j = tid + u * RB_THREADS;
            if (j >= n) break;
            const int x = jx[j];
            if (x < 0) continue;
            const int64_t cx = c[x];
            if (cx <= 0) continue;
            const int64_t d = (int64_t)jl[j] + rho;
            const int64_t g = (abs64(cx) - abs64(cx - d)) + (abs64(cm) - abs64(cm + d));
            if (g > bg) {
                bg = g;
                bj = j;
            }
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
            const int64_t og = __shfl_xor(bg, off, 64);
            const int32_t oj = __shfl_xor(bj, off, 64);
            if (rb_better(og, oj, bg, bj)) {
                bg = og;
                bj = oj;
            }
        }
        if (lane == 0) {
            wg[wv] = bg;
            wo[wv] = bj;
        }
        __syncthreads();
        // every wave finds the block's best from the per-wave ones
        int64_t g = lane < NWAVE ? wg[lane] : 0;
        int32_t jb = lane < NWAVE ? wo[lane] : INT32_MAX;
#pragma unroll
        for (int off = NWAVE / 2; off > 0; off >>= 1) {
            const int64_t og = __shfl_xor(g, off, 64);
            const int32_t oj = __shfl_xor(jb, off, 64);
            if (rb_better(og, oj, g, jb)) {
                g = og;
                jb = oj;
            }
        }
        g = rdlane64s(g, 0);
        jb = rdlane(jb, 0);
        if (g <= 0) break;  // uniform
        if (wv == 0) {
            const int64_t l = jl[jb];
            const int64_t T = -(l + rho);
            int32_t y = ci;
            if (cm <= T) {  // the lowest-index receiver at or below -d
                int32_t lo = INT32_MAX;
                for (int k = lane; k < nneg; k += 64) {
                    const int32_t w = neg[k];
                    if (negc[k] <= T && w < lo) lo = w;
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
                const int64_t cx = c[x] - (l + rho), cy = c[y] + (l + rho);
                c[x] = cx;
                c[y] = cy;
                if (cx < 0) {  // x (c_x was > 0) joins the receivers
                    pos[x] = (int16_t)s_nneg;
                    neg[s_nneg] = (int16_t)x;
                    negc[s_nneg] = cx;
                    s_nneg += 1;
                }
                const int at = pos[y];  // y (c_y was < 0) is listed
                if (cy < 0) {
                    negc[at] = cy;
                } else {  // y leaves: the last entry takes its place
                    const int last = s_nneg - 1, wl = neg[last];
                    neg[at] = (int16_t)wl;
                    negc[at] = negc[last];
                    pos[wl] = (int16_t)at;
                    pos[y] = -1;
                    s_nneg = last;
                }
                jx[jb] = (int16_t)(-2 - x);
                jy[jb] = (int16_t)y;
                a.new_worker[pr.new0 + jb] = y;
                if (a.log != nullptr) {
                    a.log[2 * (pr.new0 + moves)] = jb;
                    a.log[2 * (pr.new0 + moves) + 1] = y;
                }
            }
        }
        obj -= g;
        moves += 1;
        __syncthreads();  // the move is applied before the next step reads the lists
    }
    // the moved requests' share of the errors
    for (int j = tid; j < n; j += RB_THREADS) {
        const int v = jx[j];
        if (v > -2) continue;
        const int x = -2 - v, y = jy[j];
        const int64_t l = jl[j];
        atomicAdd((unsigned long long*)&a.le[pr.wbase + x], (unsigned long long)-l);
        atomicAdd((unsigned long long*)&a.be[pr.wbase + x], (unsigned long long)(int64_t)-1);
        atomicAdd((unsigned long long*)&a.le[pr.wbase + y], (unsigned long long)l);
        atomicAdd((unsigned long long*)&a.be[pr.wbase + y], 1ull);
    }
    if (tid == 0) {
        if (a.moves != nullptr) a.moves[p] = moves;
        if (a.obj != nullptr) {
            a.obj[2 * p] = obj0;
            a.obj[2 * p + 1] = obj;
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
