// Moves of requests placed in the current heartbeat window between loaded
// workers: one wave per affected worker stages the worker's sorted request
// columns in LDS, takes out the requests it gives up (each must be there: its
// end e = l_pred + tau and start s = l_in - tau, with the prefill sums of the
// current window holding it), inserts the ones it takes in end order, and
// writes the columns back; the prefill sums and, with constraint (d), the
// request log follow.  The worker's summaries are then stale (rebuilt by the
// next call's build).  A check launch runs first, so a move that cannot be
// applied changes nothing.
#include "ald_device.h"
#include "ald_move.h"

namespace ald {

constexpr int MOVE_THREADS = 64;

__global__ __launch_bounds__(MOVE_THREADS) void k_move(State st, MoveArgs a)
{
    __shared__ int32_t E[HOT];
    __shared__ int32_t S[HOT];
    if (a.apply && *a.err != 0) return;
    const MoveWorker mw = a.mw[blockIdx.x];
    const int gw = mw.gw, lane = threadIdx.x;
    const int s = find_scen_by_worker(st, gw);
    const Scen sc = st.scen[s];
    const int64_t base = st.slot_base[gw];
    const int head = st.head[gw], n = st.n[gw], cap = st.cap[gw];
    int B = n - head;
    const int nrm = mw.rm1 - mw.rm0, nin = mw.in1 - mw.in0;
    // the window's prefill sums must hold every request given up
    int64_t rs1 = 0, rs2 = 0;
    for (int k = mw.rm0; k < mw.rm1; ++k) {
        rs1 += a.lin[k];
        rs2 += (int64_t)a.lin[k] * a.lin[k];
    }
    const bool cur = st.hbs[gw] == a.hb;
    bool bad = nrm > 0 && (!cur || st.S1[gw] < rs1 || st.S2[gw] < rs2);
    bad = bad || B - nrm + nin > cap || B > HOT;
    if (sc.use_d) bad = bad || st.lgn[gw] - nrm + nin > cap;
    if (bad) {
        if (lane == 0) raise_error(a.err, nrm > 0 && B - nrm + nin <= cap ? DEV_EINVAL : DEV_ESLOTS);
        return;
    }
    for (int k = lane; k < B; k += MOVE_THREADS) {
        E[k] = st.e[base + head + k];
        S[k] = st.s[base + head + k];
    }
    __syncthreads();
    // removals: the first matching entry, then the tail moves down one place
    for (int r = mw.rm0; r < mw.rm1; ++r) {
        const int32_t e = a.lpred[r] + a.tau, sv = a.lin[r] - a.tau;
        int at = -1;
        for (int k0 = 0; k0 < B && at < 0; k0 += MOVE_THREADS) {
            const int k = k0 + lane;
            const uint64_t m = ballot(k < B && E[k] == e && S[k] == sv);
            if (m) at = k0 + __ffsll((unsigned long long)m) - 1;
        }
        if (at < 0) {  // not on this worker
            if (lane == 0) raise_error(a.err, DEV_EINVAL);
            return;
        }
        for (int k0 = at; k0 < B - 1; k0 += MOVE_THREADS) {
            const int k = k0 + lane;
            const int32_t ne = k < B - 1 ? E[k + 1] : 0, ns = k < B - 1 ? S[k + 1] : 0;
            __syncthreads();
            if (k < B - 1) {
                E[k] = ne;
                S[k] = ns;
            }
            __syncthreads();
        }
        B -= 1;
    }
    // insertions: after every entry with an end at or before the new one
    for (int r = mw.in0; r < mw.in1; ++r) {
        const int32_t e = a.lpred[r] + a.tau, sv = a.lin[r] - a.tau;
        int cnt = 0;  // entries with E <= e (the columns are sorted by end)
        for (int k0 = 0; k0 < B; k0 += MOVE_THREADS) cnt += __popcll(ballot(k0 + lane < B && E[k0 + lane] <= e));
        for (int k0 = B - 1 - ((B - 1 - cnt) % MOVE_THREADS + MOVE_THREADS) % MOVE_THREADS; k0 >= cnt;
             k0 -= MOVE_THREADS) {
            const int k = k0 + lane;  // lanes shift entries k -> k + 1, from the top chunk down
            const bool in = k >= cnt && k < B;
            const int32_t oe = in ? E[k] : 0, os = in ? S[k] : 0;
            __syncthreads();
            if (in) {
                E[k + 1] = oe;
                S[k + 1] = os;
            }
            __syncthreads();
        }
        if (lane == 0) {
            E[cnt] = e;
            S[cnt] = sv;
        }
        __syncthreads();
        B += 1;
    }
    if (!a.apply) return;
    const int nh = head + B <= cap ? head : 0;
    for (int k = lane; k < B; k += MOVE_THREADS) {
        st.e[base + nh + k] = E[k];
        st.s[base + nh + k] = S[k];
    }
    if (lane == 0) {
        st.head[gw] = nh;
        st.n[gw] = nh + B;
        int64_t s1 = cur ? st.S1[gw] : 0, s2 = cur ? st.S2[gw] : 0;
        s1 -= rs1;
        s2 -= rs2;
        for (int r = mw.in0; r < mw.in1; ++r) {
            s1 += a.lin[r];
            s2 += (int64_t)a.lin[r] * a.lin[r];
        }
        st.S1[gw] = s1;
        st.S2[gw] = s2;
        if (nin > 0) st.hbs[gw] = a.hb;
        if (sc.use_d) {
            // the log is unordered: a request given up leaves with its entry of
            // this window, a request taken starts at this worker's slack origin
            int32_t* lge = st.lge + base;
            int32_t* lgw = st.lgw + base;
            double* lgs = st.lgs + base;
            int L = st.lgn[gw];
            for (int r = mw.rm0; r < mw.rm1; ++r) {
                const int32_t e = a.lpred[r] + a.tau;
                for (int k = 0; k < L; ++k)
                    if (lge[k] == e && lgw[k] == a.hb) {
                        lge[k] = lge[L - 1];
                        lgw[k] = lgw[L - 1];
                        lgs[k] = lgs[L - 1];
                        L -= 1;
                        break;
                    }
            }
            for (int r = mw.in0; r < mw.in1; ++r) {
                lge[L] = a.lpred[r] + a.tau;
                lgw[L] = a.hb;
                lgs[L] = -st.phi[gw];
                L += 1;
            }
            st.lgn[gw] = L;
        }
        st.built[gw] = 0;
    }
}

hipError_t launch_move(const State& st, const MoveArgs& a, hipStream_t stream)
{
    if (a.nw == 0) return hipSuccess;
    hipLaunchKernelGGL(k_move, dim3(a.nw), dim3(MOVE_THREADS), 0, stream, st, a);
    return hipGetLastError();
}

}  // namespace ald
