// Algorithm 2 (re-balancing a heartbeat's new requests against the output-length
// prediction errors of the ongoing ones): limits, tables and launch.
#pragma once

#include "ald_internal.h"

namespace ald {

constexpr int RB_WMAX = 4096;     // workers per problem (the error accumulators live in LDS)
constexpr int RB_JMAX = 8192;     // new requests per problem
constexpr int RB_ETHREADS = 256;  // threads per error-accumulation block
constexpr int RB_CHUNK = 1024;    // ongoing requests per error-accumulation block
constexpr int32_t RB_LEN_MAX = 1 << 24;
constexpr int RB_WAVES = 4;       // waves per problem in the moves kernel

// rho = c2 / k2 of one problem, held so that the sign of a + rho * b (integer
// a, b) is exact: k2 = mk * 2^ek and c2 = mc * 2^ec with 53-bit integer
// significands (mc = 0 when c2 = 0), sh = ek - ec; rho_d = fl(c2 / k2) for
// the fp64 stand-ins; R the integer nearest rho, fs the exact sign of rho - R
// and f_up >= |rho - R| (so that a + R b = 0 decides the sign of a + rho b as
// fs * sign(b), and a small |b| f_up lets a + R b decide it alone).
struct RbRho {
    double k2, c2, rho_d, f_up;
    uint64_t mk, mc;
    int64_t R;
    int32_t sh, fs;
};

struct RbProblem {
    int64_t old0, old1;  // its ongoing requests [old0, old1)
    int64_t new0;        // its first new request
    int64_t wbase;       // its first worker in the error arrays
    RbRho rho;
    int32_t W, n_new;
};
struct RbChunk {
    int64_t begin, end;  // ongoing requests of one problem
    int32_t p, pad;
};
struct RbArgs {
    const RbProblem* prob;
    const RbChunk* chunk;
    int32_t nchunk, P;
    const int32_t* old_worker;
    const int32_t* old_lpred;
    const int32_t* old_lout;
    const int32_t* old_lreal;
    const int32_t* old_lrepred;
    const int32_t* new_lpred;
    int32_t* new_worker;  // in/out
    int64_t* le;          // per worker, zero before the launch; final errors after
    int64_t* be;
    int32_t* moves;       // per problem (nullable)
    int32_t* log;         // problem p's first log_cap (request, target) pairs at 2 * p * log_cap (nullable)
    int32_t log_cap;
    int64_t* obj;         // per problem: sum |c| before and after as pairs (a, b) = a + rho * b (nullable)
    int32_t* err;
    int32_t wmax, jmax;   // the largest W and n_new over the problems (size the moves kernel's LDS)
};
// error accumulation (nchunk + P blocks), then the greedy moves (P blocks of RB_WAVES waves)
hipError_t launch_rebalance(const RbArgs& a, hipStream_t stream);
// LDS bytes of the moves kernel for problems of at most wmax workers and jmax new requests
size_t rb_moves_lds(int32_t wmax, int32_t jmax);

// Fixed device array of the allocation-free entry point: the problem and chunk
// tables of at most RB_STATIC_P problems and RB_STATIC_CHUNKS chunks, then the
// error word.  One copy per device, held until the process ends.
constexpr int RB_STATIC_P = 4096;
constexpr int RB_STATIC_CHUNKS = 32768;
constexpr size_t RB_STATIC_TABLES = ((RB_STATIC_P * sizeof(RbProblem) + 255) & ~(size_t)255) +
                                    ((RB_STATIC_CHUNKS * sizeof(RbChunk) + 255) & ~(size_t)255);
constexpr size_t RB_STATIC_BYTES = RB_STATIC_TABLES + 256;
// Look up (once per device, with `device` current) the device address of that
// array; later calls return the cached address.  Host code uses only this
// address, never the array's own name.
hipError_t rb_static_init(int device);
void* rb_static_ptr(int device);  // null until rb_static_init succeeded for `device`

}  // namespace ald
