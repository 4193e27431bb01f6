// Moves of requests placed in the current heartbeat window between loaded
// workers (applying Algorithm 2's re-balancing to the placement): tables and
// launch.
#pragma once

#include "ald_internal.h"

namespace ald {

// One worker's share of a batch of moves: requests it gives up and takes.
struct MoveWorker {
    int32_t gw;             // global worker index
    int32_t rm0, rm1;       // its removals [rm0, rm1) in the request arrays
    int32_t in0, in1;       // its insertions [in0, in1)
    int32_t pad;
};

struct MoveArgs {
    const MoveWorker* mw;
    int32_t nw;            // affected workers
    int32_t tau, hb;       // the current decode iteration and heartbeat window
    const int32_t* lin;    // [removals then insertions, grouped by worker]
    const int32_t* lpred;
    int32_t* err;
    int32_t apply;         // 0: check only, 1: apply (after a clean check)
};

hipError_t launch_move(const State& st, const MoveArgs& a, hipStream_t stream);

}  // namespace ald
