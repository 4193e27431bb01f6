// Commit launches without decode history and without the scan's LDS copies
// (and the dispatch to the other variants).
#include "ald_commit.h"

namespace ald {

hipError_t launch_commit(const State& st, int32_t blocks, bool use_d, bool cache, hipStream_t stream)
{
    if (use_d) return launch_commit_d(st, blocks, cache, stream);
    if (cache) return launch_commit_c(st, blocks, stream);
    const dim3 g(blocks), b(COMMIT_THREADS);
    if (st.out_diag != nullptr) hipLaunchKernelGGL((k_commit<true, false, false>), g, b, 0, stream, st);
    else hipLaunchKernelGGL((k_commit<false, false, false>), g, b, 0, stream, st);
    return hipGetLastError();
}

}  // namespace ald
