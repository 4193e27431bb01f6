// Commit launches without decode history (and the dispatch to those with it).
#include "ald_commit.h"

namespace ald {

hipError_t launch_commit(const State& st, int32_t blocks, bool use_d, hipStream_t stream)
{
    if (use_d) return launch_commit_d(st, blocks, stream);
    const dim3 g(blocks), b(COMMIT_THREADS);
    if (st.out_diag != nullptr) hipLaunchKernelGGL((k_commit<true, false>), g, b, 0, stream, st);
    else hipLaunchKernelGGL((k_commit<false, false>), g, b, 0, stream, st);
    return hipGetLastError();
}

}  // namespace ald
