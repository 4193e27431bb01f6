// Commit launches that check constraint (d) against the residents' decode history.
#include "ald_commit.h"

namespace ald {

hipError_t launch_commit_d(const State& st, int32_t blocks, bool cache, hipStream_t stream)
{
    if (cache) return launch_commit_dc(st, blocks, stream);
    const dim3 g(blocks), b(COMMIT_THREADS);
    if (st.out_diag != nullptr) hipLaunchKernelGGL((k_commit<true, true, false>), g, b, 0, stream, st);
    else hipLaunchKernelGGL((k_commit<false, true, false>), g, b, 0, stream, st);
    return hipGetLastError();
}

}  // namespace ald
