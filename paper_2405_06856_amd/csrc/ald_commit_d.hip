// Commit launches that check constraint (d) against the residents' decode history.
#include "ald_commit.h"

namespace ald {

hipError_t launch_commit_d(const State& st, int32_t blocks, hipStream_t stream)
{
    const dim3 g(blocks), b(COMMIT_THREADS);
    if (st.out_diag != nullptr) hipLaunchKernelGGL((k_commit<true, true>), g, b, 0, stream, st);
    else hipLaunchKernelGGL((k_commit<false, true>), g, b, 0, stream, st);
    return hipGetLastError();
}

}  // namespace ald
