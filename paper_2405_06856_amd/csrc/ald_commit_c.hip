// Commit launches that keep the untouched-worker scan's rows and keys in LDS.
#include "ald_commit.h"

namespace ald {

hipError_t launch_commit_c(const State& st, int32_t blocks, hipStream_t stream)
{
    const dim3 g(blocks), b(COMMIT_THREADS);
    if (st.out_diag != nullptr) hipLaunchKernelGGL((k_commit<true, false, true>), g, b, 0, stream, st);
    else hipLaunchKernelGGL((k_commit<false, false, true>), g, b, 0, stream, st);
    return hipGetLastError();
}

}  // namespace ald
