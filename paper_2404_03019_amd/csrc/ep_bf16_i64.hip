// Element-parallel kernels for bf16 storage with i64 segment ids
#include "common.h"
#include "ep_kernel.h"

namespace geot {

hipError_t launch_ep_bf16_i64(const EpArgs &a, int red, int mode, int V, int NT, int L, int64_t nchunks,
                           hipStream_t stream) {
    return ep_dispatch<ELEM_BF16, int64_t, false>(a, red, mode, V, NT, L, nchunks, stream);
}

}  // namespace geot
