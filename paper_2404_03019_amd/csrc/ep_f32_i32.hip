// Element-parallel kernels for f32 storage with i32 segment ids
#include "common.h"
#include "ep_kernel.h"

namespace geot {

hipError_t launch_ep_f32_i32(const EpArgs &a, int red, int mode, int V, int NT, int L, int64_t nchunks,
                           hipStream_t stream) {
    return ep_dispatch<ELEM_F32, int32_t, false>(a, red, mode, V, NT, L, nchunks, stream);
}

}  // namespace geot
