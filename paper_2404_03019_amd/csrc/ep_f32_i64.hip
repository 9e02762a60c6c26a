// Element-parallel kernels for f32 storage with i64 segment ids, and the fp32 partial levels every storage type ends in
#include "common.h"
#include "ep_kernel.h"

namespace geot {

hipError_t launch_ep_f32_i64(const EpArgs &a, int red, int mode, int V, int NT, int L, int64_t nchunks,
                           hipStream_t stream) {
    return ep_dispatch<ELEM_F32, int64_t, true>(a, red, mode, V, NT, L, nchunks, stream);
}

hipError_t launch_ep(const EpArgs &a, int red, int mode, int V, int NT, int L, int64_t nchunks,
                     hipStream_t stream) {
    if (mode == SRC_PIECES) return launch_ep_f32_i64(a, red, mode, V, NT, L, nchunks, stream);
    const bool i32 = a.idx32 != 0;
    switch (a.elem) {
        case ELEM_F32:
            return i32 ? launch_ep_f32_i32(a, red, mode, V, NT, L, nchunks, stream)
                       : launch_ep_f32_i64(a, red, mode, V, NT, L, nchunks, stream);
        case ELEM_BF16:
            return i32 ? launch_ep_bf16_i32(a, red, mode, V, NT, L, nchunks, stream)
                       : launch_ep_bf16_i64(a, red, mode, V, NT, L, nchunks, stream);
        case ELEM_F16:
            return i32 ? launch_ep_f16_i32(a, red, mode, V, NT, L, nchunks, stream)
                       : launch_ep_f16_i64(a, red, mode, V, NT, L, nchunks, stream);
        default:
            return hipErrorInvalidValue;
    }
}

}  // namespace geot
