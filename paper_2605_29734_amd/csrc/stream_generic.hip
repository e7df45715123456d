// Bank-streaming kernel with query fragments read from global memory: any d,
// and the fp32-arithmetic path (see stream.hpp).
#include "stream.hpp"

namespace htam {
hipError_t launch_stream_generic(int key_dtype, int compute_dtype, int npl, const StreamLaunch &l) {
    const int kind = compute_dtype == kF32 ? 0 : (key_dtype == kF32 ? 1 : 2);
    switch (kind * 16 + npl) {
        case 0 * 16 + 2: return launch_stream_kernel(stream_generic<float, false, 2>, l, l.fa);
        case 0 * 16 + 4: return launch_stream_kernel(stream_generic<float, false, 4>, l, l.fa);
        case 0 * 16 + 8: return launch_stream_kernel(stream_generic<float, false, 8>, l, l.fa);
        case 1 * 16 + 2: return launch_stream_kernel(stream_generic<float, true, 2>, l, l.fa);
        case 1 * 16 + 4: return launch_stream_kernel(stream_generic<float, true, 4>, l, l.fa);
        case 1 * 16 + 8: return launch_stream_kernel(stream_generic<float, true, 8>, l, l.fa);
        case 2 * 16 + 2: return launch_stream_kernel(stream_generic<__bf16, true, 2>, l, l.fa);
        case 2 * 16 + 4: return launch_stream_kernel(stream_generic<__bf16, true, 4>, l, l.fa);
        case 2 * 16 + 8: return launch_stream_kernel(stream_generic<__bf16, true, 8>, l, l.fa);
    }
    return hipErrorInvalidValue;
}
}  // namespace htam
