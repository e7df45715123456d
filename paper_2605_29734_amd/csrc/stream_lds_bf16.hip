// Bank-streaming kernel, LDS-staged queries, bf16 key storage (see stream.hpp).
#include "stream.hpp"

namespace htam {
hipError_t launch_stream_lds_bf16(int npl, bool two_per_cu, const StreamLaunch &l) {
    return launch_stream_lds_t<__bf16>(npl, two_per_cu, l);
}
}  // namespace htam
