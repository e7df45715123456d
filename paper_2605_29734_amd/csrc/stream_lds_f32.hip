// Bank-streaming kernel, LDS-staged queries, fp32 key storage rounded to bf16
// for the MFMA (see stream.hpp).
#include "stream.hpp"

namespace htam {
hipError_t launch_stream_lds_f32(int npl, bool two_per_cu, const StreamLaunch &l) {
    return launch_stream_lds_t<float>(npl, two_per_cu, l);
}
}  // namespace htam
