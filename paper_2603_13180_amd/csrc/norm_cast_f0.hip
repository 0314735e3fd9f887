// norm_cast_f0.hip -- instantiates the norm + cast kernels for output format
// MX8_B16 (one translation unit per format keeps the build parallel).
#include "norm_cast.h"

namespace mxk {

hipError_t launch_norm_cast_MX8_B16(const Args &A, int kind, int TL, int CPL, hipStream_t stream)
{
    return launch_fmt<MX8_B16>(A, kind, TL, CPL, stream);
}

} // namespace mxk
