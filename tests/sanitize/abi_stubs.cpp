// Kernel launchers replaced by stubs that abort: the validation driver only
// makes calls the library must reject on the host, before any launch.
#include <cstdlib>

#include "../../paper_2608_01653_amd/csrc/hatq_launch.h"

namespace hatq {
[[noreturn]] static void reached() { std::abort(); }
hipError_t launch_act_quant(const float *, int, int64_t, int, const float *, float *, int8_t *, float *, hipStream_t, int) { reached(); }
hipError_t launch_act_quant_noalloc(const float *, int, int64_t, int, int8_t *, float *, hipStream_t) { reached(); }
hipError_t launch_act_quant_affine(const float *, int, int64_t, int, float *, int8_t *, float *, int32_t *, hipStream_t) { reached(); }
hipError_t launch_range_expansion(const float *, int, int64_t, int, int, float *, int32_t *, int32_t *, hipStream_t) { reached(); }
hipError_t launch_conv(const ConvArgs &, bool, hipStream_t) { reached(); }
hipError_t launch_prepare(const PrepArgs &, hipStream_t) { reached(); }
hipError_t launch_pack(const PrepArgs &, hipStream_t) { reached(); }
hipError_t launch_tapsums(const PrepArgs &, int32_t *, hipStream_t) { reached(); }
hipError_t launch_int_params(const IntParamArgs &, hipStream_t) { reached(); }
}  // namespace hatq
