// Stand-ins for the device side of libsparsp, for the host-only sanitizer
// build of the C ABI layer (api.cpp) and the host planning code
// (host_plan.cpp). Every launcher records that it was called and returns
// success without touching the pointers it gets, so the ABI layer's argument
// checks and host loops run under AddressSanitizer and
// UndefinedBehaviorSanitizer with no GPU and no HIP runtime. hipGetLastError
// and hipGetErrorString, the only runtime calls of api.cpp, are defined here
// too (the build links no HIP library).
#include <cstdint>

#include "../../paper_2609_32197_amd/csrc/sparsp_launch.h"

int g_launches = 0;  // launcher calls since the driver last reset it

extern "C" hipError_t hipGetLastError(void) { return hipSuccess; }
extern "C" const char* hipGetErrorString(hipError_t) { return "stub"; }

namespace sparsp {

static hipError_t launched() {
    ++g_launches;
    return hipSuccess;
}

hipError_t launch_pool_scores(const Geom&, const void*, const void*, float*, float*, float*,
                              hipStream_t) { return launched(); }
hipError_t launch_topk(const Geom&, const float*, int, const GlobalSet&, uint64_t*, int32_t*,
                       hipStream_t) { return launched(); }
hipError_t launch_cdf(const Geom&, const float*, float, const GlobalSet&, uint64_t*, int32_t*,
                      int32_t*, hipStream_t) { return launched(); }
hipError_t launch_demand_gather(const Geom&, const uint64_t*, const void*, const void*,
                                uint64_t*, int32_t*, int32_t*, int32_t*, void*, void*,
                                hipStream_t) { return launched(); }
hipError_t launch_gather(const Geom&, int, const int32_t*, const int32_t*, const void*,
                         const void*, void*, void*, hipStream_t) { return launched(); }
hipError_t launch_pack_for_consumers(const Geom&, const uint64_t*, int, int, int, int,
                                     const void*, const void*, uint64_t*, int32_t*, int32_t*,
                                     int32_t*, void*, void*, hipStream_t) { return launched(); }
hipError_t launch_attn_bf16(const Geom&, const void*, const int32_t*, int, const int32_t*,
                            const void*, const void*, int64_t, float, const AttnPart&, void*,
                            bool, float*, hipStream_t) { return launched(); }
int64_t attn_tail_workspace_bytes(const Geom& g, int) {
    return int64_t(512) * g.block * (g.d + 1) * 4;  // 512 resident slots
}
hipError_t launch_attn_bf16_noalloc(const Geom&, const void*, const int32_t*, int, const int32_t*,
                                    const void*, const void*, int64_t, float, void*, bool, float*,
                                    hipStream_t) { return launched(); }
hipError_t launch_attn_f32(const Geom&, const float*, const int32_t*, int, const int32_t*,
                           const float*, const float*, int64_t, float, const AttnPart&, float*,
                           float*, hipStream_t) { return launched(); }
hipError_t launch_lse_merge(const Geom&, int, int, float*, float*, const float*, const float*,
                            hipStream_t) { return launched(); }
hipError_t launch_fill_identity(float*, float*, int64_t, int, hipStream_t) { return launched(); }
hipError_t launch_permute(const Geom&, const int32_t*, const void*, void*, bool, hipStream_t) {
    return launched();
}
hipError_t run_chunks(const Geom&, const void*, const int32_t*, int, const int32_t*, const void*,
                      const void*, int64_t, float, const sparsp_chunk*, int, float*, float*,
                      hipStream_t) { return launched(); }
hipError_t launch_row_order(const int32_t*, int, int, int, int32_t*, hipStream_t) {
    return launched();
}

}  // namespace sparsp
