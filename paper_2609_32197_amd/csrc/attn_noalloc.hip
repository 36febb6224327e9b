// Attention with the last round balanced, for callers that cannot allocate
// (code under HIP graph capture, serving loops, harnesses that forbid
// hipMalloc): the float32 partials of the split last-round rows go to a fixed
// device array instead of a caller workspace.
//
// `scratch` is a file-scope device array of kScratchBytes, one copy per GPU
// the library runs on, held until the process ends. Its device address is
// looked up once per device, with that device current, on the first call
// there (hipGetSymbolAddress), and kept; host code passes that address to the
// kernels, never the array's name. Every call on a GPU shares its array and
// leaves its own partials there: nothing in it needs to start at zero (each
// partial the merge reads is written by the same call), but calls that overlap
// on one GPU race for it.
#include <mutex>

#include "sparsp_internal.h"

namespace sparsp {
namespace {

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's address of `scratch`, looked up on first use.
hipError_t scratch_address(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace

hipError_t launch_attn_bf16_noalloc(const Geom& g, const void* Q, const int32_t* sel, int keep,
                                    const int32_t* slot_of, const void* Kp, const void* Vp,
                                    int64_t capacity, float scale, void* O, bool out_bf16,
                                    float* lse, hipStream_t s) {
    void* ws = nullptr;
    if (hipError_t e = scratch_address(&ws); e != hipSuccess) return e;
    AttnPart whole{0, g.n, 0, g.H, 0};
    whole.ws = ws;
    whole.ws_bytes = kScratchBytes;
    return launch_attn_bf16(g, Q, sel, keep, slot_of, Kp, Vp, capacity, scale, whole, O, out_bf16,
                            lse, s);
}

}  // namespace sparsp
