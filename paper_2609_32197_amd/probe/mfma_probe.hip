// Measurement helper for the benchmark, not a step of the method and not
// part of libsparsp or its C ABI: the sustained rate of the
// bf16 matrix cores with every operand in registers (no memory traffic, no
// softmax), the practical ceiling the attention kernel is compared with
// beside the data-sheet peak. Each wave runs four independent accumulation
// chains of v_mfma_f32_32x32x16_bf16 over per-lane pseudo-random operands in
// [-1, 1) (random bits switch more of the datapath than constants, and the
// clock under the power limit depends on it). The sums are written out so
// that no MFMA can be dropped.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __bf16 bf16x8_p __attribute__((ext_vector_type(8)));
typedef float floatx16_p __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float lcg_unit(uint32_t& x) {
    x = x * 1664525u + 1013904223u;
    return float(int((x >> 8) & 0xffffu) - 32768) * (1.0f / 32768.0f);
}

__global__ __launch_bounds__(256) void mfma_probe_kernel(int64_t iters, float* __restrict__ sink) {
    const uint32_t t = blockIdx.x * 256u + threadIdx.x;
    uint32_t x = t * 2654435761u + 12345u;
    bf16x8_p a, b;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        a[e] = (__bf16)lcg_unit(x);
        b[e] = (__bf16)lcg_unit(x);
    }
    floatx16_p c0 = {}, c1 = {}, c2 = {}, c3 = {};
    for (int64_t i = 0; i < iters; ++i) {
        c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c0, 0, 0, 0);
        c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, a, c1, 0, 0, 0);
        c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, a, c2, 0, 0, 0);
        c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, b, c3, 0, 0, 0);
    }
    float s = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) s += c0[r] + c1[r] + c2[r] + c3[r];
    sink[t] = s;
}

}  // namespace

// Runs `workgroups` workgroups of 256 threads, each wave issuing 4 * iters
// bf16 32x32x16 matrix-core operations on register operands, i.e.
// workgroups * iters * 524,288 FLOP, on `stream` (a hipStream_t), and writes
// one float per thread to sink (device, workgroups * 256 floats; the values
// are meaningless). Returns 0, -1 for iters < 1, workgroups outside
// [1, 2^20] or a NULL sink (nothing launched), or -5 for a launch error.
extern "C" int mfma_probe_run(int64_t iters, int32_t workgroups, float* sink, void* stream) {
    if (iters < 1 || workgroups < 1 || workgroups > (1 << 20) || !sink) return -1;
    (void)hipGetLastError();
    mfma_probe_kernel<<<workgroups, 256, 0, (hipStream_t)stream>>>(iters, sink);
    return hipGetLastError() == hipSuccess ? 0 : -5;
}
