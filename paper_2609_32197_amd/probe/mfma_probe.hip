// Measurement helpers for the benchmark, not steps of the method and not
// part of libsparsp or its C ABI.
//
// mfma_probe_run: the sustained rate of the
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

namespace {

// unit_probe_run kinds: the issue rates the attention kernel's softmax and
// operand reads depend on, measured on their own.
//   0: v_exp_f32, sixteen independent chains per lane;
//   1: v_fma_f32, sixteen independent chains per lane;
//   2: ds_read_b128 from a 32 KB bf16 tile in the attention kernel's K-operand
//      pattern (lane l reads row 32 mt + sigma(l % 32), 16-byte chunk
//      (2 kt + l / 32) xor (row % 16)), 32 reads per iteration.
__global__ __launch_bounds__(256) void exp_probe_kernel(int64_t iters, float* __restrict__ sink) {
    float x[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) x[i] = -0.001f * float(threadIdx.x + i);
    for (int64_t it = 0; it < iters; ++it)
#pragma unroll
        for (int i = 0; i < 16; ++i) x[i] = __builtin_amdgcn_exp2f(x[i]) - 1.0f;
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) s += x[i];
    sink[blockIdx.x * 256u + threadIdx.x] = s;
}

__global__ __launch_bounds__(256) void fma_probe_kernel(int64_t iters, float* __restrict__ sink) {
    float x[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) x[i] = 0.001f * float(threadIdx.x + i);
    for (int64_t it = 0; it < iters; ++it)
#pragma unroll
        for (int i = 0; i < 16; ++i) x[i] = fmaf(x[i], 0.999f, 0.0001f);
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) s += x[i];
    sink[blockIdx.x * 256u + threadIdx.x] = s;
}

__device__ __forceinline__ int sigma_p(int m) { return (m & ~0xC) | ((m & 4) << 1) | ((m & 8) >> 1); }

typedef float floatx4_p __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void lds_probe_kernel(int64_t iters, float* __restrict__ sink) {
    __shared__ __attribute__((aligned(16))) uint16_t t[128 * 128];
    const int tid = threadIdx.x, lane = tid & 63, qi = lane & 31, g = lane >> 5;
    for (int i = tid; i < 128 * 128; i += 256) t[i] = uint16_t(i);
    __syncthreads();
    floatx4_p acc = {};
    for (int64_t it = 0; it < iters; ++it) {
        const int shift = int(it & 7) * 8 * 128;  // a different set of rows each iteration
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int kt = 0; kt < 8; ++kt) {
                const int row = 32 * mt + sigma_p(qi);
                const int off = (row * 128 + (((2 * kt + g) ^ (row & 15)) * 8) + shift) & (128 * 128 - 8);
                acc += *reinterpret_cast<const floatx4_p*>(&t[off]);
            }
    }
    sink[blockIdx.x * 256u + tid] = acc[0] + acc[1] + acc[2] + acc[3];
}

}  // namespace

// Runs one of the unit probes above: `workgroups` workgroups of 256 threads,
// `iters` iterations each, on `stream`; sink as for mfma_probe_run. Per
// iteration a wave issues 16 v_exp_f32 (kind 0), 16 v_fma_f32 (kind 1) or 32
// ds_read_b128 (kind 2, 32 KB of LDS per workgroup). Returns 0, -1 for a bad
// kind, iters < 1, workgroups outside [1, 2^20] or a NULL sink (nothing
// launched), or -5 for a launch error.
extern "C" int unit_probe_run(int32_t kind, int64_t iters, int32_t workgroups, float* sink,
                              void* stream) {
    if (kind < 0 || kind > 2 || iters < 1 || workgroups < 1 || workgroups > (1 << 20) || !sink)
        return -1;
    (void)hipGetLastError();
    hipStream_t s = (hipStream_t)stream;
    if (kind == 0) exp_probe_kernel<<<workgroups, 256, 0, s>>>(iters, sink);
    else if (kind == 1) fma_probe_kernel<<<workgroups, 256, 0, s>>>(iters, sink);
    else lds_probe_kernel<<<workgroups, 256, 0, s>>>(iters, sink);
    return hipGetLastError() == hipSuccess ? 0 : -5;
}
