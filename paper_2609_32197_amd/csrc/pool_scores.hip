// Step 1: pooled query/key tiles and block scores (Section 4.2).
//
// pool_kernel: one workgroup per (head, block) streams the block's rows from
// HBM with 16-byte non-temporal loads (every lane of a row group reads one
// 16-byte chunk, so a row group covers a whole token row: fully coalesced),
// accumulates float32 column sums in registers, reduces the row groups
// through LDS in a fixed order and divides by the block's valid token count.
// Q's local blocks and all of K's blocks go through one launch. The step is
// HBM-bound.
//
// score_kernel: per head, scores = pooled_q · pooled_k^T · d^-1/2 as a tiled
// float32 product (64x64 output tile per workgroup, 4x4 per thread, d staged
// through LDS in slices of 32). It is about 1 GFLOP at the largest workload.
#include "sparsp_internal.h"

namespace sparsp {
namespace {

constexpr int kPoolThreads = 256;

template <bool BF16>
__global__ __launch_bounds__(kPoolThreads) void pool_kernel(
    const void* __restrict__ Q, const void* __restrict__ K, float* __restrict__ pooled_q,
    float* __restrict__ pooled_k, int H, int L, int d, int block, int i0, int nq, int n) {
    // Elements per 16-byte chunk.
    constexpr int VEC = BF16 ? 8 : 4;
    __shared__ float part[kPoolThreads * VEC];

    const int h = blockIdx.y;
    int t = blockIdx.x;  // [0, nq) -> Q block i0+t ; [nq, nq+n) -> K block t-nq
    const bool is_q = t < nq;
    const int blk = is_q ? i0 + t : t - nq;
    const char* src = static_cast<const char*>(is_q ? Q : K);
    float* dst = is_q ? pooled_q + (int64_t(h) * nq + t) * d
                      : pooled_k + (int64_t(h) * n + (t - nq)) * d;

    const int tok0 = blk * block;
    const int cnt = min(block, L - tok0);
    const int chunks = d / VEC;                 // chunks per token row
    const int groups = kPoolThreads / chunks;   // row groups; >= 4 because d <= 256
    const int tid = threadIdx.x;
    const int ch = tid % chunks;
    const int rg = tid / chunks;

    float acc[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) acc[v] = 0.f;

    if (rg < groups) {
        const int64_t esize = BF16 ? 2 : 4;
        const char* base = src + ((int64_t(h) * L + tok0) * d + int64_t(ch) * VEC) * esize;
        const int64_t row_bytes = int64_t(d) * esize;
        int r = rg;
        // Four rows in flight per iteration. Non-temporal loads: Q and K are
        // read once here, and with the hint a cold read runs about a quarter
        // faster.
        for (; r + 3 * groups < cnt; r += 4 * groups) {
            uint4 x[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) x[u] = load_nt(base + int64_t(r + u * groups) * row_bytes);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const uint32_t w[4] = {x[u].x, x[u].y, x[u].z, x[u].w};
                if constexpr (BF16) {
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        acc[2 * v] += bf16_bits_to_f32(w[v] & 0xffffu);
                        acc[2 * v + 1] += bf16_bits_to_f32(w[v] >> 16);
                    }
                } else {
#pragma unroll
                    for (int v = 0; v < 4; ++v) acc[v] += __uint_as_float(w[v]);
                }
            }
        }
        for (; r < cnt; r += groups) {
            const uint4 x = load_nt(base + int64_t(r) * row_bytes);
            const uint32_t w[4] = {x.x, x.y, x.z, x.w};
            if constexpr (BF16) {
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    acc[2 * v] += bf16_bits_to_f32(w[v] & 0xffffu);
                    acc[2 * v + 1] += bf16_bits_to_f32(w[v] >> 16);
                }
            } else {
#pragma unroll
                for (int v = 0; v < 4; ++v) acc[v] += __uint_as_float(w[v]);
            }
        }
    }
    // part[rg][ch*VEC + v]; threads past the last full row group hold nothing.
    if (rg < groups) {
#pragma unroll
        for (int v = 0; v < VEC; ++v) part[rg * d + ch * VEC + v] = acc[v];
    }
    __syncthreads();
    for (int c = tid; c < d; c += kPoolThreads) {
        float s = 0.f;
        for (int q = 0; q < groups; ++q) s += part[q * d + c];
        dst[c] = s / float(cnt);
    }
}

constexpr int kTile = 64;   // output tile edge
constexpr int kSlice = 32;  // d slice staged per step

__global__ __launch_bounds__(256) void score_kernel(const float* __restrict__ pq,
                                                     const float* __restrict__ pk,
                                                     float* __restrict__ scores, int nq, int n,
                                                     int d, float scale) {
    // Tiles stored d-major so each thread reads 4 consecutive rows as a float4.
    // One float4 of padding per row spreads the transposing stores over the banks.
    __shared__ float4 As[kSlice][kTile / 4 + 1];
    __shared__ float4 Bs[kSlice][kTile / 4 + 1];
    const int h = blockIdx.z;
    const int row0 = blockIdx.y * kTile;  // query blocks
    const int col0 = blockIdx.x * kTile;  // key blocks
    const int tid = threadIdx.x;
    const int tr = tid / 16, tc = tid % 16;  // 16x16 threads, 4x4 outputs each
    const float* A = pq + int64_t(h) * nq * d;
    const float* B = pk + int64_t(h) * n * d;

    float acc[4][4] = {};
    for (int k0 = 0; k0 < d; k0 += kSlice) {
        // Load 64 rows x 32 columns of each operand: 2048 floats, 8 per thread.
        for (int e = tid; e < kTile * kSlice; e += 256) {
            const int r = e / kSlice, c = e % kSlice;
            const int ra = row0 + r, rb = col0 + r, k = k0 + c;
            const float a = (ra < nq && k < d) ? A[int64_t(ra) * d + k] : 0.f;
            const float b = (rb < n && k < d) ? B[int64_t(rb) * d + k] : 0.f;
            reinterpret_cast<float*>(&As[c][0])[r] = a;
            reinterpret_cast<float*>(&Bs[c][0])[r] = b;
        }
        __syncthreads();
#pragma unroll 8
        for (int c = 0; c < kSlice; ++c) {
            const float4 a = As[c][tr];
            const float4 b = Bs[c][tc];
            const float av[4] = {a.x, a.y, a.z, a.w};
            const float bv[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
            for (int x = 0; x < 4; ++x)
#pragma unroll
                for (int y = 0; y < 4; ++y) acc[x][y] = fmaf(av[x], bv[y], acc[x][y]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int x = 0; x < 4; ++x) {
        const int i = row0 + tr * 4 + x;
        if (i >= nq) continue;
#pragma unroll
        for (int y = 0; y < 4; ++y) {
            const int j = col0 + tc * 4 + y;
            if (j < n) scores[(int64_t(h) * nq + i) * n + j] = acc[x][y] * scale;
        }
    }
}

}  // namespace

hipError_t launch_pool_scores(const Geom& g, const void* Q, const void* K, float* pooled_q,
                              float* pooled_k, float* scores, hipStream_t s) {
    (void)hipGetLastError();
    dim3 pgrid(g.nq + g.n, g.H);
    if (g.bf16)
        pool_kernel<true><<<pgrid, kPoolThreads, 0, s>>>(Q, K, pooled_q, pooled_k, g.H, g.L, g.d,
                                                         g.block, g.i0, g.nq, g.n);
    else
        pool_kernel<false><<<pgrid, kPoolThreads, 0, s>>>(Q, K, pooled_q, pooled_k, g.H, g.L, g.d,
                                                          g.block, g.i0, g.nq, g.n);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    dim3 sgrid((g.n + kTile - 1) / kTile, (g.nq + kTile - 1) / kTile, g.H);
    const float scale = 1.0f / sqrtf(float(g.d));
    score_kernel<<<sgrid, 256, 0, s>>>(pooled_q, pooled_k, scores, g.nq, g.n, g.d, scale);
    return hipGetLastError();
}

}  // namespace sparsp
