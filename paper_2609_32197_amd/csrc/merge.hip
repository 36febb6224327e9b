// Online-softmax merge of partial attention results (Section 2.3: a rank folds
// the attention over each arriving KV shard into its running result).
//
// A part computed over a key set X carries O_X (the softmax-weighted mean of V
// over X) and lse_X = log sum_{t in X} exp(s_t). Two parts over disjoint key
// sets combine into the result over their union:
//   m   = max(lse_A, lse_B)
//   w_X = exp(lse_X - m)                  (0 when lse_X = -inf)
//   O   = (w_A O_A + w_B O_B) / (w_A + w_B)
//   lse = m + log(w_A + w_B)
// and a row that is empty on both sides stays O = 0, lse = -inf.
//
// Layout: O is float32 [H, nq*block, d], lse float32 [H, nq*block]; the
// accumulator is updated in place for the heads [h_lo, h_hi). Each row's d
// values are handled by d/4 consecutive lanes of one wave (float4 each), so
// the row's lse is read and rewritten inside a single wave: every lane reads
// it before the one lane that writes it. The kernel is HBM-bound: per row it
// reads 8d + 8 bytes and writes 4d + 4.
#include "sparsp_internal.h"

namespace sparsp {
namespace {

__global__ __launch_bounds__(256) void lse_merge_kernel(float* __restrict__ O_acc,
                                                        float* __restrict__ lse_acc,
                                                        const float* __restrict__ O_part,
                                                        const float* __restrict__ lse_part,
                                                        int64_t row0, int64_t rows, int d) {
    const int lane = threadIdx.x & 63;
    const int c4n = d / 4;                      // float4 per row
    const int rows_per_wave = 64 / c4n;         // >= 1 because d <= 256
    const int rw = lane / c4n, c4 = lane % c4n;
    if (rw >= rows_per_wave) return;            // lanes past the last whole row idle
    const int64_t wave = (int64_t(blockIdx.x) * blockDim.x + threadIdx.x) >> 6;
    const int64_t waves = (int64_t(gridDim.x) * blockDim.x) >> 6;
    for (int64_t r = wave * rows_per_wave + rw; r < rows; r += waves * rows_per_wave) {
        const int64_t row = row0 + r;
        const float la = lse_acc[row], lb = lse_part[row];
        const float m = fmaxf(la, lb);
        float4* oa = reinterpret_cast<float4*>(O_acc + row * d) + c4;
        const float4 xb = reinterpret_cast<const float4*>(O_part + row * d)[c4];
        if (m == -INFINITY) {  // both sides empty
            *oa = make_float4(0.f, 0.f, 0.f, 0.f);
            if (c4 == 0) lse_acc[row] = -INFINITY;
            continue;
        }
        const float wa = la == -INFINITY ? 0.f : __expf(la - m);
        const float wb = lb == -INFINITY ? 0.f : __expf(lb - m);
        const float tot = wa + wb;
        const float fa = wa / tot, fb = wb / tot;
        const float4 xa = *oa;
        *oa = make_float4(fa * xa.x + fb * xb.x, fa * xa.y + fb * xb.y, fa * xa.z + fb * xb.z,
                          fa * xa.w + fb * xb.w);
        if (c4 == 0) lse_acc[row] = m + __logf(tot);
    }
}

// rows x d floats of O set to 0 and rows entries of lse to -inf: the result
// over an empty key set, which the merge leaves to the other side.
__global__ __launch_bounds__(256) void fill_identity_kernel(float* __restrict__ O,
                                                            float* __restrict__ lse, int64_t rows,
                                                            int d) {
    const int64_t stride = int64_t(gridDim.x) * blockDim.x;
    const int64_t start = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    for (int64_t i = start; i < rows * d; i += stride) O[i] = 0.f;
    for (int64_t i = start; i < rows; i += stride) lse[i] = -INFINITY;
}

}  // namespace

hipError_t launch_fill_identity(float* O, float* lse, int64_t rows, int d, hipStream_t s) {
    (void)hipGetLastError();
    const int64_t need = (rows * d + 255) / 256;
    const int grid = int(need < 2048 ? (need > 0 ? need : 1) : 2048);
    fill_identity_kernel<<<grid, 256, 0, s>>>(O, lse, rows, d);
    return hipGetLastError();
}

hipError_t launch_lse_merge(const Geom& g, int h_lo, int h_hi, float* O_acc, float* lse_acc,
                            const float* O_part, const float* lse_part, hipStream_t s) {
    (void)hipGetLastError();
    const int64_t per_head = int64_t(g.nq) * g.block;
    const int64_t row0 = int64_t(h_lo) * per_head;
    const int64_t rows = int64_t(h_hi - h_lo) * per_head;
    const int rows_per_wave = 64 / (g.d / 4);
    const int64_t waves_needed = (rows + rows_per_wave - 1) / rows_per_wave;
    const int64_t blocks = (waves_needed + 3) / 4;  // 4 waves per workgroup
    const int grid = int(blocks < 4096 ? (blocks > 0 ? blocks : 1) : 4096);
    lse_merge_kernel<<<grid, 256, 0, s>>>(O_acc, lse_acc, O_part, lse_part, row0, rows, g.d);
    return hipGetLastError();
}

}  // namespace sparsp
