// Step 4, float32: block-sparse attention for float32 inputs (Eq. 1 over the
// kept blocks, softmax renormalised over the kept keys, online).
//
// This is the precision path: every product and sum is float32 FMA, which
// keeps the result within 1e-5 of the float64 definition at the sizes it
// serves. One workgroup per (head, local query block), one thread per query
// row; each kept block is consumed in sub-tiles of 32 keys staged in LDS (K
// rows as [key][d], V from the transposed packed layout as [d][key]), so every
// thread reads the same LDS words (broadcast reads, no bank conflicts).
#include "sparsp_internal.h"

namespace sparsp {
namespace {

constexpr int kKeys = 32;

template <int DMAX>
__global__ __launch_bounds__(256) void attn_f32_kernel(
    const float* __restrict__ Q, const int32_t* __restrict__ sel, const int32_t* __restrict__ slot_of,
    const float* __restrict__ Kp, const float* __restrict__ Vp, float* __restrict__ O,
    float* __restrict__ lse, int L, int n, int d, int block, int i0, int nq, int keep,
    int64_t capacity, float c2 /* scale * log2(e) */, int kv_lo, int kv_hi, int h_lo, int acc,
    const int32_t* __restrict__ order, int rows) {
    __shared__ float ks[kKeys][DMAX];
    __shared__ float vs[DMAX][kKeys];

    int wg = blockIdx.x;
    if (order) {  // an explicit row order (e.g. longest first)
        wg = order[blockIdx.x];
        if (wg < 0 || wg >= rows) return;
    }
    const int h = h_lo + wg / nq, r = wg % nq;
    const int tid = threadIdx.x;
    const int nthr = blockDim.x;
    const int qtok = (i0 + r) * block + tid;
    const bool qvalid = tid < block && qtok < L;

    float q[DMAX], o[DMAX];
#pragma unroll
    for (int c = 0; c < DMAX; ++c) {
        q[c] = (qvalid && c < d) ? Q[(int64_t(h) * L + qtok) * d + c] : 0.f;
        o[c] = 0.f;
    }
    float m = -INFINITY, l = 0.f;

    const int32_t* srow = sel + (int64_t(h) * nq + r) * keep;
    for (int jj = 0; jj < keep; ++jj) {
        const int j = srow[jj];
        if (j < 0 || j >= n || j < kv_lo || j >= kv_hi) continue;
        const int slot = slot_of[int64_t(h) * n + j];
        if (slot < 0 || slot >= capacity) continue;
        const int cnt = min(block, L - j * block);
        const float* kb = Kp + int64_t(slot) * block * d;
        const float* vb = Vp + int64_t(slot) * block * d;
        for (int k0 = 0; k0 < cnt; k0 += kKeys) {
            const int kn = min(kKeys, cnt - k0);
            __syncthreads();
            for (int e = tid; e < kKeys * DMAX; e += nthr) {
                const int t = e / DMAX, c = e % DMAX;
                ks[t][c] = (t < kn && c < d) ? kb[int64_t(k0 + t) * d + c] : 0.f;
            }
            for (int e = tid; e < kKeys * DMAX; e += nthr) {
                const int c = e / kKeys, t = e % kKeys;
                vs[c][t] = (t < kn && c < d) ? vb[int64_t(c) * block + k0 + t] : 0.f;
            }
            __syncthreads();
            float s[kKeys];
            float mx = -INFINITY;
#pragma unroll
            for (int t = 0; t < kKeys; ++t) {
                float acc = 0.f;
#pragma unroll
                for (int c = 0; c < DMAX; ++c) acc = fmaf(q[c], ks[t][c], acc);
                s[t] = t < kn ? acc * c2 : -INFINITY;
                mx = fmaxf(mx, s[t]);
            }
            const float m_new = fmaxf(m, mx);
            const float alpha = exp2f(m - m_new);
            m = m_new;
            l *= alpha;
#pragma unroll
            for (int c = 0; c < DMAX; ++c) o[c] *= alpha;
#pragma unroll
            for (int t = 0; t < kKeys; ++t) {
                const float p = exp2f(s[t] - m_new);
                l += p;
#pragma unroll
                for (int c = 0; c < DMAX; ++c) o[c] = fmaf(p, vs[c][t], o[c]);
            }
        }
    }
    if (tid >= block) return;
    const bool live = qvalid && l > 0.f;
    const float inv = live ? 1.0f / l : 0.f;
    const int64_t orow = (int64_t(h) * nq + r) * block + tid;
    if (acc) {
        // Fold into the stored result through the log-sum-exp (log2 units);
        // a row with no key in this part leaves it untouched.
        if (!live) return;
        const float la2 = lse[orow] * 1.4426950408889634f;
        const float lb2 = m + log2f(l);
        const float mm = fmaxf(la2, lb2);
        const float wa = la2 == -INFINITY ? 0.f : exp2f(la2 - mm);
        const float wb = exp2f(lb2 - mm);
        const float t = wa + wb;
        const float ka = wa / t, kb = wb / t * inv;
#pragma unroll
        for (int c = 0; c < DMAX; ++c)
            if (c < d) O[orow * d + c] = ka * O[orow * d + c] + kb * o[c];
        lse[orow] = (mm + log2f(t)) * 0.6931471805599453f;
        return;
    }
#pragma unroll
    for (int c = 0; c < DMAX; ++c)
        if (c < d) O[orow * d + c] = o[c] * inv;
    if (lse) lse[orow] = live ? (m + log2f(l)) * 0.6931471805599453f : -INFINITY;
}

}  // namespace

hipError_t launch_attn_f32(const Geom& g, const float* Q, const int32_t* sel, int keep,
                           const int32_t* slot_of, const float* Kp, const float* Vp,
                           int64_t capacity, float scale, const AttnPart& part, float* O,
                           float* lse, hipStream_t s) {
    (void)hipGetLastError();
    const int threads = ((g.block + 63) / 64) * 64;
    const float c2 = scale * 1.4426950408889634f;
    const int G = (part.h_hi - part.h_lo) * g.nq;
    if (g.d <= 64)
        attn_f32_kernel<64><<<G, threads, 0, s>>>(Q, sel, slot_of, Kp, Vp, O, lse, g.L, g.n, g.d,
                                                  g.block, g.i0, g.nq, keep, capacity, c2,
                                                  part.kv_lo, part.kv_hi, part.h_lo, part.acc, part.order, G);
    else
        attn_f32_kernel<128><<<G, threads, 0, s>>>(Q, sel, slot_of, Kp, Vp, O, lse, g.L, g.n,
                                                   g.d, g.block, g.i0, g.nq, keep, capacity, c2,
                                                   part.kv_lo, part.kv_hi, part.h_lo, part.acc, part.order, G);
    return hipGetLastError();
}

}  // namespace sparsp
