// Step 4, float32: block-sparse attention for float32 inputs (Eq. 1 over the
// kept blocks, softmax renormalised over the kept keys, online).
//
// This is the precision path: every product and sum is float32 FMA, which
// keeps the result within 1e-5 of the float64 definition at the sizes it
// serves. One workgroup per (head, local query block). P neighbouring lanes
// of a wave share one query row (P = 4 for blocks of up to 64 tokens, 2 up to
// 128, 1 up to 256, so a workgroup has at most 256 threads): each kept block
// is consumed in sub-tiles of 32 keys staged in LDS, lane p of a row takes keys
// p, p + P, ... of every sub-tile and runs its own online softmax over them,
// and the P partial results of a row are merged at the end through their
// maxima and sums (the online-softmax merge of Section 2.3), with lane
// shuffles inside the wave. Both tiles are staged key-major ([key][d], V
// transposed back on the way in), so a lane reads four consecutive d values
// of one key per LDS instruction; rows are padded by four words, which keeps
// those reads 16-byte aligned and puts the P lanes of a row, which read
// different keys, on different banks.
#include "sparsp_internal.h"

namespace sparsp {
namespace {

constexpr int kKeys = 32;

template <int DMAX, int P>
__global__ __launch_bounds__(256) void attn_f32_kernel(
    const float* __restrict__ Q, const int32_t* __restrict__ sel, const int32_t* __restrict__ slot_of,
    const float* __restrict__ Kp, const float* __restrict__ Vp, float* __restrict__ O,
    float* __restrict__ lse, int L, int n, int d, int block, int i0, int nq, int keep,
    int64_t capacity, float c2 /* scale * log2(e) */, int kv_lo, int kv_hi, int h_lo, int acc,
    const int32_t* __restrict__ order, int rows) {
    constexpr int KP = kKeys / P;  // keys of a sub-tile per lane
    __shared__ __attribute__((aligned(16))) float ks[kKeys][DMAX + 4];
    __shared__ __attribute__((aligned(16))) float vs[kKeys][DMAX + 4];
    // The row's kept list resolved once: slot and valid key count per entry
    // (slot -1: outside [kv_lo, kv_hi) or not packed).
    extern __shared__ int32_t kept_lds[];
    int32_t* kslot = kept_lds;
    int32_t* kcnt = kept_lds + keep;

    int wg = blockIdx.x;
    if (order) {  // an explicit row order (e.g. longest first)
        wg = order[blockIdx.x];
        if (wg < 0 || wg >= rows) return;
    }
    const int h = h_lo + wg / nq, r = wg % nq;
    const int tid = threadIdx.x;
    const int nthr = blockDim.x;
    const int part = tid % P, qrow = tid / P;
    const int qtok = (i0 + r) * block + qrow;
    const bool qvalid = qrow < block && qtok < L;

    float q[DMAX], o[DMAX];
#pragma unroll
    for (int c = 0; c < DMAX; ++c) {
        q[c] = (qvalid && c < d) ? Q[(int64_t(h) * L + qtok) * d + c] : 0.f;
        o[c] = 0.f;
    }
    float m = -INFINITY, l = 0.f;

    const int32_t* srow = sel + (int64_t(h) * nq + r) * keep;
    for (int jj = tid; jj < keep; jj += nthr) {
        const int j = srow[jj];
        int slot = -1, cnt = 0;
        if (j >= 0 && j < n && j >= kv_lo && j < kv_hi) {
            const int sl = slot_of[int64_t(h) * n + j];
            if (sl >= 0 && sl < capacity) {
                slot = sl;
                cnt = min(block, L - j * block);
            }
        }
        kslot[jj] = slot;
        kcnt[jj] = cnt;
    }
    __syncthreads();
    for (int jj = 0; jj < keep; ++jj) {
        const int slot = kslot[jj];
        if (slot < 0) continue;
        const int cnt = kcnt[jj];
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
                vs[t][c] = (t < kn && c < d) ? vb[int64_t(c) * block + k0 + t] : 0.f;
            }
            __syncthreads();
            float s[KP];
            float mx = -INFINITY;
#pragma unroll
            for (int i = 0; i < KP; ++i) {
                const int t = part + P * i;
                float dot = 0.f;
#pragma unroll
                for (int c = 0; c < DMAX; ++c) dot = fmaf(q[c], ks[t][c], dot);
                s[i] = t < kn ? dot * c2 : -INFINITY;
                mx = fmaxf(mx, s[i]);
            }
            if (mx == -INFINITY) continue;  // none of this lane's keys exist here
            const float m_new = fmaxf(m, mx);
            const float alpha = exp2f(m - m_new);
            m = m_new;
            l *= alpha;
#pragma unroll
            for (int c = 0; c < DMAX; ++c) o[c] *= alpha;
#pragma unroll
            for (int i = 0; i < KP; ++i) {
                const float pr = exp2f(s[i] - m_new);
                l += pr;
#pragma unroll
                for (int c = 0; c < DMAX; ++c) o[c] = fmaf(pr, vs[part + P * i][c], o[c]);
            }
        }
    }

    // Merge the P partial softmaxes of this row: weight each by 2^(m_p - M)
    // for the row max M (0 for a lane that saw no key), then sum.
    if constexpr (P > 1) {
        float mm = m;
#pragma unroll
        for (int x = 1; x < P; x <<= 1) mm = fmaxf(mm, __shfl_xor(mm, x));
        const float w = (m == -INFINITY) ? 0.f : exp2f(m - mm);
        l *= w;
#pragma unroll
        for (int c = 0; c < DMAX; ++c) o[c] *= w;
#pragma unroll
        for (int x = 1; x < P; x <<= 1) {
            l += __shfl_xor(l, x);
#pragma unroll
            for (int c = 0; c < DMAX; ++c) o[c] += __shfl_xor(o[c], x);
        }
        m = mm;
    }
    if (part != 0 || qrow >= block) return;
    const bool live = qvalid && l > 0.f;
    const float inv = live ? 1.0f / l : 0.f;
    const int64_t orow = (int64_t(h) * nq + r) * block + qrow;
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
    const float c2 = scale * 1.4426950408889634f;
    const int G = (part.h_hi - part.h_lo) * g.nq;
    // lanes per query row, and threads: whole waves covering block rows
    const int P = g.block <= 64 ? 4 : g.block <= 128 ? 2 : 1;
    const int rows_per_wave = 64 / P;
    const int threads = (g.block + rows_per_wave - 1) / rows_per_wave * 64;
    if (threads > 256) return hipErrorInvalidValue;
    const size_t dyn = size_t(keep) * 2 * sizeof(int32_t);  // kept slots and counts
#define SPARSP_F32_LAUNCH(DM, PP)                                                               \
    attn_f32_kernel<DM, PP><<<G, threads, dyn, s>>>(Q, sel, slot_of, Kp, Vp, O, lse, g.L, g.n, g.d, \
                                                  g.block, g.i0, g.nq, keep, capacity, c2,        \
                                                  part.kv_lo, part.kv_hi, part.h_lo, part.acc,    \
                                                  part.order, G)
    if (g.d <= 64) {
        if (P == 4) SPARSP_F32_LAUNCH(64, 4);
        else if (P == 2) SPARSP_F32_LAUNCH(64, 2);
        else SPARSP_F32_LAUNCH(64, 1);
    } else {
        if (P == 4) SPARSP_F32_LAUNCH(128, 4);
        else if (P == 2) SPARSP_F32_LAUNCH(128, 2);
        else SPARSP_F32_LAUNCH(128, 1);
    }
#undef SPARSP_F32_LAUNCH
    return hipGetLastError();
}

}  // namespace sparsp
