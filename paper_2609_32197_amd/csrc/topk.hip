// Step 2: top-k block mask (Section 4.1's M) with the diagonal and global
// blocks forced and ties broken by the lower block index; and the CDF-mode
// variant of the mask (Section 8.1), further down.
//
// One wave64 per (head, local row). Lane l holds blocks j = l + 64 s
// (s = 0 .. S-1) in registers, so the 64 lanes of chunk s are exactly the 64
// bits of mask word s: a ballot builds a mask word directly.
//
// Selection is exact and order-free. Scores become order-preserving 32-bit
// keys (-0.0 folded onto +0.0). A 32-step bitwise search finds T, the k-th
// largest candidate key (k = keep - |F|): at each bit it keeps the bit set if
// at least k candidates still reach the threshold.
// Candidates above T are taken; among those equal to T the lowest indices are
// taken until k is reached, ranked in index order with ballots and
// mbcnt. No floating point is involved, so the result is a pure function of
// the score bits. NaN scores are outside the contract: a row holding one still
// gets a well-formed selection of keep blocks, but which ones is unspecified.
#include "sparsp_internal.h"

namespace sparsp {
namespace {

__device__ __forceinline__ uint32_t order_key(float x) {
    uint32_t u = __float_as_uint(x);
    if (u == 0x80000000u) u = 0u;  // -0.0 ties +0.0
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ int popc64(uint64_t x) { return __popcll(x); }

// Number of set bits of `b` below this lane.
__device__ __forceinline__ int below_lane(uint64_t b) {
    return __builtin_amdgcn_mbcnt_hi(uint32_t(b >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(b), 0));
}

template <int S>
__global__ __launch_bounds__(256) void topk_kernel(const float* __restrict__ scores, int H, int nq,
                                                   int n, int W, int i0, int keep, GlobalSet gs,
                                                   uint64_t* __restrict__ mask,
                                                   int32_t* __restrict__ sel) {
    const int lane = threadIdx.x & 63;
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);  // h * nq + r
    if (row >= H * nq) return;  // whole wave exits together
    const int r = row % nq;
    const int i = i0 + r;  // global index of this query block: the forced diagonal

    const float* srow = scores + int64_t(row) * n;
    uint32_t key[S];
    bool cand[S], forced[S];
#pragma unroll
    for (int s = 0; s < S; ++s) {
        const int j = lane + 64 * s;
        const bool valid = j < n;
        const bool f = valid && (j == i || ((gs.w[s] >> lane) & 1));
        forced[s] = f;
        cand[s] = valid && !f;
        key[s] = valid ? order_key(srow[j]) : 0u;
    }
    const bool diag_in_g = (gs.w[i >> 6] >> (i & 63)) & 1;
    const int n_forced = gs.count + (diag_in_g ? 0 : 1);
    const int k = keep - n_forced;  // candidates to take, >= 0 (checked on the host)

    uint32_t T = 0;
    int need = 0;  // how many candidates equal to T to take
    if (k > 0) {
        for (int b = 31; b >= 0; --b) {
            const uint32_t t = T | (1u << b);
            int cnt = 0;
#pragma unroll
            for (int s = 0; s < S; ++s) cnt += popc64(__ballot(cand[s] && key[s] >= t));
            if (cnt >= k) T = t;
        }
        int gt = 0;
#pragma unroll
        for (int s = 0; s < S; ++s) gt += popc64(__ballot(cand[s] && key[s] > T));
        need = k - gt;  // >= 1 by the choice of T
    }

    uint64_t* mrow = mask + int64_t(row) * W;
    int32_t* selrow = sel + int64_t(row) * keep;
    int ties_seen = 0, written = 0;
#pragma unroll
    for (int s = 0; s < S; ++s) {
        bool take = forced[s];
        if (k > 0) {
            const bool eq = cand[s] && key[s] == T;
            const uint64_t eqb = __ballot(eq);
            const bool take_eq = eq && (ties_seen + below_lane(eqb)) < need;
            ties_seen += popc64(eqb);
            take = take || (cand[s] && key[s] > T) || take_eq;
        }
        const uint64_t word = __ballot(take);
        if (s < W && lane == 0) mrow[s] = word;
        if (take) selrow[written + below_lane(word)] = lane + 64 * s;
        written += popc64(word);
    }
}

template <int S>
hipError_t launch_s(const Geom& g, const float* scores, int keep, const GlobalSet& gs,
                    uint64_t* mask, int32_t* sel, hipStream_t st) {
    const int rows = g.H * g.nq;
    topk_kernel<S><<<(rows + 3) / 4, 256, 0, st>>>(scores, g.H, g.nq, g.n, g.W, g.i0, keep, gs,
                                                   mask, sel);
    return hipGetLastError();
}

// Wave-wide sum and max, the same value in every lane: a butterfly sum can
// differ in its last bits from lane to lane (each lane adds in its own
// order), so lane 0's result is broadcast. Every decision below therefore is
// uniform across the wave.
__device__ __forceinline__ float wave_sum(float x) {
    for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
    return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(x)));
}
__device__ __forceinline__ float wave_max(float x) {
    for (int off = 32; off > 0; off >>= 1) x = fmaxf(x, __shfl_xor(x, off, 64));
    return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(x)));
}

// CDF-mode selection (Section 8.1), one wave per (head, local row), blocks held
// as in topk_kernel. p_j = exp(s_j - max) over the row, Z = sum p. With the
// blocks ordered by (score desc, index asc), the kept prefix is the shortest
// one whose mass reaches tau Z, i.e. whose left-out mass is at most
// (1 - tau) Z. The left-out mass is summed from the blocks themselves, not
// taken as Z minus a running total, so trailing blocks far below the total
// still count. A bitwise search finds the largest order key T whose lower set
// {key < T} carries at most that budget; the blocks at or above T are kept,
// except that of the blocks equal to T (equal scores, equal p) the highest
// indices are left out while the budget allows. tau = 1 keeps every block
// (every block's mass is positive, even where float32 exp underflows). The
// diagonal and global blocks are kept in any case. sel rows list the kept
// blocks ascending, then -1 up to n. Scores must be finite.
template <int S>
__global__ __launch_bounds__(256) void cdf_kernel(const float* __restrict__ scores, int H, int nq,
                                                  int n, int W, int i0, float tau, GlobalSet gs,
                                                  uint64_t* __restrict__ mask,
                                                  int32_t* __restrict__ sel,
                                                  int32_t* __restrict__ counts) {
    const int lane = threadIdx.x & 63;
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= H * nq) return;  // whole wave exits together
    const int i = i0 + row % nq;

    const float* srow = scores + int64_t(row) * n;
    uint32_t key[S];
    float x[S], p[S];
    bool valid[S], forced[S];
    float mx = -INFINITY;
#pragma unroll
    for (int s = 0; s < S; ++s) {
        const int j = lane + 64 * s;
        valid[s] = j < n;
        forced[s] = valid[s] && (j == i || ((gs.w[s] >> lane) & 1));
        const float v = valid[s] ? srow[j] : -INFINITY;
        key[s] = valid[s] ? order_key(v) : 0u;
        x[s] = v;
        mx = fmaxf(mx, x[s]);
    }
    mx = wave_max(mx);
    float part = 0.f;
#pragma unroll
    for (int s = 0; s < S; ++s) {
        p[s] = valid[s] ? expf(x[s] - mx) : 0.f;
        part += p[s];
    }
    const bool keep_all = tau >= 1.0f;
    const float budget = (1.0f - tau) * wave_sum(part);

    uint32_t T = 0;
    int need = 0;
    if (!keep_all) {
        for (int b = 31; b >= 0; --b) {
            const uint32_t t = T | (1u << b);
            float m = 0.f;
#pragma unroll
            for (int s = 0; s < S; ++s) m += (valid[s] && key[s] < t) ? p[s] : 0.f;
            if (wave_sum(m) <= budget) T = t;
        }
        float below = 0.f, pt = 0.f;
        int ties = 0;
#pragma unroll
        for (int s = 0; s < S; ++s) {
            below += (valid[s] && key[s] < T) ? p[s] : 0.f;
            const bool eq = valid[s] && key[s] == T;
            pt = fmaxf(pt, eq ? p[s] : 0.f);
            ties += popc64(__ballot(eq));
        }
        float left = wave_sum(below);
        pt = wave_max(pt);
        int out = 0;  // ties left out, the highest indices; at least one tie stays
        while (out + 1 < ties && left + pt <= budget) {  // uniform across the wave
            left += pt;
            ++out;
        }
        need = ties - out;
    }

    uint64_t* mrow = mask + int64_t(row) * W;
    int32_t* selrow = sel + int64_t(row) * n;
    int ties_seen = 0, written = 0;
#pragma unroll
    for (int s = 0; s < S; ++s) {
        const bool eq = valid[s] && key[s] == T;
        const uint64_t eqb = __ballot(eq);
        const bool take_eq = eq && (ties_seen + below_lane(eqb)) < need;
        ties_seen += popc64(eqb);
        const bool take = forced[s] || (valid[s] && (keep_all || key[s] > T)) || take_eq;
        const uint64_t word = __ballot(take);
        if (s < W && lane == 0) mrow[s] = word;
        if (take) selrow[written + below_lane(word)] = lane + 64 * s;
        written += popc64(word);
    }
    for (int e = written + lane; e < n; e += 64) selrow[e] = -1;
    if (lane == 0) counts[row] = written;
}

template <int S>
hipError_t launch_cdf_s(const Geom& g, const float* scores, float tau, const GlobalSet& gs,
                        uint64_t* mask, int32_t* sel, int32_t* counts, hipStream_t st) {
    const int rows = g.H * g.nq;
    cdf_kernel<S><<<(rows + 3) / 4, 256, 0, st>>>(scores, g.H, g.nq, g.n, g.W, g.i0, tau, gs, mask,
                                                  sel, counts);
    return hipGetLastError();
}

// Row order for rows of unequal kept counts (CDF selection), for a launch
// whose workgroup w runs on XCD w mod 8. One workgroup:
//   1. totals per head; heads ranked by total (descending, then by index);
//   2. heads dealt to the eight XCD queues largest first, each to the least
//      loaded queue that still has room (H/8 heads per queue, the first H mod 8
//      queues one more), so every head's rows share one XCD's L2 and the
//      queues carry nearly equal work;
//   3. each queue's rows sorted by count, largest first (counting sort; rows
//      of equal count in unspecified order);
//   4. the queues interleaved: entry k of queue x goes to the position that a
//      round-robin walk over the queues gives it, i.e. x + 8k while all
//      queues are that long.
// A count outside [0, n] is clamped into it. Up to kCountCache rows the
// counts are read from memory once and kept in LDS, where one thread per head
// sums its total; past that, all rows add into the totals with LDS atomics.
// Each queue's pass walks only the rows of its own heads.
constexpr int kXcds = 8;
constexpr int kCountCache = 14336;  // rows whose counts are kept in LDS (16 bits each)
static_assert(kMaxBlocks < 65536, "counts must fit 16 bits");

// Exclusive prefix sum of v over a 1024-thread workgroup: a shuffle scan in
// each wave, then one over the 16 wave totals (wave_sums: 16 ints of LDS).
// Two barriers; every thread must call it.
__device__ __forceinline__ int block_exclusive_scan(int v, int* wave_sums) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int incl = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int t = __shfl_up(incl, off, 64);
        if (lane >= off) incl += t;
    }
    if (lane == 63) wave_sums[w] = incl;
    __syncthreads();
    if (w == 0) {
        int t = lane < 16 ? wave_sums[lane] : 0;
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) {
            const int u = __shfl_up(t, off, 64);
            if (lane >= off) t += u;
        }
        if (lane < 16) wave_sums[lane] = t;
    }
    __syncthreads();
    return (w ? wave_sums[w - 1] : 0) + incl - v;
}

__global__ __launch_bounds__(1024) void row_order_kernel(const int32_t* __restrict__ counts,
                                                         int H, int nq, int n,
                                                         int32_t* __restrict__ order) {
    __shared__ int start[kMaxBlocks + 1];
    __shared__ int wave_sums[16];
    __shared__ unsigned long long tot[kMaxHeads];
    __shared__ int head_at[kMaxHeads];   // rank -> head
    __shared__ int q_heads[kMaxHeads];   // heads grouped by queue, in dealing order
    __shared__ int q_first[kXcds + 1];   // queue x's heads: q_heads[q_first[x] .. q_first[x+1])
    __shared__ uint16_t cnt_s[kCountCache];  // the clamped counts, when they fit
    const int tid = threadIdx.x;
    auto cnt_of = [&](int row) { return min(max(counts[row], 0), n); };
    const int rows = H * nq;
    const bool cached = rows <= kCountCache;
    auto cnt_at = [&](int row) { return cached ? int(cnt_s[row]) : cnt_of(row); };

    // 1. totals per head, heads ranked by total. With the counts in LDS a
    // thread sums its head's rows there; otherwise all rows are added in
    // parallel (LDS atomics).
    for (int h = tid; h < H; h += 1024) tot[h] = 0;
    if (cached)
        for (int r = tid; r < rows; r += 1024) cnt_s[r] = uint16_t(cnt_of(r));
    __syncthreads();
    if (cached) {
        for (int h = tid; h < H; h += 1024) {
            unsigned long long t = 0;
            for (int r = 0; r < nq; ++r) t += cnt_s[h * nq + r];
            tot[h] = t;
        }
    } else {
        for (int r = tid; r < rows; r += 1024) atomicAdd(&tot[r / nq], (unsigned long long)cnt_of(r));
    }
    __syncthreads();
    for (int h = tid; h < H; h += 1024) {
        int k = 0;
        for (int o = 0; o < H; ++o) k += (tot[o] > tot[h]) || (tot[o] == tot[h] && o < h);
        head_at[k] = h;
    }
    if (tid <= kXcds) {  // queue x holds H/8 heads, the first H mod 8 queues one more
        int f = 0;
        for (int x = 0; x < tid; ++x) f += H / kXcds + (x < H % kXcds ? 1 : 0);
        q_first[tid] = f;
    }
    __syncthreads();
    // 2. heads dealt to the queues in rank order, each to the least loaded
    // queue with room (the lowest such queue on a tie); each queue's heads are
    // listed together. One wave: lane x < 8 holds queue x's load and room,
    // and a shuffle argmin over lanes 0..7 picks the queue for each head.
    if (tid < 64) {
        const int lane = tid;
        unsigned long long load = 0;
        int room = lane < kXcds ? H / kXcds + (lane < H % kXcds ? 1 : 0) : 0;
        int fill = lane < kXcds ? q_first[lane] : 0;
        for (int k = 0; k < H; ++k) {
            const int h = head_at[k];
            const unsigned long long t = tot[h];
            unsigned long long key = (lane < kXcds && room > 0) ? load : ~0ull;
            int arg = lane;
#pragma unroll
            for (int off = 1; off < kXcds; off <<= 1) {
                const uint32_t lo = __shfl_xor(uint32_t(key), off, 64);
                const uint32_t hi = __shfl_xor(uint32_t(key >> 32), off, 64);
                const int oa = __shfl_xor(arg, off, 64);
                const unsigned long long ok = (uint64_t(hi) << 32) | lo;
                if (ok < key || (ok == key && oa < arg)) {
                    key = ok;
                    arg = oa;
                }
            }
            if (lane < kXcds && lane == arg) {
                q_heads[fill++] = h;
                load += t;
                --room;
            }
        }
    }
    __syncthreads();
    int ql[kXcds];
#pragma unroll
    for (int x = 0; x < kXcds; ++x) ql[x] = (q_first[x + 1] - q_first[x]) * nq;

    // 3. per queue: counting sort of its rows by count, largest first, and
    // placement at the queue's round-robin positions
    const int per = (n + 1 + 1023) / 1024;
    for (int x = 0; x < kXcds; ++x) {
        if (ql[x] == 0) continue;
        const int* qh = q_heads + q_first[x];
        for (int c = tid; c <= n; c += 1024) start[c] = 0;
        __syncthreads();
        for (int i = tid; i < ql[x]; i += 1024) atomicAdd(&start[cnt_at(qh[i / nq] * nq + i % nq)], 1);
        __syncthreads();
        // exclusive scan over the count values n, n-1, ..., 0
        int local = 0;
        for (int k = 0; k < per; ++k) {
            const int idx = tid * per + k;
            if (idx <= n) local += start[n - idx];
        }
        int run = block_exclusive_scan(local, wave_sums);
        for (int k = 0; k < per; ++k) {
            const int idx = tid * per + k;
            if (idx <= n) {
                const int c = start[n - idx];
                start[n - idx] = run;
                run += c;
            }
        }
        __syncthreads();
        for (int i = tid; i < ql[x]; i += 1024) {
            const int r = qh[i / nq] * nq + i % nq;
            const int k = atomicAdd(&start[cnt_at(r)], 1);  // place in queue x
            int pos = 0;  // round-robin position of entry k of queue x
#pragma unroll
            for (int y = 0; y < kXcds; ++y) pos += min(k, ql[y]) + (y < x && ql[y] > k ? 1 : 0);
            order[pos] = r;
        }
        __syncthreads();
    }
}

}  // namespace

hipError_t launch_cdf(const Geom& g, const float* scores, float tau, const GlobalSet& gs,
                      uint64_t* mask, int32_t* sel, int32_t* counts, hipStream_t st) {
    (void)hipGetLastError();
    if (g.W <= 1) return launch_cdf_s<1>(g, scores, tau, gs, mask, sel, counts, st);
    if (g.W <= 2) return launch_cdf_s<2>(g, scores, tau, gs, mask, sel, counts, st);
    if (g.W <= 4) return launch_cdf_s<4>(g, scores, tau, gs, mask, sel, counts, st);
    if (g.W <= 8) return launch_cdf_s<8>(g, scores, tau, gs, mask, sel, counts, st);
    if (g.W <= 16) return launch_cdf_s<16>(g, scores, tau, gs, mask, sel, counts, st);
    if (g.W <= 32) return launch_cdf_s<32>(g, scores, tau, gs, mask, sel, counts, st);
    return launch_cdf_s<64>(g, scores, tau, gs, mask, sel, counts, st);
}

hipError_t launch_topk(const Geom& g, const float* scores, int keep, const GlobalSet& gs,
                       uint64_t* mask, int32_t* sel, hipStream_t st) {
    (void)hipGetLastError();
    if (g.W <= 1) return launch_s<1>(g, scores, keep, gs, mask, sel, st);
    if (g.W <= 2) return launch_s<2>(g, scores, keep, gs, mask, sel, st);
    if (g.W <= 4) return launch_s<4>(g, scores, keep, gs, mask, sel, st);
    if (g.W <= 8) return launch_s<8>(g, scores, keep, gs, mask, sel, st);
    if (g.W <= 16) return launch_s<16>(g, scores, keep, gs, mask, sel, st);
    if (g.W <= 32) return launch_s<32>(g, scores, keep, gs, mask, sel, st);
    return launch_s<64>(g, scores, keep, gs, mask, sel, st);
}

hipError_t launch_row_order(const int32_t* counts, int H, int nq, int n, int32_t* order,
                            hipStream_t st) {
    (void)hipGetLastError();
    row_order_kernel<<<1, 1024, 0, st>>>(counts, H, nq, n, order);
    return hipGetLastError();
}

}  // namespace sparsp
