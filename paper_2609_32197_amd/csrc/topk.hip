// Step 2: top-k block mask (Section 4.1's M) with the diagonal and global
// blocks forced and ties broken by the lower block index; and the CDF-mode
// variant of the mask (Section 8.1), further down.
//
// One wave64 per (head, local row). Lane l holds blocks j = l + 64 s
// (s = 0 .. S-1) in registers, so the 64 lanes of chunk s are exactly the 64
// bits of mask word s: a ballot builds a mask word directly.
//
// Selection is exact and order-free. Scores become order-preserving 32-bit
// keys (-0.0 folded onto +0.0, NaN below every number). A 32-step bitwise
// search finds T, the k-th largest candidate key (k = keep - |F|): at each bit
// it keeps the bit set if at least k candidates still reach the threshold.
// Candidates above T are taken; among those equal to T the lowest indices are
// taken until k is reached, ranked in index order with ballots and
// mbcnt. No floating point is involved, so the result is a pure function of
// the score bits.
#include "sparsp_internal.h"

namespace sparsp {
namespace {

__device__ __forceinline__ uint32_t order_key(float x) {
    uint32_t u = __float_as_uint(x);
    if (u == 0x80000000u) u = 0u;                                   // -0.0 ties +0.0
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return 0u;  // NaN: lowest
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
// one whose mass reaches tau Z: a bitwise search finds the largest order key T
// whose upper set {key >= T} still holds mass >= tau Z; the blocks above T
// are kept, and the blocks equal to T (equal scores, equal p) are added in
// index order until the target is met. The diagonal and global blocks are
// kept in any case. sel rows list the kept blocks ascending, then -1 up to n.
// A NaN score counts as no mass and ranks below every number.
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
        x[s] = (v != v) ? -INFINITY : v;
        mx = fmaxf(mx, x[s]);
    }
    mx = wave_max(mx);
    float part = 0.f;
#pragma unroll
    for (int s = 0; s < S; ++s) {
        p[s] = (x[s] == -INFINITY) ? 0.f : expf(x[s] - mx);
        part += p[s];
    }
    const float target = tau * wave_sum(part);

    uint32_t T = 0;
    for (int b = 31; b >= 0; --b) {
        const uint32_t t = T | (1u << b);
        float m = 0.f;
#pragma unroll
        for (int s = 0; s < S; ++s) m += (valid[s] && key[s] >= t) ? p[s] : 0.f;
        if (wave_sum(m) >= target) T = t;
    }
    float above = 0.f, pt = 0.f;
    int ties = 0;
#pragma unroll
    for (int s = 0; s < S; ++s) {
        above += (valid[s] && key[s] > T) ? p[s] : 0.f;
        const bool eq = valid[s] && key[s] == T;
        pt = fmaxf(pt, eq ? p[s] : 0.f);
        ties += popc64(__ballot(eq));
    }
    float acc = wave_sum(above);
    pt = wave_max(pt);
    int need = 0;
    while (need < ties && acc < target) {  // uniform: every lane holds the same values
        acc += pt;
        ++need;
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
        const bool take = forced[s] || (valid[s] && key[s] > T) || take_eq;
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
// A count outside [0, n] is clamped into it.
constexpr int kXcds = 8;

__global__ __launch_bounds__(1024) void row_order_kernel(const int32_t* __restrict__ counts,
                                                         int H, int nq, int n,
                                                         int32_t* __restrict__ order) {
    __shared__ int start[kMaxBlocks + 1];
    __shared__ int part[1024];
    __shared__ int64_t tot[kMaxHeads];
    __shared__ int rank_of[kMaxHeads];   // head -> rank by total
    __shared__ int head_at[kMaxHeads];   // rank -> head
    __shared__ int queue_of[kMaxHeads];  // head -> XCD queue
    __shared__ int qlen[kXcds];
    const int tid = threadIdx.x;
    auto cnt_of = [&](int row) { return min(max(counts[row], 0), n); };

    for (int h = tid; h < H; h += 1024) {
        int64_t t = 0;
        for (int r = 0; r < nq; ++r) t += cnt_of(h * nq + r);
        tot[h] = t;
    }
    __syncthreads();
    for (int h = tid; h < H; h += 1024) {
        int k = 0;
        for (int o = 0; o < H; ++o) k += (tot[o] > tot[h]) || (tot[o] == tot[h] && o < h);
        rank_of[h] = k;
        head_at[k] = h;
    }
    __syncthreads();
    if (tid == 0) {
        int64_t load[kXcds];
        int room[kXcds];
        for (int x = 0; x < kXcds; ++x) {
            load[x] = 0;
            room[x] = H / kXcds + (x < H % kXcds ? 1 : 0);
            qlen[x] = room[x] * nq;
        }
        for (int k = 0; k < H; ++k) {
            const int h = head_at[k];
            int best = -1;
            for (int x = 0; x < kXcds; ++x)
                if (room[x] > 0 && (best < 0 || load[x] < load[best])) best = x;
            queue_of[h] = best;
            load[best] += tot[h];
            --room[best];
        }
    }
    __syncthreads();
    int ql[kXcds];
#pragma unroll
    for (int x = 0; x < kXcds; ++x) ql[x] = qlen[x];

    const int rows = H * nq;
    const int per = (n + 1 + 1023) / 1024;
    for (int x = 0; x < kXcds; ++x) {
        if (ql[x] == 0) continue;
        for (int c = tid; c <= n; c += 1024) start[c] = 0;
        __syncthreads();
        for (int r = tid; r < rows; r += 1024)
            if (queue_of[r / nq] == x) atomicAdd(&start[cnt_of(r)], 1);
        __syncthreads();
        // exclusive scan over the count values n, n-1, ..., 0
        int local = 0;
        for (int k = 0; k < per; ++k) {
            const int idx = tid * per + k;
            if (idx <= n) local += start[n - idx];
        }
        part[tid] = local;
        __syncthreads();
        for (int off = 1; off < 1024; off <<= 1) {
            const int v = tid >= off ? part[tid - off] : 0;
            __syncthreads();
            part[tid] += v;
            __syncthreads();
        }
        int run = tid ? part[tid - 1] : 0;
        for (int k = 0; k < per; ++k) {
            const int idx = tid * per + k;
            if (idx <= n) {
                const int c = start[n - idx];
                start[n - idx] = run;
                run += c;
            }
        }
        __syncthreads();
        for (int r = tid; r < rows; r += 1024) {
            if (queue_of[r / nq] != x) continue;
            const int k = atomicAdd(&start[cnt_of(r)], 1);  // place in queue x
            int pos = 0;  // round-robin position of entry k of queue x
#pragma unroll
            for (int y = 0; y < kXcds; ++y) pos += min(k, ql[y]) + (y < x && ql[y] > k ? 1 : 0);
            order[pos] = r;
        }
        __syncthreads();
    }
}

// Work items for attention with long rows split (CDF rows keep from one to
// a few hundred blocks; the longest alone can outlast all the others). The
// same single-workgroup layout as the row order above, over items instead of
// rows:
//   1. which rows split: a row splits when its count c exceeds T and is at
//      least c*, the smallest threshold for which the split rows need at most
//      P pieces in all (ceil(c / T) pieces each); rows of equal count all
//      split or all stay whole;
//   2. workspace slots: split rows take consecutive slots in row order
//      (piece_base), one per piece;
//   3. piece p of a split row covers the kept blocks in [b_p, b_{p+1}), with
//      b_0 = 0, b_np = n and b_p the row's (p T)-th kept block (clamped to be
//      non-decreasing), so the pieces partition the row whatever its order;
//      with an ascending row each piece holds T kept blocks, the last the
//      rest. Its length is min(T, c - p T);
//   4. heads dealt to the eight XCD queues exactly as in the row order (by
//      their total count), each queue's items sorted longest first, the
//      queues interleaved round-robin over their item counts;
//   5. positions past the last item get row -1.
__global__ __launch_bounds__(1024) void split_plan_kernel(
    const int32_t* __restrict__ counts, const int32_t* __restrict__ sel, int H, int nq, int n,
    int keep, int T, int P, SplitItem* __restrict__ items, int32_t* __restrict__ piece_base) {
    __shared__ int hist[kMaxBlocks + 1];
    __shared__ int64_t part[1024];
    __shared__ int64_t tot[kMaxHeads];
    __shared__ int head_at[kMaxHeads];
    __shared__ int queue_of[kMaxHeads];
    __shared__ int qlen[kXcds];
    __shared__ int cstar_s;
    const int tid = threadIdx.x;
    const int R = H * nq;
    auto cnt_of = [&](int row) { return min(max(counts[row], 0), n); };
    // Block-wide inclusive scan of part[]; returns this thread's exclusive prefix.
    auto scan = [&]() -> int64_t {
        __syncthreads();
        for (int off = 1; off < 1024; off <<= 1) {
            const int64_t v = tid >= off ? part[tid - off] : 0;
            __syncthreads();
            part[tid] += v;
            __syncthreads();
        }
        return tid ? part[tid - 1] : 0;
    };

    // 1. histogram of the counts, then c* from the suffix sums of pieces.
    for (int c = tid; c <= n; c += 1024) hist[c] = 0;
    if (tid == 0) cstar_s = n + 1;
    __syncthreads();
    for (int r = tid; r < R; r += 1024) atomicAdd(&hist[cnt_of(r)], 1);
    __syncthreads();
    const int per = (n + 1 + 1023) / 1024;  // count values per thread, n downwards
    {
        int64_t local = 0;
        for (int k = 0; k < per; ++k) {
            const int c = n - (tid * per + k);
            if (c > T) local += int64_t(hist[c]) * ((c + T - 1) / T);
        }
        part[tid] = local;
        int64_t run = scan();  // pieces of the rows with a count above this thread's range
        int best = n + 1;
        for (int k = 0; k < per; ++k) {
            const int c = n - (tid * per + k);
            if (c > T) {
                run += int64_t(hist[c]) * ((c + T - 1) / T);
                if (run <= P) best = c;
            }
        }
        atomicMin(&cstar_s, best);
    }
    __syncthreads();
    const int cstar = cstar_s;
    auto npieces = [&](int c) { return (c > T && c >= cstar) ? (c + T - 1) / T : 1; };

    // 2. slots of the split rows, in row order.
    const int rper = (R + 1023) / 1024;
    {
        int64_t local = 0;
        for (int k = 0; k < rper; ++k) {
            const int r = tid * rper + k;
            if (r < R && npieces(cnt_of(r)) > 1) local += npieces(cnt_of(r));
        }
        __syncthreads();  // everyone is done reading part[] above
        part[tid] = local;
        int64_t run = scan();
        for (int k = 0; k < rper; ++k) {
            const int r = tid * rper + k;
            if (r >= R) break;
            const int np = npieces(cnt_of(r));
            piece_base[r] = np > 1 ? int32_t(run) : -1;
            if (np > 1) run += np;
        }
    }

    // 4. heads to queues, as in the row order.
    for (int h = tid; h < H; h += 1024) {
        int64_t t = 0;
        for (int r = 0; r < nq; ++r) t += cnt_of(h * nq + r);
        tot[h] = t;
    }
    if (tid < kXcds) qlen[tid] = 0;
    __syncthreads();
    for (int h = tid; h < H; h += 1024) {
        int k = 0;
        for (int o = 0; o < H; ++o) k += (tot[o] > tot[h]) || (tot[o] == tot[h] && o < h);
        head_at[k] = h;
    }
    __syncthreads();
    if (tid == 0) {
        int64_t load[kXcds];
        int room[kXcds];
        for (int x = 0; x < kXcds; ++x) {
            load[x] = 0;
            room[x] = H / kXcds + (x < H % kXcds ? 1 : 0);
        }
        for (int k = 0; k < H; ++k) {
            const int h = head_at[k];
            int best = -1;
            for (int x = 0; x < kXcds; ++x)
                if (room[x] > 0 && (best < 0 || load[x] < load[best])) best = x;
            queue_of[h] = best;
            load[best] += tot[h];
            --room[best];
        }
    }
    __syncthreads();
    for (int r = tid; r < R; r += 1024) atomicAdd(&qlen[queue_of[r / nq]], npieces(cnt_of(r)));
    __syncthreads();
    int ql[kXcds];
    int n_items = 0;
#pragma unroll
    for (int x = 0; x < kXcds; ++x) {
        ql[x] = qlen[x];
        n_items += ql[x];
    }
    // The kept block that opens piece q (q >= 1) of row r, clamped to [lo, n].
    auto bound = [&](int r, int q, int lo) {
        const int64_t e = int64_t(q) * T;
        const int j = e < keep ? sel[int64_t(r) * keep + e] : n;
        return min(max(j, lo), n);
    };

    for (int x = 0; x < kXcds; ++x) {
        if (ql[x] == 0) continue;
        for (int c = tid; c <= n; c += 1024) hist[c] = 0;
        __syncthreads();
        for (int r = tid; r < R; r += 1024) {
            if (queue_of[r / nq] != x) continue;
            const int c = cnt_of(r), np = npieces(c);
            if (np == 1) atomicAdd(&hist[c], 1);
            else
                for (int p = 0; p < np; ++p) atomicAdd(&hist[min(T, c - p * T)], 1);
        }
        __syncthreads();
        // exclusive scan over the lengths n, n-1, ..., 0
        int64_t local = 0;
        for (int k = 0; k < per; ++k) {
            const int idx = tid * per + k;
            if (idx <= n) local += hist[n - idx];
        }
        part[tid] = local;
        int64_t run = scan();
        for (int k = 0; k < per; ++k) {
            const int idx = tid * per + k;
            if (idx <= n) {
                const int c = hist[n - idx];
                hist[n - idx] = int(run);
                run += c;
            }
        }
        __syncthreads();
        auto place = [&](int len, SplitItem it) {
            const int k = atomicAdd(&hist[len], 1);  // entry k of queue x
            int pos = 0;
#pragma unroll
            for (int y = 0; y < kXcds; ++y) pos += min(k, ql[y]) + (y < x && ql[y] > k ? 1 : 0);
            items[pos] = it;
        };
        for (int r = tid; r < R; r += 1024) {
            if (queue_of[r / nq] != x) continue;
            const int c = cnt_of(r), np = npieces(c);
            if (np == 1) {
                place(c, SplitItem{r, 0, n, -1});
                continue;
            }
            const int base = piece_base[r];
            int lo = 0;
            for (int p = 0; p < np; ++p) {
                const int hi = p + 1 < np ? bound(r, p + 1, lo) : n;
                place(min(T, c - p * T), SplitItem{r, lo, hi, base + p});
                lo = hi;
            }
        }
        __syncthreads();
    }
    for (int i = n_items + tid; i < R + P; i += 1024) items[i] = SplitItem{-1, 0, 0, -1};
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

hipError_t launch_split_plan(const int32_t* counts, const int32_t* sel, int H, int nq, int n,
                             int keep, int T, int P, SplitItem* items, int32_t* piece_base,
                             hipStream_t st) {
    (void)hipGetLastError();
    split_plan_kernel<<<1, 1024, 0, st>>>(counts, sel, H, nq, n, keep, T, P, items, piece_base);
    return hipGetLastError();
}

}  // namespace sparsp
