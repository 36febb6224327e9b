// Pure host code of libsparsp: the shard-by-shard schedule (Section 2.3,
// Section 7), Eq. 4's placed order of the blocks (Section 4.3), the Eq. 3
// block count and the routing volumes of Section 5.1. Nothing here touches a
// device; the descriptions of each rule sit with their launch-side
// counterparts in chunks.hip and placement.hip.
#include <algorithm>
#include <vector>

#include "sparsp_launch.h"

namespace sparsp {

int plan_chunks(const Geom& g, const uint64_t* demand, int ranks, int rank, int heads_per_chunk,
                int tail_heads_per_chunk, sparsp_chunk* out, int max_chunks) {
    auto count = [&](int h0, int h1, int lo, int hi) {
        int c = 0;
        for (int h = h0; h < h1; ++h)
            for (int j = lo; j < hi; ++j) c += int((demand[int64_t(h) * g.W + (j >> 6)] >> (j & 63)) & 1);
        return c;
    };
    auto shard = [&](int p, int* lo, int* hi) {
        *lo = int(int64_t(p) * g.n / ranks);
        *hi = int(int64_t(p + 1) * g.n / ranks);
    };
    std::vector<sparsp_chunk> plan;
    int lo, hi;
    shard(rank, &lo, &hi);
    plan.push_back({rank, lo, hi, 0, g.H, count(0, g.H, lo, hi)});
    for (int k = 1; k < ranks; ++k) {
        const int p = (rank + k) % ranks;
        shard(p, &lo, &hi);
        const int size = k == ranks - 1 ? tail_heads_per_chunk : heads_per_chunk;
        std::vector<sparsp_chunk> part;
        for (int h0 = 0; h0 < g.H; h0 += size) {
            const int h1 = std::min(g.H, h0 + size);
            part.push_back({p, lo, hi, h0, h1, count(h0, h1, lo, hi)});
        }
        std::stable_sort(part.begin(), part.end(), [](const sparsp_chunk& a, const sparsp_chunk& b) {
            return a.blocks != b.blocks ? a.blocks > b.blocks : a.head_begin < b.head_begin;
        });
        plan.insert(plan.end(), part.begin(), part.end());
    }
    if (int(plan.size()) > max_chunks) return -int(plan.size());
    std::copy(plan.begin(), plan.end(), out);
    return int(plan.size());
}

void periodic_placement(int L, int block, int frame_tokens, int ranks, int32_t* perm,
                        int32_t* rank_begin) {
    const int n = (L + block - 1) / block;
    std::vector<int> owner(n);
    for (int j = 0; j < n; ++j)
        owner[j] = int(int64_t(ranks) * ((int64_t(j) * block) % frame_tokens) / frame_tokens);
    if (L % block) owner[n - 1] = ranks - 1;
    int k = 0;
    for (int p = 0; p < ranks; ++p) {
        rank_begin[p] = k;
        for (int j = 0; j < n; ++j)
            if (owner[j] == p) perm[k++] = j;
    }
    rank_begin[ranks] = k;
}

void remote_demand(const Geom& g, const uint64_t* demand, int64_t* remote, int64_t* demanded) {
    int64_t rem = 0, all = 0;
    for (int h = 0; h < g.H; ++h)
        for (int j = 0; j < g.n; ++j) {
            if (!((demand[int64_t(h) * g.W + (j >> 6)] >> (j & 63)) & 1)) continue;
            ++all;
            if (j < g.i0 || j >= g.i1) ++rem;
        }
    *remote = rem;
    *demanded = all;
}

void route_volume(const Geom& g, const uint64_t* demands, int ranks, int producer, int64_t* dense,
                  int64_t* relay, int64_t* direct) {
    const int lo = int(int64_t(producer) * g.n / ranks), hi = int(int64_t(producer + 1) * g.n / ranks);
    int64_t rel = 0, dir = 0;
    std::vector<uint64_t> down(g.W);
    for (int h = 0; h < g.H; ++h) {
        std::fill(down.begin(), down.end(), 0);
        for (int k = ranks - 1; k >= 1; --k) {  // farthest consumer first: down = union of distance >= k
            const int c = (producer + k) % ranks;
            const uint64_t* dm = demands + (int64_t(c) * g.H + h) * g.W;
            for (int j = lo; j < hi; ++j) {
                const uint64_t bit = uint64_t(1) << (j & 63);
                if (dm[j >> 6] & bit) {
                    ++dir;
                    down[j >> 6] |= bit;
                }
            }
            for (int j = lo; j < hi; ++j) rel += int64_t((down[j >> 6] >> (j & 63)) & 1);
        }
    }
    *dense = int64_t(ranks - 1) * g.H * (hi - lo);
    *relay = rel;
    *direct = dir;
}

}  // namespace sparsp
