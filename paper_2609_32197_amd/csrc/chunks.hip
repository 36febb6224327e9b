// Host side of shard-by-shard attention (Section 2.3, Section 7).
//
// plan_chunks orders the work of rank r over the owners' KV shards:
//   * shard p holds the blocks [floor(p n / R), floor((p+1) n / R));
//   * the local shard (p = r) comes first and stays whole: one chunk with all
//     heads (Section 7.1: it needs no transfer);
//   * the remote shards follow in ring order r+1, ..., r+R-1 (mod R), each cut
//     into runs of heads_per_chunk consecutive heads, the last remote shard
//     into finer runs of tail_heads_per_chunk heads (Section 7.1: the final
//     block of the pipeline is chunked finer to shorten the drain);
//   * inside each remote shard, chunks run by selected blocks descending, then
//     head ascending (Section 7.2: the sparsest chunk goes last, so the
//     computation left exposed after the last transfer is the smallest).
// A chunk's selected blocks are its heads' demanded blocks inside the shard,
// counted from the demand bitsets.
//
// run_chunks executes a plan in order on one stream, one attention launch per
// chunk. A chunk whose heads have no result yet writes (O, lse) directly; any
// other chunk folds itself into them through the log-sum-exp inside the
// attention kernel (query blocks with no kept block in the shard exit without
// touching memory). Heads that no chunk covers end as the empty result.
#include <algorithm>
#include <vector>

#include "sparsp_internal.h"

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

hipError_t run_chunks(const Geom& g, const void* Q, const int32_t* sel, int keep,
                      const int32_t* slot_of, const void* Kp, const void* Vp, int64_t capacity,
                      float scale, const sparsp_chunk* plan, int n_chunks, float* O, float* lse,
                      hipStream_t s) {
    const int64_t rows = int64_t(g.nq) * g.block;  // accumulator rows per head
    std::vector<bool> seen(g.H, false);             // heads whose rows hold a result
    auto clear_head = [&](int h) {
        return launch_fill_identity(O + int64_t(h) * rows * g.d, lse + int64_t(h) * rows, rows,
                                    g.d, s);
    };
    for (int c = 0; c < n_chunks; ++c) {
        const sparsp_chunk& ch = plan[c];
        bool fresh = true, mixed = false;
        for (int h = ch.head_begin; h < ch.head_end; ++h) {
            fresh = fresh && !seen[h];
            mixed = mixed || !seen[h];
        }
        hipError_t e = hipSuccess;
        if (!fresh && mixed)  // heads met for the first time start from the empty result
            for (int h = ch.head_begin; h < ch.head_end && e == hipSuccess; ++h)
                if (!seen[h]) e = clear_head(h);
        if (e != hipSuccess) return e;
        const AttnPart part{ch.kv_blk_begin, ch.kv_blk_end, ch.head_begin, ch.head_end,
                            fresh ? 0 : 1};
        e = g.bf16 ? launch_attn_bf16(g, Q, sel, keep, slot_of, Kp, Vp, capacity, scale, part, O,
                                      false, lse, s)
                   : launch_attn_f32(g, (const float*)Q, sel, keep, slot_of, (const float*)Kp,
                                     (const float*)Vp, capacity, scale, part, O, lse, s);
        if (e != hipSuccess) return e;
        for (int h = ch.head_begin; h < ch.head_end; ++h) seen[h] = true;
    }
    for (int h = 0; h < g.H; ++h)  // heads no chunk covered: the empty result
        if (!seen[h])
            if (hipError_t e = clear_head(h); e != hipSuccess) return e;
    return hipSuccess;
}

}  // namespace sparsp
