// Host side of shard-by-shard attention (Section 2.3, Section 7): running a
// plan. The plan itself (plan_chunks, in host_plan.cpp) orders the work of rank r over the owners' KV shards:
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
#include "sparsp_internal.h"

namespace sparsp {

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
