// C ABI of libsparsp: argument checking, geometry derivation and dispatch.
//
// Every check runs on the host before any launch, so a call that returns an
// error has enqueued nothing. The library holds no device state. This file is
// plain host C++ on the HIP runtime API (it calls only the launchers of
// sparsp_launch.h, hipGetLastError and hipGetErrorString), so it also builds
// with a host compiler under the address and undefined-behaviour sanitizers.
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstring>

#include "sparsp_launch.h"

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return code;
}

int ok() {
    g_err[0] = '\0';
    return SPARSP_OK;
}

int hip_status(hipError_t e, const char* what) {
    if (e == hipSuccess) e = hipGetLastError();
    if (e != hipSuccess) return fail(SPARSP_E_HIP, "%s: %s", what, hipGetErrorString(e));
    return ok();
}

// Validates the geometry shared by every call and fills `out`.
int derive(const sparsp_geom* g, sparsp::Geom* out) {
    if (!g) return fail(SPARSP_E_INVALID, "geom is NULL");
    if (g->H <= 0 || g->L <= 0 || g->d <= 0 || g->block <= 0)
        return fail(SPARSP_E_INVALID, "H, L, d and block must be positive (H=%d L=%d d=%d block=%d)",
                    g->H, g->L, g->d, g->block);
    if (g->dtype != SPARSP_F32 && g->dtype != SPARSP_BF16)
        return fail(SPARSP_E_DTYPE, "unknown dtype %d", g->dtype);
    const int64_t n = (int64_t(g->L) + g->block - 1) / g->block;
    if (g->q_blk_begin < 0 || g->q_blk_end > n || g->q_blk_begin >= g->q_blk_end)
        return fail(SPARSP_E_INVALID, "local query blocks [%d, %d) not inside [0, %lld) or empty",
                    g->q_blk_begin, g->q_blk_end, (long long)n);
    if (n > sparsp::kMaxBlocks)
        return fail(SPARSP_E_UNSUPPORTED, "n = %lld blocks exceeds the limit %d", (long long)n,
                    sparsp::kMaxBlocks);
    if (g->d > 256) return fail(SPARSP_E_UNSUPPORTED, "d = %d exceeds 256", g->d);
    if (g->H > sparsp::kMaxHeads)
        return fail(SPARSP_E_UNSUPPORTED, "H = %d exceeds %d", g->H, sparsp::kMaxHeads);
    const int vec = g->dtype == SPARSP_BF16 ? 8 : 4;
    if (g->d % vec)
        return fail(SPARSP_E_UNSUPPORTED, "d = %d must be a multiple of %d for this dtype", g->d, vec);
    if (int64_t(g->H) * g->L * g->d > (int64_t(1) << 40))
        return fail(SPARSP_E_INVALID, "H*L*d too large");
    out->H = g->H;
    out->L = g->L;
    out->d = g->d;
    out->block = g->block;
    out->i0 = g->q_blk_begin;
    out->i1 = g->q_blk_end;
    out->n = int(n);
    out->nq = g->q_blk_end - g->q_blk_begin;
    out->W = int((n + 63) / 64);
    out->bf16 = g->dtype == SPARSP_BF16;
    return SPARSP_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Packed-block kernels move 16-byte chunks: blocks must hold whole chunks.
int check_chunked(const sparsp::Geom& G) {
    const int vec = G.bf16 ? 8 : 4;
    if (G.block % vec)
        return fail(SPARSP_E_UNSUPPORTED, "block = %d must be a multiple of %d for this dtype",
                    G.block, vec);
    return SPARSP_OK;
}

// The forced global blocks as a bitset (host array of n_global indices).
int global_set(const sparsp::Geom& G, const int32_t* global_blocks, int n_global,
               sparsp::GlobalSet* gs) {
    if (n_global < 0 || (n_global > 0 && !global_blocks))
        return fail(SPARSP_E_INVALID, "global_blocks is NULL but n_global = %d", n_global);
    if (n_global > sparsp::kMaxGlobal)
        return fail(SPARSP_E_UNSUPPORTED, "n_global = %d exceeds %d", n_global, sparsp::kMaxGlobal);
    memset(gs, 0, sizeof(*gs));
    for (int t = 0; t < n_global; ++t) {
        const int j = global_blocks[t];
        if (j < 0 || j >= G.n)
            return fail(SPARSP_E_INVALID, "global block %d outside [0, %d)", j, G.n);
        gs->w[j >> 6] |= uint64_t(1) << (j & 63);
    }
    for (int w = 0; w < sparsp::kMaxWords; ++w) gs->count += __builtin_popcountll(gs->w[w]);
    return SPARSP_OK;
}

// Checks shared by every attention entry point (not the output buffers).
int check_attn(const sparsp::Geom& G, const void* Q, const int32_t* sel, int keep,
               const int32_t* slot_of, const void* Kp, const void* Vp, int64_t capacity,
               float scale) {
    if (!Q || !sel || !slot_of || !Kp || !Vp) return fail(SPARSP_E_INVALID, "NULL tensor pointer");
    if (keep < 1 || keep > G.n)
        return fail(SPARSP_E_INVALID, "keep = %d outside [1, n = %d]", keep, G.n);
    if (capacity < 1) return fail(SPARSP_E_CAPACITY, "capacity_blocks < 1");
    if (int rc = check_chunked(G)) return rc;
    if (!aligned16(Q) || !aligned16(Kp) || !aligned16(Vp))
        return fail(SPARSP_E_INVALID, "Q and the packed buffers must be 16-byte aligned");
    if (!(scale > 0.0f) || scale > 1e30f)
        return fail(SPARSP_E_INVALID, "softmax_scale must be positive and finite");
    if (G.bf16) {
        const bool ok_shape = (G.d == 64 || G.d == 128) && (G.block == 64 || G.block == 128);
        if (!ok_shape)
            return fail(SPARSP_E_UNSUPPORTED,
                        "bf16 attention needs d and block in {64, 128} (d=%d block=%d)", G.d,
                        G.block);
    } else if (G.d > 128 || G.block > 256) {
        return fail(SPARSP_E_UNSUPPORTED, "f32 attention needs d <= 128 and block <= 256");
    }
    return SPARSP_OK;
}

// A shard [kv_lo, kv_hi) of blocks and a run [h_lo, h_hi) of heads.
int check_part(const sparsp::Geom& G, int kv_lo, int kv_hi, int h_lo, int h_hi) {
    if (kv_lo < 0 || kv_hi > G.n || kv_lo > kv_hi)
        return fail(SPARSP_E_INVALID, "block range [%d, %d) not inside [0, %d]", kv_lo, kv_hi, G.n);
    if (h_lo < 0 || h_hi > G.H || h_lo >= h_hi)
        return fail(SPARSP_E_INVALID, "head range [%d, %d) not inside [0, %d) or empty", h_lo,
                    h_hi, G.H);
    return SPARSP_OK;
}

// How the bf16 launch may split the rows of its last round: not at all, into
// a caller workspace, or into the library's fixed scratch array.
enum class TailSpace { kNone, kWorkspace, kScratch };

int attn_whole(const sparsp_geom* g, const void* Q, const int32_t* sel, int32_t keep,
               const int32_t* slot_of, const void* K_packed, const void* V_packed,
               int64_t capacity_blocks, float softmax_scale, const int32_t* order, void* O,
               int32_t out_dtype, float* lse, void* stream, const char* what,
               void* workspace = nullptr, int64_t workspace_bytes = 0,
               TailSpace tail = TailSpace::kNone) {
    sparsp::Geom G;
    if (int rc = derive(g, &G)) return rc;
    if (!O) return fail(SPARSP_E_INVALID, "NULL tensor pointer");
    if (int rc = check_attn(G, Q, sel, keep, slot_of, K_packed, V_packed, capacity_blocks,
                            softmax_scale))
        return rc;
    if (!aligned16(O)) return fail(SPARSP_E_INVALID, "O must be 16-byte aligned");
    if (out_dtype != SPARSP_F32 && out_dtype != SPARSP_BF16)
        return fail(SPARSP_E_DTYPE, "unknown out_dtype %d", out_dtype);
    if (!G.bf16 && out_dtype != SPARSP_F32)
        return fail(SPARSP_E_DTYPE, "f32 inputs produce f32 output only");
    sparsp::AttnPart whole{0, G.n, 0, G.H, 0};
    whole.order = order;
    if (tail == TailSpace::kWorkspace && workspace && workspace_bytes > 0) {
        if (!aligned16(workspace)) return fail(SPARSP_E_INVALID, "workspace must be 16-byte aligned");
        whole.ws = workspace;
        whole.ws_bytes = workspace_bytes;
    }
    hipStream_t s = (hipStream_t)stream;
    if (tail == TailSpace::kScratch && G.bf16) {
        const int64_t need = sparsp::attn_tail_workspace_bytes(G, keep);
        if (need > sparsp::kScratchBytes)
            return fail(SPARSP_E_CAPACITY,
                        "%s: the tail split needs %lld bytes, the fixed scratch holds %lld", what,
                        (long long)need, (long long)sparsp::kScratchBytes);
        return hip_status(sparsp::launch_attn_bf16_noalloc(G, Q, sel, keep, slot_of, K_packed,
                                                           V_packed, capacity_blocks,
                                                           softmax_scale, O,
                                                           out_dtype == SPARSP_BF16, lse, s),
                          what);
    }
    hipError_t e =
        G.bf16 ? sparsp::launch_attn_bf16(G, Q, sel, keep, slot_of, K_packed, V_packed,
                                          capacity_blocks, softmax_scale, whole, O,
                                          out_dtype == SPARSP_BF16, lse, s)
               : sparsp::launch_attn_f32(G, (const float*)Q, sel, keep, slot_of,
                                         (const float*)K_packed, (const float*)V_packed,
                                         capacity_blocks, softmax_scale, whole, (float*)O, lse, s);
    return hip_status(e, what);
}

}  // namespace

extern "C" {

int sparsp_version(void) { return 200; }  // 0.2.0

const char* sparsp_last_error(void) { return g_err; }

int sparsp_block_scores(const sparsp_geom* g, const void* Q, const void* K, float* pooled_q,
                        float* pooled_k, float* scores, void* stream) {
    sparsp::Geom G;
    if (int rc = derive(g, &G)) return rc;
    if (!Q || !K || !pooled_q || !pooled_k || !scores)
        return fail(SPARSP_E_INVALID, "NULL tensor pointer");
    if (!aligned16(Q) || !aligned16(K))
        return fail(SPARSP_E_INVALID, "Q and K must be 16-byte aligned");
    if (G.block > 4096) return fail(SPARSP_E_UNSUPPORTED, "block %d exceeds 4096", G.block);
    hipError_t e = sparsp::launch_pool_scores(G, Q, K, pooled_q, pooled_k, scores,
                                              (hipStream_t)stream);
    return hip_status(e, "sparsp_block_scores");
}

int sparsp_topk_mask(const sparsp_geom* g, const float* scores, int32_t keep,
                     const int32_t* global_blocks, int32_t n_global, uint64_t* mask, int32_t* sel,
                     void* stream) {
    sparsp::Geom G;
    if (int rc = derive(g, &G)) return rc;
    if (!scores || !mask || !sel) return fail(SPARSP_E_INVALID, "NULL tensor pointer");
    sparsp::GlobalSet gs;
    if (int rc = global_set(G, global_blocks, n_global, &gs)) return rc;
    if (keep > G.n) return fail(SPARSP_E_INVALID, "keep = %d exceeds n = %d", keep, G.n);
    // |F_i| = |G| + (i not in G); the largest over local rows bounds keep from below.
    int max_forced = gs.count;
    for (int i = G.i0; i < G.i1; ++i)
        if (!((gs.w[i >> 6] >> (i & 63)) & 1)) { max_forced = gs.count + 1; break; }
    if (keep < max_forced)
        return fail(SPARSP_E_INVALID, "keep = %d is smaller than the forced set (%d blocks)", keep,
                    max_forced);
    hipError_t e = sparsp::launch_topk(G, scores, keep, gs, mask, sel, (hipStream_t)stream);
    return hip_status(e, "sparsp_topk_mask");
}

int sparsp_cdf_mask(const sparsp_geom* g, const float* scores, float tau,
                    const int32_t* global_blocks, int32_t n_global, uint64_t* mask, int32_t* sel,
                    int32_t* counts, void* stream) {
    sparsp::Geom G;
    if (int rc = derive(g, &G)) return rc;
    if (!scores || !mask || !sel || !counts) return fail(SPARSP_E_INVALID, "NULL tensor pointer");
    if (!(tau > 0.0f && tau <= 1.0f)) return fail(SPARSP_E_INVALID, "tau must be in (0, 1]");
    sparsp::GlobalSet gs;
    if (int rc = global_set(G, global_blocks, n_global, &gs)) return rc;
    hipError_t e = sparsp::launch_cdf(G, scores, tau, gs, mask, sel, counts, (hipStream_t)stream);
    return hip_status(e, "sparsp_cdf_mask");
}

int sparsp_demand_union_gather(const sparsp_geom* g, const uint64_t* mask, const void* K,
                               const void* V, uint64_t* demand, int32_t* head_off,
                               int32_t* slot_of, int32_t* gather_blk, void* K_packed,
                               void* V_packed, int64_t capacity_blocks, void* stream) {
    sparsp::Geom G;
    if (int rc = derive(g, &G)) return rc;
    if (!mask || !K || !V || !demand || !head_off || !slot_of || !gather_blk || !K_packed ||
        !V_packed)
        return fail(SPARSP_E_INVALID, "NULL tensor pointer");
    if (int rc = check_chunked(G)) return rc;
    if (G.block > 4096) return fail(SPARSP_E_UNSUPPORTED, "block %d exceeds 4096", G.block);
    if (!aligned16(K) || !aligned16(V) || !aligned16(K_packed) || !aligned16(V_packed))
        return fail(SPARSP_E_INVALID, "K, V and the packed buffers must be 16-byte aligned");
    const int64_t need = int64_t(G.H) * G.n;
    if (capacity_blocks < need)
        return fail(SPARSP_E_CAPACITY, "capacity_blocks = %lld < H*n = %lld",
                    (long long)capacity_blocks, (long long)need);
    hipError_t e = sparsp::launch_demand_gather(G, mask, K, V, demand, head_off, slot_of,
                                                gather_blk, K_packed, V_packed, (hipStream_t)stream);
    return hip_status(e, "sparsp_demand_union_gather");
}


int sparsp_block_sparse_attn(const sparsp_geom* g, const void* Q, const int32_t* sel, int32_t keep,
                             const int32_t* slot_of, const void* K_packed, const void* V_packed,
                             int64_t capacity_blocks, float softmax_scale, void* O,
                             int32_t out_dtype, float* lse, void* stream) {
    return attn_whole(g, Q, sel, keep, slot_of, K_packed, V_packed, capacity_blocks,
                      softmax_scale, nullptr, O, out_dtype, lse, stream,
                      "sparsp_block_sparse_attn");
}

int64_t sparsp_attn_workspace_bytes(const sparsp_geom* g, int32_t keep) {
    sparsp::Geom G;
    if (int rc = derive(g, &G)) return rc;
    if (keep < 1 || keep > G.n)
        return fail(SPARSP_E_INVALID, "keep = %d outside [1, n = %d]", keep, G.n);
    ok();
    if (!G.bf16) return 0;
    const bool shape = (G.d == 64 || G.d == 128) && (G.block == 64 || G.block == 128);
    return shape ? sparsp::attn_tail_workspace_bytes(G, keep) : 0;
}

int sparsp_block_sparse_attn_balanced(const sparsp_geom* g, const void* Q, const int32_t* sel,
                                      int32_t keep, const int32_t* slot_of, const void* K_packed,
                                      const void* V_packed, int64_t capacity_blocks,
                                      float softmax_scale, void* workspace,
                                      int64_t workspace_bytes, void* O, int32_t out_dtype,
                                      float* lse, void* stream) {
    if (workspace_bytes < 0) return fail(SPARSP_E_INVALID, "workspace_bytes < 0");
    return attn_whole(g, Q, sel, keep, slot_of, K_packed, V_packed, capacity_blocks,
                      softmax_scale, nullptr, O, out_dtype, lse, stream,
                      "sparsp_block_sparse_attn_balanced", workspace, workspace_bytes,
                      TailSpace::kWorkspace);
}

int sparsp_block_sparse_attn_balanced_noalloc(const sparsp_geom* g, const void* Q,
                                              const int32_t* sel, int32_t keep,
                                              const int32_t* slot_of, const void* K_packed,
                                              const void* V_packed, int64_t capacity_blocks,
                                              float softmax_scale, void* O, int32_t out_dtype,
                                              float* lse, void* stream) {
    return attn_whole(g, Q, sel, keep, slot_of, K_packed, V_packed, capacity_blocks,
                      softmax_scale, nullptr, O, out_dtype, lse, stream,
                      "sparsp_block_sparse_attn_balanced_noalloc", nullptr, 0,
                      TailSpace::kScratch);
}

int sparsp_block_sparse_attn_ordered(const sparsp_geom* g, const void* Q, const int32_t* sel,
                                     int32_t keep, const int32_t* slot_of, const void* K_packed,
                                     const void* V_packed, int64_t capacity_blocks,
                                     float softmax_scale, const int32_t* row_order, void* O,
                                     int32_t out_dtype, float* lse, void* stream) {
    if (!row_order) return fail(SPARSP_E_INVALID, "row_order is NULL");
    return attn_whole(g, Q, sel, keep, slot_of, K_packed, V_packed, capacity_blocks,
                      softmax_scale, row_order, O, out_dtype, lse, stream,
                      "sparsp_block_sparse_attn_ordered");
}

int sparsp_row_order(const sparsp_geom* g, const int32_t* counts, int32_t* order, void* stream) {
    sparsp::Geom G;
    if (int rc = derive(g, &G)) return rc;
    if (!counts || !order) return fail(SPARSP_E_INVALID, "NULL tensor pointer");
    return hip_status(sparsp::launch_row_order(counts, G.H, G.nq, G.n, order, (hipStream_t)stream),
                      "sparsp_row_order");
}

int sparsp_chunk_plan(const sparsp_geom* g, const uint64_t* demand, int32_t ranks, int32_t rank,
                      int32_t heads_per_chunk, int32_t tail_heads_per_chunk, sparsp_chunk* chunks,
                      int32_t max_chunks) {
    sparsp::Geom G;
    if (int rc = derive(g, &G)) return rc;
    if (!demand || !chunks) return fail(SPARSP_E_INVALID, "NULL pointer");
    if (ranks < 1 || ranks > G.n)
        return fail(SPARSP_E_INVALID, "ranks = %d outside [1, n = %d]", ranks, G.n);
    if (rank < 0 || rank >= ranks)
        return fail(SPARSP_E_INVALID, "rank = %d outside [0, %d)", rank, ranks);
    if (heads_per_chunk < 1 || tail_heads_per_chunk < 1)
        return fail(SPARSP_E_INVALID, "chunk sizes must be at least one head");
    if (max_chunks < 0) return fail(SPARSP_E_INVALID, "max_chunks < 0");
    const int r = sparsp::plan_chunks(G, demand, ranks, rank, heads_per_chunk,
                                      tail_heads_per_chunk, chunks, max_chunks);
    if (r < 0)
        return fail(SPARSP_E_CAPACITY, "the schedule has %d chunks, max_chunks = %d", -r,
                    max_chunks);
    ok();
    return r;
}

int sparsp_block_sparse_attn_part(const sparsp_geom* g, const void* Q, const int32_t* sel,
                                  int32_t keep, const int32_t* slot_of, const void* K_packed,
                                  const void* V_packed, int64_t capacity_blocks,
                                  float softmax_scale, int32_t kv_blk_begin, int32_t kv_blk_end,
                                  int32_t head_begin, int32_t head_end, float* O, float* lse,
                                  int32_t accumulate, void* stream) {
    sparsp::Geom G;
    if (int rc = derive(g, &G)) return rc;
    if (!O || !lse) return fail(SPARSP_E_INVALID, "NULL tensor pointer");
    if (int rc = check_attn(G, Q, sel, keep, slot_of, K_packed, V_packed, capacity_blocks,
                            softmax_scale))
        return rc;
    if (int rc = check_part(G, kv_blk_begin, kv_blk_end, head_begin, head_end)) return rc;
    if (!aligned16(O)) return fail(SPARSP_E_INVALID, "O must be 16-byte aligned");
    const sparsp::AttnPart part{kv_blk_begin, kv_blk_end, head_begin, head_end,
                                accumulate ? 1 : 0};
    hipStream_t s = (hipStream_t)stream;
    hipError_t e =
        G.bf16 ? sparsp::launch_attn_bf16(G, Q, sel, keep, slot_of, K_packed, V_packed,
                                          capacity_blocks, softmax_scale, part, O, false, lse, s)
               : sparsp::launch_attn_f32(G, (const float*)Q, sel, keep, slot_of,
                                         (const float*)K_packed, (const float*)V_packed,
                                         capacity_blocks, softmax_scale, part, O, lse, s);
    return hip_status(e, "sparsp_block_sparse_attn_part");
}

int sparsp_lse_merge(const sparsp_geom* g, int32_t head_begin, int32_t head_end, float* O_acc,
                     float* lse_acc, const float* O_part, const float* lse_part, void* stream) {
    sparsp::Geom G;
    if (int rc = derive(g, &G)) return rc;
    if (!O_acc || !lse_acc || !O_part || !lse_part)
        return fail(SPARSP_E_INVALID, "NULL tensor pointer");
    if (int rc = check_part(G, 0, G.n, head_begin, head_end)) return rc;
    if (G.d % 4) return fail(SPARSP_E_UNSUPPORTED, "d = %d must be a multiple of 4", G.d);
    if (!aligned16(O_acc) || !aligned16(O_part))
        return fail(SPARSP_E_INVALID, "O_acc and O_part must be 16-byte aligned");
    if (O_acc == O_part || lse_acc == lse_part)
        return fail(SPARSP_E_INVALID, "the part may not alias the accumulator");
    hipError_t e = sparsp::launch_lse_merge(G, head_begin, head_end, O_acc, lse_acc, O_part,
                                            lse_part, (hipStream_t)stream);
    return hip_status(e, "sparsp_lse_merge");
}

int sparsp_chunked_attn(const sparsp_geom* g, const void* Q, const int32_t* sel, int32_t keep,
                        const int32_t* slot_of, const void* K_packed, const void* V_packed,
                        int64_t capacity_blocks, float softmax_scale, const sparsp_chunk* plan,
                        int32_t n_chunks, float* O, float* lse, void* stream) {
    sparsp::Geom G;
    if (int rc = derive(g, &G)) return rc;
    if (!O || !lse || (n_chunks > 0 && !plan)) return fail(SPARSP_E_INVALID, "NULL pointer");
    if (n_chunks < 0) return fail(SPARSP_E_INVALID, "n_chunks < 0");
    if (int rc = check_attn(G, Q, sel, keep, slot_of, K_packed, V_packed, capacity_blocks,
                            softmax_scale))
        return rc;
    for (int c = 0; c < n_chunks; ++c)
        if (int rc = check_part(G, plan[c].kv_blk_begin, plan[c].kv_blk_end, plan[c].head_begin,
                                plan[c].head_end))
            return rc;
    if (!aligned16(O)) return fail(SPARSP_E_INVALID, "O must be 16-byte aligned");
    hipError_t e = sparsp::run_chunks(G, Q, sel, keep, slot_of, K_packed, V_packed,
                                      capacity_blocks, softmax_scale, plan, n_chunks, O, lse,
                                      (hipStream_t)stream);
    return hip_status(e, "sparsp_chunked_attn");
}

int sparsp_periodic_placement(int32_t L, int32_t block, int32_t frame_tokens, int32_t ranks,
                              int32_t* perm, int32_t* rank_begin) {
    if (!perm || !rank_begin) return fail(SPARSP_E_INVALID, "NULL pointer");
    if (L <= 0 || block <= 0 || frame_tokens <= 0 || ranks <= 0)
        return fail(SPARSP_E_INVALID, "L, block, frame_tokens and ranks must be positive");
    const int64_t n = (int64_t(L) + block - 1) / block;
    if (n > sparsp::kMaxBlocks)
        return fail(SPARSP_E_UNSUPPORTED, "n = %lld blocks exceeds %d", (long long)n,
                    sparsp::kMaxBlocks);
    if (ranks > n) return fail(SPARSP_E_INVALID, "ranks = %d exceeds n = %lld", ranks, (long long)n);
    sparsp::periodic_placement(L, block, frame_tokens, ranks, perm, rank_begin);
    return ok();
}

int sparsp_permute_blocks(const sparsp_geom* g, const int32_t* perm, const void* X, void* Y,
                          int32_t inverse, void* stream) {
    sparsp::Geom G;
    if (int rc = derive(g, &G)) return rc;
    if (!perm || !X || !Y) return fail(SPARSP_E_INVALID, "NULL tensor pointer");
    if (X == Y) return fail(SPARSP_E_INVALID, "X and Y must not overlap");
    if (!aligned16(X) || !aligned16(Y))
        return fail(SPARSP_E_INVALID, "X and Y must be 16-byte aligned");
    hipError_t e = sparsp::launch_permute(G, perm, X, Y, inverse != 0, (hipStream_t)stream);
    return hip_status(e, "sparsp_permute_blocks");
}

int sparsp_remote_demand(const sparsp_geom* g, const uint64_t* demand, int64_t* remote,
                         int64_t* demanded) {
    sparsp::Geom G;
    if (int rc = derive(g, &G)) return rc;
    if (!demand || !remote || !demanded) return fail(SPARSP_E_INVALID, "NULL pointer");
    sparsp::remote_demand(G, demand, remote, demanded);
    return ok();
}

int sparsp_pack_for_consumers(const sparsp_geom* g, const uint64_t* demands, int32_t ranks,
                              int32_t producer, const void* K, const void* V, uint64_t* provide,
                              int32_t* head_off, int32_t* slot_of, int32_t* gather_blk,
                              void* K_packed, void* V_packed, int64_t capacity_blocks,
                              void* stream) {
    sparsp::Geom G;
    if (int rc = derive(g, &G)) return rc;
    if (!demands || !K || !V || !provide || !head_off || !slot_of || !gather_blk || !K_packed ||
        !V_packed)
        return fail(SPARSP_E_INVALID, "NULL tensor pointer");
    if (ranks < 2 || ranks > G.n)
        return fail(SPARSP_E_INVALID, "ranks = %d outside [2, n = %d]", ranks, G.n);
    if (producer < 0 || producer >= ranks)
        return fail(SPARSP_E_INVALID, "producer = %d outside [0, %d)", producer, ranks);
    if (int64_t(ranks - 1) * G.H > sparsp::kMaxHeads)
        return fail(SPARSP_E_UNSUPPORTED, "(ranks-1) * H = %lld exceeds %d",
                    (long long)(int64_t(ranks - 1) * G.H), sparsp::kMaxHeads);
    if (int rc = check_chunked(G)) return rc;
    if (G.block > 4096) return fail(SPARSP_E_UNSUPPORTED, "block %d exceeds 4096", G.block);
    if (!aligned16(K) || !aligned16(V) || !aligned16(K_packed) || !aligned16(V_packed))
        return fail(SPARSP_E_INVALID, "K, V and the packed buffers must be 16-byte aligned");
    const int lo = int(int64_t(producer) * G.n / ranks), hi = int(int64_t(producer + 1) * G.n / ranks);
    const int64_t need = int64_t(ranks - 1) * G.H * (hi - lo);
    if (capacity_blocks < need)
        return fail(SPARSP_E_CAPACITY, "capacity_blocks = %lld < %lld", (long long)capacity_blocks,
                    (long long)need);
    hipError_t e = sparsp::launch_pack_for_consumers(G, demands, ranks, producer, lo, hi, K, V,
                                                     provide, head_off, slot_of, gather_blk,
                                                     K_packed, V_packed, (hipStream_t)stream);
    return hip_status(e, "sparsp_pack_for_consumers");
}

int sparsp_route_volume(const sparsp_geom* g, const uint64_t* demands, int32_t ranks,
                        int32_t producer, int64_t* dense, int64_t* relay, int64_t* direct) {
    sparsp::Geom G;
    if (int rc = derive(g, &G)) return rc;
    if (!demands || !dense || !relay || !direct) return fail(SPARSP_E_INVALID, "NULL pointer");
    if (ranks < 2 || ranks > G.n)
        return fail(SPARSP_E_INVALID, "ranks = %d outside [2, n = %d]", ranks, G.n);
    if (producer < 0 || producer >= ranks)
        return fail(SPARSP_E_INVALID, "producer = %d outside [0, %d)", producer, ranks);
    sparsp::route_volume(G, demands, ranks, producer, dense, relay, direct);
    return ok();
}

}  // extern "C"
