// Host interface between the C ABI layer (api.cpp) and the HIP translation
// units that launch the kernels: derived geometry, limits and launcher
// declarations. It uses only the HIP runtime API's types (hipError_t,
// hipStream_t), no device code, so the ABI layer and the pure host planning
// code compile with a plain host compiler as well; every argument check of
// the ABI happens before any launcher is called.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include "../../include/sparsp.h"

namespace sparsp {

constexpr int kMaxBlocks = 4096;        // n limit: 64 mask words per row
constexpr int kMaxWords = kMaxBlocks / 64;
constexpr int kMaxGlobal = 64;          // global (always-kept) blocks per call
constexpr int kMaxHeads = 1024;         // H limit (head offsets are staged in LDS)

// Derived geometry, computed once on the host.
struct Geom {
    int H, L, d, block, i0, i1, n, nq, W;
    bool bf16;
};

// Forced global blocks as a bitset, passed by value as a kernel argument.
struct GlobalSet {
    uint64_t w[kMaxWords];
    int count;  // distinct global blocks
};

hipError_t launch_pool_scores(const Geom& g, const void* Q, const void* K, float* pooled_q,
                              float* pooled_k, float* scores, hipStream_t s);

hipError_t launch_topk(const Geom& g, const float* scores, int keep, const GlobalSet& gs,
                       uint64_t* mask, int32_t* sel, hipStream_t s);

hipError_t launch_cdf(const Geom& g, const float* scores, float tau, const GlobalSet& gs,
                      uint64_t* mask, int32_t* sel, int32_t* counts, hipStream_t s);

hipError_t launch_demand_gather(const Geom& g, const uint64_t* mask, const void* K, const void* V,
                                uint64_t* demand, int32_t* head_off, int32_t* slot_of,
                                int32_t* gather_blk, void* Kp, void* Vp, hipStream_t s);

// Which part of the attention a launch computes: the heads [h_lo, h_hi) and,
// of every kept list, only the blocks inside [kv_lo, kv_hi) (one owner's
// shard). The whole attention is {0, n, 0, H, 0}. With acc set, the float32
// (O, lse) already hold a running result and the part is folded into it
// through the log-sum-exp instead of overwriting it; rows without a kept key
// in the part are left untouched.
struct AttnPart {
    int kv_lo, kv_hi, h_lo, h_hi, acc;
    const int32_t* order = nullptr;  // workgroup w takes row order[w] (longest first), if set
    // Workspace for the tail split of the bf16 kernels (whole launches only):
    // the rows of the last, partial round of workgroups are split into pieces
    // whose float32 partials go here and are merged by a second kernel.
    void* ws = nullptr;
    int64_t ws_bytes = 0;
};

// Packed K/V copies of n_vheads virtual heads (virtual head v reads head v % g.H).
hipError_t launch_gather(const Geom& g, int n_vheads, const int32_t* head_off,
                         const int32_t* gather_blk, const void* K, const void* V, void* Kp,
                         void* Vp, hipStream_t s);

// Producer p's packing for every other rank (demands: device [ranks, H, W]).
hipError_t launch_pack_for_consumers(const Geom& g, const uint64_t* demands, int ranks,
                                     int producer, int lo, int hi, const void* K, const void* V,
                                     uint64_t* provide, int32_t* head_off, int32_t* slot_of,
                                     int32_t* gather_blk, void* Kp, void* Vp, hipStream_t s);

// Host: block-hops of producer p's shard under dense ring, relay and direct routing.
void route_volume(const Geom& g, const uint64_t* demands, int ranks, int producer, int64_t* dense,
                  int64_t* relay, int64_t* direct);

hipError_t launch_attn_bf16(const Geom& g, const void* Q, const int32_t* sel, int keep,
                            const int32_t* slot_of, const void* Kp, const void* Vp,
                            int64_t capacity, float scale, const AttnPart& part, void* O,
                            bool out_bf16, float* lse, hipStream_t s);

// Bytes of workspace the tail split of a bf16 attention launch can use (0
// when it does not apply): one float32 partial block per resident slot.
int64_t attn_tail_workspace_bytes(const Geom& g, int keep);

// Size of the fixed device array that the no-allocation attention entry point
// uses in place of a workspace (per GPU). 36 MiB holds the largest tail split
// of the supported shapes on a 256-CU part (512 slots x 128 x 129 x 4 bytes =
// 33.8 MB) plus the row order of up to 983,040 local rows.
constexpr int64_t kScratchBytes = int64_t(36) << 20;

// The bf16 attention of the whole geometry with the tail split's partials in
// that fixed array (the caller has checked attn_tail_workspace_bytes against
// kScratchBytes).
hipError_t launch_attn_bf16_noalloc(const Geom& g, const void* Q, const int32_t* sel, int keep,
                                    const int32_t* slot_of, const void* Kp, const void* Vp,
                                    int64_t capacity, float scale, void* O, bool out_bf16,
                                    float* lse, hipStream_t s);

hipError_t launch_attn_f32(const Geom& g, const float* Q, const int32_t* sel, int keep,
                           const int32_t* slot_of, const float* Kp, const float* Vp,
                           int64_t capacity, float scale, const AttnPart& part, float* O,
                           float* lse, hipStream_t s);

hipError_t launch_lse_merge(const Geom& g, int h_lo, int h_hi, float* O_acc, float* lse_acc,
                            const float* O_part, const float* lse_part, hipStream_t s);

hipError_t launch_fill_identity(float* O, float* lse, int64_t rows, int d, hipStream_t s);

// Host: the chunk schedule of rank `rank` (count of chunks written, or minus
// the count needed when it exceeds max_chunks). demand is host memory [H, W].
int plan_chunks(const Geom& g, const uint64_t* demand, int ranks, int rank, int heads_per_chunk,
                int tail_heads_per_chunk, sparsp_chunk* out, int max_chunks);

// Host: Eq. 4's placed order of the blocks (perm [n], rank_begin [ranks+1]).
void periodic_placement(int L, int block, int frame_tokens, int ranks, int32_t* perm,
                        int32_t* rank_begin);

hipError_t launch_permute(const Geom& g, const int32_t* perm, const void* X, void* Y, bool inverse,
                          hipStream_t s);

// Host: demanded blocks outside [i0, i1) and in total, over all heads.
void remote_demand(const Geom& g, const uint64_t* demand, int64_t* remote, int64_t* demanded);

// Host: runs a validated plan on stream s (one attention launch per chunk,
// folding into (O, lse)).
hipError_t run_chunks(const Geom& g, const void* Q, const int32_t* sel, int keep,
                      const int32_t* slot_of, const void* Kp, const void* Vp, int64_t capacity,
                      float scale, const sparsp_chunk* plan, int n_chunks, float* O, float* lse,
                      hipStream_t s);

// Rows (h * nq + r) on eight XCD queues by head, each queue longest first, interleaved.
hipError_t launch_row_order(const int32_t* counts, int H, int nq, int n, int32_t* order,
                            hipStream_t s);

}  // namespace sparsp
