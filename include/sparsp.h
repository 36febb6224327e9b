/*
 * sparsp.h - C ABI of the MI355X (gfx950) library for one rank's share of
 * SparSP sparse sequence-parallel attention (arXiv 2609.32197).
 *
 * The four calls are the four steps of the per-rank hot path:
 *
 *   sparsp_block_scores        pool Q and K per token block, score block pairs
 *                              (Section 4.2: the mask comes from pooled tiles)
 *   sparsp_topk_mask           block mask M[h,i,j] (Section 4.1) by top-k per
 *                              query block, diagonal and global blocks forced
 *   sparsp_demand_union_gather per-head demand union (Eq. 2, Section 5.2) and
 *                              row-major compaction of the demanded K/V blocks
 *   sparsp_block_sparse_attn   attention (Eq. 1) of the local query blocks over
 *                              their kept blocks, read from the packed buffers
 *
 * Conventions shared by every call
 * --------------------------------
 * - Tensors are DEVICE pointers owned by the caller. The library allocates
 *   nothing, keeps no state between calls (except a per-thread error string)
 *   and never synchronizes: work is enqueued on `stream` (a hipStream_t passed
 *   as void*, NULL meaning the default stream) and completes in stream order.
 * - Q, K, V are [H, L, d] row-major with d contiguous, either float32 or
 *   bfloat16 (geom.dtype). Tokens are cut into n = ceil(L / block) blocks;
 *   block j covers tokens [j*block, min((j+1)*block, L)).
 * - The local query blocks are the global block indices [q_blk_begin,
 *   q_blk_end); nq = q_blk_end - q_blk_begin. W = ceil(n / 64).
 * - Block masks are bitsets: bit (j % 64) of 64-bit word (j / 64) is block j.
 * - Every call returns SPARSP_OK (0) or a negative sparsp_status. Argument
 *   errors are found on the host before anything is launched, so a failing
 *   call leaves every output untouched. SPARSP_E_HIP reports a launch error;
 *   sparsp_last_error() gives the message of the calling thread's last error.
 * - Indices are int32; byte offsets are computed in 64-bit inside the library.
 * - Limits: n <= 4096 blocks; H <= 1024; d <= 256; block <= 4096; d must be
 *   a multiple of 8 (bf16) or 4 (f32), and so must block for the packed-block
 *   calls; bf16 attention needs d and block in {64, 128}; f32 attention needs
 *   d <= 128 and block <= 256.
 */
#ifndef SPARSP_H
#define SPARSP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    SPARSP_OK = 0,
    SPARSP_E_INVALID = -1,     /* bad geometry, NULL pointer, out-of-range value */
    SPARSP_E_DTYPE = -2,       /* unknown or mismatched element type */
    SPARSP_E_UNSUPPORTED = -3, /* valid but outside the compiled kernel variants */
    SPARSP_E_CAPACITY = -4,    /* packed buffers smaller than H * n blocks */
    SPARSP_E_HIP = -5          /* the HIP runtime reported a launch error */
} sparsp_status;

typedef enum { SPARSP_F32 = 0, SPARSP_BF16 = 1 } sparsp_dtype;

/* Geometry of one rank's share. */
typedef struct {
    int32_t H;           /* heads */
    int32_t L;           /* tokens per head (the whole sequence) */
    int32_t d;           /* head dimension */
    int32_t block;       /* tokens per block, b */
    int32_t q_blk_begin; /* first local query block (global index), i0 */
    int32_t q_blk_end;   /* one past the last local query block, i1 */
    int32_t dtype;       /* sparsp_dtype of Q, K, V */
} sparsp_geom;

/*
 * Step 1 - pooled tiles and block scores (Section 4.2; mask M of Section 4.1).
 *
 *   pooled_q[h,i,:] = mean of Q[h,t,:] over the valid tokens t of block i0+i
 *   pooled_k[h,j,:] = mean of K[h,t,:] over the valid tokens t of block j
 *   scores[h,i,j]   = <pooled_q[h,i,:], pooled_k[h,j,:]> * d^-1/2
 *
 * Q, K: [H, L, d] in geom.dtype (only the local blocks of Q are read).
 * pooled_q: float32 [H, nq, d]; pooled_k: float32 [H, n, d]; both are written
 * (they are outputs, and the working storage of the score step).
 * scores: float32 [H, nq, n]. Sums are accumulated in float32.
 */
int sparsp_block_scores(const sparsp_geom* g, const void* Q, const void* K, float* pooled_q,
                        float* pooled_k, float* scores, void* stream);

/*
 * Step 2 - top-k block mask (Section 4.1's M).
 *
 * For local row i (global block i0+i) of head h, the forced set is
 * F = {i0+i} U global_blocks. The row keeps F and the first keep - |F| other
 * blocks ordered by score descending, then block index ascending. Scores are
 * compared as float32 values (+0.0 equals -0.0; infinities order as usual).
 * `keep` counts every kept block, forced ones included. A NaN score is outside
 * the contract: the device cannot report it without a host round trip, so the
 * call still writes a well-formed row of `keep` blocks, but which blocks is
 * unspecified.
 *
 * scores: float32 [H, nq, n] device. global_blocks: HOST array of n_global
 * block indices (may be NULL when n_global == 0; duplicates are ignored;
 * n_global <= 64). Outputs: mask uint64 [H, nq, W] (bits past n are zero) and
 * sel int32 [H, nq, keep], each row the kept block indices ascending.
 * Errors: keep > n, keep < |F| for some row, a global block outside [0, n).
 * The outputs are a pure function of the score bits.
 */
int sparsp_topk_mask(const sparsp_geom* g, const float* scores, int32_t keep,
                     const int32_t* global_blocks, int32_t n_global, uint64_t* mask,
                     int32_t* sel, void* stream);

/*
 * Step 2, CDF mode - the selection rule of the paper's evaluation (Section
 * 8.1): keep, per query block, the highest-scoring blocks until their
 * cumulative attention mass reaches tau.
 *
 * For local row i of head h: p_j = exp(S[h,i,j] - max_j S) / sum_j exp(...)
 * over all n blocks (float32); with the blocks ordered by score descending,
 * then index ascending, the row keeps the shortest prefix whose mass reaches
 * tau, plus F = {i0+i} U global_blocks. "Reaches tau" is decided on the mass
 * the prefix leaves out: at most (1 - tau) of the total, summed from the
 * left-out blocks themselves, so blocks far below the total still count;
 * tau = 1 keeps every block. Scores compare as in sparsp_topk_mask and must
 * be finite (an infinite or NaN score is outside the contract: the row is
 * well-formed, its cut unspecified).
 *
 * tau in (0, 1]. Outputs: mask uint64 [H, nq, W]; sel int32 [H, nq, n], each
 * row the kept blocks ascending then -1 (attention skips -1, so pass n as
 * `keep` with this sel); counts int32 [H, nq], the kept blocks per row.
 * Errors as for sparsp_topk_mask (no keep), and tau outside (0, 1].
 */
int sparsp_cdf_mask(const sparsp_geom* g, const float* scores, float tau,
                    const int32_t* global_blocks, int32_t n_global, uint64_t* mask, int32_t* sel,
                    int32_t* counts, void* stream);

/*
 * Step 3 - per-head demand union and compaction (Eq. 2 taken over all owners;
 * Section 5.2: per-head demand, row-major packing, locally derived offsets).
 *
 *   demand[h,:]  = OR over local rows i of mask[h,i,:]          uint64 [H, W]
 *   head_off     = exclusive scan of U_h = popcount(demand[h])  int32 [H+1]
 *   gather_blk   = each head's demanded blocks ascending, heads
 *                  concatenated (entries past head_off[H] untouched)
 *                                                               int32 [capacity]
 *   slot_of[h,j] = slot of block j of head h, or -1             int32 [H, n]
 *   K_packed[s]  = K[h, block gather_blk[s]] as [block, d]
 *   V_packed[s]  = V[h, block gather_blk[s]] TRANSPOSED, as [d, block]
 *
 * Token rows past L are zero in both packed buffers. Element type of K, V,
 * K_packed, V_packed is geom.dtype. capacity_blocks is the number of blocks the
 * packed buffers and gather_blk can hold; it must be at least H * n so that
 * the worst case fits without a host round trip (SPARSP_E_CAPACITY otherwise).
 */
int sparsp_demand_union_gather(const sparsp_geom* g, const uint64_t* mask, const void* K,
                               const void* V, uint64_t* demand, int32_t* head_off,
                               int32_t* slot_of, int32_t* gather_blk, void* K_packed,
                               void* V_packed, int64_t capacity_blocks, void* stream);

/*
 * Step 4 - block-sparse attention (Eq. 1 over the kept blocks; the softmax is
 * renormalised over the kept keys, online, in float32).
 *
 * For every valid local query token q of block i0+i, head h:
 *   T  = valid tokens of the blocks listed in sel[h,i,:]
 *   O[h, i*block + (q - (i0+i)*block), :] = sum_t softmax_t(Q[h,q]·K[h,t] * scale) V[h,t]
 *   lse[h, same row] = log sum_t exp(Q[h,q]·K[h,t] * scale)      (natural log)
 * Query rows past L get O = 0 and lse = -inf.
 *
 * Q: [H, L, d] in geom.dtype. sel: int32 [H, nq, keep]. slot_of: int32 [H, n].
 * K_packed [capacity, block, d] and V_packed [capacity, d, block] as written by
 * sparsp_demand_union_gather. O: [H, nq*block, d] of out_dtype (F32 always
 * allowed; BF16, rounded to nearest even, when geom.dtype is BF16).
 * lse: float32 [H, nq*block] or NULL. A sel entry outside [0, n), or whose
 * slot is -1 or >= capacity_blocks, is skipped (it contributes nothing).
 * bf16 inputs use bf16 matrix-core products with float32 accumulation.
 * Q, K_packed and V_packed must hold finite values: the bf16 kernels are
 * compiled without NaN semantics, so an infinite or NaN input gives
 * unspecified outputs for the rows it reaches (memory accesses stay in
 * bounds whatever the values).
 */
int sparsp_block_sparse_attn(const sparsp_geom* g, const void* Q, const int32_t* sel,
                             int32_t keep, const int32_t* slot_of, const void* K_packed,
                             const void* V_packed, int64_t capacity_blocks, float softmax_scale,
                             void* O, int32_t out_dtype, float* lse, void* stream);

/*
 * Bytes of device workspace that sparsp_block_sparse_attn_balanced can use for
 * this geometry and keep on the current device: the row order (4 bytes per
 * local row, padded to a multiple of 256), then one float32 partial block
 * (block x (d + 1) x 4 bytes) per workgroup the attention kernel keeps
 * resident at once. 0 when neither applies (float32 inputs). Returns the size
 * (>= 0) or a negative sparsp_status for a bad geometry or keep. Host only.
 */
int64_t sparsp_attn_workspace_bytes(const sparsp_geom* g, int32_t keep);

/*
 * sparsp_block_sparse_attn with a workspace that lets the workgroups share
 * the L2 better and the last round of workgroups fill the GPU.
 *   - Row order: the first 4 * H * nq bytes (padded to 256) receive, per head,
 *     the local rows ordered by their first kept block (sel[h, r, 0]; ties by
 *     row index), and the rows are launched in that order. The positions are
 *     dealt to the XCDs in contiguous ranges as in sparsp_block_sparse_attn,
 *     so the workgroups an XCD runs together walk overlapping, ascending tile
 *     sequences in step. A row's arithmetic does not depend on its position.
 * The launch runs one workgroup per local row: R = H*nq rows on the P
 * workgroups the device holds at once, so the last round (the last positions
 * of that order) has only S = R mod P rows and most of the GPU idles while they
 * run. With the rest of the workspace, each of those S rows is split into
 * k = min(4, P / S) workgroups,
 * each over a consecutive part of the row's kept blocks. The pieces write
 * float32 partials (O normalised by its own sum, and lse) to the workspace,
 * and a second kernel merges each row's pieces through the log-sum-exp: the
 * online-softmax merge of Section 2.3. k shrinks to fit workspace_bytes.
 *   - Rows outside the last round are computed exactly as by
 *     sparsp_block_sparse_attn, bit for bit; split rows differ from it by
 *     float32 rounding only.
 *   - workspace: caller-owned device memory, 16-byte aligned; contents on entry
 *     do not matter and on return are unspecified. Calls that share a workspace
 *     must not overlap. A workspace too small for the row order leaves the
 *     natural order; one too small for k = 2 after the row order, or S = 0,
 *     leaves no split. With workspace NULL or float32 inputs the call is
 *     exactly sparsp_block_sparse_attn.
 * Errors: those of sparsp_block_sparse_attn; SPARSP_E_INVALID for a
 * misaligned workspace or workspace_bytes < 0.
 */
int sparsp_block_sparse_attn_balanced(const sparsp_geom* g, const void* Q, const int32_t* sel,
                                      int32_t keep, const int32_t* slot_of, const void* K_packed,
                                      const void* V_packed, int64_t capacity_blocks,
                                      float softmax_scale, void* workspace,
                                      int64_t workspace_bytes, void* O, int32_t out_dtype,
                                      float* lse, void* stream);

/*
 * sparsp_block_sparse_attn_balanced for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the float32 partials of the split last-round rows go to a
 * fixed device array of the library instead of a caller workspace. The array
 * holds 36 MiB per GPU the library runs on and stays allocated until the
 * process ends; the call itself allocates and frees nothing.
 *   - Outputs are those of sparsp_block_sparse_attn_balanced with a workspace
 *     of sparsp_attn_workspace_bytes(g, keep) bytes, bit for bit.
 *   - Every call on a GPU shares that GPU's array. Calls that overlap on one
 *     GPU (different streams, or different host threads without ordering)
 *     race for it and must not be issued; stream-ordered calls are fine.
 * Errors: those of sparsp_block_sparse_attn; SPARSP_E_CAPACITY when the row
 * order and the tail split would need more than the fixed array
 * (sparsp_attn_workspace_bytes above 36 MiB: on a 256-CU part, more than
 * 983,040 local rows at d = 128 with 128-token blocks); SPARSP_E_HIP when the
 * array's device address cannot be obtained.
 */
int sparsp_block_sparse_attn_balanced_noalloc(const sparsp_geom* g, const void* Q,
                                              const int32_t* sel, int32_t keep,
                                              const int32_t* slot_of, const void* K_packed,
                                              const void* V_packed, int64_t capacity_blocks,
                                              float softmax_scale, void* O, int32_t out_dtype,
                                              float* lse, void* stream);

/*
 * Longest-first row order, for selections whose rows keep different numbers of
 * blocks (CDF mode, Section 8.1): a row whose kept list is several times the
 * mean otherwise starts late and sets the attention time alone.
 *
 * counts: int32 [H, nq], the kept blocks of each local row (as written by
 * sparsp_cdf_mask); a count outside [0, n] is clamped into it.
 * order: int32 [H * nq] out, a permutation of the rows h * nq + r for a
 * launch whose workgroup w runs on XCD w mod 8:
 *   - heads, by total count (largest first, then lower index), go to the
 *     least loaded of eight queues that still has room (H/8 heads each, the
 *     first H mod 8 queues one more), so a head's rows share one XCD's L2;
 *   - each queue's rows are sorted by count, largest first (rows of equal
 *     count in unspecified order);
 *   - the queues are interleaved round-robin: entry k of queue x is at
 *     position x + 8k while every queue is longer than k.
 * Device pointers; one workgroup on `stream`.
 */
int sparsp_row_order(const sparsp_geom* g, const int32_t* counts, int32_t* order, void* stream);

/*
 * sparsp_block_sparse_attn with the local rows launched in the order given by
 * row_order (int32 [H * nq], a permutation of 0 .. H*nq-1, device): workgroup w
 * computes row row_order[w], and consecutive workgroups go to different XCDs.
 * Every row's arithmetic is the same as in sparsp_block_sparse_attn, so the
 * outputs are identical bit for bit; only the schedule changes. Entries
 * outside [0, H*nq) are skipped, and rows missing from row_order are not
 * written. Errors: those of sparsp_block_sparse_attn, and a NULL row_order.
 */
int sparsp_block_sparse_attn_ordered(const sparsp_geom* g, const void* Q, const int32_t* sel,
                                     int32_t keep, const int32_t* slot_of, const void* K_packed,
                                     const void* V_packed, int64_t capacity_blocks,
                                     float softmax_scale, const int32_t* row_order, void* O,
                                     int32_t out_dtype, float* lse, void* stream);

/*
 * Shard-by-shard attention (Section 2.3: a rank attends to one owner's KV
 * shard at a time and folds the partial result in with the online softmax;
 * Section 7: shards are cut into chunks of heads and ordered to shorten the
 * pipeline tail). Owner p of R holds the blocks [floor(p n / R),
 * floor((p+1) n / R)). Chunk results are float32.
 */

/* One chunk of a schedule. */
typedef struct {
    int32_t owner;        /* rank that owns the shard */
    int32_t kv_blk_begin; /* the shard: blocks [kv_blk_begin, kv_blk_end) */
    int32_t kv_blk_end;
    int32_t head_begin;   /* the chunk's heads [head_begin, head_end) */
    int32_t head_end;
    int32_t blocks;       /* demanded blocks of those heads inside the shard */
} sparsp_chunk;

/*
 * The chunk schedule of rank `rank` of `ranks` (Section 7.1, Section 7.2):
 * the local shard first, whole (all heads); then the remote shards in ring
 * order rank+1, ..., rank+ranks-1 (mod ranks), each cut into runs of
 * heads_per_chunk consecutive heads, the last one into runs of
 * tail_heads_per_chunk heads; inside each remote shard the chunks run by
 * `blocks` descending, then head_begin ascending, so the sparsest chunk ends
 * the pipeline.
 *
 * demand: HOST uint64 [H, W] as written by sparsp_demand_union_gather (copy it
 * back first). chunks: HOST array of max_chunks entries. Returns the number of
 * chunks written (>= 1), SPARSP_E_CAPACITY if max_chunks is too small (the
 * message gives the count needed; 1 + (ranks-1) * ceil(H / min chunk size)
 * always suffices), or SPARSP_E_INVALID for ranks outside [1, n], rank
 * outside [0, ranks), a chunk size below 1 or a NULL pointer. Pure host code.
 */
int sparsp_chunk_plan(const sparsp_geom* g, const uint64_t* demand, int32_t ranks, int32_t rank,
                      int32_t heads_per_chunk, int32_t tail_heads_per_chunk, sparsp_chunk* chunks,
                      int32_t max_chunks);

/*
 * Attention of the local query blocks of heads [head_begin, head_end) over
 * the kept blocks that lie inside [kv_blk_begin, kv_blk_end) only: Step 4
 * restricted to one shard and one chunk of heads. The softmax and lse run over
 * those keys alone. Arguments as for sparsp_block_sparse_attn, except that O
 * is float32 [H, nq*block, d] and lse float32 [H, nq*block] is required; only
 * the rows of the chunk's heads are touched. 0 <= kv_blk_begin <= kv_blk_end
 * <= n and 0 <= head_begin < head_end <= H.
 *
 * accumulate == 0: (O, lse) are overwritten with the part's result; a row with
 * no kept key in the part gets O = 0, lse = -inf (the merge identity).
 * accumulate != 0: (O, lse) hold a running result (from an earlier call, or
 * O = 0 and lse = -inf) and the part is folded into it exactly as
 * sparsp_lse_merge would; rows with no kept key in the part are left as they
 * are, and query blocks with none are not read or written at all.
 */
int sparsp_block_sparse_attn_part(const sparsp_geom* g, const void* Q, const int32_t* sel,
                                  int32_t keep, const int32_t* slot_of, const void* K_packed,
                                  const void* V_packed, int64_t capacity_blocks,
                                  float softmax_scale, int32_t kv_blk_begin, int32_t kv_blk_end,
                                  int32_t head_begin, int32_t head_end, float* O, float* lse,
                                  int32_t accumulate, void* stream);

/*
 * Folds a part (O_part, lse_part) into the accumulator (O_acc, lse_acc), in
 * place, for the rows of heads [head_begin, head_end): with m the larger lse
 * and w = exp(lse - m) per side, O = (w_a O_a + w_b O_b) / (w_a + w_b) and
 * lse = m + log(w_a + w_b); a side with lse = -inf contributes nothing. All
 * four are float32, O [H, nq*block, d], lse [H, nq*block], 16-byte aligned;
 * the part may not alias the accumulator.
 */
int sparsp_lse_merge(const sparsp_geom* g, int32_t head_begin, int32_t head_end, float* O_acc,
                     float* lse_acc, const float* O_part, const float* lse_part, void* stream);

/*
 * Runs a schedule on `stream`, one attention launch per chunk in plan order: a
 * chunk whose heads have no result yet writes (O, lse) (accumulate = 0), every
 * other chunk is folded in (accumulate = 1); heads that no chunk covers end
 * with O = 0, lse = -inf. plan: HOST array of n_chunks chunks (each range
 * checked as above). O float32 [H, nq*block, d], lse float32 [H, nq*block].
 * Allocates nothing.
 */
int sparsp_chunked_attn(const sparsp_geom* g, const void* Q, const int32_t* sel, int32_t keep,
                        const int32_t* slot_of, const void* K_packed, const void* V_packed,
                        int64_t capacity_blocks, float softmax_scale, const sparsp_chunk* plan,
                        int32_t n_chunks, float* O, float* lse, void* stream);

/*
 * Dependency-aware placement (Section 4.3, Eq. 4): spatial interval
 * floor(G s / B) of every frame goes to the same rank. Block j (tokens in
 * frame-major raster order, F = frame_tokens per frame) goes to rank
 * floor(ranks * ((j * block) mod F) / F), which is Eq. 4 when F is a multiple
 * of block; a ragged last block stays last and belongs to the last rank. The
 * placed order lists rank 0's blocks in logical order, then rank 1's, ...
 *
 * Outputs (HOST): perm [n] with perm[k] = the logical block at placed position
 * k, and rank_begin [ranks + 1]: rank p holds placed blocks [rank_begin[p],
 * rank_begin[p+1]) (use them as q_blk_begin / q_blk_end of that rank's geometry
 * over placed tensors). Errors: non-positive sizes, ranks > n, NULL pointers.
 * Pure host code.
 */
int sparsp_periodic_placement(int32_t L, int32_t block, int32_t frame_tokens, int32_t ranks,
                              int32_t* perm, int32_t* rank_begin);

/*
 * Moves whole token blocks of X [H, L, d] (geom.dtype) into Y: Y block k =
 * X block perm[k] (inverse == 0, into placed order) or Y block perm[k] =
 * X block k (inverse != 0, back to logical order). perm: DEVICE int32 [n], a
 * permutation of [0, n) that keeps a ragged last block last (as
 * sparsp_periodic_placement returns); an entry outside [0, n) leaves its
 * destination block untouched, and blocks of unequal valid rows copy the
 * smaller count, so a malformed perm cannot make the kernel leave the tensors.
 * X and Y must not overlap and must be 16-byte aligned.
 */
int sparsp_permute_blocks(const sparsp_geom* g, const int32_t* perm, const void* X, void* Y,
                          int32_t inverse, void* stream);

/*
 * Eq. 3's block count for the rank whose own blocks are the geometry's
 * [q_blk_begin, q_blk_end) (in whatever layout, placed or contiguous, the
 * tensors are in): *remote = sum over heads of the demanded blocks outside that
 * range (sum_{p != r} |D_{r,h,p}|; times 2 * block * d * w it is V_r), and
 * *demanded = all demanded blocks (sum of U_h). demand: HOST uint64 [H, W] as
 * sparsp_demand_union_gather writes it. Pure host code.
 */
int sparsp_remote_demand(const sparsp_geom* g, const uint64_t* demand, int64_t* remote,
                         int64_t* demanded);

/*
 * Demand-directed KV routing, producer side (Section 5.1: each consumer gets
 * exactly the blocks it selected, directly; Section 5.2: per head, packed
 * row-major, offsets derivable from the shared mask on both ends).
 *
 * demands: DEVICE uint64 [ranks, H, W], rank c's demand bitset (the `demand`
 * output of sparsp_demand_union_gather for c's query blocks). The producer
 * owns the blocks [floor(producer n / ranks), floor((producer+1) n / ranks)).
 * Consumers c = producer+1, ..., producer+ranks-1 (mod ranks), in that ring
 * order, are packed one after another; within a consumer, head-major, block
 * ascending. With C = ranks - 1 and virtual head v = (distance - 1) * H + h:
 *   provide   uint64 [C*H, W]  consumer's demand cut to the producer's shard
 *   head_off  int32 [C*H + 1]  first slot of each (consumer, head) run
 *   slot_of   int32 [C*H, n]   slot of block j in run v, or -1
 *   gather_blk int32 [capacity] block of each slot
 *   K_packed [capacity, block, d], V_packed [capacity, d, block] (transposed)
 * Consumer c's blocks are slots [head_off[(k-1)*H], head_off[k*H]) for its
 * distance k; the consumer rebuilds the same offsets from its own demand. The
 * geometry's local range is not used (it must still be valid). capacity_blocks
 * must be at least C * H * (shard blocks). Errors: ranks outside [2, n],
 * producer outside [0, ranks), C * H > 1024, NULL or misaligned pointers.
 */
int sparsp_pack_for_consumers(const sparsp_geom* g, const uint64_t* demands, int32_t ranks,
                              int32_t producer, const void* K, const void* V, uint64_t* provide,
                              int32_t* head_off, int32_t* slot_of, int32_t* gather_blk,
                              void* K_packed, void* V_packed, int64_t capacity_blocks,
                              void* stream);

/*
 * Block transfers of the producer's shard to the other ranks (Section 5.1),
 * summed over heads, in block-hops: *dense = the whole shard over each of the
 * ranks-1 ring hops; *relay = ring forwarding of selected blocks only (hop k
 * carries what consumers at distance >= k need); *direct = each consumer's
 * own blocks once. Bytes are 2 * block * d * w per block-hop. demands: HOST
 * uint64 [ranks, H, W]. Pure host code.
 */
int sparsp_route_volume(const sparsp_geom* g, const uint64_t* demands, int32_t ranks,
                        int32_t producer, int64_t* dense, int64_t* relay, int64_t* direct);

/* Message of the calling thread's most recent error ("" if none). */
const char* sparsp_last_error(void);

/* Library version, major * 10000 + minor * 100 + patch. */
int sparsp_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SPARSP_H */
