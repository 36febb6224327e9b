// Step 4, bf16: block-sparse flash attention of the local query blocks over
// the packed K/V buffers (Eq. 1 over the kept blocks; softmax renormalised
// over the kept keys, computed online in float32).
//
// Two kernels, one workgroup per (head, local query block) in both; the
// block size picks the kernel.
//
// attn_rows_kernel (128-token blocks): four waves, wave w owns queries
// 32 w .. +31 against all 128 keys of every kept block; single K and V tile
// buffers (64 KB of LDS at d = 128), two workgroups per CU. The waves that
// share a SIMD come from different workgroups and are not tied by a barrier,
// so one wave's MFMAs overlap the other's softmax. The copy of the next
// block's K is issued once the scores of the current block are done, the
// next V once its output product is done.
//
// attn_bf16_kernel (64-token blocks): 2*BLK/32 waves: wave w owns query group
// w % (BLK/32) (32 queries) and key half w / (BLK/32) of every kept block
// (BLK/2 keys). Each wave runs its own online softmax over its key halves
// (running max, running sum, output accumulator) and the two halves of a
// query group are merged once at the end through their log-sum-exp, so waves
// never wait on each other inside a tile. Tiles are double-buffered: the copy
// of block jj+1 is issued right after the barrier that opens block jj and has
// the whole of block jj's compute to land. One barrier per block.
//
// Data movement (both). The kept blocks' K tile ([BLK, D]) and transposed V
// tile ([D, BLK]) are copied HBM -> LDS with direct-to-LDS buffer loads
// (buffer_load_dwordx4 ... lds); each wave waits for its own copies before the
// barrier that publishes them. The split-key kernel reads all MFMA operands
// of a phase from LDS up front (K before the score MFMAs, V^T before the
// softmax); the rows kernel reads them one k step ahead of the MFMAs that use
// them. LDS rows carry an XOR
// swizzle of their 16-byte chunks (applied through the source addresses of the
// copies) so the MFMA operand reads are bank-conflict free. Workgroup ids are
// remapped so that each of the eight XCDs walks a contiguous range of (head,
// query block): neighbouring query blocks select overlapping KV blocks, which
// then hit in that XCD's L2.
//
// Products use v_mfma_f32_32x32x16_bf16 with the score tile computed
// transposed, S^T = K Q^T (A = K from LDS, B = Q^T from registers):
//   * each lane holds one query column (q = lane % 32) and 16 keys per 32x32
//     tile, so the row max and row sum are in-lane except for one exchange
//     between lanes l and l^32;
//   * the output is accumulated transposed too, O^T = V^T P^T (A = V^T from
//     the transposed V tile, B = P^T): the B operand is exactly the lane's own
//     probabilities converted to bf16, no shuffles. For that to line up, the
//     lane that feeds A-row m of the K product reads key sigma(m), sigma
//     swapping bits 2 and 3 of m; then the 8 values a lane holds for each
//     16-key step of P^T are 8 consecutive keys.
// MFMA operand layout (32x32x16, wave64): A lane l holds row l%32, k values
// 8*(l/32) .. +7; B lane l holds column l%32, same k values; the 16 results
// of lane l are column l%32, rows 8*(r/4) + 4*(l/32) + r%4.
//
// The running max m moves (and the accumulator is rescaled) when some lane's
// block max exceeds it by more than a per-lane threshold t (log2 units). t is
// 8 at most, which keeps every probability below 2^8, and smaller while the
// mass the lane has accumulated is small: at each rescale, t = clamp(log2(l) -
// 2, 0, 8) for the lane's mass l (rescaled to the new max, before the block is
// added). A block whose top probability 2^(max - m) would carry more than a
// quarter of the accumulated mass therefore enters with its max exactly at m,
// i.e. probability exactly 1, which bf16 represents exactly. On peaked rows,
// where O is close to a few V rows, the bf16 rounding of those few
// probabilities would otherwise be the largest error of O. Between rescales l
// only grows, so t errs on the side of moving the max; on spread rows t
// reaches several units after the first blocks, and most blocks skip the
// rescale (and the logarithm, which only rescale blocks compute).
#include <type_traits>

#include "sparsp_internal.h"

namespace sparsp {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float floatx8 __attribute__((ext_vector_type(8)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kRescaleThreshold = 8.0f;  // log2 units

// The rescale threshold for a lane that has accumulated mass l (units of its
// running max): moving the max pays off once a block's top probability would
// exceed l / 4, and is forced beyond 2^8.
__device__ __forceinline__ float rescale_threshold(float l) {
    return fminf(kRescaleThreshold, fmaxf(0.f, __log2f(l) - 2.f));
}

__device__ __forceinline__ int sigma(int m) {  // swap bits 2 and 3
    return (m & ~0xC) | ((m & 4) << 1) | ((m & 8) >> 1);
}

// XOR swizzle of the 16-byte chunk index for a tile whose rows are COLS bf16
// wide: the 16 rows read together by one quarter-wave land on distinct banks.
template <int COLS>
__device__ __forceinline__ int swz(int row) {
    constexpr int NCH = COLS / 8;                          // chunks per row
    constexpr int RP = (128 / COLS) > 1 ? 128 / COLS : 1;  // rows per 256 bytes
    return (row / RP) & (NCH - 1);
}

// v_permlane32_swap with x in both operands returns, in lane l, the pair
// {x[l], x[l^32]} in some order; max and sum of the pair are the same in both
// lanes of the pair, bit for bit.
__device__ __forceinline__ float pair_max(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// XCD-aware row of workgroup index w: consecutive workgroups go to the eight
// XCDs in turn, so XCD x runs indices x, x+8, ...; they get the x-th
// contiguous range of rows, where neighbouring query blocks share KV blocks in
// that XCD's L2.
__device__ __forceinline__ int xcd_row(int w, int G) {
    const int xcd = w & 7, idx = w >> 3, per = G >> 3, rem = G & 7;
    return xcd * per + min(xcd, rem) + idx;
}

// With row_sort (the balanced launch), position k of head h's rows holds row
// row_sort[h * nq + k] of that head: the rows in the order of their first kept
// block, so that the workgroups an XCD runs together walk overlapping tile
// sequences in step and share more of its L2. Without it, positions are rows.
__device__ __forceinline__ int sorted_row(int p, int nq, const int32_t* row_sort) {
    if (!row_sort) return p;
    const int r = row_sort[p];
    return (p / nq) * nq + ((r >= 0 && r < nq) ? r : p % nq);
}

// Per head (one workgroup of 1024 threads): the local rows ordered by their
// first kept block (sel rows are ascending, so that is sel[h, r, 0]; a row
// whose list starts with -1 sorts last), ties by row index. row_sort[h * nq +
// k] is the row at position k. Each rank is a count of smaller keys, so the
// order is deterministic.
__global__ __launch_bounds__(1024) void row_sort_kernel(const int32_t* __restrict__ sel, int keep,
                                                        int nq, int n,
                                                        int32_t* __restrict__ row_sort) {
    __shared__ uint32_t key[kMaxBlocks];  // nq <= n <= kMaxBlocks
    const int h = blockIdx.x;
    const int32_t* srow = sel + int64_t(h) * nq * keep;
    for (int r = threadIdx.x; r < nq; r += 1024) {
        int j = srow[int64_t(r) * keep];
        if (j < 0 || j >= n) j = n;
        key[r] = uint32_t(j) * uint32_t(kMaxBlocks) + uint32_t(r);  // unique per row
    }
    __syncthreads();
    for (int r = threadIdx.x; r < nq; r += 1024) {
        const uint32_t mine = key[r];
        int rank = 0;
        for (int q = 0; q < nq; ++q) rank += key[q] < mine;
        row_sort[int64_t(h) * nq + rank] = r;
    }
}

// Bytes of the row order at the start of a balanced launch's workspace.
int64_t row_sort_bytes(int rows) { return (int64_t(rows) * 4 + 255) / 256 * 256; }

// Tail split: the rows of the last, partial round of workgroups (indices
// tail_first .. G-1) run as tail_k workgroups each, so that round fills the
// GPU. Workgroup tail_first + t*tail_k + p is piece p of tail row t, which
// has index tail_first + t; index is the row index a workgroup works on.
struct TailPiece {
    int index, piece;
};
__device__ __forceinline__ TailPiece tail_piece(int w, int tail_first, int tail_k) {
    if (tail_k > 1 && w >= tail_first)
        return {tail_first + (w - tail_first) / tail_k, (w - tail_first) % tail_k};
    return {w, -1};
}

template <int D, int BLK>
struct Cfg {
    static constexpr int NQG = BLK / 32;          // query groups of 32
    static constexpr int NW = 2 * NQG;            // waves: query group x key half
    static constexpr int THREADS = 64 * NW;
    static constexpr int HALF = BLK / 2;          // keys per wave per block
    static constexpr int MTW = HALF / 32;         // 32-key tiles per wave
    static constexpr int KT = D / 16;             // k steps of the score product
    static constexpr int DT = D / 32;             // d tiles of the output product
    static constexpr int PTW = HALF / 16;         // k steps of the output product
    static constexpr int TILE = BLK * D;          // elements per K (or V) tile
    static constexpr int CHUNKS = TILE / 8;       // 16-byte chunks per tile
    static constexpr int DMA = CHUNKS / THREADS;  // copies per lane per tile
    static_assert(CHUNKS % THREADS == 0, "tile must split evenly");
    static_assert(4 * TILE * 2 >= NQG * 64 * (DT * 16 + 2) * 4, "merge area must fit");
};

typedef __attribute__((address_space(3))) void lds_void;

// s_waitcnt vmcnt(0), leaving the other counters alone (gfx9 encoding:
// vmcnt bits [3:0] and [15:14], expcnt [6:4], lgkmcnt [11:8]).
__device__ __forceinline__ void wait_vmem_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Byte offset, within a packed tile of rows COLS bf16 wide, of the 16-byte
// chunk that lands at LDS chunk position p: LDS row p/NCH, physical chunk
// p%NCH holds logical chunk (p%NCH) ^ swz(row). Constant for the whole
// kernel, so each lane computes its copy offsets once.
template <int COLS>
__device__ __forceinline__ int chunk_src_offset(int p) {
    constexpr int NCH = COLS / 8;
    const int row = p / NCH, pc = p % NCH;
    return (row * COLS + ((pc ^ swz<COLS>(row)) * 8)) * 2;
}

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

// Direct-to-LDS copy of one tile (buffer_load_dwordx4 ... lds) through a
// buffer descriptor rooted at the tile, 16 bytes per lane per instruction:
// the LDS destination of each instruction is this wave's 1 KB of the tile (in
// M0), the source a precomputed per-lane offset. Reads outside the tile return
// zero instead of faulting.
//
// The copies are issued as inline assembly on purpose. When the compiler
// sees direct-to-LDS loads it protects every later LDS read with a wait for
// all of them, which makes each block wait for the copy of the next one and
// undoes the double buffering. Issued this way they are invisible to it, and
// the only wait is the explicit vmcnt(0) that opens each block, which covers
// exactly the copies issued one block earlier. One assembly block issues all
// of a lane's copies of the tile, stepping M0 from one destination to the
// next; M0 is saved and restored around it, and one wait state separates
// each M0 write from its use.
template <int NW, int DMA>
__device__ __forceinline__ void copy_tile(const uint16_t* tile, int tile_bytes, uint16_t* dst,
                                          const int (&voff)[DMA], int wave) {
    static_assert(DMA == 2 || DMA == 4 || DMA == 8, "copies per lane per tile");
#if defined(__HIP_DEVICE_COMPILE__)
    const uint64_t b = reinterpret_cast<uint64_t>(tile);
    u32x4_t desc;
    desc.x = __builtin_amdgcn_readfirstlane(uint32_t(b));
    desc.y = __builtin_amdgcn_readfirstlane(uint32_t(b >> 32) & 0xffffu);  // stride 0
    desc.z = uint32_t(tile_bytes);                                         // num_records
    desc.w = 0x00020000u;
    // This wave's first 1 KB of the tile; its next ones follow every NW KB.
    const uint32_t lds = __builtin_amdgcn_readfirstlane(
        uint32_t(reinterpret_cast<uintptr_t>(dst + wave * 64 * 8)));
    constexpr uint32_t kStep = NW * 64 * 16;
    uint32_t saved;
#define SPARSP_COPY_HEAD "s_mov_b32 %[sv], m0\n\ts_mov_b32 m0, %[lds]\n\ts_nop 0\n\t"
#define SPARSP_COPY(o) "buffer_load_dwordx4 %[" #o "], %[desc], 0 offen lds\n\t"
#define SPARSP_STEP "s_add_u32 m0, m0, %[st]\n\ts_nop 0\n\t"
#define SPARSP_COPY_TAIL "s_mov_b32 m0, %[sv]"
    if constexpr (DMA == 2) {
        asm volatile(SPARSP_COPY_HEAD SPARSP_COPY(o0) SPARSP_STEP SPARSP_COPY(o1) SPARSP_COPY_TAIL
                     : [sv] "=&s"(saved)
                     : [lds] "s"(lds), [desc] "s"(desc), [st] "n"(kStep), [o0] "v"(voff[0]),
                       [o1] "v"(voff[1])
                     : "memory", "scc");
    } else if constexpr (DMA == 4) {
        asm volatile(SPARSP_COPY_HEAD SPARSP_COPY(o0) SPARSP_STEP SPARSP_COPY(o1) SPARSP_STEP
                         SPARSP_COPY(o2) SPARSP_STEP SPARSP_COPY(o3) SPARSP_COPY_TAIL
                     : [sv] "=&s"(saved)
                     : [lds] "s"(lds), [desc] "s"(desc), [st] "n"(kStep), [o0] "v"(voff[0]),
                       [o1] "v"(voff[1]), [o2] "v"(voff[2]), [o3] "v"(voff[3])
                     : "memory", "scc");
    } else {
        asm volatile(SPARSP_COPY_HEAD SPARSP_COPY(o0) SPARSP_STEP SPARSP_COPY(o1) SPARSP_STEP
                         SPARSP_COPY(o2) SPARSP_STEP SPARSP_COPY(o3) SPARSP_STEP SPARSP_COPY(o4)
                             SPARSP_STEP SPARSP_COPY(o5) SPARSP_STEP SPARSP_COPY(o6) SPARSP_STEP
                                 SPARSP_COPY(o7) SPARSP_COPY_TAIL
                     : [sv] "=&s"(saved)
                     : [lds] "s"(lds), [desc] "s"(desc), [st] "n"(kStep), [o0] "v"(voff[0]),
                       [o1] "v"(voff[1]), [o2] "v"(voff[2]), [o3] "v"(voff[3]),
                       [o4] "v"(voff[4]), [o5] "v"(voff[5]), [o6] "v"(voff[6]), [o7] "v"(voff[7])
                     : "memory", "scc");
    }
#undef SPARSP_COPY_HEAD
#undef SPARSP_COPY
#undef SPARSP_STEP
#undef SPARSP_COPY_TAIL
#endif
}

template <int D, int BLK, bool OUT_BF16>
__global__ __launch_bounds__(4 * BLK) __attribute__((amdgpu_waves_per_eu(2)))
void attn_bf16_kernel(const uint16_t* __restrict__ Q, const int32_t* __restrict__ sel,
                      const int32_t* __restrict__ slot_of, const uint16_t* __restrict__ Kp,
                      const uint16_t* __restrict__ Vp, void* __restrict__ O,
                      float* __restrict__ lse, int L, int n, int i0, int nq, int keep,
                      int64_t capacity, float c2 /* scale * log2(e) */, int kv_lo, int kv_hi,
                      int h_lo, int n_heads, int acc, int remap,
                      const int32_t* __restrict__ order, int tail_first, int tail_k,
                      float* __restrict__ part_o, float* __restrict__ part_lse,
                      const int32_t* __restrict__ row_sort) {
    using C = Cfg<D, BLK>;
    // [buffer][K tile | V tile]; reused for the final merge.
    __shared__ __attribute__((aligned(16))) uint16_t lds[2][2][C::TILE];
    // Per kept entry: 2 * slot + (block is the partial last one), or -1 to skip.
    extern __shared__ int32_t codes[];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int qi = lane & 31, g = lane >> 5;
    const int qg = wave % C::NQG, kh = wave / C::NQG;

    // Workgroup -> (head, local query block), XCD-contiguous when remap is on.
    const int G = n_heads * nq;
    int wg = blockIdx.x;
    const TailPiece tp = tail_piece(wg, tail_first, tail_k);
    if (order) {  // an explicit row order (e.g. longest first); no XCD remap
        wg = order[blockIdx.x];
        if (wg < 0 || wg >= G) return;
    } else if (remap) {
        wg = sorted_row(xcd_row(tp.index, G), nq, row_sort);
    } else {
        wg = tp.index;
    }
    const int h = h_lo + wg / nq, r = wg % nq;
    const int qtok = (i0 + r) * BLK + qg * 32 + qi;
    const bool qvalid = qtok < L;

    // Resolve the kept list once: sel -> slot (and partial-block flag), keeping
    // only the usable entries inside [kv_lo, kv_hi), compacted in list order.
    __shared__ int wave_cnt[C::NW];
    int nkeep = 0;
    {
        const int32_t* srow = sel + (int64_t(h) * nq + r) * keep;
        const int32_t* hslot = slot_of + int64_t(h) * n;
        const bool ragged = (L % BLK) != 0;
        for (int base = 0; base < keep; base += C::THREADS) {
            const int jj = base + tid;
            int code = -1;
            if (jj < keep) {
                const int j = srow[jj];
                if (j >= kv_lo && j < kv_hi && j >= 0 && j < n) {
                    const int sl = hslot[j];
                    if (sl >= 0 && sl < capacity && sl < (1 << 30))
                        code = 2 * sl + ((ragged && j == n - 1) ? 1 : 0);
                }
            }
            const uint64_t bal = __ballot(code >= 0);
            if (lane == 0) wave_cnt[wave] = __popcll(bal);
            __syncthreads();
            int off = nkeep, total = 0;
#pragma unroll
            for (int w = 0; w < C::NW; ++w) {
                off += w < wave ? wave_cnt[w] : 0;
                total += wave_cnt[w];
            }
            const int below = __builtin_amdgcn_mbcnt_hi(
                uint32_t(bal >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(bal), 0));
            if (code >= 0) codes[off + below] = code;
            nkeep += total;
            __syncthreads();  // wave_cnt is rewritten by the next round
        }
    }

    int kvoff[C::DMA], vvoff[C::DMA];
#pragma unroll
    for (int u = 0; u < C::DMA; ++u) {
        const int p = (u * C::NW + wave) * 64 + lane;
        kvoff[u] = chunk_src_offset<D>(p);
        vvoff[u] = chunk_src_offset<BLK>(p);
    }
    auto issue = [&](int code, int buf) {
        code = __builtin_amdgcn_readfirstlane(code);  // wave-uniform: scalar address arithmetic
        const int64_t off = int64_t(code < 0 ? 0 : (code >> 1)) * C::TILE;
        copy_tile<C::NW, C::DMA>(Kp + off, C::TILE * 2, &lds[buf][0][0], kvoff, wave);
        copy_tile<C::NW, C::DMA>(Vp + off, C::TILE * 2, &lds[buf][1][0], vvoff, wave);
    };

    // Q^T operand: lane holds Q[qtok][16 kt + 8 g .. +7] for every k step.
    bf16x8 qf[C::KT];
    {
        const uint16_t* qp = Q + (int64_t(h) * L + (qvalid ? qtok : 0)) * D + 8 * g;
#pragma unroll
        for (int kt = 0; kt < C::KT; ++kt) {
            uint4 v = qvalid ? *reinterpret_cast<const uint4*>(qp + 16 * kt) : make_uint4(0, 0, 0, 0);
            qf[kt] = __builtin_bit_cast(bf16x8, v);
        }
    }
    // Folding into a running result: nothing to add when no block is kept here.
    if (acc && nkeep == 0) return;
    const int32_t* kept = codes;  // this workgroup's kept list
    if (tp.piece >= 0) {          // its share of a split tail row
        const int e0 = tp.piece * nkeep / tail_k, e1 = (tp.piece + 1) * nkeep / tail_k;
        kept = codes + e0;
        nkeep = e1 - e0;
    }
    // (the last compaction round ended with a barrier: codes are visible)
    int code = nkeep > 0 ? kept[0] : -1;
    if (nkeep > 0) issue(code, 0);
    int next_code = nkeep > 1 ? kept[1] : -1;

    floatx16 oacc[C::DT];
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt) oacc[dt] = floatx16{};
    float m_run = -INFINITY;  // running max of scaled scores, log2 units
    float l_run = 0.f;        // this lane's partial row sum
    // Set only where the max moves: lim = m_run + the rescale threshold (see
    // above), neg_m = -m_run, or 0 while the lane has seen no finite score.
    float lim = -INFINITY, neg_m = 0.f;
    const int last_cnt = L - (L / BLK) * BLK;  // valid keys of a partial last block

    // One block of the loop. The buffer index is a compile-time constant (the
    // loop below is unrolled by two), so the LDS operand addresses of both
    // buffers are per-lane constants plus an immediate offset, with no address
    // arithmetic inside the loop.
    auto step = [&](int jj, auto buf_c) {
        constexpr int buf = decltype(buf_c)::value;
        const int cur = code;
        // A workgroup barrier does not wait for outstanding vector-memory
        // loads, and the compiler does not add that wait for direct-to-LDS
        // copies: each wave waits for its own copies of block jj (the only
        // ones in flight) before the barrier publishes the whole tile.
        wait_vmem_all();
        __syncthreads();  // block jj in LDS; everyone is done with block jj-1
        if (jj + 1 < nkeep) {
            issue(next_code, buf ^ 1);
            code = next_code;
            next_code = (jj + 2 < nkeep) ? kept[jj + 2] : -1;
        }
        if (cur < 0) return;

        const uint16_t* lk = &lds[buf][0][0];
        const uint16_t* lv = &lds[buf][1][0];

        // S^T for this wave's key half: s[mt][rr] is key
        // HALF*kh + 32 mt + 16 (rr/8) + 8 g + rr%8 of query qi.
        floatx16 s[C::MTW];
#pragma unroll
        for (int mt = 0; mt < C::MTW; ++mt) s[mt] = floatx16{};
        // The score MFMAs run at raised wave priority, so the matrix pipe is
        // fed first while the SIMD's other wave fills in with softmax work.
        // All K operands of the block are read from LDS before the first MFMA,
        // so the LDS latency is paid once per block instead of once per pair
        // of MFMAs (the scheduler would otherwise sink each read to its use).
        bf16x8 ka[C::KT][C::MTW];
#pragma unroll
        for (int kt = 0; kt < C::KT; ++kt)
#pragma unroll
            for (int mt = 0; mt < C::MTW; ++mt) {
                const int krow = C::HALF * kh + 32 * mt + sigma(qi);
                ka[kt][mt] = *reinterpret_cast<const bf16x8*>(
                    lk + krow * D + (((2 * kt + g) ^ swz<D>(krow)) * 8));
            }
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int kt = 0; kt < C::KT; ++kt)
#pragma unroll
            for (int mt = 0; mt < C::MTW; ++mt)
                s[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[kt][mt], qf[kt], s[mt], 0, 0, 0);
        __builtin_amdgcn_s_setprio(0);
        // The V^T operands of the whole block, read before the softmax so that
        // the LDS latency overlaps the exponentials.
        bf16x8 va[C::PTW][C::DT];
#pragma unroll
        for (int t = 0; t < C::PTW; ++t)
#pragma unroll
            for (int dt = 0; dt < C::DT; ++dt) {
                const int tg = C::PTW * kh + t;
                const int vrow = 32 * dt + qi;
                va[t][dt] = *reinterpret_cast<const bf16x8*>(
                    lv + vrow * BLK + (((2 * tg + g) ^ swz<BLK>(vrow)) * 8));
            }
        __builtin_amdgcn_sched_barrier(0);
        if (cur & 1) {  // partial last block: keys past L do not exist
#pragma unroll
            for (int mt = 0; mt < C::MTW; ++mt)
#pragma unroll
                for (int rr = 0; rr < 16; ++rr) {
                    const int key = C::HALF * kh + 32 * mt + 16 * (rr >> 3) + 8 * g + (rr & 7);
                    if (key >= last_cnt) s[mt][rr] = -INFINITY;
                }
        }

        float mx = -INFINITY;
#pragma unroll
        for (int mt = 0; mt < C::MTW; ++mt)
#pragma unroll
            for (int rr = 0; rr < 16; rr += 2) mx = fmaxf(fmaxf(mx, s[mt][rr]), s[mt][rr + 1]);
        mx = pair_max(mx) * c2;
        // The max moves by the rule above (always on the first block a lane sees).
        const bool moved = __ballot(mx > lim) != 0;
        if (moved) {
            const float m_new = fmaxf(m_run, mx);
            const float alpha = (m_new == -INFINITY) ? 1.0f : __builtin_amdgcn_exp2f(m_run - m_new);
            m_run = m_new;
            l_run *= alpha;
            lim = m_run + rescale_threshold(l_run);
            neg_m = (m_run == -INFINITY) ? 0.f : -m_run;
#pragma unroll
            for (int dt = 0; dt < C::DT; ++dt) oacc[dt] *= alpha;
        }

        // (the two partial sums start from the first two probabilities, not
        // from 0 + p, which the compiler cannot drop)
        float lsum[2];
#pragma unroll
        for (int t = 0; t < C::PTW; ++t) {
            const int mt = t >> 1, hf = t & 1;
            floatx8 p;
#pragma unroll
            for (int v = 0; v < 8; ++v) {
                p[v] = __builtin_amdgcn_exp2f(fmaf(s[mt][8 * hf + v], c2, neg_m));
                if (t == 0 && v < 2)
                    lsum[v] = p[v];
                else
                    lsum[v & 1] += p[v];
            }
            const bf16x8 pb = __builtin_convertvector(p, bf16x8);
#pragma unroll
            for (int dt = 0; dt < C::DT; ++dt)
                oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[t][dt], pb, oacc[dt], 0, 0, 0);
        }
        l_run += lsum[0] + lsum[1];
    };
    for (int jj = 0; jj < nkeep; jj += 2) {
        step(jj, std::integral_constant<int, 0>{});
        if (jj + 1 < nkeep) step(jj + 1, std::integral_constant<int, 1>{});
    }

    // Merge the two key halves of each query group through their log-sum-exp.
    const float l_half = pair_sum(l_run);
    __syncthreads();  // every wave is done with the tiles
    float* mrg = reinterpret_cast<float*>(&lds[0][0][0]);
    constexpr int REGS = C::DT * 16;
    float* mine = mrg + qg * 64 * (REGS + 2);
    if (kh == 1) {
#pragma unroll
        for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
            for (int rr = 0; rr < 16; ++rr) mine[(dt * 16 + rr) * 64 + lane] = oacc[dt][rr];
        mine[REGS * 64 + lane] = m_run;
        mine[(REGS + 1) * 64 + lane] = l_half;
    }
    __syncthreads();
    if (kh == 1) return;

    const float m_b = mine[REGS * 64 + lane];
    const float l_b = mine[(REGS + 1) * 64 + lane];
    const float m = fmaxf(m_run, m_b);
    const float w_a = (m_run == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m_run - m);
    const float w_b = (m_b == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m_b - m);
    const float l_tot = l_half * w_a + l_b * w_b;
    const bool live = qvalid && l_tot > 0.f;
    const float inv = live ? 1.0f / l_tot : 0.f;
    const float fa = w_a * inv, fb = w_b * inv;
    const int64_t orow = int64_t(h) * nq * BLK + int64_t(r) * BLK + qg * 32 + qi;
    float lse_out = live ? (m + __log2f(l_tot)) * kLn2 : -INFINITY;
    if (tp.piece >= 0) {  // a piece of a split tail row: float32 partial into the workspace
        const int64_t prow = int64_t(blockIdx.x - tail_first) * BLK + qg * 32 + qi;
#pragma unroll
        for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                float o4[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int rr = 4 * q4 + u;
                    o4[u] = live ? oacc[dt][rr] * fa + mine[(dt * 16 + rr) * 64 + lane] * fb : 0.f;
                }
                *reinterpret_cast<float4*>(part_o + prow * D + 32 * dt + 8 * q4 + 4 * g) =
                    make_float4(o4[0], o4[1], o4[2], o4[3]);
            }
        if (g == 0) part_lse[prow] = lse_out;
        return;
    }
    // Folding into a running result (O, lse, float32): with both log-sum-exps
    // in log2 units, the stored rows weigh ka and this part kb. Both lanes of
    // a row pair read the stored lse before the g == 0 lane rewrites it (the
    // rewrite depends on the value read).
    float ka = 0.f, kb = 1.f;
    bool store = true;
    if (!OUT_BF16 && acc) {
        store = live;
        if (live) {
            const float la2 = lse[orow] * kLog2e;
            const float lb2 = m + __log2f(l_tot);
            const float mm = fmaxf(la2, lb2);
            const float wa = (la2 == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(la2 - mm);
            const float wb = __builtin_amdgcn_exp2f(lb2 - mm);
            const float t = wa + wb;
            ka = wa / t;
            kb = wb / t;
            lse_out = (mm + __log2f(t)) * kLn2;
        }
    }
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt) {
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
            const int d0 = 32 * dt + 8 * q4 + 4 * g;
            float o4[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int rr = 4 * q4 + u;
                o4[u] = live ? oacc[dt][rr] * fa + mine[(dt * 16 + rr) * 64 + lane] * fb : 0.f;
            }
            if (!store) continue;
            if constexpr (OUT_BF16) {
                uint16_t* op = static_cast<uint16_t*>(O) + orow * D + d0;
                uint2 w;
                w.x = f32_to_bf16_bits(o4[0]) | (f32_to_bf16_bits(o4[1]) << 16);
                w.y = f32_to_bf16_bits(o4[2]) | (f32_to_bf16_bits(o4[3]) << 16);
                *reinterpret_cast<uint2*>(op) = w;
            } else {
                float* op = static_cast<float*>(O) + orow * D + d0;
                if (acc) {
                    const float4 prev = *reinterpret_cast<const float4*>(op);
                    o4[0] = ka * prev.x + kb * o4[0];
                    o4[1] = ka * prev.y + kb * o4[1];
                    o4[2] = ka * prev.z + kb * o4[2];
                    o4[3] = ka * prev.w + kb * o4[3];
                }
                *reinterpret_cast<float4*>(op) = make_float4(o4[0], o4[1], o4[2], o4[3]);
            }
        }
    }
    if (lse && g == 0 && store) lse[orow] = lse_out;
}

// Kernel for 128-token blocks: two independent workgroups per CU. Four waves
// per workgroup, wave w owning queries 32 w .. +31 and every key of each kept
// block, so each wave runs one online softmax and no merge is needed; single
// K and V tile buffers (64 KB of LDS at d = 128). The two waves that share a
// SIMD belong to different workgroups and are not held in step by a common
// barrier, so one can run its MFMAs while the other runs its softmax. The K
// copy of block j+1 is issued once every wave has finished the scores of
// block j, the V copy once the output product of block j is done; each copy
// thus has half a block of compute to land.
template <int D, int BLK_>
struct CfgRows {
    static constexpr int BLK = BLK_;
    static constexpr int NW = BLK / 32;          // one wave per 32 queries
    static constexpr int THREADS = 64 * NW;
    static constexpr int MT = BLK / 32;          // 32-key tiles of the score product
    static constexpr int PT = BLK / 16;          // 16-key steps of the output product
    static constexpr int KT = D / 16;
    static constexpr int DT = D / 32;
    static constexpr int TILE = BLK * D;
    static constexpr int CHUNKS = TILE / 8;
    static constexpr int DMA = CHUNKS / THREADS;
    static_assert(CHUNKS % THREADS == 0, "tile must split evenly");
};

// s_waitcnt vmcnt(n) for the n copies issued last, other counters untouched.
template <int N>
__device__ __forceinline__ void wait_vmem_keep() {
    static_assert(N >= 0 && N < 16, "vmcnt field");
    __builtin_amdgcn_s_waitcnt(0x0F70 | N);
}

template <int D, int BLK, bool OUT_BF16>
__global__ __launch_bounds__(64 * (BLK / 32)) __attribute__((amdgpu_waves_per_eu(2)))
void attn_rows_kernel(const uint16_t* __restrict__ Q, const int32_t* __restrict__ sel,
                    const int32_t* __restrict__ slot_of, const uint16_t* __restrict__ Kp,
                    const uint16_t* __restrict__ Vp, void* __restrict__ O,
                    float* __restrict__ lse, int L, int n, int i0, int nq, int keep,
                    int64_t capacity, float c2 /* scale * log2(e) */, int kv_lo, int kv_hi,
                    int h_lo, int n_heads, int acc, int remap,
                    const int32_t* __restrict__ order, int tail_first, int tail_k,
                    float* __restrict__ part_o, float* __restrict__ part_lse,
                    const int32_t* __restrict__ row_sort) {
    using C = CfgRows<D, BLK>;
    __shared__ __attribute__((aligned(16))) uint16_t lk[C::TILE];
    __shared__ __attribute__((aligned(16))) uint16_t lv[C::TILE];
    extern __shared__ int32_t codes[];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int qi = lane & 31, g = lane >> 5;

    const int G = n_heads * nq;
    int wg = blockIdx.x;
    const TailPiece tp = tail_piece(wg, tail_first, tail_k);
    if (order) {  // an explicit row order (e.g. longest first); no XCD remap
        wg = order[blockIdx.x];
        if (wg < 0 || wg >= G) return;
    } else if (remap) {
        wg = sorted_row(xcd_row(tp.index, G), nq, row_sort);
    } else {
        wg = tp.index;
    }
    const int h = h_lo + wg / nq, r = wg % nq;
    const int qtok = (i0 + r) * BLK + 32 * wave + qi;
    const bool qvalid = qtok < L;

    __shared__ int wave_cnt[C::NW];
    int nkeep = 0;
    {
        const int32_t* srow = sel + (int64_t(h) * nq + r) * keep;
        const int32_t* hslot = slot_of + int64_t(h) * n;
        const bool ragged = (L % BLK) != 0;
        for (int base = 0; base < keep; base += C::THREADS) {
            const int jj = base + tid;
            int code = -1;
            if (jj < keep) {
                const int j = srow[jj];
                if (j >= kv_lo && j < kv_hi && j >= 0 && j < n) {
                    const int sl = hslot[j];
                    if (sl >= 0 && sl < capacity && sl < (1 << 30))
                        code = 2 * sl + ((ragged && j == n - 1) ? 1 : 0);
                }
            }
            const uint64_t bal = __ballot(code >= 0);
            if (lane == 0) wave_cnt[wave] = __popcll(bal);
            __syncthreads();
            int off = nkeep, total = 0;
#pragma unroll
            for (int w = 0; w < C::NW; ++w) {
                off += w < wave ? wave_cnt[w] : 0;
                total += wave_cnt[w];
            }
            const int below = __builtin_amdgcn_mbcnt_hi(
                uint32_t(bal >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(bal), 0));
            if (code >= 0) codes[off + below] = code;
            nkeep += total;
            __syncthreads();
        }
    }
    if (acc && nkeep == 0) return;
    const int32_t* kept = codes;  // this workgroup's kept list
    if (tp.piece >= 0) {          // its share of a split tail row
        const int e0 = tp.piece * nkeep / tail_k, e1 = (tp.piece + 1) * nkeep / tail_k;
        kept = codes + e0;
        nkeep = e1 - e0;
    }

    int kvoff[C::DMA], vvoff[C::DMA];
#pragma unroll
    for (int u = 0; u < C::DMA; ++u) {
        const int p = (u * C::NW + wave) * 64 + lane;
        kvoff[u] = chunk_src_offset<D>(p);
        vvoff[u] = chunk_src_offset<BLK>(p);
    }
    // (codes are wave-uniform; taking them into scalar registers keeps the
    // copies' address arithmetic on the scalar unit)
    auto copy_k = [&](int code) {
        code = __builtin_amdgcn_readfirstlane(code);
        copy_tile<C::NW, C::DMA>(Kp + int64_t(code >> 1) * C::TILE, C::TILE * 2, lk, kvoff, wave);
    };
    auto copy_v = [&](int code) {
        code = __builtin_amdgcn_readfirstlane(code);
        copy_tile<C::NW, C::DMA>(Vp + int64_t(code >> 1) * C::TILE, C::TILE * 2, lv, vvoff, wave);
    };

    bf16x8 qf[C::KT];
    {
        const uint16_t* qp = Q + (int64_t(h) * L + (qvalid ? qtok : 0)) * D + 8 * g;
#pragma unroll
        for (int kt = 0; kt < C::KT; ++kt) {
            uint4 v = qvalid ? *reinterpret_cast<const uint4*>(qp + 16 * kt) : make_uint4(0, 0, 0, 0);
            qf[kt] = __builtin_bit_cast(bf16x8, v);
        }
    }
    // From here on nothing the compiler tracks is in flight: the Q loads are
    // waited for here, and the copies are issued behind its back (copy_tile).
    wait_vmem_all();
    if (nkeep > 0) {
        copy_k(kept[0]);
        copy_v(kept[0]);
    }

    floatx16 oacc[C::DT];
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt) oacc[dt] = floatx16{};
    float m_run = -INFINITY, l_run = 0.f;
    // Set only where the max moves: lim = m_run + the rescale threshold,
    // neg_m = -m_run, or 0 while the lane has seen no finite score.
    float lim = -INFINITY, neg_m = 0.f;
    const int last_cnt = L - (L / BLK) * BLK;

    // Entering block jj: K(jj) and V(jj) are in flight, K issued first.
    if (nkeep > 0) {
        wait_vmem_keep<C::DMA>();  // K(0) landed (V(0) may still be in flight)
        __syncthreads();
    }
    for (int jj = 0; jj < nkeep; ++jj) {
        const int cur = kept[jj];
        // Scores: S^T for the wave's 32 queries over all 128 keys of the block;
        // s[mt][rr] is key 32 mt + 16 (rr/8) + 8 g + rr%8.
        // k step outermost, so the four accumulators advance together and no
        // MFMA waits on the one before it; the K operands of step kt+1 are
        // read while the four MFMAs of step kt run.
        floatx16 s[C::MT];
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt) s[mt] = floatx16{};
        bf16x8 kb[2][C::MT];
        auto kread = [&](int kt, bf16x8 (&dst)[C::MT]) {
#pragma unroll
            for (int mt = 0; mt < C::MT; ++mt) {
                const int krow = 32 * mt + sigma(qi);
                dst[mt] = *reinterpret_cast<const bf16x8*>(
                    lk + krow * D + (((2 * kt + g) ^ swz<D>(krow)) * 8));
            }
        };
        kread(0, kb[0]);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int kt = 0; kt < C::KT; ++kt) {
            if (kt + 1 < C::KT) kread(kt + 1, kb[(kt + 1) & 1]);
#pragma unroll
            for (int mt = 0; mt < C::MT; ++mt)
                s[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kb[kt & 1][mt], qf[kt], s[mt], 0, 0, 0);
        }
        // Keep that order: the reads of step kt+1 ahead of the MFMAs of step kt.
#pragma unroll
        for (int kt = 0; kt < C::KT; ++kt) {
            if (kt + 1 < C::KT) __builtin_amdgcn_sched_group_barrier(0x100, C::MT, 0);  // LDS reads
            __builtin_amdgcn_sched_group_barrier(0x008, C::MT, 0);                      // MFMAs
        }
        __builtin_amdgcn_sched_barrier(0);
        wait_vmem_all();   // V(jj) landed
        __syncthreads();   // V(jj) visible; every wave is done with K(jj)
        if (jj + 1 < nkeep) copy_k(kept[jj + 1]);

        // Softmax and output product at raised priority: where the other wave
        // on the SIMD is in its score MFMAs, this wave's VALU work issues first
        // and the matrix pipe stays fed by both.
        __builtin_amdgcn_s_setprio(1);
        if (cur & 1) {
#pragma unroll
            for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
                for (int rr = 0; rr < 16; ++rr) {
                    const int key = 32 * mt + 16 * (rr >> 3) + 8 * g + (rr & 7);
                    if (key >= last_cnt) s[mt][rr] = -INFINITY;
                }
        }
        float mx = -INFINITY;
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
            for (int rr = 0; rr < 16; rr += 2) mx = fmaxf(fmaxf(mx, s[mt][rr]), s[mt][rr + 1]);
        mx = pair_max(mx) * c2;
        const bool moved = __ballot(mx > lim) != 0;
        if (moved) {
            const float m_new = fmaxf(m_run, mx);
            const float alpha = (m_new == -INFINITY) ? 1.0f : __builtin_amdgcn_exp2f(m_run - m_new);
            m_run = m_new;
            l_run *= alpha;
            lim = m_run + rescale_threshold(l_run);
            neg_m = (m_run == -INFINITY) ? 0.f : -m_run;
#pragma unroll
            for (int dt = 0; dt < C::DT; ++dt) oacc[dt] *= alpha;
        }

        // 16-key steps; the V^T operands of step t+1 are read one step ahead.
        // (the two partial sums start from the first two probabilities, not
        // from 0 + p, which the compiler cannot drop)
        float lsum[2];
        bf16x8 vb[2][C::DT];
        auto vread = [&](int t, bf16x8 (&dst)[C::DT]) {
#pragma unroll
            for (int dt = 0; dt < C::DT; ++dt) {
                const int vrow = 32 * dt + qi;
                dst[dt] = *reinterpret_cast<const bf16x8*>(
                    lv + vrow * BLK + (((2 * t + g) ^ swz<BLK>(vrow)) * 8));
            }
        };
        // Step t+1's probabilities are computed while step t's MFMAs run: the
        // scheduling groups interleave each MFMA with about seven VALU
        // instructions of the next step.
        auto pstep = [&](int t) -> bf16x8 {
            const int mt = t >> 1, hf = t & 1;
            floatx8 p;
#pragma unroll
            for (int v = 0; v < 8; ++v) {
                p[v] = __builtin_amdgcn_exp2f(fmaf(s[mt][8 * hf + v], c2, neg_m));
                if (t == 0 && v < 2)
                    lsum[v] = p[v];
                else
                    lsum[v & 1] += p[v];
            }
            return __builtin_convertvector(p, bf16x8);
        };
        vread(0, vb[0]);
        bf16x8 pbn = pstep(0);
#pragma unroll
        for (int t = 0; t < C::PT; ++t) {
            if (t + 1 < C::PT) vread(t + 1, vb[(t + 1) & 1]);
            __builtin_amdgcn_sched_barrier(0);
            const bf16x8 pb = pbn;
            if (t + 1 < C::PT) pbn = pstep(t + 1);
#pragma unroll
            for (int dt = 0; dt < C::DT; ++dt)
                oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vb[t & 1][dt], pb, oacc[dt], 0, 0, 0);
            if (t + 1 < C::PT) {
#pragma unroll
                for (int k = 0; k < C::DT; ++k) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x002, 7, 0);
                }
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        __builtin_amdgcn_s_setprio(0);
        l_run += lsum[0] + lsum[1];

        wait_vmem_all();   // K(jj+1) landed
        __syncthreads();   // K(jj+1) visible; every wave is done with V(jj)
        if (jj + 1 < nkeep) copy_v(kept[jj + 1]);
    }

    const float l_tot = pair_sum(l_run);
    const bool live = qvalid && l_tot > 0.f;
    const float inv = live ? 1.0f / l_tot : 0.f;
    const int64_t orow = int64_t(h) * nq * BLK + int64_t(r) * BLK + 32 * wave + qi;
    float lse_out = live ? (m_run + __log2f(l_tot)) * kLn2 : -INFINITY;
    if (tp.piece >= 0) {  // a piece of a split tail row: float32 partial into the workspace
        const int64_t prow = int64_t(blockIdx.x - tail_first) * BLK + 32 * wave + qi;
#pragma unroll
        for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                float4 o;
                o.x = live ? oacc[dt][4 * q4] * inv : 0.f;
                o.y = live ? oacc[dt][4 * q4 + 1] * inv : 0.f;
                o.z = live ? oacc[dt][4 * q4 + 2] * inv : 0.f;
                o.w = live ? oacc[dt][4 * q4 + 3] * inv : 0.f;
                *reinterpret_cast<float4*>(part_o + prow * D + 32 * dt + 8 * q4 + 4 * g) = o;
            }
        if (g == 0) part_lse[prow] = lse_out;
        return;
    }
    float ka = 0.f, kb = 1.f;
    bool store = true;
    if (!OUT_BF16 && acc) {
        store = live;
        if (live) {
            const float la2 = lse[orow] * kLog2e;
            const float lb2 = m_run + __log2f(l_tot);
            const float mm = fmaxf(la2, lb2);
            const float wa = (la2 == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(la2 - mm);
            const float wb = __builtin_amdgcn_exp2f(lb2 - mm);
            const float t = wa + wb;
            ka = wa / t;
            kb = wb / t;
            lse_out = (mm + __log2f(t)) * kLn2;
        }
    }
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt) {
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
            const int d0 = 32 * dt + 8 * q4 + 4 * g;
            float o4[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) o4[u] = live ? oacc[dt][4 * q4 + u] * inv : 0.f;
            if (!store) continue;
            if constexpr (OUT_BF16) {
                uint16_t* op = static_cast<uint16_t*>(O) + orow * D + d0;
                uint2 w;
                w.x = f32_to_bf16_bits(o4[0]) | (f32_to_bf16_bits(o4[1]) << 16);
                w.y = f32_to_bf16_bits(o4[2]) | (f32_to_bf16_bits(o4[3]) << 16);
                *reinterpret_cast<uint2*>(op) = w;
            } else {
                float* op = static_cast<float*>(O) + orow * D + d0;
                if (acc) {
                    const float4 prev = *reinterpret_cast<const float4*>(op);
                    o4[0] = ka * prev.x + kb * o4[0];
                    o4[1] = ka * prev.y + kb * o4[1];
                    o4[2] = ka * prev.z + kb * o4[2];
                    o4[3] = ka * prev.w + kb * o4[3];
                }
                *reinterpret_cast<float4*>(op) = make_float4(o4[0], o4[1], o4[2], o4[3]);
            }
        }
    }
    if (lse && g == 0 && store) lse[orow] = lse_out;
}

constexpr int kMaxTailSplit = 4;  // pieces per split tail row, at most

// Merge of the pieces of the split tail rows. Piece p of tail row t sits in
// workspace slot t * tail_k + p as (O_p normalised by its own sum, lse_p in
// natural log); the pieces cover disjoint parts of the row's kept blocks, so
// with m = max_p lse_p and w_p = exp(lse_p - m)
//   O = sum_p w_p O_p / sum_p w_p,   lse = m + log sum_p w_p
// (the online-softmax merge of Section 2.3). Rows whose pieces are all
// empty (padded queries) get O = 0, lse = -inf. One thread per float4 of
// output: a workgroup covers 256 / (D/4) query rows of one tail row, and each
// thread issues the loads of all the row's pieces at once.
template <int D, int BLK, bool OUT_BF16>
__global__ __launch_bounds__(256) void tail_merge_kernel(
    const float* __restrict__ part_o, const float* __restrict__ part_lse, void* __restrict__ O,
    float* __restrict__ lse, int G, int nq, int h_lo, int tail_first, int tail_k,
    const int32_t* __restrict__ row_sort) {
    constexpr int C4 = D / 4;             // float4 per query row
    constexpr int QPW = 256 / C4;         // query rows per workgroup
    constexpr int WPR = BLK / QPW;        // workgroups per tail row
    const int t = blockIdx.x / WPR;
    const int q = (blockIdx.x % WPR) * QPW + threadIdx.x / C4, c4 = threadIdx.x % C4;
    const int row = sorted_row(xcd_row(tail_first + t, G), nq, row_sort);
    const int h = h_lo + row / nq, r = row % nq;
    const int64_t orow = (int64_t(h) * nq + r) * BLK + q;
    float lp[kMaxTailSplit];
    float4 x[kMaxTailSplit];
    float m = -INFINITY;
#pragma unroll
    for (int p = 0; p < kMaxTailSplit; ++p) {
        if (p < tail_k) {
            const int64_t prow = (int64_t(t) * tail_k + p) * BLK + q;
            lp[p] = part_lse[prow];
            x[p] = reinterpret_cast<const float4*>(part_o + prow * D)[c4];
            m = fmaxf(m, lp[p]);
        } else {
            lp[p] = -INFINITY;
        }
    }
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    float wsum = 0.f;
    if (m != -INFINITY) {
#pragma unroll
        for (int p = 0; p < kMaxTailSplit; ++p) {
            if (lp[p] == -INFINITY) continue;
            const float w = expf(lp[p] - m);
            wsum += w;
            acc.x += w * x[p].x;
            acc.y += w * x[p].y;
            acc.z += w * x[p].z;
            acc.w += w * x[p].w;
        }
    }
    const float inv = wsum > 0.f ? 1.0f / wsum : 0.f;
    const int64_t at = orow * D + 4 * c4;
    if constexpr (OUT_BF16) {
        uint2 wv;
        wv.x = f32_to_bf16_bits(acc.x * inv) | (f32_to_bf16_bits(acc.y * inv) << 16);
        wv.y = f32_to_bf16_bits(acc.z * inv) | (f32_to_bf16_bits(acc.w * inv) << 16);
        *reinterpret_cast<uint2*>(static_cast<uint16_t*>(O) + at) = wv;
    } else {
        *reinterpret_cast<float4*>(static_cast<float*>(O) + at) =
            make_float4(acc.x * inv, acc.y * inv, acc.z * inv, acc.w * inv);
    }
    if (c4 == 0 && lse) lse[orow] = wsum > 0.f ? m + logf(wsum) : -INFINITY;
}


// Workgroups of `kernel` that are resident at once on the current device.
template <typename Kernel>
int resident_slots(Kernel kernel, int threads, size_t dyn) {
    int per_cu = 0, dev = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, dyn) != hipSuccess)
        return 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return 0;
    return per_cu * cus;
}

// The tail split of a launch of G rows on `slots` resident workgroups: the S
// = G mod slots rows of the last, partial round run as k pieces each, k as
// large as the round's free slots, kMaxTailSplit and the workspace allow.
struct TailPlan {
    int first, k;
    const int32_t* row_sort = nullptr;
};
TailPlan plan_tail(int G, int slots, int64_t piece_bytes, int64_t ws_bytes) {
    if (slots <= 0) return {G, 1};
    const int S = G % slots;
    if (S == 0) return {G, 1};
    int k = min(kMaxTailSplit, slots / S);
    while (k > 1 && int64_t(S) * k * piece_bytes > ws_bytes) --k;
    if (k < 2) return {G, 1};
    return {G - S, k};
}

template <int D, int BLK, bool OUT>
hipError_t launch_tail_merge(const Geom& g, const AttnPart& part, const TailPlan& tp, int G,
                             const float* part_o, const float* part_lse, void* O, float* lse,
                             hipStream_t s) {
    const int S = G - tp.first;
    constexpr int wpr = BLK / (256 / (D / 4));  // workgroups per tail row
    tail_merge_kernel<D, BLK, OUT><<<S * wpr, 256, 0, s>>>(part_o, part_lse, O, lse, G, g.nq,
                                                           part.h_lo, tp.first, tp.k, tp.row_sort);
    return hipGetLastError();
}

// Workspace layout of a tail split: the partial outputs, then their lse.
struct TailSpace {
    float* part_o;
    float* part_lse;
};
TailSpace tail_space(void* ws, const TailPlan& tp, int G, int D, int BLK) {
    const int64_t pieces = int64_t(G - tp.first) * tp.k;
    float* o = static_cast<float*>(ws);
    return {o, o + pieces * BLK * D};
}

// The balanced launch's workspace holds the row order first (when it fits),
// then the float32 partials of the tail split. Writes the order (one small
// kernel on stream s) and returns the tail plan and where the partials go.
template <typename Kernel>
hipError_t balanced_plan(Kernel kernel, int threads, size_t dyn, const Geom& g,
                         const AttnPart& part, const int32_t* sel, int keep, int G,
                         int64_t piece_bytes, hipStream_t s, TailPlan* tp, void** partials) {
    *tp = TailPlan{G, 1};
    *partials = nullptr;
    if (!part.ws || part.order || part.acc) return hipSuccess;
    char* ws = static_cast<char*>(part.ws);
    int64_t bytes = part.ws_bytes;
    const int32_t* order = nullptr;
    const int64_t sb = row_sort_bytes(G);
    if (bytes >= sb) {
        row_sort_kernel<<<part.h_hi - part.h_lo, 1024, 0, s>>>(
            sel + int64_t(part.h_lo) * g.nq * keep, keep, g.nq, g.n, reinterpret_cast<int32_t*>(ws));
        if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
        order = reinterpret_cast<const int32_t*>(ws);
        ws += sb;
        bytes -= sb;
    }
    *tp = plan_tail(G, resident_slots(kernel, threads, dyn), piece_bytes, bytes);
    tp->row_sort = order;
    *partials = ws;
    return hipSuccess;
}

template <int D, int BLK>
hipError_t launch_rows(const Geom& g, const void* Q, const int32_t* sel, int keep,
                     const int32_t* slot_of, const void* Kp, const void* Vp, int64_t cap,
                     float scale, const AttnPart& part, void* O, bool out_bf16, float* lse,
                     hipStream_t s) {
    const int n_heads = part.h_hi - part.h_lo;
    const int G = n_heads * g.nq;
    const float c2 = scale * kLog2e;
    const size_t dyn = size_t(keep) * sizeof(int32_t);
    constexpr int THREADS = CfgRows<D, BLK>::THREADS;
    TailPlan tp;
    void* partials = nullptr;
    if (hipError_t e = balanced_plan(attn_rows_kernel<D, BLK, true>, THREADS, dyn, g, part, sel,
                                     keep, G, int64_t(BLK) * (D + 1) * 4, s, &tp, &partials);
        e != hipSuccess)
        return e;
    const TailSpace ts = tp.k > 1 ? tail_space(partials, tp, G, D, BLK) : TailSpace{nullptr, nullptr};
    const int grid = tp.first + (G - tp.first) * tp.k;
    if (out_bf16)
        attn_rows_kernel<D, BLK, true><<<grid, THREADS, dyn, s>>>(
            (const uint16_t*)Q, sel, slot_of, (const uint16_t*)Kp, (const uint16_t*)Vp, O, lse,
            g.L, g.n, g.i0, g.nq, keep, cap, c2, part.kv_lo, part.kv_hi, part.h_lo, n_heads,
            part.acc, 1, part.order, tp.first, tp.k, ts.part_o, ts.part_lse, tp.row_sort);
    else
        attn_rows_kernel<D, BLK, false><<<grid, THREADS, dyn, s>>>(
            (const uint16_t*)Q, sel, slot_of, (const uint16_t*)Kp, (const uint16_t*)Vp, O, lse,
            g.L, g.n, g.i0, g.nq, keep, cap, c2, part.kv_lo, part.kv_hi, part.h_lo, n_heads,
            part.acc, 1, part.order, tp.first, tp.k, ts.part_o, ts.part_lse, tp.row_sort);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || tp.k < 2) return e;
    return out_bf16 ? launch_tail_merge<D, BLK, true>(g, part, tp, G, ts.part_o, ts.part_lse, O, lse, s)
                    : launch_tail_merge<D, BLK, false>(g, part, tp, G, ts.part_o, ts.part_lse, O, lse, s);
}

template <int D, int BLK>
hipError_t launch_shape(const Geom& g, const void* Q, const int32_t* sel, int keep,
                        const int32_t* slot_of, const void* Kp, const void* Vp, int64_t cap,
                        float scale, const AttnPart& part, void* O, bool out_bf16, float* lse,
                        hipStream_t s) {
    using C = Cfg<D, BLK>;
    const int n_heads = part.h_hi - part.h_lo;
    const int G = n_heads * g.nq;
    const float c2 = scale * kLog2e;
    const int remap = 1;
    const size_t dyn = size_t(keep) * sizeof(int32_t);
    TailPlan tp;
    void* partials = nullptr;
    if (hipError_t e = balanced_plan(attn_bf16_kernel<D, BLK, true>, C::THREADS, dyn, g, part,
                                     sel, keep, G, int64_t(BLK) * (D + 1) * 4, s, &tp, &partials);
        e != hipSuccess)
        return e;
    const TailSpace ts = tp.k > 1 ? tail_space(partials, tp, G, D, BLK) : TailSpace{nullptr, nullptr};
    const int grid = tp.first + (G - tp.first) * tp.k;
    if (out_bf16)
        attn_bf16_kernel<D, BLK, true><<<grid, C::THREADS, dyn, s>>>(
            (const uint16_t*)Q, sel, slot_of, (const uint16_t*)Kp, (const uint16_t*)Vp, O, lse,
            g.L, g.n, g.i0, g.nq, keep, cap, c2, part.kv_lo, part.kv_hi, part.h_lo, n_heads,
            part.acc, remap, part.order, tp.first, tp.k, ts.part_o, ts.part_lse,
            tp.row_sort);
    else
        attn_bf16_kernel<D, BLK, false><<<grid, C::THREADS, dyn, s>>>(
            (const uint16_t*)Q, sel, slot_of, (const uint16_t*)Kp, (const uint16_t*)Vp, O, lse,
            g.L, g.n, g.i0, g.nq, keep, cap, c2, part.kv_lo, part.kv_hi, part.h_lo, n_heads,
            part.acc, remap, part.order, tp.first, tp.k, ts.part_o, ts.part_lse,
            tp.row_sort);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || tp.k < 2) return e;
    return out_bf16 ? launch_tail_merge<D, BLK, true>(g, part, tp, G, ts.part_o, ts.part_lse, O, lse, s)
                    : launch_tail_merge<D, BLK, false>(g, part, tp, G, ts.part_o, ts.part_lse, O, lse, s);
}

}  // namespace

hipError_t launch_attn_bf16(const Geom& g, const void* Q, const int32_t* sel, int keep,
                            const int32_t* slot_of, const void* Kp, const void* Vp,
                            int64_t capacity, float scale, const AttnPart& part, void* O,
                            bool out_bf16, float* lse, hipStream_t s) {
    (void)hipGetLastError();
    if (g.d == 128 && g.block == 128)
        return launch_rows<128, 128>(g, Q, sel, keep, slot_of, Kp, Vp, capacity, scale, part, O,
                              out_bf16, lse, s);
    if (g.d == 64 && g.block == 128)
        return launch_rows<64, 128>(g, Q, sel, keep, slot_of, Kp, Vp, capacity, scale, part, O,
                             out_bf16, lse, s);
    if (g.d == 64 && g.block == 64)
        return launch_shape<64, 64>(g, Q, sel, keep, slot_of, Kp, Vp, capacity, scale, part, O,
                                    out_bf16, lse, s);
    if (g.d == 128 && g.block == 64)
        return launch_shape<128, 64>(g, Q, sel, keep, slot_of, Kp, Vp, capacity, scale, part, O,
                                     out_bf16, lse, s);
    return hipErrorInvalidValue;
}

int64_t attn_tail_workspace_bytes(const Geom& g, int keep) {
    const size_t dyn = size_t(keep) * sizeof(int32_t);
    int slots = 0;
    if (g.d == 128 && g.block == 128)
        slots = resident_slots(attn_rows_kernel<128, 128, true>, CfgRows<128, 128>::THREADS, dyn);
    else if (g.d == 64 && g.block == 128)
        slots = resident_slots(attn_rows_kernel<64, 128, true>, CfgRows<64, 128>::THREADS, dyn);
    else if (g.d == 64 && g.block == 64)
        slots = resident_slots(attn_bf16_kernel<64, 64, true>, Cfg<64, 64>::THREADS, dyn);
    else if (g.d == 128 && g.block == 64)
        slots = resident_slots(attn_bf16_kernel<128, 64, true>, Cfg<128, 64>::THREADS, dyn);
    if (slots <= 0) return 0;
    // the row order, then the tail pieces, which never outnumber the resident slots
    return row_sort_bytes(g.H * g.nq) + int64_t(slots) * g.block * (g.d + 1) * 4;
}

}  // namespace sparsp
