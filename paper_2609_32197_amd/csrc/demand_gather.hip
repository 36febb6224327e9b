// Step 3: per-head demand union (Eq. 2 over all owners, kept per head as
// Section 5.2 requires) and row-major compaction of the demanded blocks.
//
// union_kernel   one workgroup per head: OR of the nq mask rows, word-parallel.
// offsets_kernel one workgroup per head: head_off[h] is the popcount of all
//                earlier heads' demand words (integer sums, so exact and
//                deterministic without a cross-workgroup scan); then every
//                block's slot = head_off[h] + rank of the block in D_h, which
//                fills slot_of and gather_blk. Both ends of an exchange could
//                derive these offsets locally from the same bitsets.
// gather_stream_kernel / gather_kernel
//                copy the demanded blocks, reading the slot count and the
//                slot -> (head, block) map from head_off and gather_blk on the
//                device, so the grid is fixed and no host round trip is needed.
//                K blocks are copied with 16-byte loads and stores; V blocks
//                are written transposed ([d, block]) so the attention kernel
//                reads V^T MFMA operands with contiguous 16-byte loads (each
//                thread moves a VEC x VEC sub-block and transposes it in
//                registers). Rows past L are written as zero. The streaming
//                kernel strides over the packed buffers as flat arrays (the
//                usual shapes); the windowed kernel walks the slots in windows
//                (any other shape).
#include "sparsp_internal.h"

namespace sparsp {
namespace {

constexpr int kGatherGrid = 256;  // one workgroup per CU of an MI355X

// Plain loads and stores for the windowed kernel (the streaming kernel below
// uses non-temporal ones).
__device__ __forceinline__ uint4 load_stream(const char* p) {
    return *reinterpret_cast<const uint4*>(p);
}
__device__ __forceinline__ void store_stream(char* p, uint4 v) {
    *reinterpret_cast<uint4*>(p) = v;
}

// Thread t ORs word t % W over the rows t / W, t / W + RG, ... (RG = 256 / W
// row groups), so every thread has work even when a row is a few words.
__global__ __launch_bounds__(256) void union_kernel(const uint64_t* __restrict__ mask, int nq,
                                                    int W, uint64_t* __restrict__ demand) {
    __shared__ uint64_t part[256];
    const int h = blockIdx.x;
    const int tid = threadIdx.x;
    const int rg_count = 256 / W;  // W <= 64, so at least 4 row groups
    const int w = tid % W, rg = tid / W;
    uint64_t acc = 0;
    if (rg < rg_count) {
        const uint64_t* m = mask + int64_t(h) * nq * W + w;
        for (int i = rg; i < nq; i += rg_count) acc |= m[int64_t(i) * W];
    }
    part[tid] = acc;
    __syncthreads();
    if (tid < W) {
        uint64_t r = 0;
        for (int g = 0; g < rg_count; ++g) r |= part[g * W + tid];
        demand[int64_t(h) * W + tid] = r;
    }
}

__global__ __launch_bounds__(256) void offsets_kernel(const uint64_t* __restrict__ demand, int H,
                                                      int n, int W, int32_t* __restrict__ head_off,
                                                      int32_t* __restrict__ slot_of,
                                                      int32_t* __restrict__ gather_blk) {
    __shared__ int red[256];
    __shared__ int word_prefix[kMaxWords];
    const int h = blockIdx.x;
    const int tid = threadIdx.x;

    // Demanded blocks of all earlier heads.
    int c = 0;
    for (int e = tid; e < h * W; e += 256) c += __popcll(demand[e]);
    red[tid] = c;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
        if (tid < s) red[tid] += red[tid + s];
        __syncthreads();
    }
    const int prefix = red[0];
    const uint64_t* dh = demand + int64_t(h) * W;
    if (tid == 0) {
        int run = 0;
        for (int w = 0; w < W; ++w) {
            word_prefix[w] = run;
            run += __popcll(dh[w]);
        }
        head_off[h] = prefix;
        if (h == H - 1) head_off[H] = prefix + run;
    }
    __syncthreads();
    for (int j = tid; j < n; j += 256) {
        const uint64_t word = dh[j >> 6];
        const int bit = j & 63;
        int32_t slot = -1;
        if ((word >> bit) & 1) {
            const uint64_t below = bit ? (word & ((uint64_t(1) << bit) - 1)) : 0;
            slot = prefix + word_prefix[j >> 6] + __popcll(below);
            gather_blk[slot] = j;
        }
        slot_of[int64_t(h) * n + j] = slot;
    }
}

// 16-bit transpose of an 8x8 tile held as 8 rows of uint4: out[c] holds column c.
__device__ __forceinline__ void transpose8x8_b16(const uint4 (&in)[8], uint4 (&out)[8]) {
    uint32_t a[8][4];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
        a[r][0] = in[r].x; a[r][1] = in[r].y; a[r][2] = in[r].z; a[r][3] = in[r].w;
    }
#pragma unroll
    for (int c = 0; c < 8; ++c) {
        uint32_t o[4];
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            // element (row 2p, col c) -> low half; (row 2p+1, col c) -> high half
            const uint32_t lo = (a[2 * p][c >> 1] >> ((c & 1) * 16)) & 0xffffu;
            const uint32_t hi = (a[2 * p + 1][c >> 1] >> ((c & 1) * 16)) & 0xffffu;
            o[p] = lo | (hi << 16);
        }
        out[c] = make_uint4(o[0], o[1], o[2], o[3]);
    }
}

__device__ __forceinline__ void transpose4x4_b32(const uint4 (&in)[4], uint4 (&out)[4]) {
    out[0] = make_uint4(in[0].x, in[1].x, in[2].x, in[3].x);
    out[1] = make_uint4(in[0].y, in[1].y, in[2].y, in[3].y);
    out[2] = make_uint4(in[0].z, in[1].z, in[2].z, in[3].z);
    out[3] = make_uint4(in[0].w, in[1].w, in[2].w, in[3].w);
}

constexpr int kMaxWS = 64;  // slots per window, at most

// e / div for 0 <= e < 2^24 and div >= 1, with inv = 1.0f / div: the float
// quotient is off by at most one, which the two corrections remove.
__device__ __forceinline__ int div_small(int e, int div, float inv) {
    int q = __float2int_rz(float(e) * inv);
    if (q * div > e) --q;
    if ((q + 1) * div <= e) ++q;
    return q;
}

// The packed buffers are filled window by window. A window covers a group of
// WS consecutive slots (WS > 1 only for small blocks, so that a window still
// gives every thread work): window 2g copies the group's K blocks, window
// 2g+1 writes its V blocks transposed. The group's source offsets and valid
// row counts are looked up once per window into LDS. A grid-stride walk over
// the windows keeps all resident workgroups on neighbouring slots, i.e. inside
// one contiguous stretch of source and destination at any moment, which is
// what lets the copy stream at full HBM rate; each thread keeps four 16-byte
// loads in flight per pass for K (eight rows for the V transpose).
template <bool BF16>
__global__ __launch_bounds__(256) void gather_kernel(const int32_t* __restrict__ head_off,
                                                     const int32_t* __restrict__ gather_blk,
                                                     const char* __restrict__ K,
                                                     const char* __restrict__ V,
                                                     char* __restrict__ Kp, char* __restrict__ Vp,
                                                     int H, int L, int d, int block, int WS,
                                                     int H_src) {
    constexpr int ES = BF16 ? 2 : 4;  // element size
    constexpr int VEC = 16 / ES;      // elements per 16-byte chunk
    constexpr int T = 256;
    __shared__ int32_t hoff[kMaxHeads + 1];
    __shared__ int64_t win_src[kMaxWS];  // byte offset of the block's first row in K and V
    __shared__ int32_t win_cnt[kMaxWS];  // valid token rows of the block
    for (int i = threadIdx.x; i <= H; i += T) hoff[i] = head_off[i];
    __syncthreads();
    const int total_slots = hoff[H];
    const int groups = (total_slots + WS - 1) / WS;
    const int64_t blk_bytes = int64_t(block) * d * ES;
    const int tid = threadIdx.x;
    const int row_chunks = d / VEC;             // 16-byte chunks per token row
    const int k_items = block * row_chunks;     // chunks per K block
    const int dblocks = d / VEC, kblocks = block / VEC;
    const int v_items = dblocks * kblocks;      // VEC x VEC sub-blocks per V block
    const float inv_k = 1.0f / float(k_items), inv_v = 1.0f / float(v_items);
    int h = 0;  // this thread's table slot's head; its slots only grow along the walk
    for (int w = blockIdx.x; w < 2 * groups; w += gridDim.x) {
        const int s0 = (w >> 1) * WS;
        const int ns = min(WS, total_slots - s0);
        __syncthreads();  // the previous window is done with the table
        if (tid < ns) {
            const int slot = s0 + tid;
            while (slot >= hoff[h + 1]) ++h;
            const int tok0 = gather_blk[slot] * block;
            win_src[tid] = (int64_t(h % H_src) * L + tok0) * d * ES;
            win_cnt[tid] = min(block, L - tok0);
        }
        __syncthreads();
        if ((w & 1) == 0) {
            // K: straight copy of the valid token rows, zero rows after.
            const int total = ns * k_items;
            for (int e0 = tid; e0 < total; e0 += 4 * T) {
                uint4 x[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int e = e0 + u * T;
                    x[u] = make_uint4(0, 0, 0, 0);
                    if (e < total) {
                        const int ls = WS == 1 ? 0 : div_small(e, k_items, inv_k);
                        const int c = e - ls * k_items;
                        if (c < win_cnt[ls] * row_chunks)
                            x[u] = load_stream(K + win_src[ls] + int64_t(c) * 16);
                    }
                }
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int e = e0 + u * T;
                    if (e < total) store_stream(Kp + int64_t(s0) * blk_bytes + int64_t(e) * 16, x[u]);
                }
            }
        } else {
            // V: transposed copy by VEC x VEC sub-blocks. Sub-block (kb, db)
            // covers tokens kb*VEC .. +VEC-1 and dims db*VEC .. +VEC-1.
            // Consecutive threads take consecutive db, so each load
            // instruction reads whole token rows.
            const int total = ns * v_items;
            for (int e = tid; e < total; e += T) {
                const int ls = WS == 1 ? 0 : div_small(e, v_items, inv_v);
                const int r = e - ls * v_items;
                const int db = r % dblocks, kb = r / dblocks;
                const int cnt = win_cnt[ls];
                const char* vsrc = V + win_src[ls];
                char* vdst = Vp + int64_t(s0 + ls) * blk_bytes;
                uint4 rows[VEC], cols[VEC];
#pragma unroll
                for (int rr = 0; rr < VEC; ++rr) {
                    const int t = kb * VEC + rr;
                    rows[rr] = make_uint4(0, 0, 0, 0);
                    if (t < cnt) rows[rr] = load_stream(vsrc + (int64_t(t) * d + db * VEC) * ES);
                }
                if constexpr (BF16) transpose8x8_b16(rows, cols);
                else transpose4x4_b32(rows, cols);
                // cols[c] = dim db*VEC+c, tokens kb*VEC .. +VEC-1 -> V_packed[slot][dim][token]
#pragma unroll
                for (int c = 0; c < VEC; ++c)
                    store_stream(vdst + (int64_t(db * VEC + c) * block + kb * VEC) * ES, cols[c]);
            }
        }
    }
}

// Streaming form of the same copy. A grid of two workgroups per CU strides
// over the packed buffers as flat arrays, so at any moment the workgroups
// read and write neighbouring pieces of memory, the way a plain streaming
// copy does; loads and stores are non-temporal (the data is used once, by
// the next kernel). K moves in groups of 256 16-byte chunks and V in groups
// of 64 VEC x VEC sub-blocks (one wave); a group never straddles two slots,
// which holds when a K block is a multiple of 256 chunks and a V block of 64
// sub-blocks with 8 | block / VEC and 8 | d / VEC. The V transpose places
// eight consecutive sub-blocks of a row (8 VEC tokens) in eight consecutive
// lanes, so every store instruction writes whole 128-byte row segments.
constexpr int kStreamGrid = 512;


template <bool BF16, bool WHOLE>  // WHOLE: a K block is a multiple of 1,024 chunks
__global__ __launch_bounds__(256) void gather_stream_kernel(
    const int32_t* __restrict__ head_off, const int32_t* __restrict__ gather_blk,
    const char* __restrict__ K, const char* __restrict__ V, char* __restrict__ Kp,
    char* __restrict__ Vp, int H, int L, int d, int block, int H_src) {
    constexpr int ES = BF16 ? 2 : 4;
    constexpr int VEC = 16 / ES;
    __shared__ int32_t hoff[kMaxHeads + 1];
    const int tid = threadIdx.x;
    for (int i = tid; i <= H; i += 256) hoff[i] = head_off[i];
    __syncthreads();
    const int total_slots = hoff[H];
    const int64_t blk_bytes = int64_t(block) * d * ES;
    const int row_chunks = d / VEC;
    const int k_items = block * row_chunks;        // chunks per K block
    const int kblocks = block / VEC, dblocks = d / VEC;
    const int v_items = kblocks * dblocks;         // sub-blocks per V block
    const int kgroups = kblocks / 8;

    // K: step u covers chunks [1024 u, 1024 u + 1024) of the flat K buffer.
    // Flat indices fit 31 bits (checked by the launcher).
    int h = 0;
    const uint32_t k_total = uint32_t(total_slots) * uint32_t(k_items);
    for (uint32_t e0 = blockIdx.x * 1024u; e0 < k_total; e0 += gridDim.x * 1024u) {
        uint4 x[4];
        int64_t dst_off[4];
        // slot and in-slot offset of each group; a group of 256 chunks never
        // straddles slots and k_items >= 256, so the next group wraps at most once
        int slot = int(e0 / uint32_t(k_items));
        int cbase = int(e0 - uint32_t(slot) * uint32_t(k_items));
        if constexpr (WHOLE) {  // the step lies in one slot
            while (slot >= hoff[h + 1]) ++h;
            const int tok0 = gather_blk[slot] * block;
            const int valid = min(block, L - tok0) * row_chunks;
            const char* src = K + (int64_t(h % H_src) * L + tok0) * d * ES;
            char* dst = Kp + int64_t(e0) * 16;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int c = cbase + i * 256 + tid;
                x[i] = c < valid ? load_nt(src + int64_t(c) * 16) : make_uint4(0, 0, 0, 0);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) store_nt(dst + (i * 256 + tid) * 16, x[i]);
            continue;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t eg = e0 + i * 256u;  // first chunk of the group
            if (i > 0) {
                cbase += 256;
                if (cbase >= k_items) {
                    cbase -= k_items;
                    ++slot;
                }
            }
            dst_off[i] = -1;
            x[i] = make_uint4(0, 0, 0, 0);
            if (eg < k_total) {
                const int c = cbase + tid;
                while (slot >= hoff[h + 1]) ++h;
                const int tok0 = gather_blk[slot] * block;
                const int valid = min(block, L - tok0) * row_chunks;
                if (c < valid)
                    x[i] = load_nt(K + (int64_t(h % H_src) * L + tok0) * d * ES + int64_t(c) * 16);
                dst_off[i] = int64_t(eg + tid) * 16;
            }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (dst_off[i] >= 0) store_nt(Kp + dst_off[i], x[i]);
    }

    // V: step u covers sub-blocks [256 u, 256 u + 256) of the flat V buffer,
    // one group of 64 per wave. Sub-block t of a slot: kb = t % 8 + 8 ((t / 64)
    // % kgroups), db = (t / 8) % 8 + 8 ((t / 64) / kgroups).
    h = 0;
    const uint32_t v_total = uint32_t(total_slots) * uint32_t(v_items);
    for (uint32_t t0 = blockIdx.x * 256u; t0 < v_total; t0 += gridDim.x * 256u) {
        const uint32_t tt = t0 + tid;
        if (tt >= v_total) continue;  // whole waves: v_total is a multiple of 64
        const int slot = int(tt / uint32_t(v_items));
        const int t = int(tt - uint32_t(slot) * uint32_t(v_items));
        while (slot >= hoff[h + 1]) ++h;
        const int tok0 = gather_blk[slot] * block;
        const int cnt = min(block, L - tok0);
        const char* src = V + (int64_t(h % H_src) * L + tok0) * d * ES;
        char* dst = Vp + int64_t(slot) * blk_bytes;
        const int grp = t >> 6;
        const int kb = (t & 7) + 8 * (grp % kgroups);
        const int db = ((t >> 3) & 7) + 8 * (grp / kgroups);
        uint4 rows[VEC], cols[VEC];
#pragma unroll
        for (int rr = 0; rr < VEC; ++rr) {
            const int tk = kb * VEC + rr;
            rows[rr] = tk < cnt ? load_nt(src + (int64_t(tk) * d + db * VEC) * ES) : make_uint4(0, 0, 0, 0);
        }
        if constexpr (BF16) transpose8x8_b16(rows, cols);
        else transpose4x4_b32(rows, cols);
#pragma unroll
        for (int c = 0; c < VEC; ++c)
            store_nt(dst + (int64_t(db * VEC + c) * block + kb * VEC) * ES, cols[c]);
    }
}

}  // namespace

hipError_t launch_demand_gather(const Geom& g, const uint64_t* mask, const void* K, const void* V,
                                uint64_t* demand, int32_t* head_off, int32_t* slot_of,
                                int32_t* gather_blk, void* Kp, void* Vp, hipStream_t s) {
    (void)hipGetLastError();
    union_kernel<<<g.H, 256, 0, s>>>(mask, g.nq, g.W, demand);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    offsets_kernel<<<g.H, 256, 0, s>>>(demand, g.H, g.n, g.W, head_off, slot_of, gather_blk);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    // One workgroup per CU walks the windows (measured best against 128..2048
    // workgroups); the demand total is read on the device, so the grid is fixed.
    return launch_gather(g, g.H, head_off, gather_blk, K, V, Kp, Vp, s);
}

// Packed copies of `slots` (virtual) heads: virtual head v reads K/V head v % g.H.
hipError_t launch_gather(const Geom& g, int n_vheads, const int32_t* head_off,
                         const int32_t* gather_blk, const void* K, const void* V, void* Kp,
                         void* Vp, hipStream_t s) {
    const int vec = g.bf16 ? 8 : 4;
    const int v_items = (g.d / vec) * (g.block / vec);  // V sub-blocks per slot
    const int k_items = g.block * (g.d / vec);            // K chunks per slot
    const int64_t max_slots = int64_t(n_vheads) * g.n;
    if (k_items % 256 == 0 && v_items % 64 == 0 && (g.block / vec) % 8 == 0 &&
        (g.d / vec) % 8 == 0 && max_slots * k_items + int64_t(kStreamGrid) * 1024 < (int64_t(1) << 31)) {
        const bool whole = k_items % 1024 == 0;
        auto* kern = g.bf16 ? (whole ? gather_stream_kernel<true, true> : gather_stream_kernel<true, false>)
                            : (whole ? gather_stream_kernel<false, true> : gather_stream_kernel<false, false>);
        kern<<<kStreamGrid, 256, 0, s>>>(head_off, gather_blk, (const char*)K, (const char*)V,
                                         (char*)Kp, (char*)Vp, n_vheads, g.L, g.d, g.block, g.H);
        return hipGetLastError();
    }
    const int grid = kGatherGrid;
    const int ws = v_items >= 256 ? 1 : min(kMaxWS, (256 + v_items - 1) / v_items);
    if (g.bf16)
        gather_kernel<true><<<grid, 256, 0, s>>>(head_off, gather_blk, (const char*)K,
                                                 (const char*)V, (char*)Kp, (char*)Vp, n_vheads,
                                                 g.L, g.d, g.block, ws, g.H);
    else
        gather_kernel<false><<<grid, 256, 0, s>>>(head_off, gather_blk, (const char*)K,
                                                  (const char*)V, (char*)Kp, (char*)Vp, n_vheads,
                                                  g.L, g.d, g.block, ws, g.H);
    return hipGetLastError();
}

// Producer side of demand-directed routing (Section 5.1, Section 5.2): what
// producer p sends each consumer c = p+1, ..., p+R-1 (ring order) is c's
// demand cut to p's shard [lo, hi). The cut bitsets are laid out as virtual
// heads v = (consumer distance - 1) * H + h, after which the offsets and gather
// kernels above pack every consumer's blocks per head, row-major, consumer
// after consumer, in one pass.
__global__ __launch_bounds__(256) void provide_kernel(const uint64_t* __restrict__ demands,
                                                      int ranks, int producer, int H, int W,
                                                      int lo, int hi,
                                                      uint64_t* __restrict__ provide) {
    const int64_t total = int64_t(ranks - 1) * H * W;
    for (int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x; e < total;
         e += int64_t(gridDim.x) * 256) {
        const int w = int(e % W);
        const int64_t vh = e / W;
        const int h = int(vh % H), k = int(vh / H) + 1;
        const int c = (producer + k) % ranks;
        // bits of word w inside [lo, hi)
        const int b0 = w * 64;
        uint64_t keep = 0;
        const int from = max(lo, b0), to = min(hi, b0 + 64);
        if (from < to) {
            const int len = to - from;
            keep = (len == 64 ? ~uint64_t(0) : ((uint64_t(1) << len) - 1)) << (from - b0);
        }
        provide[e] = demands[(int64_t(c) * H + h) * W + w] & keep;
    }
}

hipError_t launch_pack_for_consumers(const Geom& g, const uint64_t* demands, int ranks,
                                     int producer, int lo, int hi, const void* K, const void* V,
                                     uint64_t* provide, int32_t* head_off, int32_t* slot_of,
                                     int32_t* gather_blk, void* Kp, void* Vp, hipStream_t s) {
    (void)hipGetLastError();
    const int nv = (ranks - 1) * g.H;
    const int64_t words = int64_t(nv) * g.W;
    const int64_t want = (words + 255) / 256;
    const int grid = int(want < 1024 ? (want > 0 ? want : 1) : 1024);
    provide_kernel<<<grid, 256, 0, s>>>(demands, ranks, producer, g.H, g.W, lo, hi, provide);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    offsets_kernel<<<nv, 256, 0, s>>>(provide, nv, g.n, g.W, head_off, slot_of, gather_blk);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_gather(g, nv, head_off, gather_blk, K, V, Kp, Vp, s);
}

}  // namespace sparsp
