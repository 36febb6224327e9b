// Dependency-aware placement (Section 4.3, Eq. 4): the block permutation on
// the device. The host parts live in host_plan.cpp:
//
// periodic_placement (host): rank floor(G s / B) of Eq. 4 for every block, with
// s / B read as the in-frame offset of the block's first token over the frame
// size F, i.e. rank floor(G ((j b) mod F) / F) for block j (Eq. 4 exactly when
// F is a multiple of b). A ragged last block stays last and belongs to the last
// rank, so every placed block keeps its size and the kernels' block structure
// holds. The placed order lists rank 0's blocks in logical order, then rank
// 1's, ...; perm[k] is the logical block at placed position k.
//
// permute_kernel: moves whole token blocks of a [H, L, d] tensor into placed
// order (Y block k = X block perm[k]) or back (Y block perm[k] = X block k).
// One workgroup per (head, block) copies the block's rows with 16-byte loads
// and stores, four in flight per thread. Every index read from perm is bounds
// checked, and a block pair of unequal valid rows copies the smaller count, so
// a malformed perm cannot make the kernel leave the tensors. HBM-bound: it
// reads and writes H L d w bytes.
//
// route_volume (host): the block transfers of producer p's shard (Section
// 5.1), summed over heads: dense ring forwarding moves the whole shard over
// each of the R-1 hops; relay forwarding moves, over hop k, the blocks that a
// consumer at distance >= k still needs; direct delivery moves each
// consumer's own blocks once.
//
// remote_demand (host): sum over heads of the demanded blocks outside the
// rank's own range [i0, i1) of the geometry, i.e. sum_{p != r} |D_{r,h,p}|
// of Eq. 3 in the layout (placed or contiguous) the geometry describes.
#include "sparsp_internal.h"

namespace sparsp {
namespace {

__global__ __launch_bounds__(256) void permute_kernel(const int32_t* __restrict__ perm,
                                                      const char* __restrict__ X,
                                                      char* __restrict__ Y, int n, int L,
                                                      int block, int row_bytes, int inverse) {
    const int k = blockIdx.x, h = blockIdx.y;
    const int j = perm[k];
    if (j < 0 || j >= n) return;
    const int src = inverse ? k : j, dst = inverse ? j : k;
    const int c_src = min(block, L - src * block), c_dst = min(block, L - dst * block);
    const int rows = min(c_src, c_dst);
    const int64_t head = int64_t(h) * L * row_bytes;
    const char* s = X + head + int64_t(src) * block * row_bytes;
    char* d = Y + head + int64_t(dst) * block * row_bytes;
    const int chunks = rows * (row_bytes / 16);
    for (int e0 = threadIdx.x; e0 < chunks; e0 += 4 * 256) {
        uint4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int e = e0 + u * 256;
            if (e < chunks) v[u] = reinterpret_cast<const uint4*>(s)[e];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int e = e0 + u * 256;
            if (e < chunks) reinterpret_cast<uint4*>(d)[e] = v[u];
        }
    }
}

}  // namespace

hipError_t launch_permute(const Geom& g, const int32_t* perm, const void* X, void* Y, bool inverse,
                          hipStream_t s) {
    (void)hipGetLastError();
    const int row_bytes = g.d * (g.bf16 ? 2 : 4);
    permute_kernel<<<dim3(g.n, g.H), 256, 0, s>>>(perm, (const char*)X, (char*)Y, g.n, g.L,
                                                  g.block, row_bytes, inverse ? 1 : 0);
    return hipGetLastError();
}

}  // namespace sparsp
