// Host-only driver for the sanitizer build of the C ABI layer: the argument
// checks of every entry point (the same rejection cases as the ctypes suite
// in test_abi_cpu.py), the success paths into the stub launchers, and the
// host planning code (chunk schedule, placement, Eq. 3 count, routing
// volumes) on real host arrays. Built with -fsanitize=address,undefined by
// test_host_sanitizers.py; any sanitizer report aborts the run, any wrong
// status makes it exit non-zero.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "../../include/sparsp.h"

extern int g_launches;

namespace {

int failures = 0;
int cases = 0;

// A 16-byte aligned dummy device address; the stubs never dereference it.
void* const P = reinterpret_cast<void*>(uintptr_t(1) << 20);
template <typename T = void>
T* at(uintptr_t off = 0) { return reinterpret_cast<T*>(reinterpret_cast<uintptr_t>(P) + off); }

void expect(const char* what, int line, long long rc, long long want, int launches_want) {
    ++cases;
    const bool msg_ok = want >= 0 || std::strlen(sparsp_last_error()) > 0;
    if (rc != want || g_launches != launches_want || !msg_ok) {
        ++failures;
        std::printf("FAIL line %d %s: rc %lld (want %lld), launches %d (want %d), error \"%s\"\n",
                    line, what, rc, want, g_launches, launches_want, sparsp_last_error());
    }
    g_launches = 0;
}
#define REJECT(call, want) expect(#call, __LINE__, (call), (want), 0)
#define ACCEPT(call, launches) expect(#call, __LINE__, (call), 0, (launches))

sparsp_geom geom(int H = 2, int L = 1024, int d = 128, int block = 128, int i0 = 0, int i1 = 8,
                 int dtype = SPARSP_BF16) {
    return sparsp_geom{H, L, d, block, i0, i1, dtype};
}

int scores(const sparsp_geom* g) {
    return sparsp_block_scores(g, P, P, at<float>(), at<float>(), at<float>(), nullptr);
}

int topk(sparsp_geom g, int keep, std::vector<int32_t> glob = {}, int n_global = -1) {
    return sparsp_topk_mask(&g, at<float>(), keep, glob.empty() ? nullptr : glob.data(),
                            n_global < 0 ? int(glob.size()) : n_global, at<uint64_t>(),
                            at<int32_t>(), nullptr);
}

int gather(sparsp_geom g, long long cap, uintptr_t koff = 0) {
    return sparsp_demand_union_gather(&g, at<uint64_t>(), at(koff), P, at<uint64_t>(),
                                      at<int32_t>(), at<int32_t>(), at<int32_t>(), P, P, cap,
                                      nullptr);
}

int attn(sparsp_geom g, int keep = 2, long long cap = 16, float scale = 0.125f,
         int out = SPARSP_BF16, void* Q = P) {
    return sparsp_block_sparse_attn(&g, Q, at<int32_t>(), keep, at<int32_t>(), P, P, cap, scale, P,
                                    out, nullptr, nullptr);
}

}  // namespace

int main() {
    const int E_INVALID = SPARSP_E_INVALID, E_DTYPE = SPARSP_E_DTYPE,
              E_UNSUPPORTED = SPARSP_E_UNSUPPORTED, E_CAPACITY = SPARSP_E_CAPACITY;

    // geometry
    REJECT(sparsp_block_scores(nullptr, P, P, at<float>(), at<float>(), at<float>(), nullptr),
           E_INVALID);
    { auto g = geom(0); REJECT(scores(&g), E_INVALID); }
    { auto g = geom(2, -5); REJECT(scores(&g), E_INVALID); }
    { auto g = geom(2, 1024, 128, 128, 0, 8, 7); REJECT(scores(&g), E_DTYPE); }
    { auto g = geom(2, 1024, 128, 128, 3, 3); REJECT(scores(&g), E_INVALID); }
    { auto g = geom(2, 1024, 128, 128, 0, 9); REJECT(scores(&g), E_INVALID); }
    { auto g = geom(2, 1024, 128, 128, -1, 2); REJECT(scores(&g), E_INVALID); }
    { auto g = geom(2, 4097 * 16, 128, 16, 0, 1); REJECT(scores(&g), E_UNSUPPORTED); }
    { auto g = geom(2, 1024, 100); REJECT(scores(&g), E_UNSUPPORTED); }
    { auto g = geom(2, 1024, 320); REJECT(scores(&g), E_UNSUPPORTED); }
    { auto g = geom(1024, 4096 * 4096, 128, 4096, 0, 1, SPARSP_F32); REJECT(scores(&g), E_INVALID); }
    { auto g = geom(); REJECT(sparsp_block_scores(&g, at(4), P, at<float>(), at<float>(),
                                                  at<float>(), nullptr), E_INVALID); }
    { auto g = geom(); REJECT(sparsp_block_scores(&g, P, nullptr, at<float>(), at<float>(),
                                                  at<float>(), nullptr), E_INVALID); }
    { auto g = geom(); ACCEPT(scores(&g), 1); }

    // top-k mask: n = 8, rows 2..5
    {
        const auto g = geom(2, 1024, 128, 128, 2, 6);
        REJECT(topk(g, 9), E_INVALID);
        REJECT(topk(g, 0), E_INVALID);
        REJECT(topk(g, 2, {7, 0}), E_INVALID);
        REJECT(topk(g, 2, {8}), E_INVALID);
        REJECT(topk(g, 2, {-1}), E_INVALID);
        REJECT(topk(g, 2, {}, 3), E_INVALID);
        std::vector<int32_t> many;
        for (int j = 10; j < 75; ++j) many.push_back(j);
        REJECT(topk(geom(2, 128 * 100, 128, 128, 0, 4), 90, many), E_UNSUPPORTED);
        auto gg = g;
        REJECT(sparsp_topk_mask(&gg, nullptr, 3, nullptr, 0, at<uint64_t>(), at<int32_t>(),
                                nullptr), E_INVALID);
        ACCEPT(topk(g, 3, {7, 7, 1}), 1);
        ACCEPT(topk(g, 8), 1);
    }

    // CDF mask
    {
        auto g = geom(2, 1024, 128, 128, 2, 6);
        auto cdf = [&](float tau, std::vector<int32_t> glob = {}, int ng = -1) {
            return sparsp_cdf_mask(&g, at<float>(), tau, glob.empty() ? nullptr : glob.data(),
                                   ng < 0 ? int(glob.size()) : ng, at<uint64_t>(), at<int32_t>(),
                                   at<int32_t>(), nullptr);
        };
        REJECT(cdf(0.0f), E_INVALID);
        REJECT(cdf(-0.5f), E_INVALID);
        REJECT(cdf(1.01f), E_INVALID);
        REJECT(cdf(std::nanf("")), E_INVALID);
        REJECT(cdf(0.9f, {8}), E_INVALID);
        REJECT(cdf(0.9f, {}, 2), E_INVALID);
        REJECT(sparsp_cdf_mask(&g, at<float>(), 0.9f, nullptr, 0, at<uint64_t>(), at<int32_t>(),
                               nullptr, nullptr), E_INVALID);
        ACCEPT(cdf(1.0f, {0}), 1);
    }

    // demand union and gather: H = 3, n = 8
    {
        const auto g = geom(3, 1000, 128, 128, 0, 8);
        REJECT(gather(g, 23), E_CAPACITY);
        REJECT(gather(g, 24, 8), E_INVALID);
        REJECT(gather(geom(3, 1000, 128, 100, 0, 10), 1000), E_UNSUPPORTED);
        REJECT(gather(geom(2, 300, 64, 30, 0, 10, SPARSP_F32), 1000), E_UNSUPPORTED);
        ACCEPT(gather(g, 24), 1);
    }

    // attention
    REJECT(attn(geom(), 0), E_INVALID);
    REJECT(attn(geom(), 9), E_INVALID);
    REJECT(attn(geom(), 2, 0), E_CAPACITY);
    REJECT(attn(geom(), 2, 16, 0.0f), E_INVALID);
    REJECT(attn(geom(), 2, 16, std::nanf("")), E_INVALID);
    REJECT(attn(geom(), 2, 16, 0.125f, 3), E_DTYPE);
    REJECT(attn(geom(2, 1024, 96)), E_UNSUPPORTED);
    REJECT(attn(geom(2, 256, 128, 32)), E_UNSUPPORTED);
    REJECT(attn(geom(2, 1024, 192, 128, 0, 8, SPARSP_F32), 2, 16, 0.125f, SPARSP_F32),
           E_UNSUPPORTED);
    REJECT(attn(geom(2, 1024, 64, 128, 0, 8, SPARSP_F32), 2, 16, 0.125f, SPARSP_BF16), E_DTYPE);
    REJECT(attn(geom(2, 4096, 64, 512, 0, 8, SPARSP_F32), 2, 16, 0.125f, SPARSP_F32),
           E_UNSUPPORTED);
    REJECT(attn(geom(), 2, 16, 0.125f, SPARSP_BF16, nullptr), E_INVALID);
    ACCEPT(attn(geom()), 1);
    ACCEPT(attn(geom(2, 1024, 64, 128, 0, 8, SPARSP_F32), 2, 16, 0.125f, SPARSP_F32), 1);

    // balanced and ordered attention, workspace size
    {
        auto g = geom();
        auto bal = [&](void* ws, long long ws_bytes, int keep = 4, int out = SPARSP_BF16) {
            return sparsp_block_sparse_attn_balanced(&g, P, at<int32_t>(), keep, at<int32_t>(), P,
                                                     P, 16, 0.1f, ws, ws_bytes, P, out, nullptr,
                                                     nullptr);
        };
        REJECT(bal(at(8), 1 << 20), E_INVALID);
        REJECT(bal(P, -1), E_INVALID);
        REJECT(bal(P, 1 << 20, 0), E_INVALID);
        REJECT(bal(P, 1 << 20, 9), E_INVALID);
        REJECT(bal(P, 1 << 20, 4, 7), E_DTYPE);
        ACCEPT(bal(P, 1 << 20), 1);
        ACCEPT(bal(nullptr, 0), 1);
        auto noalloc = [&](int keep, int out, const sparsp_geom* gg) {
            return sparsp_block_sparse_attn_balanced_noalloc(gg, P, at<int32_t>(), keep,
                                                             at<int32_t>(), P, P, 16, 0.1f, P, out,
                                                             nullptr, nullptr);
        };
        REJECT(noalloc(0, SPARSP_BF16, &g), E_INVALID);
        REJECT(noalloc(9, SPARSP_BF16, &g), E_INVALID);
        REJECT(noalloc(4, 7, &g), E_DTYPE);
        REJECT(noalloc(4, SPARSP_BF16, nullptr), E_INVALID);
        ACCEPT(noalloc(4, SPARSP_BF16, &g), 1);
        // the stand-in's workspace for 512 slots at d = 128 (33.8 MB) fits the fixed
        // 36 MiB array; at d = 256 (f32 only) the call takes the f32 path, no scratch
        auto g32 = geom(2, 1024, 64, 128, 0, 8, SPARSP_F32);
        ACCEPT(noalloc(4, SPARSP_F32, &g32), 1);
        REJECT(sparsp_attn_workspace_bytes(&g, 0), E_INVALID);
        auto bad = geom(2, 1024, 128, 128, 3, 3);
        REJECT(sparsp_attn_workspace_bytes(&bad, 4), E_INVALID);
        const long long wsb = sparsp_attn_workspace_bytes(&g, 4);
        expect("workspace bytes > 0", __LINE__, wsb > 0 ? 0 : -1, 0, 0);
        auto ord = [&](const int32_t* order, int keep = 4) {
            return sparsp_block_sparse_attn_ordered(&g, P, at<int32_t>(), keep, at<int32_t>(), P,
                                                    P, 16, 0.1f, order, P, SPARSP_BF16, nullptr,
                                                    nullptr);
        };
        REJECT(ord(nullptr), E_INVALID);
        REJECT(ord(at<int32_t>(), 0), E_INVALID);
        REJECT(ord(at<int32_t>(), 9), E_INVALID);
        ACCEPT(ord(at<int32_t>()), 1);
        REJECT(sparsp_row_order(&g, nullptr, at<int32_t>(), nullptr), E_INVALID);
        REJECT(sparsp_row_order(&g, at<int32_t>(), nullptr, nullptr), E_INVALID);
        REJECT(sparsp_row_order(&bad, at<int32_t>(), at<int32_t>(), nullptr), E_INVALID);
        ACCEPT(sparsp_row_order(&g, at<int32_t>(), at<int32_t>(), nullptr), 1);
    }

    // shard-by-shard calls, with the chunk schedule on real host arrays
    {
        auto g = geom(4, 1024, 128, 128, 0, 8);  // n = 8, W = 1
        std::vector<uint64_t> dem = {0x0fu, 0xf0u, 0xffu, 0x81u};
        std::vector<sparsp_chunk> arr(64);
        auto plan = [&](int R, int r, int a, int b, int cap = 64) {
            return sparsp_chunk_plan(&g, dem.data(), R, r, a, b, arr.data(), cap);
        };
        REJECT(plan(0, 0, 1, 1), E_INVALID);
        REJECT(plan(9, 0, 1, 1), E_INVALID);
        REJECT(plan(4, 4, 1, 1), E_INVALID);
        REJECT(plan(4, -1, 1, 1), E_INVALID);
        REJECT(plan(4, 0, 0, 1), E_INVALID);
        REJECT(plan(4, 0, 1, 0), E_INVALID);
        REJECT(plan(4, 0, 1, 1, 12), E_CAPACITY);
        REJECT(plan(4, 0, 1, 1, -1), E_INVALID);
        REJECT(sparsp_chunk_plan(&g, nullptr, 4, 0, 1, 1, arr.data(), 64), E_INVALID);
        expect("plan(4, 0, 1, 1) = 13 chunks", __LINE__, plan(4, 0, 1, 1), 13, 0);
        expect("plan(4, 3, 3, 2) = 1 + 2 + 2 + 2 chunks", __LINE__, plan(4, 3, 3, 2), 7, 0);
        expect("plan(1, 0, 1, 1) = 1 chunk", __LINE__, plan(1, 0, 1, 1), 1, 0);
        ACCEPT(sparsp_chunked_attn(&g, P, at<int32_t>(), 2, at<int32_t>(), P, P, 16, 0.125f,
                                   arr.data(), 7, at<float>(), at<float>(), nullptr), 1);

        auto g2 = geom();  // H = 2, n = 8
        auto part = [&](int lo, int hi, int h0, int h1, float* lse) {
            return sparsp_block_sparse_attn_part(&g2, P, at<int32_t>(), 2, at<int32_t>(), P, P, 16,
                                                 0.125f, lo, hi, h0, h1, at<float>(), lse, 0,
                                                 nullptr);
        };
        REJECT(part(0, 9, 0, 2, at<float>()), E_INVALID);
        REJECT(part(-1, 4, 0, 2, at<float>()), E_INVALID);
        REJECT(part(5, 4, 0, 2, at<float>()), E_INVALID);
        REJECT(part(0, 8, 1, 1, at<float>()), E_INVALID);
        REJECT(part(0, 8, 0, 3, at<float>()), E_INVALID);
        REJECT(part(0, 8, 0, 2, nullptr), E_INVALID);
        ACCEPT(part(2, 6, 1, 2, at<float>()), 1);
        auto merge = [&](int h0, int h1, uintptr_t a, uintptr_t b) {
            return sparsp_lse_merge(&g2, h0, h1, at<float>(a), at<float>(a + 8192), at<float>(b),
                                    at<float>(b + 8192), nullptr);
        };
        REJECT(merge(0, 3, 0, 4096), E_INVALID);
        REJECT(merge(1, 1, 0, 4096), E_INVALID);
        REJECT(merge(0, 2, 0, 0), E_INVALID);
        REJECT(merge(0, 2, 4, 4096), E_INVALID);
        ACCEPT(merge(0, 2, 0, 1 << 16), 1);
        sparsp_chunk bad{0, 0, 9, 0, 2, 0};
        REJECT(sparsp_chunked_attn(&g2, P, at<int32_t>(), 2, at<int32_t>(), P, P, 16, 0.125f, &bad,
                                   1, at<float>(), at<float>(), nullptr), E_INVALID);
    }

    // placement, Eq. 3 count and routing on real host arrays
    {
        std::vector<int32_t> perm(64), begin(9);
        auto place = [&](int L, int b, int F, int R) {
            return sparsp_periodic_placement(L, b, F, R, perm.data(), begin.data());
        };
        REJECT(place(0, 8, 64, 2), E_INVALID);
        REJECT(place(64, 0, 64, 2), E_INVALID);
        REJECT(place(64, 8, 0, 2), E_INVALID);
        REJECT(place(64, 8, 64, 0), E_INVALID);
        REJECT(place(64, 8, 64, 9), E_INVALID);
        REJECT(sparsp_periodic_placement(64, 8, 64, 2, nullptr, begin.data()), E_INVALID);
        ACCEPT(place(500, 8, 120, 8), 0);  // 63 blocks, ragged last block
        std::vector<int> seen(63, 0);
        for (int k = 0; k < 63; ++k) ++seen[perm[k]];
        int bad = 0;
        for (int j = 0; j < 63; ++j) bad += seen[j] != 1;
        expect("placement is a permutation", __LINE__, bad, 0, 0);
        expect("rank_begin[8] = 63", __LINE__, begin[8], 63, 0);

        auto g = geom();
        REJECT(sparsp_permute_blocks(&g, at<int32_t>(), P, P, 0, nullptr), E_INVALID);
        REJECT(sparsp_permute_blocks(&g, at<int32_t>(), P, at(8), 0, nullptr), E_INVALID);
        REJECT(sparsp_permute_blocks(&g, nullptr, P, at(4096), 0, nullptr), E_INVALID);
        ACCEPT(sparsp_permute_blocks(&g, at<int32_t>(), P, at(1 << 16), 1, nullptr), 1);

        auto gr = geom(3, 200 * 16, 64, 16, 50, 100, SPARSP_F32);  // n = 200, W = 4
        std::vector<uint64_t> dem(3 * 4, 0x5555555555555555ull);
        dem[3] = dem[7] = dem[11] = 0x55ull;  // bits past n stay clear
        long long remote = -1, total = -1;
        int64_t r64 = 0, t64 = 0;
        ACCEPT(sparsp_remote_demand(&gr, dem.data(), &r64, &t64), 0);
        remote = r64;
        total = t64;
        expect("demanded = 3 x 100", __LINE__, total, 300, 0);
        expect("remote = 300 - 3 x 25", __LINE__, remote, 225, 0);
        REJECT(sparsp_remote_demand(&gr, nullptr, &r64, &t64), E_INVALID);

        auto g4 = geom(4, 1024, 128, 128, 0, 8);  // n = 8
        std::vector<uint64_t> dems(4 * 4, 0xffull);
        int64_t dense = 0, relay = 0, direct = 0;
        ACCEPT(sparsp_route_volume(&g4, dems.data(), 4, 1, &dense, &relay, &direct), 0);
        expect("dense = 3 x 4 x 2", __LINE__, dense, 24, 0);
        expect("direct = 3 x 4 x 2", __LINE__, direct, 24, 0);
        expect("relay = 3 hops x 4 heads x 2 blocks", __LINE__, relay, 24, 0);
        REJECT(sparsp_route_volume(&g4, dems.data(), 1, 0, &dense, &relay, &direct), E_INVALID);
        auto pack = [&](int R, int p, long long cap, uintptr_t koff = 0) {
            return sparsp_pack_for_consumers(&g4, dems.data(), R, p, at(koff), P, at<uint64_t>(),
                                             at<int32_t>(), at<int32_t>(), at<int32_t>(), P, P,
                                             cap, nullptr);
        };
        REJECT(pack(1, 0, 1 << 20), E_INVALID);
        REJECT(pack(9, 0, 1 << 20), E_INVALID);
        REJECT(pack(4, 4, 1 << 20), E_INVALID);
        REJECT(pack(4, 0, 23), E_CAPACITY);
        REJECT(pack(4, 0, 1 << 20, 8), E_INVALID);
        ACCEPT(pack(4, 0, 24), 1);
        auto big = geom(300, 1024, 128, 128, 0, 8);
        REJECT(sparsp_pack_for_consumers(&big, dems.data(), 8, 0, P, P, at<uint64_t>(),
                                         at<int32_t>(), at<int32_t>(), at<int32_t>(), P, P,
                                         1 << 30, nullptr), E_UNSUPPORTED);
    }

    expect("version", __LINE__, sparsp_version(), 200, 0);
    std::printf("%d cases, %d failures\n", cases, failures);
    return failures ? 1 : 0;
}
