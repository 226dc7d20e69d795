// Exercises the shard library's pure host functions on random inputs, for a
// build under AddressSanitizer and UndefinedBehaviorSanitizer (no GPU
// needed): the host plan of a batch (validation and grouping of tokens by
// adapter), the host adapter packer and the sizing functions, each checked
// against a plain re-statement of what it must return, plus their argument
// errors.  Exit status 0 when every check passes.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <vector>

#include "bdlora.h"

static int g_fail = 0;
#define CHECK(c)                                                                 \
    do {                                                                         \
        if (!(c)) {                                                              \
            std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
            ++g_fail;                                                            \
        }                                                                        \
    } while (0)

// the plan, stated plainly: an id is kept when it names a loaded slot;
// groups are the slots in use, ascending; perm lists each group's tokens in
// token order
static void plan_reference(const std::vector<int>& loaded, const std::vector<int>& ids, std::vector<int>& vid,
                           std::vector<int>& gs, std::vector<int>& gst, std::vector<int>& gc, std::vector<int>& perm,
                           bool& bad) {
    const int S = (int)loaded.size(), T = (int)ids.size();
    vid.assign(T, -1);
    bad = false;
    for (int t = 0; t < T; ++t) {
        const int a = ids[t];
        if (a >= 0 && a < S && loaded[a]) vid[t] = a;
        else if (a != -1) bad = true;
    }
    gs.clear(); gst.clear(); gc.clear(); perm.clear();
    for (int s = 0; s < S; ++s) {
        const int start = (int)perm.size();
        for (int t = 0; t < T; ++t)
            if (vid[t] == s) perm.push_back(t);
        if ((int)perm.size() > start) {
            gs.push_back(s);
            gst.push_back(start);
            gc.push_back((int)perm.size() - start);
        }
    }
}

static void check_plan(std::mt19937& rng) {
    const int sizes[][2] = {{0, 1}, {1, 1}, {7, 3}, {64, 32}, {333, 20}, {4288, 512}, {5000, 8192}};
    for (auto& sz : sizes) {
        const int T = sz[0], S = sz[1];
        std::vector<int> loaded(S), ids(T);
        for (int s = 0; s < S; ++s) loaded[s] = (rng() % 10) != 0;
        for (int t = 0; t < T; ++t) ids[t] = (int)(rng() % (S + 4)) - 2;
        std::vector<int> vid(T + 1), gs(S + 1), gst(S + 1), gc(S + 1), perm(T + 1);
        int ng = -1;
        const int rc = bdlora_build_plan(loaded.data(), S, ids.data(), T, vid.data(), gs.data(), gst.data(), gc.data(),
                                         perm.data(), &ng);
        std::vector<int> rv, rgs, rgst, rgc, rp;
        bool bad;
        plan_reference(loaded, ids, rv, rgs, rgst, rgc, rp, bad);
        CHECK(rc == (bad ? BDLORA_ERR_BAD_ADAPTER : BDLORA_OK));
        CHECK(ng == (int)rgs.size());
        for (int t = 0; t < T; ++t) CHECK(vid[t] == rv[t]);
        for (int g = 0; g < ng && g < (int)rgs.size(); ++g) {
            CHECK(gs[g] == rgs[g]);
            CHECK(gst[g] == rgst[g]);
            CHECK(gc[g] == rgc[g]);
        }
        for (size_t i = 0; i < rp.size(); ++i) CHECK(perm[i] == rp[i]);
    }
    int ng = 0;
    const int loaded1[1] = {1};
    CHECK(bdlora_build_plan(loaded1, 1, nullptr, -1, nullptr, nullptr, nullptr, nullptr, nullptr, &ng) ==
          BDLORA_ERR_INVALID_ARG);
    CHECK(bdlora_build_plan(nullptr, 1, nullptr, 0, nullptr, nullptr, nullptr, nullptr, nullptr, &ng) ==
          BDLORA_ERR_INVALID_ARG);
    CHECK(bdlora_build_plan(loaded1, 0, nullptr, 0, nullptr, nullptr, nullptr, nullptr, nullptr, &ng) ==
          BDLORA_ERR_INVALID_ARG);
}

static bdlora_proj_desc proj(int kind, int d_in, std::vector<int> slices) {
    bdlora_proj_desc d;
    std::memset(&d, 0, sizeof(d));
    d.kind = kind;
    d.d_in = d_in;
    d.n_slices = (int)slices.size();
    for (size_t i = 0; i < slices.size(); ++i) d.slice_out[i] = slices[i];
    d.weight_format = BDLORA_WEIGHT_BF16;
    return d;
}

static long long up(long long v, long long m) { return (v + m - 1) / m * m; }

// the slot layout, stated element by element (see bdlora_pack_adapter_host)
static std::vector<uint16_t> layout_reference(const std::vector<bdlora_proj_desc>& P, int max_rank, int rank,
                                              const std::vector<std::vector<uint16_t>>& A,
                                              const std::vector<std::vector<uint16_t>>& B) {
    const int r8max = std::max(8, (max_rank + 7) / 8 * 8), r8 = (rank + 7) / 8 * 8;
    long long off = 0;
    std::vector<long long> aoff, boff;
    for (auto& d : P) {
        int N = 0;
        for (int s = 0; s < d.n_slices; ++s) N += d.slice_out[s];
        aoff.push_back(off);
        off = up(off + up((long long)d.n_slices * r8max, 16) * d.d_in, 128);
        boff.push_back(off);
        off = up(off + (long long)N * r8max, 128);
    }
    std::vector<uint16_t> out((size_t)off, 0);
    size_t k = 0;
    for (size_t p = 0; p < P.size(); ++p) {
        const auto& d = P[p];
        const int KS = d.d_in / 32;
        int col = 0;
        for (int s = 0; s < d.n_slices; ++s, ++k) {
            for (int j = 0; j < rank; ++j) {
                const int row = s * r8 + j, rb = row / 16, lr = row % 16;
                for (int kk = 0; kk < d.d_in; ++kk) {
                    const int ks = kk / 32, w = kk % 32, lane = lr + 16 * (w / 8);
                    out[(size_t)aoff[p] + ((size_t)rb * KS + ks) * 512 + lane * 8 + w % 8] = A[k][(size_t)kk * rank + j];
                }
            }
            for (int j = 0; j < rank; ++j)
                for (int n = 0; n < d.slice_out[s]; ++n)
                    out[(size_t)boff[p] + (size_t)(col + n) * r8 + j] = B[k][(size_t)j * d.slice_out[s] + n];
            col += d.slice_out[s];
        }
    }
    return out;
}

static void check_packer(std::mt19937& rng) {
    const std::vector<std::vector<bdlora_proj_desc>> sets = {
        {proj(BDLORA_COLUMN, 64, {32, 16, 16}), proj(BDLORA_ROW, 32, {48})},
        {proj(BDLORA_COLUMN, 96, {16})},
        {proj(BDLORA_COLUMN, 128, {64, 16, 16, 32}), proj(BDLORA_ROW, 64, {128}), proj(BDLORA_COLUMN, 32, {16})},
    };
    const int cases[][2] = {{8, 0}, {8, 3}, {16, 16}, {24, 9}, {40, 33}};
    for (auto& P : sets)
        for (auto& c : cases) {
            const int max_rank = c[0], rank = c[1];
            std::vector<std::vector<uint16_t>> A, B;
            std::vector<const uint16_t*> pa, pb;
            for (auto& d : P)
                for (int s = 0; s < d.n_slices; ++s) {
                    std::vector<uint16_t> a((size_t)d.d_in * rank), b((size_t)rank * d.slice_out[s]);
                    for (auto& v : a) v = (uint16_t)(1 + rng() % 0x3f00);
                    for (auto& v : b) v = (uint16_t)(1 + rng() % 0x3f00);
                    A.push_back(std::move(a));
                    B.push_back(std::move(b));
                }
            for (size_t i = 0; i < A.size(); ++i) {
                pa.push_back(A[i].data());
                pb.push_back(B[i].data());
            }
            int64_t bytes = 0;
            CHECK(bdlora_layout_slot_bytes(P.data(), (int)P.size(), max_rank, &bytes) == BDLORA_OK);
            int64_t slab = 0, ws = 0;
            CHECK(bdlora_pool_size(P.data(), (int)P.size(), 3, max_rank, 16, &slab, &ws) == BDLORA_OK);
            CHECK(slab == 3 * bytes);
            std::vector<uint16_t> got((size_t)bytes / 2, 0xffff);
            CHECK(bdlora_pack_adapter_layout(P.data(), (int)P.size(), max_rank, rank, pa.data(), pb.data(),
                                             got.data()) == BDLORA_OK);
            const auto ref = layout_reference(P, max_rank, rank, A, B);
            CHECK(ref.size() == got.size());
            CHECK(ref.size() == got.size() && std::memcmp(ref.data(), got.data(), got.size() * 2) == 0);
            int64_t elems = 0;
            CHECK(bdlora_adapter_elems(P.data(), (int)P.size(), rank, &elems) == BDLORA_OK);
            long long want = 0;
            for (auto& d : P)
                for (int s = 0; s < d.n_slices; ++s) want += (long long)d.d_in * rank + (long long)rank * d.slice_out[s];
            CHECK(elems == want);
            // errors: rank above max_rank, a non-finite value, null arrays
            CHECK(bdlora_pack_adapter_layout(P.data(), (int)P.size(), max_rank, max_rank + 1, pa.data(), pb.data(),
                                             got.data()) == BDLORA_ERR_INVALID_ARG);
            if (rank > 0) {
                const uint16_t keep = A[0][0];
                A[0][0] = 0x7fc0;
                CHECK(bdlora_pack_adapter_layout(P.data(), (int)P.size(), max_rank, rank, pa.data(), pb.data(),
                                                 got.data()) == BDLORA_ERR_INVALID_ARG);
                A[0][0] = keep;
                CHECK(bdlora_pack_adapter_layout(P.data(), (int)P.size(), max_rank, rank, nullptr, pb.data(),
                                                 got.data()) == BDLORA_ERR_INVALID_ARG);
            }
        }
    // descriptor errors
    bdlora_proj_desc bad = proj(BDLORA_COLUMN, 48, {16});
    int64_t b = 0, w = 0;
    CHECK(bdlora_layout_slot_bytes(&bad, 1, 8, &b) == BDLORA_ERR_SHAPE);
    bad = proj(BDLORA_COLUMN, 64, {24});
    CHECK(bdlora_pool_size(&bad, 1, 4, 8, 16, &b, &w) == BDLORA_ERR_SHAPE);
    bad = proj(7, 64, {16});
    CHECK(bdlora_pool_size(&bad, 1, 4, 8, 16, &b, &w) == BDLORA_ERR_INVALID_ARG);
    bdlora_proj_desc ok = proj(BDLORA_COLUMN, 64, {16});
    CHECK(bdlora_pool_size(&ok, 1, 0, 8, 16, &b, &w) == BDLORA_ERR_INVALID_ARG);
    CHECK(bdlora_pool_size(&ok, 1, 4, BDLORA_MAX_RANK + 1, 16, &b, &w) == BDLORA_ERR_INVALID_ARG);
    CHECK(bdlora_pool_size(nullptr, 1, 4, 8, 16, &b, &w) == BDLORA_ERR_INVALID_ARG);
    CHECK(bdlora_pool_size(&ok, 9, 4, 8, 16, &b, &w) == BDLORA_ERR_INVALID_ARG);
    // an adapter budget too small for the slots fails before any device work
    bdlora_pool_t pool = nullptr;
    CHECK(bdlora_layout_slot_bytes(&ok, 1, 8, &b) == BDLORA_OK);
    CHECK(bdlora_create_pool(&ok, 1, 0, 8, 16, b - 1, 0, &pool) == BDLORA_ERR_OOM && pool == nullptr);
    CHECK(bdlora_create_pool(&ok, 1, 4, 8, 16, 4 * b - 1, 0, &pool) == BDLORA_ERR_OOM && pool == nullptr);
    CHECK(bdlora_create_pool(&ok, 1, 4, 8, 16, -1, 0, &pool) == BDLORA_ERR_INVALID_ARG);
    CHECK(bdlora_last_error() != nullptr && std::strlen(bdlora_last_error()) > 0);
    // null pools
    int32_t v = 0;
    CHECK(bdlora_pool_slots(nullptr, &v) == BDLORA_ERR_INVALID_ARG);
    CHECK(bdlora_last_path(nullptr, &v) == BDLORA_ERR_INVALID_ARG);
    CHECK(bdlora_slot_bytes(nullptr) == 0);
    CHECK(bdlora_destroy_pool(nullptr) == BDLORA_ERR_INVALID_ARG);
}

int main() {
    std::mt19937 rng(12345);
    check_plan(rng);
    check_packer(rng);
    std::printf("host sanitizer driver: %d failed checks\n", g_fail);
    return g_fail == 0 ? 0 : 1;
}
