// host_checks.cpp -- drives the host layer of libsom.so (paper_2608_24067_amd/csrc/som_api.cpp,
// built for the CPU alone with host_stubs.cpp) under AddressSanitizer and
// UndefinedBehaviorSanitizer: the CSR validator over valid and broken batches, the
// workspace queries over the whole size range, the schedule, and every argument check
// that must reject a call before it reaches a device.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "../../include/som.h"

static int failures = 0;

#define CHECK(cond)                                                                      \
    do {                                                                                 \
        if (!(cond)) {                                                                   \
            std::fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond); \
            ++failures;                                                                  \
        }                                                                                \
    } while (0)

static uint64_t lcg = 88172645463325252ull;
static uint32_t rnd(uint32_t n)
{
    lcg = lcg * 6364136223846793005ull + 1442695040888963407ull;
    return (uint32_t)((lcg >> 33) % n);
}

// A valid batch of N rows over V features, in heap arrays sized exactly.
static void make_batch(int64_t N, int64_t V, std::vector<int32_t> &rp, std::vector<int32_t> &ci)
{
    rp.assign((size_t)N + 1, 0);
    ci.clear();
    for (int64_t s = 0; s < N; ++s) {
        int32_t v = -1;
        const uint32_t len = rnd(6);
        for (uint32_t k = 0; k < len && v + 1 < V; ++k) {
            v += 1 + (int32_t)rnd((uint32_t)((V - 1 - v) < 5 ? (V - 1 - v) : 5));
            ci.push_back(v);
        }
        rp[(size_t)s + 1] = (int32_t)ci.size();
    }
}

static void validator()
{
    for (int round = 0; round < 200; ++round) {
        const int64_t N = rnd(40), V = 1 + rnd(50);
        std::vector<int32_t> rp, ci;
        make_batch(N, V, rp, ci);
        CHECK(som_validate_csr_host(rp.data(), ci.data(), N, V) == SOM_OK);
        CHECK(som_last_error()[0] == '\0');
        if (!ci.empty()) {
            std::vector<int32_t> bad = ci;
            const size_t p = rnd((uint32_t)bad.size());
            bad[p] = (round & 1) ? (int32_t)V : -1;  // outside [0, V)
            CHECK(som_validate_csr_host(rp.data(), bad.data(), N, V) == SOM_ERR_BAD_CSR);
            CHECK(std::strlen(som_last_error()) > 0);
        }
        if (N > 0 && rp[(size_t)N] >= 2) {
            // a repeated id: the row holding positions p-1, p
            for (int64_t s = 0; s < N; ++s)
                if (rp[(size_t)s + 1] - rp[(size_t)s] >= 2) {
                    std::vector<int32_t> dup = ci;
                    dup[(size_t)rp[(size_t)s] + 1] = dup[(size_t)rp[(size_t)s]];
                    CHECK(som_validate_csr_host(rp.data(), dup.data(), N, V) == SOM_ERR_BAD_CSR);
                    break;
                }
        }
        if (N >= 2) {
            std::vector<int32_t> drp = rp;
            drp[1] = drp[2] + 1;  // row pointers that decrease
            CHECK(som_validate_csr_host(drp.data(), ci.data(), N, V) == SOM_ERR_BAD_CSR);
        }
        // a slice of the batch: rows [1, N) keep the same id array as their base
        if (N >= 2) CHECK(som_validate_csr_host(rp.data() + 1, ci.data(), N - 1, V) == SOM_OK);
    }
    // offsets before the start of the id array, or past its declared end, are rejected before any id is read
    std::vector<int32_t> ids = {0, 1};
    std::vector<int32_t> neg = {-2, 0};
    CHECK(som_validate_csr_host(neg.data(), ids.data(), 1, 4) == SOM_ERR_BAD_CSR);
    std::vector<int32_t> empty_rp = {0, 0, 0};
    CHECK(som_validate_csr_host(empty_rp.data(), nullptr, 2, 3) == SOM_OK);
    CHECK(som_validate_csr_host(nullptr, nullptr, 0, 3) == SOM_ERR_INVALID_ARG);
    CHECK(som_validate_csr_host(empty_rp.data(), nullptr, -1, 3) == SOM_ERR_INVALID_ARG);
    CHECK(som_validate_csr_host(empty_rp.data(), nullptr, 2, 0) == SOM_ERR_INVALID_ARG);
    std::vector<int32_t> one = {0, 1};
    CHECK(som_validate_csr_host(one.data(), nullptr, 1, 3) == SOM_ERR_INVALID_ARG);
}

static void workspace_queries()
{
    const int64_t Ns[] = {0, 1, 7, 1000, 29900000, INT32_MAX - 1, INT32_MAX, -1};
    const int64_t Ms[] = {1, 255, 4096, 1 << 20, (1 << 20) + 1, 0};
    const int64_t Vs[] = {1, 30000, INT32_MAX - 1, INT32_MAX, 0};
    const int64_t nnzs[] = {0, 12, INT32_MAX, (int64_t)INT32_MAX + 1, -1};
    som_bmu_config cfgs[6] = {};
    cfgs[1].tile_samples = 16;
    cfgs[2].tile_samples = 32;
    cfgs[3].keep_order = 1;
    cfgs[4].tile_samples = 7;    // invalid
    cfgs[5].reserved[3] = 1;     // invalid
    for (int64_t N : Ns)
        for (int64_t M : Ms)
            for (int64_t V : Vs)
                for (int64_t nnz : nnzs)
                    for (int c = 0; c < 6; ++c) {
                        const bool valid = N >= 0 && N < INT32_MAX && M >= 1 && M <= (1 << 20) && V >= 1 &&
                                           V < INT32_MAX && nnz >= 0 && nnz <= INT32_MAX && c < 4;
                        const size_t a = som_bmu_workspace_bytes(N, M, V, nnz, &cfgs[c]);
                        const size_t b = som_bmu2_workspace_bytes(N, M, V, nnz, &cfgs[c]);
                        const size_t r = som_bmu_sf_workspace_bytes(N, M, V, nnz, &cfgs[c]);
                        CHECK((a != 0) == valid && (b != 0) == valid);
                        CHECK(!valid || (a % 256 == 0 && b >= a));
                        CHECK(r == 0 || (valid && r >= b));
                    }
    CHECK(som_bmu_workspace_bytes(10, 64, 100, 50, nullptr) == som_bmu_workspace_bytes(10, 64, 100, 50, &cfgs[0]));
    CHECK(som_update_workspace_bytes(30000, 1024, 500000, 16) > 0);
    CHECK(som_update_workspace_bytes(30000, 1025, 500000, 16) == 0);
    CHECK(som_update_workspace_bytes(0, 4, 10, 0) == 0);
    CHECK(som_update_workspace_bytes(10, 4, -1, 0) == 0);
    CHECK(som_update_workspace_bytes(10, 4, 10, -1) == 0);
}

static void rejected_calls()
{
    // fake device addresses: never dereferenced, every call below fails its host checks first
    float *W = reinterpret_cast<float *>(uintptr_t(1) << 20);
    uint16_t *H = reinterpret_cast<uint16_t *>(uintptr_t(1) << 20);
    double *d = reinterpret_cast<double *>(uintptr_t(2) << 20);
    int32_t *i = reinterpret_cast<int32_t *>(uintptr_t(3) << 20);
    float *f = reinterpret_cast<float *>(uintptr_t(4) << 20);
    void *ws = reinterpret_cast<void *>(uintptr_t(5) << 20);
    void *ws_odd = reinterpret_cast<void *>((uintptr_t(5) << 20) + 64);
    const size_t big = size_t(1) << 40;
    som_bmu_config bad = {};
    bad.keep_order = 2;
    som_bmu_config t16 = {};
    t16.tile_samples = 16;

    CHECK(som_codebook_norms(nullptr, 10, 10, d, nullptr) == SOM_ERR_INVALID_ARG);
    CHECK(som_codebook_norms(W, 10, 0, d, nullptr) == SOM_ERR_INVALID_ARG);
    CHECK(som_codebook_norms(W, 0, 10, d, nullptr) == SOM_ERR_INVALID_ARG);
    CHECK(som_codebook_norms(W, 10, (1 << 20) + 1, d, nullptr) == SOM_ERR_INVALID_ARG);
    CHECK(som_codebook_norms(W + 0, 10, 10, nullptr, nullptr) == SOM_ERR_INVALID_ARG);
    CHECK(som_codebook_norms(reinterpret_cast<float *>(uintptr_t(W) + 2), 10, 10, d, nullptr) == SOM_ERR_INVALID_ARG);
    CHECK(som_codebook_norms_f16(reinterpret_cast<uint16_t *>(uintptr_t(H) + 1), 10, 10, d, nullptr) ==
          SOM_ERR_INVALID_ARG);

    // N == 0 is a no-op for every phase
    CHECK(som_bmu_search(nullptr, nullptr, 10, 10, nullptr, nullptr, 0, 0, nullptr, nullptr, nullptr, 0, nullptr,
                         nullptr) == SOM_OK);
    CHECK(som_bmu_plan(nullptr, nullptr, 0, 0, 10, 10, nullptr, 0, nullptr, nullptr) == SOM_OK);
    CHECK(som_bmu_sweep(W, d, 10, 10, 0, 0, nullptr, 0, nullptr, nullptr) == SOM_OK);
    CHECK(som_bmu_finalize(d, 10, 10, i, 0, 0, i, d, nullptr, 0, nullptr, nullptr) == SOM_OK);
    CHECK(som_bmu2_search(W, d, 10, 10, i, i, 0, 0, i, d, i, d, nullptr, 0, nullptr, nullptr) == SOM_OK);
    CHECK(som_bmu_sf_search(W, d, 10, 10, i, i, f, 0, 0, i, d, nullptr, nullptr, nullptr, 0, nullptr, nullptr) ==
          SOM_OK);

    // sizes, pointers, configs and workspaces
    CHECK(som_bmu_search(W, d, 10, 10, i, i, -1, 0, i, d, ws, big, nullptr, nullptr) == SOM_ERR_INVALID_ARG);
    CHECK(som_bmu_search(W, d, 10, (1 << 20) + 1, i, i, 5, 5, i, d, ws, big, nullptr, nullptr) == SOM_ERR_INVALID_ARG);
    CHECK(som_bmu_search(W, d, 0, 10, i, i, 5, 5, i, d, ws, big, nullptr, nullptr) == SOM_ERR_INVALID_ARG);
    CHECK(som_bmu_search(W, d, 10, 10, i, i, 5, -5, i, d, ws, big, nullptr, nullptr) == SOM_ERR_INVALID_ARG);
    CHECK(som_bmu_search(W, d, 10, 10, i, nullptr, 5, 5, i, d, ws, big, nullptr, nullptr) == SOM_ERR_INVALID_ARG);
    CHECK(som_bmu_search(W, d, 10, 10, i, i, 5, 5, nullptr, d, ws, big, nullptr, nullptr) == SOM_ERR_INVALID_ARG);
    CHECK(som_bmu_search(W, d, 10, 10, i, i, 5, 5, i, d, nullptr, big, nullptr, nullptr) == SOM_ERR_WORKSPACE);
    CHECK(som_bmu_search(W, d, 10, 10, i, i, 5, 5, i, d, ws_odd, big, nullptr, nullptr) == SOM_ERR_WORKSPACE);
    CHECK(som_bmu_search(W, d, 10, 10, i, i, 5, 5, i, d, ws, 256, nullptr, nullptr) == SOM_ERR_WORKSPACE);
    CHECK(som_bmu_search(W, d, 10, 10, i, i, 5, 5, i, d, ws, big, &bad, nullptr) == SOM_ERR_INVALID_ARG);
    CHECK(som_bmu2_search(W, d, 10, 10, i, i, 5, 5, i, d, nullptr, d, ws, big, nullptr, nullptr) == SOM_ERR_INVALID_ARG);
    CHECK(som_bmu2_sweep(W, d, 10, 10, 5, 5, ws, som_bmu_workspace_bytes(5, 10, 10, 5, nullptr), nullptr, nullptr) ==
          SOM_ERR_WORKSPACE);
    CHECK(som_bmu_sf_search(W, d, 10, 10, i, i, nullptr, 5, 5, i, d, nullptr, nullptr, ws, big, nullptr, nullptr) ==
          SOM_ERR_INVALID_ARG);
    CHECK(som_bmu_sf_plan(i, i, f, 5, 5, 10, 10, ws, big, &t16, nullptr) == SOM_ERR_INVALID_ARG);
    CHECK(som_bmu_sweep_f16(reinterpret_cast<uint16_t *>(uintptr_t(H) + 1), d, 10, 10, 5, 5, ws, big, nullptr,
                            nullptr) == SOM_ERR_INVALID_ARG);
    uint32_t flags = 7;
    CHECK(som_bmu_input_flags(ws, big, 5, 10, 10, 5, nullptr, nullptr, nullptr) == SOM_ERR_INVALID_ARG);
    CHECK(som_bmu_input_flags(ws, 256, 5, 10, 10, 5, nullptr, &flags, nullptr) == SOM_ERR_WORKSPACE);
    CHECK(som_bmu_input_flags(ws, big, 0, 10, 10, 5, nullptr, &flags, nullptr) == SOM_OK && flags == 0);

    CHECK(som_update(nullptr, 10, 4, i, i, 5, 5, i, 1, 0, ws, big, nullptr) == SOM_ERR_INVALID_ARG);
    CHECK(som_update(W, 10, 4, i, i, 5, 5, i, 0, 0, ws, big, nullptr) == SOM_ERR_INVALID_ARG);
    CHECK(som_update(W, 10, 1025, i, i, 5, 5, i, 1, 0, ws, big, nullptr) == SOM_ERR_INVALID_ARG);
    CHECK(som_update(W, 10, 4, nullptr, i, 5, 5, i, 1, 0, ws, big, nullptr) == SOM_ERR_INVALID_ARG);
    CHECK(som_update(W, 10, 4, i, i, 5, 5, i, 1, -1, ws, big, nullptr) == SOM_ERR_INVALID_ARG);
    CHECK(som_update(W, 10, 4, i, i, 5, 5, i, 1, 0, ws_odd, big, nullptr) == SOM_ERR_WORKSPACE);
    CHECK(som_update(W, 10, 4, i, i, 5, 5, i, 1, 0, ws, 256, nullptr) == SOM_ERR_WORKSPACE);
    CHECK(som_update_f16(reinterpret_cast<uint16_t *>(uintptr_t(H) + 1), 10, 4, i, i, 5, 5, i, 1, 0, ws, big,
                         nullptr) == SOM_ERR_INVALID_ARG);
    CHECK(std::strlen(som_last_error()) > 0);
}

static void schedule()
{
    CHECK(som_sigma(1, 512.0, 0.5, 0.3) == 512.0);
    CHECK(som_sigma(-5, 8.0, 1.0, 0.3) == 8.0);
    CHECK(som_sigma(INT32_MAX, 8.0, 1.0, 0.3) == 1.0);
    const double odd[] = {NAN, INFINITY, -INFINITY, -1.0, 0.0, 0.5, 1.5, 2.4999, 1e300, 2147483647.4, 2147483648.0};
    for (double s : odd) {
        const int32_t r = som_radius(s);
        CHECK(r >= 1);
    }
    CHECK(som_radius(1e300) == INT32_MAX && som_radius(1.5) == 2 && som_radius(NAN) == 1);
}

int main()
{
    validator();
    workspace_queries();
    rejected_calls();
    schedule();
    if (failures) {
        std::fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    std::printf("host layer checks passed\n");
    return 0;
}
