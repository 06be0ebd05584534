// Drives the host planner (csrc/plan.cpp) over a grid of shapes, edge cases included, for the
// AddressSanitizer / UndefinedBehaviorSanitizer build that tests/test_sanitizers.py makes.
// Exits non-zero when a plan breaks one of the invariants below (the sanitizers abort on their
// own findings).
#include <cstdio>
#include <cstdint>
#include <initializer_list>

#include "nmm_internal.h"

using namespace nmm;

static int fails = 0, checked = 0;
#define EXPECT(c)                                                                   \
    do {                                                                            \
        if (!(c)) {                                                                 \
            std::fprintf(stderr, "invariant failed: %s (line %d)\n", #c, __LINE__); \
            ++fails;                                                                \
        }                                                                           \
    } while (0)

static void check_gemv(int64_t batch, int64_t M, int64_t K, int64_t N, int dt, int path) {
    GemvPlan p;
    const nmm_status st = plan_gemv(batch, M, K, N, dt, path, &p);
    if (st != NMM_OK) return;
    if (batch == 0 || M == 0 || N == 0 || K == 0) return;
    ++checked;
    EXPECT(p.grid > 0);
    EXPECT(p.mt >= 1 && int64_t(p.mblocks) * p.mt >= M);
    if (p.path == NMM_PATH_MFMA) {
        EXPECT(int64_t(p.ks_full) * p.rows_full >= K);
        EXPECT(int64_t(p.ks_full - 1) * p.rows_full < K);
        EXPECT(int64_t(p.n_full) * kMfmaPanelCols >= N);
    } else {
        const int64_t chunks = (N + 7) / 8;
        EXPECT(int64_t(p.n_full) * p.cw_full + p.tail_chunks == chunks);
        if (p.n_full) EXPECT(int64_t(p.ks_full) * p.rows_full >= K && int64_t(p.ks_full - 1) * p.rows_full < K);
        if (p.tail_chunks) EXPECT(int64_t(p.ks_tail) * p.rows_tail >= K && int64_t(p.ks_tail - 1) * p.rows_tail < K);
        EXPECT(p.grid == batch * p.mblocks * int64_t(p.items));
    }
    if (p.split()) {
        EXPECT(p.n_tickets <= kMaxTickets);
        EXPECT(p.ws_bytes >= size_t(kTicketBytes) + size_t(p.part_floats) * 4);
    }
}

static void check_nt(int64_t M, int64_t K, int64_t N) {
    NtPlan q;
    if (plan_gemv_nt(M, K, N, &q) != NMM_OK || M == 0 || N == 0 || K == 0) return;
    EXPECT(int64_t(q.ks) * q.slice_k >= K);
    EXPECT(int64_t(q.row_blocks) * 4 * q.r >= N);
    EXPECT(q.grid == int64_t(q.mblocks) * q.row_blocks * q.ks);
}

int main() {
    const int64_t Ms[] = {0, 1, 2, 3, 4, 5, 8, 9, 16, 17, 32, 33, 100};
    const int64_t Ks[] = {0, 1, 7, 8, 13, 513, 1536, 4099, 7168, 16384, 33000};
    const int64_t Ns[] = {0, 1, 3, 8, 24, 64, 520, 576, 2112, 7168, 24576};
    const int64_t Bs[] = {0, 1, 3, 128};
    for (int64_t b : Bs)
        for (int64_t m : Ms)
            for (int64_t k : Ks)
                for (int64_t n : Ns)
                    for (int dt : {int(NMM_F16), int(NMM_BF16)})
                        for (int path : {int(NMM_PATH_AUTO), int(NMM_PATH_GEMV), int(NMM_PATH_MFMA)})
                            check_gemv(b, m, k, n, dt, path);
    for (int64_t m : Ms)
        for (int64_t k : Ks)
            for (int64_t n : Ns) check_nt(m, k, n);
    // argument checks on the limits, and invalid arguments
    GemvPlan p;
    EXPECT(plan_gemv(1, 1, int64_t(1) << 31, 8, NMM_BF16, NMM_PATH_AUTO, &p) == NMM_ERR_SHAPE);
    EXPECT(plan_gemv(1, -1, 8, 8, NMM_BF16, NMM_PATH_AUTO, &p) == NMM_ERR_SHAPE);
    EXPECT(plan_gemv(1, 1, 8, 8, 7, NMM_PATH_AUTO, &p) == NMM_ERR_DTYPE);
    EXPECT(plan_gemv(1, 1, 8, 8, NMM_BF16, 9, &p) == NMM_ERR_PATH);
    EXPECT(plan_gemv(2, 4, 8, 8, NMM_BF16, NMM_PATH_MFMA, &p) == NMM_ERR_PATH);
    EXPECT(plan_gemv(1, 1, 8, 8, NMM_BF16, NMM_PATH_AUTO, nullptr) == NMM_ERR_NULL);
    GemvArgs a;
    a.M = 1; a.K = 1024; a.N = 1000; a.dt = NMM_BF16; a.ldx = 1024; a.ldw = 1000; a.ldy = 1000;
    alignas(16) static uint16_t x[8], w[8];
    alignas(16) static float y[8];
    a.x = x; a.w = w; a.y = y;
    EXPECT(validate_gemv(a, NMM_PATH_AUTO) == NMM_OK);
    a.ldw = 1004;
    EXPECT(validate_gemv(a, NMM_PATH_AUTO) == NMM_ERR_ALIGN);
    a.ldw = 1000; a.w = w + 1;
    EXPECT(validate_gemv(a, NMM_PATH_AUTO) == NMM_ERR_ALIGN);
    a.w = w; a.K = int64_t(1) << 21; a.ldx = a.K; a.ldw = 1024;
    EXPECT(validate_gemv(a, NMM_PATH_AUTO) == NMM_ERR_SHAPE);   // W's extent reaches 2^31 bytes
    a.w = nullptr; a.K = 8; a.ldx = 8;
    EXPECT(validate_gemv(a, NMM_PATH_AUTO) == NMM_ERR_NULL);
    EXPECT(validate_workspace(nullptr, 0, 64) == NMM_ERR_WORKSPACE);
    std::printf("plan driver: %d plans checked, %d failures\n", checked, fails);
    return (fails || checked < 1000) ? 1 : 0;
}
