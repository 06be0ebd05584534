// Host-side argument checks and the GEMV partition.  Pure functions: no HIP calls, no device
// access, so they run (and are tested) on a machine without a GPU.
//
// The partition plays the role of Algorithm 2's init stage (Section IV-E), which splits a
// [K, N] weight into kParts K-slices x fractalNum 16-column fractals and spreads them evenly over
// at most 2P vector units.  Here the unit of work is a K-slice of a column panel (64 to 512
// columns; one 16-byte chunk per lane per row).  Panel width and K-split count follow rules
// fitted to measurements on MI355X over the decode shapes (see the comments below).
#include <algorithm>
#include <cstdlib>

#include "nmm_internal.h"

namespace nmm {
namespace {

constexpr int64_t kLimit = int64_t(1) << 31;

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
int64_t rup(int64_t a, int64_t b) { return cdiv(a, b) * b; }

int next_pow2(int64_t v) {
    int p = 1;
    while (p < v) p <<= 1;
    return p;
}

// The partition's tuning constants are fixed in the library, so a plan (and with it the order of
// every sum) depends on the shape alone.  Only a library built with -DNMM_TUNING_ENV, for tuning
// sweeps, lets the environment override them; the library as built for use reads no environment.
int64_t tuned(const char* name, int64_t dflt) {
#ifdef NMM_TUNING_ENV
    const char* s = std::getenv(name);
    if (!s || !*s) return dflt;
    char* end = nullptr;
    long long v = std::strtoll(s, &end, 10);
    return (end && *end == '\0' && v > 0) ? v : dflt;
#else
    (void)name;
    return dflt;
#endif
}

bool tuned_set(const char* name) {
#ifdef NMM_TUNING_ENV
    return std::getenv(name) != nullptr;
#else
    (void)name;
    return false;
#endif
}

int m_tile_for(int64_t M) {
    if (M <= 1) return 1;
    if (M <= 2) return 2;
    if (M <= 4) return 4;
    if (M <= 8) return 8;
    return kMaxMTile;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

nmm_status validate_workspace(const void* ws, size_t bytes, size_t need) {
    if (need == 0) return NMM_OK;
    if (!ws || bytes < need || (reinterpret_cast<uintptr_t>(ws) & 255u) != 0) return NMM_ERR_WORKSPACE;
    return NMM_OK;
}

nmm_status validate_gemv(const GemvArgs& a, int path) {
    if (path != NMM_PATH_AUTO && path != NMM_PATH_GEMV && path != NMM_PATH_MFMA) return NMM_ERR_PATH;
    if (a.dt != NMM_F16 && a.dt != NMM_BF16) return NMM_ERR_DTYPE;
    if (a.batch < 0 || a.M < 0 || a.K < 0 || a.N < 0) return NMM_ERR_SHAPE;
    if (a.M >= kLimit || a.K >= kLimit || a.N >= kLimit) return NMM_ERR_SHAPE;
    if (a.ldx < 0 || a.ldw < 0 || a.ldy < 0 || a.ldx >= kLimit || a.ldw >= kLimit || a.ldy >= kLimit)
        return NMM_ERR_SHAPE;
    if (a.sx < 0 || a.sw < 0 || a.sy < 0) return NMM_ERR_SHAPE;
    if (a.batch == 0 || a.M == 0 || a.N == 0) return NMM_OK;          // nothing is touched
    if (!a.y && !a.ybf) return NMM_ERR_NULL;                         // some output is required
    if (a.y && a.ldy < a.N) return NMM_ERR_SHAPE;
    if (a.ybf && (a.ybf_ldm < 0 || a.ybf_ldm >= kLimit)) return NMM_ERR_SHAPE;
    if (a.ybf && (a.ybf_group <= 0 || a.ybf_keep <= 0 || a.ybf_keep > a.ybf_group)) return NMM_ERR_ARG;
    if (a.ybf_away != 0 && a.ybf_away != 1) return NMM_ERR_ARG;
    if ((a.y && (reinterpret_cast<uintptr_t>(a.y) & 3u)) || (reinterpret_cast<uintptr_t>(a.ybf) & 1u))
        return NMM_ERR_ALIGN;
    if (a.K == 0) return NMM_OK;                                      // y = 0; x and W unused
    if (!a.x || !a.w) return NMM_ERR_NULL;
    if (a.ldx < a.K || a.ldw < a.N) return NMM_ERR_SHAPE;
    if (!aligned16(a.x) || !aligned16(a.w) || a.ldx % 8 || a.ldw % 8 || a.sx % 8 || a.sw % 8)
        return NMM_ERR_ALIGN;
    const int64_t extent = ((a.K - 1) * a.ldw + rup(a.N, 8)) * 2;    // bytes of one W
    if (extent >= kLimit) return NMM_ERR_SHAPE;
    // bytes of x one row block reads (blocks are at most 32 rows)
    const int64_t x_extent = ((std::min<int64_t>(a.M, 32) - 1) * a.ldx + rup(a.K, 8)) * 2;
    if (x_extent >= kLimit) return NMM_ERR_SHAPE;
    return NMM_OK;
}

// The matrix-core partition: 128-column panels, K-slices of whole 64-row stages, x tiles of
// 16 or 32 rows.  Splits are added only until the grid reaches about 256 workgroups: every
// workgroup pays a fixed start-up latency and split-K tail, so one round of long streams beats
// more, shorter ones (measured on the W_UQ, W_O and down shapes).
nmm_status plan_mfma(int64_t M, int64_t K, int64_t N, GemvPlan* p) {
    GemvPlan q;
    q.path = NMM_PATH_MFMA;
    q.mt = M <= 16 ? 16 : 32;
    q.mblocks = static_cast<int>(std::max<int64_t>(1, cdiv(M, q.mt)));
    q.unroll = 1;
    q.cw_full = kMfmaPanelCols / 8;
    q.n_full = static_cast<int>(cdiv(N, kMfmaPanelCols));
    if (M == 0 || N == 0 || K == 0) {
        *p = q;
        return NMM_OK;
    }
    const int64_t panels = int64_t(q.mblocks) * q.n_full;
    const int64_t want = tuned("NMM_GEMV_TARGET", kMfmaTargetGrid);
    const int64_t ks_cap = tuned("NMM_GEMV_MAXSPLIT", 16);
    int64_t ks_want = 1;
    const double ratio = double(want) / double(panels);
    while (ks_want < ks_cap && double(ks_want) * 1.41421356 < ratio) ks_want *= 2;
    int64_t r = rup(cdiv(K, ks_want), kMfmaStageRows);
    int64_t k = cdiv(K, r);
    if (panels > kMaxTickets) {
        k = 1;
        r = rup(K, kMfmaStageRows);
    }
    q.ks_full = static_cast<int>(k);
    q.rows_full = static_cast<int>(r);
    q.ks_max = q.ks_full;
    q.items = q.n_full * q.ks_full;
    q.grid = int64_t(q.mblocks) * q.items;
    if (q.split()) {
        q.n_tickets = panels;
        q.part_floats = panels * q.ks_max * int64_t(q.mt) * kMfmaPanelCols;
        q.ws_bytes = static_cast<size_t>(kTicketBytes + q.part_floats * 4);
    }
    *p = q;
    return NMM_OK;
}

nmm_status plan_gemv(int64_t batch, int64_t M, int64_t K, int64_t N, int dt, int path, GemvPlan* p,
                     int unroll) {
    if (!p) return NMM_ERR_NULL;
    if (dt != NMM_F16 && dt != NMM_BF16) return NMM_ERR_DTYPE;
    if (path != NMM_PATH_AUTO && path != NMM_PATH_GEMV && path != NMM_PATH_MFMA) return NMM_ERR_PATH;
    if (batch < 0 || M < 0 || K < 0 || N < 0 || M >= kLimit || K >= kLimit || N >= kLimit)
        return NMM_ERR_SHAPE;
    GemvPlan q;
    // AUTO (single matrices; batched calls always stream): the streaming GEMV for one row, the
    // matrix cores from kMfmaMinMDefault rows on.  At two rows the matrix-core launch wins only
    // where its plan needs no K-split: its split-K tail (16-row partials) costs more than the
    // GEMV's second row.  Measured on MI355X: W_UQ [1536, 24576] (one slice) 15.8 against
    // 16.3 us; W_O [16384, 7168] (4 slices) 42.2 against 41.1; down [7168, 2112] (16 slices)
    // 14.0 against 10.3.
    if (path == NMM_PATH_AUTO) {
        const int64_t mfma_min_m = tuned("NMM_MFMA_MIN_M", kMfmaMinMDefault);
        path = NMM_PATH_GEMV;
        if (batch <= 1 && M >= mfma_min_m) {
            path = NMM_PATH_MFMA;
        } else if (batch <= 1 && M == 2 && K > 0 && N > 0) {
            GemvPlan m;
            if (plan_mfma(M, K, N, &m) == NMM_OK && m.ks_full == 1) path = NMM_PATH_MFMA;
        }
    }
    if (path == NMM_PATH_MFMA) {
        if (batch > 1) return NMM_ERR_PATH;
        return plan_mfma(M, K, N, p);
    }
    q.path = NMM_PATH_GEMV;
    q.mt = m_tile_for(M);
    q.mblocks = static_cast<int>(std::max<int64_t>(1, cdiv(M, q.mt)));
    const int64_t chunks = cdiv(N, 8);
    const int64_t mats = std::max<int64_t>(batch, 1) * q.mblocks;
    const int64_t w_bytes = mats * K * chunks * 16;
    // Measured on MI355X over the decode shapes: 1- and 2-row tiles stream best with about one
    // workgroup per compute unit -- for weights up to 100 MB with 16 row-steps in flight per lane
    // and as few K-slices as the panel count allows (the split-K gather is a serial tail), for
    // larger weights with 8 in flight and panels up to 512 columns.  Taller tiles keep 4 in
    // flight and more workgroups.
    const bool narrow_m = q.mt <= 2;
    const bool deep = narrow_m && w_bytes <= int64_t(100) << 20;
    q.unroll = unroll > 0 ? unroll : static_cast<int>(tuned("NMM_GEMV_UNROLL", deep ? 16 : narrow_m ? 8 : 4));
    if (q.unroll != 2 && q.unroll != 4 && q.unroll != 8 && q.unroll != 16) q.unroll = 8;
    if (q.unroll == 16 && q.mt > 2) q.unroll = 8;                  // 16 only for 1- and 2-row tiles
    const int U = q.unroll;
    // Panel width (measured on MI355X over the decode shapes): as wide as possible, up to 32
    // chunks (64 for 16-row tiles and for 1-2-row tiles of weights over 100 MB), while the launch
    // still has >= 24 panels in total and every row is split into >= 2 panels; never narrower
    // than 8 chunks (128-byte row segments).
    int min_cw = static_cast<int>(tuned("NMM_GEMV_MINCW", 8));
    if (min_cw > kPanelChunks || (min_cw & (min_cw - 1))) min_cw = 8;
    int cw = static_cast<int>(tuned("NMM_GEMV_MAXCW", (q.mt >= 16 || (narrow_m && !deep)) ? 64 : 32));
    if (cw > kPanelChunks || (cw & (cw - 1)) || cw < min_cw) cw = std::max(min_cw, 32);
    // Workgroups wanted: one per ~100 KB of W, between 256 and 768 (fewer leave HBM idle; more
    // only add split-K gather work); 256 for the deep-prefetch plans.
    const int64_t want = tuned("NMM_GEMV_TARGET",
                                 narrow_m ? 256 : std::max<int64_t>(256, std::min<int64_t>(768, w_bytes / 100000)));
    while (cw > min_cw && (mats * cdiv(chunks, cw) < 24 || chunks < 2 * cw)) cw /= 2;
    // deep plans trade K-slices for narrower panels while twice the panels still fit the target
    if (deep && U == 16 && !tuned_set("NMM_GEMV_MAXCW"))
        while (cw > min_cw && 2 * mats * cdiv(chunks, cw) <= want) cw /= 2;
    // K-slices per panel: the power of two nearest want / panels, capped (fewer for tall row
    // tiles, whose partial sums are MT times larger)
    const int64_t ks_cap = tuned("NMM_GEMV_MAXSPLIT", q.mt >= 8 ? 8 : 16);
    q.cw_full = cw;
    q.n_full = static_cast<int>(chunks / cw);
    q.tail_chunks = static_cast<int>(chunks % cw);
    if (q.tail_chunks) {
        // the staged x slice of a tail item must fit the LDS budget: rows_tail * mt * 4 bytes,
        // with rows_tail >= kWaves * (64 / tail_cw) * U
        int lds_cw = 1;
        while (int64_t(kWaves) * (kPanelChunks / lds_cw) * U * q.mt * 4 > kXStageBytes) lds_cw <<= 1;
        q.tail_cw = std::max(next_pow2(q.tail_chunks), lds_cw);
    }
    if (batch == 0 || M == 0 || N == 0 || K == 0) {
        q.items = 0;
        q.grid = 0;
        *p = q;
        return NMM_OK;
    }

    const int64_t rstep_full = int64_t(kWaves) * (kPanelChunks / q.cw_full);   // rows per WG step
    const int64_t rstep_tail = q.tail_chunks ? int64_t(kWaves) * (kPanelChunks / q.tail_cw) : 1;
    const int64_t steps_per_matrix = q.n_full * cdiv(K, rstep_full) +
                                     (q.tail_chunks ? cdiv(K, rstep_tail) : 0);
    (void)steps_per_matrix;
    const int64_t panels_all = mats * (q.n_full + (q.tail_chunks ? 1 : 0));
    int64_t ks_want = 1;
    {
        const double ratio = double(want) / double(std::max<int64_t>(panels_all, 1));
        if (tuned("NMM_GEMV_KS_ANY", 0) > 0) {
            ks_want = std::max<int64_t>(1, std::min<int64_t>(ks_cap, int64_t(ratio + 0.5)));
        } else {
            while (ks_want < ks_cap && double(ks_want) * 1.41421356 < ratio) ks_want *= 2;   // nearest power of two
            ks_want = std::min(ks_want, ks_cap);
        }
    }

    auto slice = [&](int64_t rstep, int& ks, int& rows) {
        const int64_t unit = rstep * U;
        const int64_t cap = std::max<int64_t>(unit, (kXStageBytes / (4 * q.mt * rstep)) / U * unit);
        int64_t r = std::min<int64_t>(std::min<int64_t>(rup(cdiv(K, ks_want), unit), cap), rup(K, unit));
        int64_t k = cdiv(K, r);
        r = std::min<int64_t>(cap, rup(cdiv(K, k), unit));   // rebalance the slices
        k = cdiv(K, r);
        ks = static_cast<int>(k);
        rows = static_cast<int>(r);
    };
    if (q.n_full) slice(rstep_full, q.ks_full, q.rows_full);
    if (q.tail_chunks) slice(rstep_tail, q.ks_tail, q.rows_tail);
    const int64_t panels = q.n_full + (q.tail_chunks ? 1 : 0);
    if (mats * panels > kMaxTickets) {
        // more panels than arrival counters: give every panel a single K-slice instead
        auto whole = [&](int64_t rstep, int& ks, int& rows) {
            const int64_t unit = rstep * U;
            ks = 1;
            rows = static_cast<int>(rup(K, unit));
        };
        if (q.n_full) whole(rstep_full, q.ks_full, q.rows_full);
        if (q.tail_chunks) whole(rstep_tail, q.ks_tail, q.rows_tail);
        if (std::max(q.rows_full, q.rows_tail) * int64_t(q.mt) * 4 > kXStageBytes) return NMM_ERR_SHAPE;
    }
    q.ks_max = std::max(q.ks_full, q.ks_tail);
    q.items = q.n_full * q.ks_full + (q.tail_chunks ? q.ks_tail : 0);
    q.grid = batch * q.mblocks * int64_t(q.items);
    if (q.split()) {
        q.n_tickets = mats * panels;
        q.part_floats = mats * panels * q.ks_max * int64_t(q.mt) * kPanelCols;
        q.ws_bytes = static_cast<size_t>(kTicketBytes + q.part_floats * 4);
    }
    *p = q;
    return NMM_OK;
}


// ---------------------------------------------------------------------------------------------
// The transposed-weight GEMV.  x's K-slice is staged in LDS as 16-bit values (at most
// kXStageBytes), so a slice holds at most 16384 / mt values of k; rows are dealt so that at
// least one workgroup per CU streams (4 r rows each, r at most 8).
// ---------------------------------------------------------------------------------------------
nmm_status validate_gemv_nt(const GemvArgs& a) {
    if (a.dt != NMM_F16 && a.dt != NMM_BF16) return NMM_ERR_DTYPE;
    if (a.M < 0 || a.K < 0 || a.N < 0 || a.M >= kLimit || a.K >= kLimit || a.N >= kLimit) return NMM_ERR_SHAPE;
    if (a.ldx < 0 || a.ldw < 0 || a.ldy < 0 || a.ldx >= kLimit || a.ldw >= kLimit || a.ldy >= kLimit)
        return NMM_ERR_SHAPE;
    if (a.M == 0 || a.N == 0) return NMM_OK;
    if (!a.y) return NMM_ERR_NULL;
    if (a.ldy < a.N) return NMM_ERR_SHAPE;
    if (reinterpret_cast<uintptr_t>(a.y) & 3u) return NMM_ERR_ALIGN;
    if (a.K == 0) return NMM_OK;
    if (!a.x || !a.w) return NMM_ERR_NULL;
    if (a.ldx < a.K || a.ldw < a.K) return NMM_ERR_SHAPE;
    if (!aligned16(a.x) || !aligned16(a.w) || a.ldx % 8 || a.ldw % 8) return NMM_ERR_ALIGN;
    const int64_t extent = ((a.N - 1) * a.ldw + rup(a.K, 8)) * 2;     // bytes of Wt
    if (extent >= kLimit) return NMM_ERR_SHAPE;
    const int64_t x_extent = ((std::min<int64_t>(a.M, 4) - 1) * a.ldx + rup(a.K, 8)) * 2;
    if (x_extent >= kLimit) return NMM_ERR_SHAPE;
    return NMM_OK;
}

nmm_status plan_gemv_nt(int64_t M, int64_t K, int64_t N, NtPlan* p) {
    NtPlan q;
    q.mt = M <= 1 ? 1 : M <= 2 ? 2 : 4;
    q.mblocks = static_cast<int>(std::max<int64_t>(1, cdiv(M, q.mt)));
    if (M == 0 || N == 0 || K == 0) {
        *p = q;
        return NMM_OK;
    }
    const int64_t slice_max = kXStageBytes / 2 / q.mt;          // 16384, 8192 or 4096 (16-bit x in LDS)
    int64_t ks = cdiv(K, slice_max);
    const int64_t slice = rup(cdiv(K, ks), 512);
    ks = cdiv(K, slice);
    q.slice_k = static_cast<int>(slice);
    q.ks = static_cast<int>(ks);
    const int64_t target_rb = std::max<int64_t>(1, 256 / (ks * q.mblocks));
    // at most 8 rows per wave: short rows (small K) then spread over more workgroups, which
    // measured faster for W_UQ's [24576, 1536] (768 workgroups) than 24 rows per wave
    int r = static_cast<int>(std::min<int64_t>(8, std::max<int64_t>(1, N / (4 * target_rb))));
    r = static_cast<int>(std::min<int64_t>(32, std::max<int64_t>(1, tuned("NMM_NT_ROWS", r))));
    // rows per load step (rgroup) times steps in flight is 8 loads per lane.  With eight rows per
    // step only one step is in flight, so the next step's loads wait for this step's multiply-adds;
    // with one row per step x is read from LDS for every load.  Measured on MI355X: one-row tiles
    // take two rows per step (four steps in flight; W_O [7168, 16384] 39.0 against 41.7 us with
    // eight, W_UQ [24576, 1536] 14.7 against 15.1), taller tiles, whose x reads per step grow with
    // MT, four (two steps in flight; at M = 2 W_O 46.6 against 49.1, W_UQ 15.6 against 16.7, down
    // [2112, 7168] 12.2 against 13.5 with its rows per wave raised from 2 to 4; at M = 4 W_O 55.8
    // against 61.7).  One row per wave (small N) keeps one.
    q.rgroup = r < 2 ? 1 : q.mt == 1 ? 2 : 4;
    const int rg = tuned("NMM_NT_GROUP", q.rgroup);
    if (rg == 1 || rg == 2 || rg == 4 || rg == 8) q.rgroup = rg;
    q.depth = (q.mt == 1 && tuned("NMM_NT_DEPTH", 8) == 16) ? 16 : 8;
    q.r = (r + q.rgroup - 1) / q.rgroup * q.rgroup;
    const int64_t rb = cdiv(N, 4 * q.r);
    if (rb >= kLimit) return NMM_ERR_SHAPE;
    q.row_blocks = static_cast<int>(rb);
    q.grid = int64_t(q.mblocks) * rb * ks;
    if (q.grid >= kLimit) return NMM_ERR_SHAPE;
    if (ks > 1) {
        q.n_tickets = int64_t(q.mblocks) * rb;
        if (q.n_tickets > kMaxTickets) return NMM_ERR_SHAPE;
        q.ws_bytes = size_t(kTicketBytes) + size_t(q.grid) * q.mt * 4 * q.r * 4;
    }
    *p = q;
    return NMM_OK;
}

}  // namespace nmm
