// Host side of the DIGEST per-partition library: argument validation, the
// partition's index maps (Eq. 2; halo and push sets of Sec. 3.2), the
// workspace layout, and the launch sequence of each C-ABI call.
#include "digest.h"
#include "kernels.h"

#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>
#include <numeric>
#include <string>
#include <vector>

using digest::SpmmBlock;

namespace {

thread_local std::string g_last_error;

digest_status fail(digest_status st, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return st;
}

// Kernel kinds reported by the instrumentation.
enum Kind : int32_t {
    K_PULL = 0,
    K_PUSH,
    K_SPMM_FWD,
    K_GEMM_FWD,
    K_GEMM_DW,
    K_REDUCE_DW,
    K_GEMM_DH,
    K_SPMM_BWD,
    K_LOSS,
    K_LOSS_MEAN,
    K_HALO_GRAD,
    K_GRAD_PUSH,
    K_GRAD_PULL,
    K_GAT_TRANSFORM,
    K_GAT_SCORES,
    K_GAT_SOFTMAX,
    K_GAT_AGG,
    K_GAT_EDGE_GRAD,
    K_GAT_PERM,
    K_GAT_AGG_T,
    K_GAT_SCORE_GRAD,
    K_GAT_SCORE_SUMS,
    K_GAT_DATT,
    K_GAT_DW,
    K_GAT_DGRAD,
    K_PAD_ROWS,
    K_SPMM_GEMM_FWD,
    K_SPMM_GEMM_BWD,
    K_RELU_MASK,
    K_TRANSPOSE_W,
    K_HALO_AGG,
    K_BND_ROWS,
    K_COUNT
};
const char *const kKindNames[K_COUNT] = {
    "pull_gather", "push_scatter", "spmm_fwd", "gemm_fwd_relu", "gemm_dw_splitk",
    "splitk_reduce_dw", "gemm_dgrad", "spmm_bwd_transposed", "softmax_xent", "loss_mean",
    "halo_gradient", "grad_push_add", "grad_pull_add", "gat_transform", "gat_scores",
    "gat_softmax", "gat_aggregate", "gat_edge_grad", "gat_transpose_edges",
    "gat_aggregate_transposed", "gat_score_grad", "gat_score_sums", "gat_datt", "gat_dw",
    "gat_dgrad", "pad_rows", "spmm_gemm_fwd", "spmm_gemm_bwd", "relu_mask", "transpose_w",
    "halo_aggregate", "boundary_rows"};

constexpr size_t kAlign = 256;
constexpr int32_t kMaxWidth = 65536;
constexpr int32_t kMaxLayers = 64;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Row stride of a library-owned buffer of rows `d` floats wide: a multiple
// of 4 floats, so that its rows hold whole 16-byte vectors.
int32_t padded_width(int32_t d) { return (d + 3) / 4 * 4; }

// Split-K factor for a contraction with an M x N result over K: at least
// `target` workgroups in all (kSplitTarget, or kSideSplitTarget on the side
// stream), at least kSplitMinRows rows of K per split,
// split starts on GEMM K-tile boundaries.  From that count up to twice it,
// the split whose workgroups fill whole rounds of the chip's kCUs compute
// units best is taken (the fewest splits among equals): a round of 800
// workgroups on 256 CUs leaves most CUs idle for its last quarter.
constexpr int64_t kSplitTarget = 768;
// A weight gradient on the side stream runs next to the memory-bound
// aggregations of the same backward: one workgroup per CU leaves them the
// rest of each CU (OGB-Products-shaped round 6.82 -> 6.70 ms against 768).
constexpr int64_t kSideSplitTarget = 256;
constexpr int64_t kSplitMinRows = 256;
constexpr int64_t kCUs = 256;

void splitk_plan(int64_t M, int64_t N, int64_t K, int32_t &splits, int32_t &kchunk,
                 int64_t target = kSplitTarget)
{
    const int64_t tiles = std::max<int64_t>(1, ((M + digest::kGemmBM - 1) / digest::kGemmBM) *
                                                   ((N + digest::kGemmBN - 1) / digest::kGemmBN));
    const int64_t cap = std::min<int64_t>(256, std::max<int64_t>(1, K / kSplitMinRows));
    const int64_t lo = std::max<int64_t>(1, std::min<int64_t>((target + tiles - 1) / tiles, cap));
    // the split count and K-chunk that a requested count rounds to
    auto realise = [&](int64_t want, int64_t &chunk) {
        chunk = (K + want - 1) / want;
        chunk = (chunk + digest::kGemmBK - 1) / digest::kGemmBK * digest::kGemmBK;
        if (chunk <= 0)
            chunk = digest::kGemmBK;
        return std::max<int64_t>(1, (K + chunk - 1) / chunk);
    };
    int64_t best_chunk = 0;
    int64_t best = realise(lo, best_chunk);
    auto fill = [&](int64_t sp) {
        const int64_t wg = tiles * sp;
        return (double)wg / (double)(((wg + kCUs - 1) / kCUs) * kCUs);
    };
    for (int64_t want = lo + 1; want <= std::min<int64_t>(cap, 2 * lo); ++want) {
        int64_t chunk = 0;
        const int64_t sp = realise(want, chunk);
        if (fill(sp) > fill(best) + 1e-9) {
            best = sp;
            best_chunk = chunk;
        }
    }
    splits = (int32_t)best;
    kchunk = (int32_t)best_chunk;
}

// Workgroup tile of C for a GEMM (see GemmArgs::tile): 64x64 keeps enough
// workgroups for the partition-sized products and for every split-K weight
// gradient; tall products (>= 20,000 rows) run faster on 128x128 tiles,
// whose waves each own a 64x64 block (one LDS fragment read per MFMA).
int32_t gemm_tile_for(int64_t M, int64_t N, int64_t K, bool contraction_over_rows)
{
    if (contraction_over_rows)
        return 0;
    return (M >= 20000 && N >= 128) ? 3 : 0;
}

// A CSR's first n_rows rows split at kFuseLong entries, for the fused
// passes: the long rows (count, entries), the distinct source rows (of
// n_cols) that the short and the long rows read, and per tile of kFuseRows
// rows the order in which its waves take the rows: by descending entry
// count, long rows (read back, cheap) last, so that the waves' shares are
// even.
void fuse_stats(const std::vector<int32_t> &rowptr, const std::vector<int32_t> &col,
                int32_t n_rows, int64_t n_cols, int64_t &long_rows, int64_t &long_nnz,
                int64_t &src_short, int64_t &src_long, std::vector<uint8_t> &order)
{
    long_rows = long_nnz = src_short = src_long = 0;
    std::vector<uint8_t> seen((size_t)n_cols, 0);
    for (int32_t i = 0; i < n_rows; ++i) {
        const int32_t len = rowptr[i + 1] - rowptr[i];
        const bool lng = len > digest::kFuseLong;
        long_rows += lng;
        long_nnz += lng ? len : 0;
        for (int32_t k = rowptr[i]; k < rowptr[i + 1]; ++k)
            seen[col[k]] |= lng ? 2 : 1;
    }
    for (const uint8_t v : seen) {
        src_short += v & 1;
        src_long += v >> 1;
    }
    static_assert(digest::kFuseRows <= 256, "tile offsets fit a byte");
    order.resize(n_rows);
    for (int32_t t0 = 0; t0 < n_rows; t0 += digest::kFuseRows) {
        const int32_t nr = std::min(digest::kFuseRows, n_rows - t0);
        auto work = [&](int32_t i) {
            const int32_t len = rowptr[t0 + i + 1] - rowptr[t0 + i];
            return len > digest::kFuseLong ? -1 : len;
        };
        std::vector<int32_t> idx(nr);
        for (int32_t i = 0; i < nr; ++i)
            idx[i] = i;
        std::stable_sort(idx.begin(), idx.end(),
                         [&](int32_t a, int32_t b) { return work(a) > work(b); });
        for (int32_t i = 0; i < nr; ++i)
            order[t0 + i] = (uint8_t)idx[i];
    }
}

// Aggregation blocks of a CSR: every long row gets a block of its own (those
// come first, by default longest first, so that the longest start earliest
// and do not set the launch's tail; else in row order); runs of consecutive
// short rows are packed one per wave.  Returns the number of long-row
// blocks.
int32_t build_blocks(const std::vector<int32_t> &rowptr, int32_t n_rows,
                     std::vector<SpmmBlock> &blocks, bool longest_first = true,
                     int32_t long_row = digest::kSpmmLongRow)
{
    const int32_t waves = digest::kSpmmThreads / 64;
    blocks.clear();
    for (int32_t r = 0; r < n_rows; ++r)
        if (rowptr[r + 1] - rowptr[r] > long_row)
            blocks.push_back({r, 0, rowptr[r], rowptr[r + 1]});
    if (longest_first)
        std::stable_sort(blocks.begin(), blocks.end(),
                         [](const SpmmBlock &a, const SpmmBlock &b) {
                             return a.ke - a.kb > b.ke - b.kb;
                         });
    const int32_t n_long = (int32_t)blocks.size();
    int32_t first = -1, count = 0;
    for (int32_t r = 0; r <= n_rows; ++r) {
        const bool short_row = r < n_rows && rowptr[r + 1] - rowptr[r] <= long_row;
        if (short_row) {
            if (count == 0)
                first = r;
            ++count;
        }
        if (count > 0 && (!short_row || count == waves || r == n_rows - 1)) {
            blocks.push_back({first, count, 0, 0});
            count = 0;
        }
    }
    return n_long;
}

// A tiered plan of one aggregation (one sparse operand at one width).  The
// source rows (columns of the operand) are ranked by how many entries read
// them; tier t holds the rows ranked [t H, (t+1) H), where H rows of one
// XCD's share of the column slices fit the L2 budget of one XCD.  The
// aggregation then runs as one sliced pass per tier (each XCD gathering its
// column slices of the tier's rows, which stay in its L2) and one ordinary
// pass over the remaining entries, each pass adding into the output, in
// tier order.  The entries are split into T + 1 CSRs over the same rows,
// stored one after another in `col` / `val` (row pointers are offsets into
// them); a row's entries keep their order within each CSR.
struct TierPlan {
    int32_t which = 0;       // the sparse operand (Csr)
    int32_t width = 0;       // aggregation width the plan is for
    int32_t tiers = 0;       // sliced passes (the last CSR is the rest)
    int32_t rows_per_tier = 0;
    int64_t tier_entries = 0;   // entries in the sliced passes
    std::vector<int32_t> rowptr;   // (tiers + 1) x (n_rows + 1), absolute offsets
    std::vector<int32_t> col;
    std::vector<float> val;
    std::vector<SpmmBlock> blocks;   // per CSR: long-row blocks first
    std::vector<int32_t> blk_off, blk_cnt, blk_long;   // per CSR
    size_t off_rowptr = 0, off_col = 0, off_val = 0, off_blocks = 0;   // workspace
};

// Cost model of a tier: the gathers of its entries hit the L2 (kTierHitBytesPerS)
// instead of going past it (the measured random-gather rate); in exchange
// the pass re-reads the tier's index arrays once per column slice and the
// output (and writes it) once more, and costs one more launch.
constexpr double kTierHitBytesPerS = 18.0e12;
constexpr double kTierMissBytesPerS = 7.0e12;
constexpr double kStreamBytesPerS = 6.5e12;
constexpr double kLaunchSeconds = 4.0e-6;
constexpr int32_t kMaxTiers = 32;
// Tiering is off unless DIGEST_SPMM_TIER_BYTES gives the per-XCD L2 budget
// (about 3 MiB of the 4 MiB L2 suits it): on the measured workloads the
// sliced passes do hit the L2 (82-84% of their requests), but the one-pass
// kernel already finds the most-read rows in the Infinity Cache, the
// remaining pass then runs at the lower rate of rows that miss it, and the
// tiered aggregation was no faster (OGB-Products-shaped, 256 wide) or
// slower (Reddit-shaped, 602 wide, 15 tiers).
constexpr int64_t kTierBudgetBytes = 0;

int64_t env_int(const char *name, int64_t dflt)
{
    const char *v = std::getenv(name);
    if (!v || !*v)
        return dflt;
    char *end = nullptr;
    const long long x = std::strtoll(v, &end, 10);
    return (end && *end == 0) ? (int64_t)x : dflt;
}

// Plan the tiers of the CSR (rowptr, col, val) with n_rows rows over
// n_cols source rows, aggregated at `width`.  DIGEST_SPMM_TIER_BYTES sets
// the per-XCD L2 budget (unset or 0: no tiers) and DIGEST_SPMM_TIERS forces
// that many tiers regardless of the cost model (tuning and tests).
TierPlan plan_one_tier(int32_t which, const std::vector<int32_t> &rowptr,
                       const std::vector<int32_t> &col, const std::vector<float> &val,
                       int32_t n_rows, int64_t n_cols, int32_t width)
{
    TierPlan t;
    t.which = which;
    t.width = width;
    const int64_t budget = env_int("DIGEST_SPMM_TIER_BYTES", kTierBudgetBytes);
    const int64_t force = env_int("DIGEST_SPMM_TIERS", -1);
    const int64_t slices = (width + digest::kSliceFloats - 1) / digest::kSliceFloats;
    // a sliced pass needs a slice for every XCD and rows of an even width
    if (budget <= 0 || force == 0 || slices < 8 || width % 2 != 0 || n_rows == 0)
        return t;
    const int64_t per_xcd = (slices + 7) / 8;
    const int64_t H = std::max<int64_t>(1, budget / (per_xcd * digest::kSliceFloats * 4));
    const int64_t nnz = rowptr[n_rows];
    std::vector<int64_t> count((size_t)n_cols, 0);
    for (int64_t k = 0; k < nnz; ++k)
        count[col[k]] += 1;
    std::vector<int32_t> order((size_t)n_cols);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(),
                     [&](int32_t a, int32_t b) { return count[a] > count[b]; });
    // tier of each source row (-1: the rest); rows read once stay in the rest
    std::vector<int32_t> tier_of((size_t)n_cols, -1);
    const double row_bytes = 4.0 * width;
    const double per_pass = 2.0 * n_rows * row_bytes / kStreamBytesPerS + kLaunchSeconds;
    int32_t T = 0;
    for (int64_t t0 = 0; t0 < n_cols && T < kMaxTiers; t0 += H) {
        if (force > 0 && T >= force)
            break;
        const int64_t t1 = std::min<int64_t>(n_cols, t0 + H);
        int64_t refs = 0;
        for (int64_t r = t0; r < t1; ++r)
            refs += count[order[r]] >= 2 ? count[order[r]] : 0;
        if (refs == 0)
            break;
        const double saving =
            refs * row_bytes * (1.0 / kTierMissBytesPerS - 1.0 / kTierHitBytesPerS);
        const double cost = per_pass + refs * 8.0 * slices / kTierHitBytesPerS;
        if (force < 0 && saving <= cost)
            break;
        for (int64_t r = t0; r < t1; ++r)
            if (count[order[r]] >= 2)
                tier_of[order[r]] = T;
        t.tier_entries += refs;
        ++T;
    }
    if (T == 0)
        return t;
    t.tiers = T;
    t.rows_per_tier = (int32_t)H;
    // split the entries into T + 1 CSRs (tiers, then the rest), each row's
    // entries in their original order
    const int32_t C = T + 1;
    std::vector<int64_t> per((size_t)C * (n_rows + 1), 0);   // counts, then offsets
    for (int32_t i = 0; i < n_rows; ++i)
        for (int32_t k = rowptr[i]; k < rowptr[i + 1]; ++k) {
            const int32_t c = tier_of[col[k]] < 0 ? T : tier_of[col[k]];
            per[(size_t)c * (n_rows + 1) + i + 1] += 1;
        }
    t.rowptr.assign((size_t)C * (n_rows + 1), 0);
    int64_t base = 0;
    for (int32_t c = 0; c < C; ++c) {
        int32_t *rp = &t.rowptr[(size_t)c * (n_rows + 1)];
        rp[0] = (int32_t)base;
        for (int32_t i = 0; i < n_rows; ++i)
            rp[i + 1] = rp[i] + (int32_t)per[(size_t)c * (n_rows + 1) + i + 1];
        base = rp[n_rows];
    }
    t.col.resize((size_t)nnz);
    t.val.resize((size_t)nnz);
    for (int32_t i = 0; i < n_rows; ++i) {
        int32_t next[kMaxTiers + 1];
        for (int32_t c = 0; c < C; ++c)
            next[c] = t.rowptr[(size_t)c * (n_rows + 1) + i];
        for (int32_t k = rowptr[i]; k < rowptr[i + 1]; ++k) {
            const int32_t c = tier_of[col[k]] < 0 ? T : tier_of[col[k]];
            t.col[next[c]] = col[k];
            t.val[next[c]] = val[k];
            ++next[c];
        }
    }
    for (int32_t c = 0; c < C; ++c) {
        std::vector<int32_t> rp(t.rowptr.begin() + (size_t)c * (n_rows + 1),
                                t.rowptr.begin() + (size_t)(c + 1) * (n_rows + 1));
        std::vector<SpmmBlock> b;
        // the sliced passes' strip kernel takes every row up to
        // kTierLongRow entries; only longer rows get a workgroup each
        const int32_t n_long = build_blocks(rp, n_rows, b, true,
                                            c < T ? digest::kTierLongRow : digest::kSpmmLongRow);
        t.blk_off.push_back((int32_t)t.blocks.size());
        t.blk_cnt.push_back((int32_t)b.size());
        t.blk_long.push_back(n_long);
        t.blocks.insert(t.blocks.end(), b.begin(), b.end());
    }
    return t;
}

}  // namespace

struct digest_partition {
    int64_t n_global = 0;
    int32_t n_own = 0, n_halo = 0, n_bnd = 0;
    int64_t nnz = 0, nnz_in = 0;
    int32_t L = 0;
    std::vector<int32_t> widths;

    // host copies of everything uploaded at bind time
    std::vector<int32_t> rowptr, col, t_rowptr, t_src, halo_gid, bnd_local, bnd_gid, owned_gid;
    std::vector<float> val, t_val;
    // blocks_t covers the first n_own rows of the transpose (P_in^T),
    // blocks_tf all n_own + n_halo rows (P_m^T), blocks_th its n_halo halo rows
    // (P_out^T, numbered from 0).
    std::vector<SpmmBlock> blocks_f, blocks_t, blocks_tf, blocks_th;
    int32_t long_f = 0, long_t = 0, long_tf = 0, long_th = 0;   // leading long-row blocks
    // The GCN forward's operands.  Between two pulls of a level its halo rows
    // are constants, and so is their share of every owned row's aggregate,
    // P_out halo.  P_b holds the halo entries of the boundary rows (n_bnd
    // rows; columns are halo slots), which a pull multiplies into the halo
    // aggregate S = P_b halo ([n_bnd] rows).  P_s = [P_in | E] holds each
    // owned row's owned-column entries, then, for boundary row b, one entry
    // of 1 in column n_own + b, which reads S's row b: P_s [h; S] = P_m [h; halo].
    int64_t nnz_s = 0, nnz_b = 0;
    std::vector<int32_t> s_rowptr, s_col, b_rowptr, b_col;
    std::vector<int32_t> b_gcol;   // P_b's columns as global ids (the store's rows)
    std::vector<float> s_val, b_val;
    std::vector<SpmmBlock> blocks_s, blocks_b;
    int32_t long_s = 0, long_b = 0;
    // P_s and P_in^T with their long rows in row order, for the aggregations
    // of rows of at most kNarrowWide floats (whose long rows are short work:
    // longest first measured 10-13 us slower on the OGB-Products-shaped
    // 48-float layer)
    std::vector<SpmmBlock> blocks_s_rows, blocks_t_rows;
    // DIGEST_PULL_ROWS: a pull fills the halo buffer, then S from it;
    // DIGEST_PULL_AGGREGATE: a pull forms S straight from the store and
    // leaves the halo buffer alone (the calls that read it refuse).
    int32_t pull_mode = DIGEST_PULL_ROWS;
    // P_s split at kFuseLong entries per row: the long rows (their count and
    // entries) and the distinct source rows the short and the long rows read
    int64_t long_rows_f = 0, long_nnz_f = 0, src_short_f = 0, src_long_f = 0;
    // the fused forward's row order: tile t's rows t kFuseRows + fuse_order[..]
    // by descending entry count (long rows, read back, last), so that the
    // rows the waves take last are the short ones
    std::vector<uint8_t> fuse_order;
    // the same for P_in^T (the input gradient's aggregation)
    int64_t long_rows_t = 0, long_nnz_t = 0, src_short_t = 0, src_long_t = 0;
    std::vector<uint8_t> fuse_order_t;

    // Tiered plans of the aggregations (see TierPlan), at most one per
    // (sparse operand, width).
    std::vector<TierPlan> tier_plans;

    struct Layout {
        size_t rowptr, col, val, t_rowptr, t_src, t_val, halo_gid, bnd_local, bnd_gid, owned_gid;
        size_t blocks_f, blocks_t, blocks_tf, blocks_th;
        size_t s_rowptr, s_col, s_val, b_rowptr, b_col, b_gcol, b_val, blocks_s, blocks_b;
        size_t blocks_s_rows, blocks_t_rows;
        size_t fuse_order, fuse_order_t;   // per owned row, uint8 (see fuse_order below)
        size_t fz;                      // the fused input gradient's D and long rows
        size_t wt;                      // W^T of the fused input gradient
        std::vector<size_t> halo_buf;   // per level 0..L-1, rows padded_width(d_level) apart
        std::vector<size_t> hagg;       // per level 0..L-1: S, n_bnd rows padded like halo_buf
        std::vector<size_t> ah;         // per layer 1..L (index 0 unused), padded rows
        size_t tmp, tmp_halo, tbuf, gemm_part, loss_part;
        size_t hpad;                    // a padded copy of h_in for widths not a multiple of 4
        size_t total;
    } lay{};

    char *ws = nullptr;
    std::vector<char> pulled;       // per level
    std::vector<int64_t> pull_gen;  // per level: number of pulls since create
    std::vector<char> fwd_done;     // per layer
    std::vector<int32_t> act;       // per layer
    std::vector<char> tf;           // per layer: forward ran transform-first
    std::vector<int64_t> fwd_gen;   // per layer: pull_gen of level layer-1 at forward

    // GAT state, in a workspace of its own (digest_gat_bind_workspace)
    std::vector<int32_t> t_perm;    // entry k of P_m^T is entry t_perm[k] of P_m
    struct GatLayout {
        size_t t_perm, ones;
        std::vector<size_t> z, s, alpha;   // per layer 1..L (index 0 unused)
        size_t alpha_t, dpre, dpre_t, d_o, dz, ds_src, g2, part;
        size_t total;
    } glay{};
    char *gws = nullptr;
    std::vector<char> gat_done;      // per layer: a GAT forward since the GAT bind
    std::vector<int64_t> gat_gen;    // per layer: pull_gen of level layer-1 at that forward
    std::vector<int32_t> gat_act;
    std::vector<float> gat_slope;

    template <class T>
    T *gat(size_t off) const
    {
        return reinterpret_cast<T *>(gws + off);
    }

    // A second stream of the library for the weight gradient, which runs
    // concurrently with the input-gradient chain of the same backward call
    // (forked from and joined back into the caller's stream by events).
    hipStream_t side = nullptr;
    hipEvent_t ev_fork = nullptr, ev_join = nullptr;
    int side_dev = -1;

    bool prof = false;
    struct Rec {
        int32_t kind, layer;
        hipEvent_t a, b;
    };
    std::vector<Rec> recs;
    std::vector<hipEvent_t> pool;

    template <class T>
    T *at(size_t off) const
    {
        return reinterpret_cast<T *>(ws + off);
    }
};

namespace {

// Order of the two products of a layer (the same result, associated the
// other way; a ReLU applies to the aggregated product either way).  Both
// orders read the halo rows through their aggregate S (nb boundary rows,
// formed at the pull).  Aggregate-first gathers the nnz_s entries of P_s at
// width d_in (and, for layers > 1, nnz_in entries of width min(d_in, d_out)
// for the input gradient) and multiplies the n_own aggregated rows.
// Transform-first, Z = P_s ([H_in; S] W), multiplies the n_own + nb rows of
// [H_in; S] (its weight gradient runs over them too), gathers nnz_s + nnz_in
// entries of width d_out (P_s and P_in^T) and copies D's boundary rows; a
// ReLU layer forms the masked D once, an identity layer pads D when d_out
// is not a multiple of 4.  The rates are those measured for the aggregation
// kernels (random row gathers), the fp32 MFMA GEMM and row copies on MI355X.
constexpr double kGatherBytesPerS = 7.0e12;
constexpr double kGemmFlopsPerS = 80.0e12;

bool transform_first_cheaper(const digest_partition &p, int32_t layer, bool relu)
{
    const double di = p.widths[layer - 1], dout = p.widths[layer];
    const double n = p.n_own, R = (double)p.n_own + (double)p.n_bnd;
    const double nnz_s = (double)p.nnz_s, nnz_in = (double)p.nnz_in;
    const bool dgrad = layer > 1;
    const double af =
        (nnz_s * di + (dgrad ? nnz_in * std::min(di, dout) : 0.0)) * 4.0 / kGatherBytesPerS +
        2.0 * n * di * dout * (dgrad ? 3.0 : 2.0) / kGemmFlopsPerS;
    const double copies = 8.0 * p.n_bnd * dout +
                          (relu ? 12.0 * n * dout
                                : p.widths[layer] % 4
                                      ? 4.0 * n * (dout + padded_width(p.widths[layer]))
                                      : 0.0);
    const double tf = (nnz_s + nnz_in) * dout * 4.0 / kGatherBytesPerS +
                      (4.0 * R * di * dout + (dgrad ? 2.0 * n * di * dout : 0.0)) /
                          kGemmFlopsPerS +
                      copies / kStreamBytesPerS;
    return tf < af;
}

// The kernels for a narrow side (<= kNarrow columns): the dgrad one keeps a
// 256-column slice of W per wave, the weight-gradient one 64 features per
// wave; d_in is bounded to keep their launch shapes sane.
bool narrow_valu(int64_t d_in, int64_t d_out)
{
    return d_out <= digest::kNarrow && d_in <= 1024;
}

// The forward's product for outputs up to kNarrowN wide, with W in LDS.
bool narrow_out(int64_t d_in, int64_t d_out)
{
    return d_out <= digest::kNarrowN &&
           digest::narrow_n_lds((int32_t)d_in, (int32_t)d_out) <= digest::kNarrowNLds;
}

// Split-K slices of a narrow-output weight gradient over R rows, F features
// (about 2,048 waves: F / 64 feature blocks x slices of >= 32 rows): rows
// per slice and the number of slices.
void narrow_rows_plan(int64_t R, int64_t F, int32_t &chunk, int32_t &slices)
{
    const int64_t fblocks = (F + 63) / 64;
    const int64_t target = std::max<int64_t>(1, 2048 / fblocks);
    int64_t c = std::max<int64_t>(32, (R + target - 1) / target);
    c = (c + 31) / 32 * 32;
    chunk = (int32_t)c;
    slices = (int32_t)std::max<int64_t>(1, (R + c - 1) / c);
}

// Split-K slices of the transform-first weight gradient H_mix^T G over the
// n_own owned rows and n_halo rows of a second block (the halo rows, or the
// halo aggregate's boundary rows).  Narrow outputs (<= kNarrow) use the MFMA
// kernel with `chunk` rows per slice; wider ones use the MFMA GEMM twice
// (owned rows, then the second block) with their own split plans.
struct TfPlan {
    bool valu;
    int32_t chunk, slices;           // VALU: rows per slice, number of slices
    int32_t s_own, k_own, s_halo, k_halo;   // MFMA: splits and chunks (owned, second block)
};

TfPlan tf_plan(int64_t n_own, int64_t n2, int64_t d_in, int64_t d_out)
{
    TfPlan t{};
    const int64_t R = n_own + n2;
    t.valu = d_out <= digest::kNarrow;
    if (t.valu) {
        narrow_rows_plan(R, d_in, t.chunk, t.slices);
    } else {
        splitk_plan(d_in, d_out, n_own, t.s_own, t.k_own);
        if (n2 > 0)
            splitk_plan(d_in, d_out, n2, t.s_halo, t.k_halo);
        t.slices = t.s_own + (n2 > 0 ? t.s_halo : 0);
    }
    return t;
}

void plan_layout(digest_partition &p)
{
    auto &l = p.lay;
    size_t o = 0;
    auto take = [&](size_t bytes) {
        const size_t r = o;
        o += align_up(std::max<size_t>(bytes, 1));
        return r;
    };
    l.rowptr = take(sizeof(int32_t) * (p.n_own + 1));
    l.col = take(sizeof(int32_t) * p.nnz);
    l.val = take(sizeof(float) * p.nnz);
    l.t_rowptr = take(sizeof(int32_t) * ((size_t)p.n_own + p.n_halo + 1));
    l.t_src = take(sizeof(int32_t) * p.nnz);
    l.t_val = take(sizeof(float) * p.nnz);
    l.halo_gid = take(sizeof(int32_t) * p.n_halo);
    l.bnd_local = take(sizeof(int32_t) * p.n_bnd);
    l.bnd_gid = take(sizeof(int32_t) * p.n_bnd);
    l.owned_gid = take(sizeof(int32_t) * p.n_own);
    l.blocks_f = take(sizeof(SpmmBlock) * p.blocks_f.size());
    l.fuse_order = take(p.fuse_order.size());
    l.fuse_order_t = take(p.fuse_order_t.size());
    l.blocks_t = take(sizeof(SpmmBlock) * p.blocks_t.size());
    l.blocks_tf = take(sizeof(SpmmBlock) * p.blocks_tf.size());
    l.blocks_th = take(sizeof(SpmmBlock) * p.blocks_th.size());
    l.s_rowptr = take(sizeof(int32_t) * p.s_rowptr.size());
    l.s_col = take(sizeof(int32_t) * p.s_col.size());
    l.s_val = take(sizeof(float) * p.s_val.size());
    l.b_rowptr = take(sizeof(int32_t) * p.b_rowptr.size());
    l.b_col = take(sizeof(int32_t) * p.b_col.size());
    l.b_gcol = take(sizeof(int32_t) * p.b_gcol.size());
    l.b_val = take(sizeof(float) * p.b_val.size());
    l.blocks_s = take(sizeof(SpmmBlock) * p.blocks_s.size());
    l.blocks_s_rows = take(sizeof(SpmmBlock) * p.blocks_s_rows.size());
    l.blocks_t_rows = take(sizeof(SpmmBlock) * p.blocks_t_rows.size());
    l.blocks_b = take(sizeof(SpmmBlock) * p.blocks_b.size());
    l.halo_buf.assign(p.L, 0);
    l.hagg.assign(p.L, 0);
    for (int32_t lev = 0; lev < p.L; ++lev) {
        l.halo_buf[lev] = take(sizeof(float) * (size_t)p.n_halo * padded_width(p.widths[lev]));
        l.hagg[lev] = take(sizeof(float) * (size_t)p.n_bnd * padded_width(p.widths[lev]));
    }
    l.ah.assign(p.L + 1, 0);
    // padded copies of h_in (odd d_in) or dh_out (odd d_out), and a
    // transform-first ReLU layer's masked D
    int64_t hpad = 0;
    for (int32_t k = 1; k <= p.L; ++k) {
        l.ah[k] = take(sizeof(float) * (size_t)p.n_own * padded_width(p.widths[k - 1]));
        for (int32_t d : {p.widths[k - 1], p.widths[k]})
            if (d % 4)
                hpad = std::max<int64_t>(hpad, (int64_t)p.n_own * padded_width(d));
        if (transform_first_cheaper(p, k, true))
            hpad = std::max<int64_t>(hpad, (int64_t)p.n_own * padded_width(p.widths[k]));
    }
    l.hpad = take(sizeof(float) * (size_t)hpad);
    int64_t wmax = 0, gemm_part = 0, tbuf = 0;
    for (int32_t k = 1; k <= p.L; ++k) {
        const int64_t di = p.widths[k - 1], dout = p.widths[k];
        wmax = std::max({wmax, di, dout});
        int32_t splits, kchunk;
        splitk_plan(di, dout, p.n_own, splits, kchunk);
        if (splits > 1)
            gemm_part = std::max<int64_t>(gemm_part, (int64_t)splits * di * dout);
        // (the order depends on the activation the caller passes: room for
        // either)
        if (transform_first_cheaper(p, k, false) || transform_first_cheaper(p, k, true)) {
            // the second block of rows is the halo (with the halo gradient)
            // or the halo aggregate's boundary rows
            for (const int64_t n2 : {(int64_t)p.n_halo, (int64_t)p.n_bnd}) {
                tbuf = std::max<int64_t>(tbuf, ((int64_t)p.n_own + n2) * padded_width(dout));
                const TfPlan t = tf_plan(p.n_own, n2, di, dout);
                gemm_part = std::max<int64_t>(gemm_part, (int64_t)t.slices * di * dout);
            }
        }
    }
    // the fused input gradient's D and long rows (two n_own x padded rows)
    // and W^T, for every layer whose width allows it
    int64_t fz = 0, wt = 0;
    for (int32_t k = 2; k <= p.L; ++k)
        if (p.widths[k] >= digest::kFuseMinWidth && p.widths[k] <= digest::kFuseMaxWidth) {
            fz = std::max<int64_t>(fz, 2 * (int64_t)p.n_own * padded_width(p.widths[k]));
            wt = std::max<int64_t>(wt, (int64_t)p.widths[k - 1] * p.widths[k]);
        }
    l.fz = take(sizeof(float) * (size_t)fz);
    l.wt = take(sizeof(float) * (size_t)wt);
    l.tmp = take(sizeof(float) * (size_t)p.n_own * wmax);
    l.tmp_halo = take(sizeof(float) * (size_t)p.n_halo * wmax);
    l.tbuf = take(sizeof(float) * (size_t)tbuf);
    l.gemm_part = take(sizeof(float) * (size_t)gemm_part);
    l.loss_part = take(sizeof(float) * (size_t)digest::softmax_xent_blocks(p.n_own, p.widths[p.L]));
    for (TierPlan &t : p.tier_plans) {
        t.off_rowptr = take(sizeof(int32_t) * t.rowptr.size());
        t.off_col = take(sizeof(int32_t) * t.col.size());
        t.off_val = take(sizeof(float) * t.val.size());
        t.off_blocks = take(sizeof(SpmmBlock) * t.blocks.size());
    }
    l.total = o;
}

// The GAT workspace: the transposed-entry permutation, a column of ones,
// per layer the transformed rows z, their scores and the attention
// weights (kept from the forward for the backward), and the backward's
// scratch, sized for the widest layer.
void plan_gat_layout(digest_partition &p)
{
    auto &l = p.glay;
    size_t o = 0;
    auto take = [&](size_t bytes) {
        const size_t r = o;
        o += align_up(std::max<size_t>(bytes, 1));
        return r;
    };
    const int64_t R = (int64_t)p.n_own + p.n_halo;
    l.t_perm = take(sizeof(int32_t) * p.nnz);
    l.ones = take(sizeof(float) * p.n_own);
    l.z.assign(p.L + 1, 0);
    l.s.assign(p.L + 1, 0);
    l.alpha.assign(p.L + 1, 0);
    int64_t dmax = 0, part = 0;
    for (int32_t k = 1; k <= p.L; ++k) {
        const int64_t di = p.widths[k - 1], dout = p.widths[k];
        l.z[k] = take(sizeof(float) * (size_t)(R * dout));
        l.s[k] = take(sizeof(float) * (size_t)(R * 2));
        l.alpha[k] = take(sizeof(float) * (size_t)p.nnz);
        dmax = std::max(dmax, dout);
        const TfPlan t = tf_plan(p.n_own, p.n_halo, di, dout);
        part = std::max<int64_t>(part, (int64_t)t.slices * di * dout);
        int32_t chunk, slices;
        narrow_rows_plan(R, dout, chunk, slices);
        part = std::max<int64_t>(part, (int64_t)slices * dout * 2);
    }
    l.alpha_t = take(sizeof(float) * p.nnz);
    l.dpre = take(sizeof(float) * p.nnz);
    l.dpre_t = take(sizeof(float) * p.nnz);
    l.d_o = take(sizeof(float) * (size_t)(p.n_own * dmax));
    l.dz = take(sizeof(float) * (size_t)(R * dmax));
    l.ds_src = take(sizeof(float) * (size_t)R);
    l.g2 = take(sizeof(float) * (size_t)(R * 2));
    l.part = take(sizeof(float) * (size_t)part);
    l.total = o;
}

// RAII bracket of one kernel launch for the instrumentation.
struct Timed {
    digest_partition *p;
    hipStream_t s;
    hipEvent_t b = nullptr;
    Timed(digest_partition *p_, int32_t kind, int32_t layer, hipStream_t s_) : p(p_), s(s_)
    {
        if (!p->prof)
            return;
        auto get = [&]() {
            hipEvent_t e = nullptr;
            if (!p->pool.empty()) {
                e = p->pool.back();
                p->pool.pop_back();
            } else if (hipEventCreate(&e) != hipSuccess) {
                e = nullptr;
            }
            return e;
        };
        hipEvent_t a = get();
        b = get();
        if (!a || !b) {
            if (a)
                p->pool.push_back(a);
            if (b)
                p->pool.push_back(b);
            b = nullptr;
            return;
        }
        (void)hipEventRecord(a, s);
        p->recs.push_back({kind, layer, a, b});
    }
    ~Timed()
    {
        if (b)
            (void)hipEventRecord(b, s);
    }
};

digest_status hip_check(hipError_t e, const char *what)
{
    if (e != hipSuccess)
        return fail(DIGEST_EHIP, "%s: %s", what, hipGetErrorString(e));
    return DIGEST_OK;
}

// Weight gradients of at least this many flops run on the side stream,
// concurrently with the input-gradient chain (smaller ones lose more to the
// fork and join than the overlap gives).  DIGEST_SIDE_STREAM=0 keeps all
// work on the caller's stream, =2 uses the side stream at any size.
constexpr double kSideFlops = 8.0e9;

bool side_pays(double flops)
{
    const char *v = std::getenv("DIGEST_SIDE_STREAM");
    if (v && v[0] == '0')
        return false;
    if (v && v[0] == '2')
        return true;
    return flops >= kSideFlops;
}

// Start work on the side stream after everything enqueued on s so far; *sw
// becomes the side stream, or stays s when s belongs to another device than
// the current one (the side stream is created on the current device).
digest_status fork_side(digest_partition *p, hipStream_t s, hipStream_t *sw)
{
    *sw = s;
    int dev = -1;
    if (digest_status st = hip_check(hipGetDevice(&dev), "current device"))
        return st;
    if (s) {
        hipDevice_t sdev = -1;
        if (digest_status st = hip_check(hipStreamGetDevice(s, &sdev), "stream device"))
            return st;
        if (sdev != dev)
            return DIGEST_OK;
    }
    if (!p->side || p->side_dev != dev) {
        if (p->side)
            return DIGEST_OK;   // created for another device: stay on s
        if (digest_status st = hip_check(hipStreamCreateWithFlags(&p->side, hipStreamNonBlocking),
                                         "side stream"))
            return st;
        p->side_dev = dev;
        if (digest_status st =
                hip_check(hipEventCreateWithFlags(&p->ev_fork, hipEventDisableTiming), "event"))
            return st;
        if (digest_status st =
                hip_check(hipEventCreateWithFlags(&p->ev_join, hipEventDisableTiming), "event"))
            return st;
    }
    if (digest_status st = hip_check(hipEventRecord(p->ev_fork, s), "fork"))
        return st;
    if (digest_status st = hip_check(hipStreamWaitEvent(p->side, p->ev_fork, 0), "fork"))
        return st;
    *sw = p->side;
    return DIGEST_OK;
}

// Make s wait for everything enqueued on the side stream so far.
digest_status join_side(digest_partition *p, hipStream_t s)
{
    if (digest_status st = hip_check(hipEventRecord(p->ev_join, p->side), "join"))
        return st;
    return hip_check(hipStreamWaitEvent(s, p->ev_join, 0), "join");
}

digest_status need_bound(const digest_partition *p)
{
    if (!p)
        return fail(DIGEST_EINVAL, "NULL partition handle");
    if (!p->ws)
        return fail(DIGEST_ESTATE, "no workspace bound");
    return DIGEST_OK;
}

// Sparse aggregation over the local CSR (P_m), the CSR of P_in^T (the first
// n_own rows of the transpose), of P_m^T (all of it), of P_out^T (its
// n_halo halo rows, numbered from 0) or of P_s (owned columns, then the
// halo aggregate's).  `val` replaces the matrix's values (edge weights in
// the same entry order); relu stores max(x, 0).
enum class Csr { Fwd, InT, FullT, HaloT, InH };

// Tiered plans for the aggregations a standard round runs at widths where
// slicing applies: the forward's P_s at d_in of every aggregate-first layer
// and the backward's P_in^T at its width for layers >= 2 (the layer plan's
// orders, ReLU below the last layer).  Operands or widths that gain nothing
// get no plan and run as one pass.
void plan_tiers(digest_partition &p)
{
    p.tier_plans.clear();
    std::vector<std::pair<int32_t, int32_t>> tried;
    auto want = [&](Csr which, int32_t w) {
        for (const auto &tw : tried)
            if (tw.first == (int32_t)which && tw.second == w)
                return;
        tried.push_back({(int32_t)which, w});
        TierPlan t = which == Csr::InH
                         ? plan_one_tier((int32_t)which, p.s_rowptr, p.s_col, p.s_val, p.n_own,
                                         (int64_t)p.n_own + p.n_bnd, w)
                         : plan_one_tier((int32_t)which, p.t_rowptr, p.t_src, p.t_val, p.n_own,
                                         p.n_own, w);
        if (t.tiers > 0)
            p.tier_plans.push_back(std::move(t));
    };
    for (int32_t l = 1; l <= p.L; ++l) {
        const int32_t d_in = p.widths[l - 1], d_out = p.widths[l];
        const bool relu = l < p.L;
        if (p.n_own > 0 && transform_first_cheaper(p, l, relu))
            continue;
        want(Csr::InH, padded_width(d_in));
        if (l > 1)
            want(Csr::InT, (!relu && d_out < d_in) ? d_out : d_in);
    }
}

const TierPlan *find_tiers(const digest_partition &p, Csr which, int32_t width)
{
    for (const TierPlan &t : p.tier_plans)
        if (t.which == (int32_t)which && t.width == width)
            return &t;
    return nullptr;
}

// Aggregate-first forwards of at least this many owned rows run as one pass
// that multiplies each aggregated row tile by W while other tiles gather
// (launch_spmm_gemm).  DIGEST_FUSE=0 never fuses, =2 fuses at any size.
constexpr int64_t kFuseMinRows = 16384;

// The input gradient of a ReLU aggregate-first layer (layer >= 2, 129..256
// output floats) runs as P_in^T (D W^T) = (P_in^T D) W^T in one pass over
// D = dh_out masked by the ReLU derivative (launch_spmm_gemm): the same
// rules and switch as the fused forward.
bool fuse_backward(const digest_partition &p, int32_t layer, bool transform_first)
{
    const int32_t d_out = p.widths[layer];
    const int64_t mode = env_int("DIGEST_FUSE", 1);
    if (mode == 0 || transform_first || layer < 2 || layer >= p.L || p.n_own <= 0 ||
        d_out < digest::kFuseMinWidth || d_out > digest::kFuseMaxWidth ||
        (mode == 1 && p.n_own < kFuseMinRows))
        return false;
    return find_tiers(p, Csr::InT, p.widths[layer - 1]) == nullptr;
}

bool fuse_forward(const digest_partition &p, int32_t layer, bool transform_first)
{
    const int32_t d_in = p.widths[layer - 1], d_out = p.widths[layer];
    const int64_t mode = env_int("DIGEST_FUSE", 1);
    // a product with a narrow output (the narrow-output kernel) is too
    // cheap for the fusion to pay: the halo-dominated partition's 256 -> 47
    // layer took 557 + 696 us fused against 1,087 + 70 us
    if (mode == 0 || transform_first || p.n_own <= 0 || narrow_out(d_in, d_out) ||
        d_in < digest::kFuseMinWidth || d_in > digest::kFuseMaxWidth ||
        (mode == 1 && p.n_own < kFuseMinRows))
        return false;
    return find_tiers(p, Csr::InH, padded_width(d_in)) == nullptr;
}

digest_status run_spmm(digest_partition *p, Csr which, const float *src0, const float *src1,
                       int32_t n_src0, int32_t d, float *out, int32_t layer, hipStream_t s,
                       const digest::SpmmEpilogue *ep = nullptr, int32_t kind = -1,
                       float *out1 = nullptr, int32_t n_out0 = INT32_MAX,
                       const float *val = nullptr, bool relu = false,
                       const digest::SpmmRank1 *r1 = nullptr, int32_t lds = 0,
                       int32_t out_ld = 0, int32_t out_w = 0)
{
    const bool fwd = which == Csr::Fwd;
    const std::vector<SpmmBlock> *blocks = &p->blocks_f;
    size_t boff = p->lay.blocks_f;
    int32_t n_long = p->long_f;
    size_t o_rowptr = fwd ? p->lay.rowptr : p->lay.t_rowptr;
    size_t o_col = fwd ? p->lay.col : p->lay.t_src;
    size_t o_val = fwd ? p->lay.val : p->lay.t_val;
    const bool narrow = d <= digest::kNarrowWide;
    if (which == Csr::InH) {
        blocks = &p->blocks_s, boff = narrow ? p->lay.blocks_s_rows : p->lay.blocks_s;
        n_long = p->long_s;
        o_rowptr = p->lay.s_rowptr, o_col = p->lay.s_col, o_val = p->lay.s_val;
    } else if (which == Csr::InT) {
        blocks = &p->blocks_t, boff = narrow ? p->lay.blocks_t_rows : p->lay.blocks_t;
        n_long = p->long_t;
    } else if (which == Csr::FullT) {
        blocks = &p->blocks_tf, boff = p->lay.blocks_tf, n_long = p->long_tf;
    } else if (which == Csr::HaloT) {
        blocks = &p->blocks_th, boff = p->lay.blocks_th, n_long = p->long_th;
    }
    const int32_t *rowptr = p->at<int32_t>(o_rowptr);
    if (which == Csr::HaloT)
        rowptr += p->n_own;
    Timed t(p, kind >= 0 ? kind : (fwd || which == Csr::InH ? K_SPMM_FWD : K_SPMM_BWD), layer,
            s);
    const TierPlan *tp = find_tiers(*p, which, d);
    if (tp && !ep && !val && !relu && !(r1 && r1->a) && n_out0 == INT32_MAX && !out1 &&
        (lds == 0 || lds == d) && (out_ld == 0 || out_ld == d) && (out_w == 0 || out_w == d) &&
        digest::spmm_sliced_ok(d, src0, src1, out)) {
        // sliced passes over the tiers, then the rest, each adding into out
        const int32_t n_rows = p->n_own;
        const int32_t *trp = p->at<int32_t>(tp->off_rowptr);
        const int32_t *tcol = p->at<int32_t>(tp->off_col);
        const float *tval = p->at<float>(tp->off_val);
        const SpmmBlock *tblk = p->at<SpmmBlock>(tp->off_blocks);
        for (int32_t c = 0; c <= tp->tiers; ++c) {
            const int32_t *rp = trp + (int64_t)c * (n_rows + 1);
            const SpmmBlock *b = tblk + tp->blk_off[c];
            const hipError_t e =
                c < tp->tiers
                    ? digest::launch_spmm_sliced(b, tp->blk_cnt[c], tp->blk_long[c], rp, tcol,
                                                 tval, (int64_t)tp->col.size(), src0, src1,
                                                 n_src0, n_rows, d, out, c > 0, s)
                    : digest::launch_spmm(b, tp->blk_cnt[c], tp->blk_long[c], rp, tcol, tval,
                                          src0, src1, n_src0, d, out, s, nullptr, nullptr,
                                          INT32_MAX, false, nullptr, true);
            if (digest_status st = hip_check(e, "tiered spmm"))
                return st;
        }
        return DIGEST_OK;
    }
    return hip_check(
        digest::launch_spmm(p->at<SpmmBlock>(boff), (int32_t)blocks->size(), n_long, rowptr,
                            p->at<int32_t>(o_col), val ? val : p->at<float>(o_val), src0, src1,
                            n_src0, d, out, s, ep, out1, n_out0, relu, r1, false, lds, out_ld,
                            out_w),
        "spmm");
}

// S = P_b halo_buf[level]: the halo aggregate of level `level` (the halo
// rows' share of each boundary row's aggregate in the forward of layer
// level + 1), rows padded like the halo buffer.  With `store` (the level's
// [n_global, d] rows) the same sum is gathered from the store by global id
// instead; S then stores the d columns of each row.
digest_status halo_aggregate(digest_partition *p, int32_t level, hipStream_t s,
                             const float *store = nullptr)
{
    if (p->n_bnd == 0)
        return DIGEST_OK;
    const int32_t d = p->widths[level], lw = padded_width(d);
    const int32_t *rowptr = p->at<int32_t>(p->lay.b_rowptr);
    const float *val = p->at<float>(p->lay.b_val);
    const SpmmBlock *blocks = p->at<SpmmBlock>(p->lay.blocks_b);
    const int32_t nb = (int32_t)p->blocks_b.size();
    float *out = p->at<float>(p->lay.hagg[level]);
    Timed t(p, K_HALO_AGG, level, s);
    if (store)
        return hip_check(digest::launch_spmm(blocks, nb, p->long_b, rowptr,
                                             p->at<int32_t>(p->lay.b_gcol), val, store, nullptr,
                                             INT32_MAX, d, out, s, nullptr, nullptr, INT32_MAX,
                                             false, nullptr, false, d, lw, d),
                         "halo aggregate");
    return hip_check(digest::launch_spmm(blocks, nb, p->long_b, rowptr,
                                         p->at<int32_t>(p->lay.b_col), val,
                                         p->at<float>(p->lay.halo_buf[level]), nullptr,
                                         p->n_halo, lw, out, s),
                     "halo aggregate");
}

// T = [h_own; h2] W over the n_own owned rows and the n2 rows of a second
// block h2 (the halo rows, or the halo aggregate's boundary rows; rows
// padded_width(d_in) apart), T row-major [n_own + n2][ldt]: the
// narrow-output kernel with W in LDS when the widths allow, else the MFMA
// GEMM for the owned and for the second block's rows.
digest_status transform_rows(digest_partition *p, int32_t layer, const float *h_own,
                             const float *h2, int32_t n2, const float *w, float *T, int32_t ldt,
                             hipStream_t s)
{
    const int32_t d_in = p->widths[layer - 1], d_out = p->widths[layer];
    if (narrow_out(d_in, d_out))
        return hip_check(digest::launch_narrow_n(p->n_own + n2, p->n_own, d_in, d_out, h_own,
                                                 h2, d_in, w, T, ldt, false, s,
                                                 padded_width(d_in)),
                         "transform");
    digest::GemmArgs g{};
    g.N = d_out;
    g.K = d_in;
    g.lda = d_in;
    g.B = w;
    g.ldb = d_out;
    g.ldc = ldt;
    g.splits = 1;
    g.kchunk = d_in;
    if (p->n_own > 0) {
        g.M = p->n_own;
        g.A = h_own;
        g.C = T;
        g.tile = gemm_tile_for(g.M, d_out, d_in, false);
        if (digest_status st = hip_check(digest::launch_gemm(g, s), "transform"))
            return st;
    }
    if (n2 > 0) {
        g.M = n2;
        g.tile = gemm_tile_for(g.M, d_out, d_in, false);
        g.A = h2;
        g.lda = padded_width(d_in);
        g.C = T + (int64_t)p->n_own * ldt;
        if (digest_status st = hip_check(digest::launch_gemm(g, s), "transform"))
            return st;
    }
    return DIGEST_OK;
}

}  // namespace

extern "C" {

const char *digest_last_error(void) { return g_last_error.c_str(); }

digest_status digest_partition_create(int64_t n_global, const int64_t *indptr,
                                      const int64_t *indices, const float *values,
                                      const int64_t *owned, int64_t n_owned,
                                      const int64_t *halo, int64_t n_halo,
                                      int32_t n_layers, const int32_t *widths,
                                      digest_partition **out)
{
    if (!out)
        return fail(DIGEST_EINVAL, "out is NULL");
    if (n_global < 1 || n_global >= INT32_MAX)
        return fail(DIGEST_EINVAL, "n_global must be in [1, 2^31-1)");
    if (n_owned < 0 || n_owned > n_global || n_halo < 0 || n_halo > n_global ||
        n_owned + n_halo > n_global)
        return fail(DIGEST_EINVAL, "n_owned / n_halo out of range");
    if (!indptr || (n_owned > 0 && !owned) || (n_halo > 0 && !halo))
        return fail(DIGEST_EINVAL, "NULL id or indptr array");
    if (n_layers < 1 || n_layers > kMaxLayers || !widths)
        return fail(DIGEST_EINVAL, "n_layers must be in [1, %d] and widths non-NULL", kMaxLayers);
    for (int32_t k = 0; k <= n_layers; ++k)
        if (widths[k] < 1 || widths[k] > kMaxWidth)
            return fail(DIGEST_EINVAL, "widths[%d] = %d outside [1, %d]", k, widths[k], kMaxWidth);
    if (indptr[0] != 0)
        return fail(DIGEST_EINVAL, "indptr[0] must be 0");
    for (int64_t i = 0; i < n_owned; ++i)
        if (indptr[i + 1] < indptr[i])
            return fail(DIGEST_EINVAL, "indptr decreases at row %lld", (long long)i);
    const int64_t nnz = indptr[n_owned];
    if (nnz >= INT32_MAX)
        return fail(DIGEST_EINVAL, "nnz must be < 2^31");
    if (nnz > 0 && (!indices || !values))
        return fail(DIGEST_EINVAL, "NULL indices or values");

    digest_partition *p = new (std::nothrow) digest_partition();
    if (!p)
        return fail(DIGEST_ENOMEM, "out of host memory");
    try {
        p->n_global = n_global;
        p->n_own = (int32_t)n_owned;
        p->n_halo = (int32_t)n_halo;
        p->nnz = nnz;
        p->L = n_layers;
        p->widths.assign(widths, widths + n_layers + 1);

        // global id -> local number (owned i -> i, halo j -> n_own + j)
        std::vector<int32_t> local((size_t)n_global, -1);
        p->owned_gid.resize(n_owned);
        for (int64_t i = 0; i < n_owned; ++i) {
            const int64_t g = owned[i];
            if (g < 0 || g >= n_global || local[g] != -1) {
                delete p;
                return fail(DIGEST_EINVAL, "owned[%lld] = %lld is out of range or repeated",
                            (long long)i, (long long)g);
            }
            local[g] = (int32_t)i;
            p->owned_gid[i] = (int32_t)g;
        }
        p->halo_gid.resize(n_halo);
        for (int64_t j = 0; j < n_halo; ++j) {
            const int64_t g = halo[j];
            if (g < 0 || g >= n_global || local[g] != -1) {
                delete p;
                return fail(DIGEST_EINVAL,
                            "halo[%lld] = %lld is out of range, repeated or owned",
                            (long long)j, (long long)g);
            }
            local[g] = (int32_t)(n_owned + j);
            p->halo_gid[j] = (int32_t)g;
        }

        // local CSR and the boundary (rows that read at least one halo column)
        p->rowptr.resize(n_owned + 1);
        p->col.resize(nnz);
        p->val.assign(values, values + nnz);
        p->rowptr[0] = 0;
        for (int64_t i = 0; i < n_owned; ++i) {
            bool reads_halo = false;
            for (int64_t k = indptr[i]; k < indptr[i + 1]; ++k) {
                const int64_t g = indices[k];
                if (g < 0 || g >= n_global || local[g] < 0) {
                    delete p;
                    return fail(DIGEST_EINVAL,
                                "column %lld of row %lld is neither owned nor halo",
                                (long long)g, (long long)i);
                }
                const int32_t c = local[g];
                p->col[k] = c;
                reads_halo |= c >= n_owned;
            }
            p->rowptr[i + 1] = (int32_t)indptr[i + 1];
            if (reads_halo) {
                p->bnd_local.push_back((int32_t)i);
                p->bnd_gid.push_back((int32_t)owned[i]);
            }
        }
        p->n_bnd = (int32_t)p->bnd_local.size();

        // CSR of P_m^T by a stable counting sort on the local column: row c
        // lists the owned rows i with an entry in column c, i ascending.  Its
        // first n_own rows are P_in^T.
        const int64_t n_loc = n_owned + n_halo;
        p->t_rowptr.assign(n_loc + 1, 0);
        for (int64_t k = 0; k < nnz; ++k)
            p->t_rowptr[p->col[k] + 1] += 1;
        for (int64_t c = 0; c < n_loc; ++c)
            p->t_rowptr[c + 1] += p->t_rowptr[c];
        p->nnz_in = p->t_rowptr[n_owned];
        p->t_src.resize(nnz);
        p->t_val.resize(nnz);
        p->t_perm.resize(nnz);
        std::vector<int32_t> next(p->t_rowptr.begin(), p->t_rowptr.end() - 1);
        for (int32_t i = 0; i < (int32_t)n_owned; ++i)
            for (int32_t k = p->rowptr[i]; k < p->rowptr[i + 1]; ++k) {
                const int32_t c = p->col[k];
                p->t_src[next[c]] = i;
                p->t_val[next[c]] = p->val[k];
                p->t_perm[next[c]] = k;
                ++next[c];
            }

        // P_s and P_b (entries in P_m's order within each row)
        p->nnz_b = nnz - p->nnz_in;
        p->nnz_s = p->nnz_in + p->n_bnd;
        p->s_rowptr.assign(n_owned + 1, 0);
        p->s_col.reserve(p->nnz_s);
        p->s_val.reserve(p->nnz_s);
        p->b_rowptr.assign(p->n_bnd + 1, 0);
        p->b_col.reserve(p->nnz_b);
        p->b_val.reserve(p->nnz_b);
        for (int32_t i = 0, b = 0; i < (int32_t)n_owned; ++i) {
            for (int32_t k = p->rowptr[i]; k < p->rowptr[i + 1]; ++k)
                if (p->col[k] < n_owned) {
                    p->s_col.push_back(p->col[k]);
                    p->s_val.push_back(p->val[k]);
                }
            if (b < p->n_bnd && p->bnd_local[b] == i) {
                for (int32_t k = p->rowptr[i]; k < p->rowptr[i + 1]; ++k)
                    if (p->col[k] >= n_owned) {
                        p->b_col.push_back(p->col[k] - (int32_t)n_owned);
                        p->b_val.push_back(p->val[k]);
                    }
                p->b_rowptr[b + 1] = (int32_t)p->b_col.size();
                p->s_col.push_back((int32_t)n_owned + b);
                p->s_val.push_back(1.0f);
                ++b;
            }
            p->s_rowptr[i + 1] = (int32_t)p->s_col.size();
        }
        p->b_gcol.resize(p->b_col.size());
        for (size_t k = 0; k < p->b_col.size(); ++k)
            p->b_gcol[k] = p->halo_gid[p->b_col[k]];
        p->long_f = build_blocks(p->rowptr, p->n_own, p->blocks_f);
        p->long_s = build_blocks(p->s_rowptr, p->n_own, p->blocks_s);
        build_blocks(p->s_rowptr, p->n_own, p->blocks_s_rows, false);
        p->long_b = build_blocks(p->b_rowptr, p->n_bnd, p->blocks_b);
        fuse_stats(p->s_rowptr, p->s_col, (int32_t)n_owned, p->n_own + p->n_bnd, p->long_rows_f,
                   p->long_nnz_f, p->src_short_f, p->src_long_f, p->fuse_order);
        p->long_t = build_blocks(p->t_rowptr, p->n_own, p->blocks_t);
        build_blocks(p->t_rowptr, p->n_own, p->blocks_t_rows, false);
        fuse_stats(p->t_rowptr, p->t_src, (int32_t)n_owned, p->n_own, p->long_rows_t,
                   p->long_nnz_t, p->src_short_t, p->src_long_t, p->fuse_order_t);
        p->long_tf = build_blocks(p->t_rowptr, p->n_own + p->n_halo, p->blocks_tf);
        {
            const std::vector<int32_t> halo_rows(p->t_rowptr.begin() + n_owned,
                                                 p->t_rowptr.end());
            p->long_th = build_blocks(halo_rows, p->n_halo, p->blocks_th);
        }
        plan_tiers(*p);
        plan_layout(*p);
        plan_gat_layout(*p);
        p->gat_done.assign(p->L + 1, 0);
        p->gat_gen.assign(p->L + 1, 0);
        p->gat_act.assign(p->L + 1, 0);
        p->gat_slope.assign(p->L + 1, 0.f);
        p->pulled.assign(p->L, 0);
        p->pull_gen.assign(p->L, 0);
        p->fwd_done.assign(p->L + 1, 0);
        p->tf.assign(p->L + 1, 0);
        p->fwd_gen.assign(p->L + 1, 0);
        p->act.assign(p->L + 1, DIGEST_ACT_RELU);
    } catch (const std::bad_alloc &) {
        delete p;
        return fail(DIGEST_ENOMEM, "out of host memory");
    }
    *out = p;
    return DIGEST_OK;
}

void digest_partition_destroy(digest_partition *p)
{
    if (!p)
        return;
    for (auto &r : p->recs) {
        (void)hipEventDestroy(r.a);
        (void)hipEventDestroy(r.b);
    }
    for (auto e : p->pool)
        (void)hipEventDestroy(e);
    if (p->side)
        (void)hipStreamDestroy(p->side);
    if (p->ev_fork)
        (void)hipEventDestroy(p->ev_fork);
    if (p->ev_join)
        (void)hipEventDestroy(p->ev_join);
    delete p;
}

digest_status digest_partition_query(const digest_partition *p, int64_t *n_boundary,
                                     int64_t *nnz, int64_t *nnz_in, size_t *workspace_bytes)
{
    if (!p)
        return fail(DIGEST_EINVAL, "NULL partition handle");
    if (n_boundary)
        *n_boundary = p->n_bnd;
    if (nnz)
        *nnz = p->nnz;
    if (nnz_in)
        *nnz_in = p->nnz_in;
    if (workspace_bytes)
        *workspace_bytes = p->lay.total;
    return DIGEST_OK;
}

digest_status digest_partition_bind_workspace(digest_partition *p, void *dev_ptr, size_t bytes,
                                              void *hip_stream)
{
    if (!p || !dev_ptr)
        return fail(DIGEST_EINVAL, "NULL handle or workspace");
    if ((uintptr_t)dev_ptr % kAlign)
        return fail(DIGEST_EINVAL, "workspace must be %zu-byte aligned", kAlign);
    if (bytes < p->lay.total)
        return fail(DIGEST_ENOMEM, "workspace has %zu bytes, needs %zu", bytes, p->lay.total);
    hipStream_t s = (hipStream_t)hip_stream;
    char *ws = (char *)dev_ptr;
    struct Up {
        size_t off;
        const void *src;
        size_t bytes;
    };
    const auto &l = p->lay;
    const Up ups[] = {
        {l.rowptr, p->rowptr.data(), sizeof(int32_t) * p->rowptr.size()},
        {l.col, p->col.data(), sizeof(int32_t) * p->col.size()},
        {l.val, p->val.data(), sizeof(float) * p->val.size()},
        {l.t_rowptr, p->t_rowptr.data(), sizeof(int32_t) * p->t_rowptr.size()},
        {l.t_src, p->t_src.data(), sizeof(int32_t) * p->t_src.size()},
        {l.t_val, p->t_val.data(), sizeof(float) * p->t_val.size()},
        {l.halo_gid, p->halo_gid.data(), sizeof(int32_t) * p->halo_gid.size()},
        {l.bnd_local, p->bnd_local.data(), sizeof(int32_t) * p->bnd_local.size()},
        {l.bnd_gid, p->bnd_gid.data(), sizeof(int32_t) * p->bnd_gid.size()},
        {l.owned_gid, p->owned_gid.data(), sizeof(int32_t) * p->owned_gid.size()},
        {l.blocks_f, p->blocks_f.data(), sizeof(SpmmBlock) * p->blocks_f.size()},
        {l.fuse_order, p->fuse_order.data(), p->fuse_order.size()},
        {l.fuse_order_t, p->fuse_order_t.data(), p->fuse_order_t.size()},
        {l.blocks_t, p->blocks_t.data(), sizeof(SpmmBlock) * p->blocks_t.size()},
        {l.blocks_tf, p->blocks_tf.data(), sizeof(SpmmBlock) * p->blocks_tf.size()},
        {l.blocks_th, p->blocks_th.data(), sizeof(SpmmBlock) * p->blocks_th.size()},
        {l.s_rowptr, p->s_rowptr.data(), sizeof(int32_t) * p->s_rowptr.size()},
        {l.s_col, p->s_col.data(), sizeof(int32_t) * p->s_col.size()},
        {l.s_val, p->s_val.data(), sizeof(float) * p->s_val.size()},
        {l.b_rowptr, p->b_rowptr.data(), sizeof(int32_t) * p->b_rowptr.size()},
        {l.b_col, p->b_col.data(), sizeof(int32_t) * p->b_col.size()},
        {l.b_gcol, p->b_gcol.data(), sizeof(int32_t) * p->b_gcol.size()},
        {l.b_val, p->b_val.data(), sizeof(float) * p->b_val.size()},
        {l.blocks_s, p->blocks_s.data(), sizeof(SpmmBlock) * p->blocks_s.size()},
        {l.blocks_s_rows, p->blocks_s_rows.data(), sizeof(SpmmBlock) * p->blocks_s_rows.size()},
        {l.blocks_t_rows, p->blocks_t_rows.data(), sizeof(SpmmBlock) * p->blocks_t_rows.size()},
        {l.blocks_b, p->blocks_b.data(), sizeof(SpmmBlock) * p->blocks_b.size()},
    };
    for (const Up &u : ups) {
        if (!u.bytes)
            continue;
        digest_status st = hip_check(
            hipMemcpyAsync(ws + u.off, u.src, u.bytes, hipMemcpyHostToDevice, s), "upload");
        if (st)
            return st;
    }
    for (const TierPlan &t : p->tier_plans) {
        const Up tu[] = {
            {t.off_rowptr, t.rowptr.data(), sizeof(int32_t) * t.rowptr.size()},
            {t.off_col, t.col.data(), sizeof(int32_t) * t.col.size()},
            {t.off_val, t.val.data(), sizeof(float) * t.val.size()},
            {t.off_blocks, t.blocks.data(), sizeof(SpmmBlock) * t.blocks.size()},
        };
        for (const Up &u : tu) {
            if (!u.bytes)
                continue;
            digest_status st = hip_check(
                hipMemcpyAsync(ws + u.off, u.src, u.bytes, hipMemcpyHostToDevice, s), "upload");
            if (st)
                return st;
        }
    }
    p->ws = ws;
    // The halo buffers and AH of the old workspace are gone: no level counts
    // as pulled and no forward (GCN or GAT) as done.  Pull generations keep
    // counting across binds, so a forward recorded before the bind can never
    // match a later pull count.
    std::fill(p->pulled.begin(), p->pulled.end(), 0);
    std::fill(p->fwd_done.begin(), p->fwd_done.end(), 0);
    std::fill(p->gat_done.begin(), p->gat_done.end(), 0);
    return DIGEST_OK;
}

digest_status digest_partition_export_maps(const digest_partition *p, int32_t *col_local,
                                           int64_t *boundary_gid, int32_t *boundary_local)
{
    if (!p)
        return fail(DIGEST_EINVAL, "NULL partition handle");
    if (col_local)
        std::copy(p->col.begin(), p->col.end(), col_local);
    if (boundary_gid)
        for (int32_t b = 0; b < p->n_bnd; ++b)
            boundary_gid[b] = p->bnd_gid[b];
    if (boundary_local)
        std::copy(p->bnd_local.begin(), p->bnd_local.end(), boundary_local);
    return DIGEST_OK;
}

digest_status digest_partition_export_transpose(const digest_partition *p, int64_t *t_indptr,
                                                int32_t *t_src, float *t_vals)
{
    if (!p)
        return fail(DIGEST_EINVAL, "NULL partition handle");
    if (t_indptr)
        for (int64_t c = 0; c <= p->n_own; ++c)
            t_indptr[c] = p->t_rowptr[c];
    if (t_src)
        std::copy(p->t_src.begin(), p->t_src.begin() + p->nnz_in, t_src);
    if (t_vals)
        std::copy(p->t_val.begin(), p->t_val.begin() + p->nnz_in, t_vals);
    return DIGEST_OK;
}

digest_status digest_partition_read_halo(const digest_partition *p, int32_t level, float *out,
                                         void *hip_stream)
{
    if (digest_status st = need_bound(p))
        return st;
    if (level < 0 || level >= p->L || !out)
        return fail(DIGEST_EINVAL, "bad level %d or NULL output", level);
    if (p->n_halo == 0)
        return DIGEST_OK;
    if (p->pull_mode != DIGEST_PULL_ROWS)
        return fail(DIGEST_ESTATE, "the pull mode keeps no halo rows");
    const int32_t d = p->widths[level];
    return hip_check(digest::launch_copy_rows(nullptr, nullptr, p->n_halo, d,
                                              p->at<float>(p->lay.halo_buf[level]), out,
                                              (hipStream_t)hip_stream, padded_width(d), d),
                     "read halo");
}

digest_status digest_partition_set_pull_mode(digest_partition *p, int32_t mode)
{
    if (!p)
        return fail(DIGEST_EINVAL, "NULL partition handle");
    if (mode != DIGEST_PULL_ROWS && mode != DIGEST_PULL_AGGREGATE)
        return fail(DIGEST_EINVAL, "unknown pull mode %d", mode);
    if (mode != p->pull_mode)
        std::fill(p->pulled.begin(), p->pulled.end(), 0);
    p->pull_mode = mode;
    return DIGEST_OK;
}

digest_status digest_pull(digest_partition *p, int32_t level, const float *store,
                          void *hip_stream)
{
    if (digest_status st = need_bound(p))
        return st;
    if (level < 0 || level >= p->L)
        return fail(DIGEST_EINVAL, "pull level %d outside [0, %d)", level, p->L);
    if (!store)
        return fail(DIGEST_EINVAL, "store is NULL");
    hipStream_t s = (hipStream_t)hip_stream;
    if (p->n_halo > 0 && p->pull_mode == DIGEST_PULL_AGGREGATE) {
        if (digest_status st = halo_aggregate(p, level, s, store))
            return st;
    } else if (p->n_halo > 0) {
        {
            Timed t(p, K_PULL, level, s);
            digest_status st = hip_check(
                digest::launch_copy_rows(p->at<int32_t>(p->lay.halo_gid), nullptr, p->n_halo,
                                         p->widths[level], store,
                                         p->at<float>(p->lay.halo_buf[level]), s,
                                         p->widths[level], padded_width(p->widths[level])),
                "pull");
            if (st)
                return st;
        }
        // the halo aggregate for the next layer's GCN forward (a partition
        // with a GAT workspace forms it in each GCN forward instead)
        if (!p->gws)
            if (digest_status st = halo_aggregate(p, level, s))
                return st;
    }
    p->pulled[level] = 1;
    p->pull_gen[level] += 1;
    return DIGEST_OK;
}

digest_status digest_push(digest_partition *p, int32_t level, const float *h_own, float *store,
                          int32_t mode, void *hip_stream)
{
    if (digest_status st = need_bound(p))
        return st;
    if (level < 1 || level >= p->L)
        return fail(DIGEST_EINVAL, "push level %d outside [1, %d)", level, p->L);
    if (!h_own || !store)
        return fail(DIGEST_EINVAL, "h_own or store is NULL");
    if (mode != DIGEST_PUSH_BOUNDARY && mode != DIGEST_PUSH_ALL_OWNED)
        return fail(DIGEST_EINVAL, "unknown push mode %d", mode);
    hipStream_t s = (hipStream_t)hip_stream;
    const bool all = mode == DIGEST_PUSH_ALL_OWNED;
    const int32_t rows = all ? p->n_own : p->n_bnd;
    if (rows == 0)
        return DIGEST_OK;
    Timed t(p, K_PUSH, level, s);
    return hip_check(digest::launch_copy_rows(
                         all ? nullptr : p->at<int32_t>(p->lay.bnd_local),
                         p->at<int32_t>(all ? p->lay.owned_gid : p->lay.bnd_gid), rows,
                         p->widths[level], h_own, store, s),
                     "push");
}

digest_status digest_layer_forward(digest_partition *p, int32_t layer, const float *h_in,
                                   const float *w, float *h_out, int32_t act, void *hip_stream)
{
    if (digest_status st = need_bound(p))
        return st;
    if (layer < 1 || layer > p->L)
        return fail(DIGEST_EINVAL, "layer %d outside [1, %d]", layer, p->L);
    if (act != DIGEST_ACT_RELU && act != DIGEST_ACT_IDENTITY)
        return fail(DIGEST_EINVAL, "unknown activation %d", act);
    if (p->n_own > 0 && (!h_in || !w || !h_out))
        return fail(DIGEST_EINVAL, "NULL h_in, w or h_out");
    if (p->n_halo > 0 && !p->pulled[layer - 1])
        return fail(DIGEST_ESTATE, "level %d was never pulled", layer - 1);
    hipStream_t s = (hipStream_t)hip_stream;
    const int32_t d_in = p->widths[layer - 1], d_out = p->widths[layer];
    // The halo rows enter through their aggregate S = P_out halo (n_bnd rows),
    // formed by the pull of level layer-1, or here when a GAT workspace is
    // bound (its pulls skip it).
    const float *hs = p->n_bnd > 0 ? p->at<float>(p->lay.hagg[layer - 1]) : nullptr;
    if (p->gws && p->pull_mode == DIGEST_PULL_ROWS && p->n_own > 0)
        if (digest_status st = halo_aggregate(p, layer - 1, s))
            return st;
    const bool tf = transform_first_cheaper(*p, layer, act == DIGEST_ACT_RELU);
    if (p->n_own > 0 && tf) {
        // T = [h_in; S] W over the owned and the boundary rows, then
        // h_out = act(P_s T).  T's rows are padded to a multiple of 4 floats
        // so that the aggregation gathers whole float4 vectors; it stores
        // d_out columns
        float *T = p->at<float>(p->lay.tbuf);
        const int32_t ldt = padded_width(d_out);
        {
            Timed t(p, K_GEMM_FWD, layer, s);
            if (digest_status st = transform_rows(p, layer, h_in, hs, p->n_bnd, w, T, ldt, s))
                return st;
        }
        if (digest_status st = run_spmm(p, Csr::InH, T, nullptr, p->n_own + p->n_bnd, ldt,
                                        h_out, layer, s, nullptr, -1, nullptr, INT32_MAX,
                                        nullptr, act == DIGEST_ACT_RELU, nullptr, ldt, d_out,
                                        d_out))
            return st;
    } else if (p->n_own > 0) {
        // AH = P_s [h_in; S] = P_in h_in + P_out halo (kept for the backward),
        // then act(AH W).  Rows whose width is not a multiple of 4 floats are
        // gathered from padded copies (S is padded, h_in is copied), so that
        // the aggregation loads whole float4 vectors; AH keeps the padding.
        float *ah = p->at<float>(p->lay.ah[layer]);
        const int32_t lh = padded_width(d_in);
        const float *src0 = h_in;
        if (lh != d_in) {
            float *hp = p->at<float>(p->lay.hpad);
            Timed t(p, K_PAD_ROWS, layer, s);
            if (digest_status st = hip_check(digest::launch_copy_rows(nullptr, nullptr, p->n_own,
                                                                      d_in, h_in, hp, s, d_in, lh),
                                             "pad rows"))
                return st;
            src0 = hp;
        }
        if (fuse_forward(*p, layer, tf) &&
            digest::spmm_gemm_ok(d_in, lh, lh, src0, hs, ah, ah)) {
            // the long rows through the ordinary kernel's long-row blocks,
            // then every row tile aggregated and multiplied by W in one pass
            const int32_t *rowptr = p->at<int32_t>(p->lay.s_rowptr);
            const int32_t *col = p->at<int32_t>(p->lay.s_col);
            const float *val = p->at<float>(p->lay.s_val);
            if (p->long_s > 0) {
                Timed t(p, K_SPMM_FWD, layer, s);
                if (digest_status st = hip_check(
                        digest::launch_spmm(p->at<SpmmBlock>(p->lay.blocks_s), p->long_s,
                                            p->long_s, rowptr, col, val, src0, hs, p->n_own,
                                            lh, ah, s),
                        "spmm long rows"))
                    return st;
            }
            Timed t(p, K_SPMM_GEMM_FWD, layer, s);
            if (digest_status st = hip_check(
                    digest::launch_spmm_gemm(p->n_own, rowptr, col, val,
                                             p->at<uint8_t>(p->lay.fuse_order), src0, hs,
                                             p->n_own, lh, d_in, ah, ah, lh, w, d_out, h_out,
                                             d_out, act == DIGEST_ACT_RELU, s),
                    "fused forward"))
                return st;
            p->fwd_done[layer] = 1;
            p->act[layer] = act;
            p->tf[layer] = tf;
            p->fwd_gen[layer] = p->pull_gen[layer - 1];
            return DIGEST_OK;
        }
        if (digest_status st = run_spmm(p, Csr::InH, src0, hs, p->n_own, lh, ah, layer, s))
            return st;
        Timed t(p, K_GEMM_FWD, layer, s);
        if (narrow_out(d_in, d_out)) {
            if (digest_status st = hip_check(
                    digest::launch_narrow_n(p->n_own, p->n_own, d_in, d_out, ah, nullptr, lh, w,
                                            h_out, d_out, act == DIGEST_ACT_RELU, s),
                    "forward transform"))
                return st;
        } else {
            digest::GemmArgs g{};
            g.M = p->n_own;
            g.N = d_out;
            g.K = d_in;
            g.A = ah;
            g.lda = lh;
            g.B = w;
            g.ldb = d_out;
            g.C = h_out;
            g.ldc = d_out;
            g.relu = act == DIGEST_ACT_RELU;
            g.splits = 1;
            g.kchunk = d_in;
            g.tile = gemm_tile_for(g.M, d_out, d_in, false);
            if (digest_status st = hip_check(digest::launch_gemm(g, s), "forward gemm"))
                return st;
        }
    }
    p->fwd_done[layer] = 1;
    p->act[layer] = act;
    p->tf[layer] = tf;
    p->fwd_gen[layer] = p->pull_gen[layer - 1];
    return DIGEST_OK;
}

namespace {

// C[rows][d_in] = A[rows][d_out] W^T (W row-major [d_in][d_out]): the VALU
// kernel for contractions up to kNarrow long, the MFMA kernel with W in LDS
// up to kTimesWtK, else the MFMA GEMM.
digest_status times_wt(int32_t rows, int32_t d_in, int32_t d_out, const float *A, int32_t lda,
                       const float *w, float *C, hipStream_t s)
{
    if (narrow_valu(d_in, d_out))
        return hip_check(digest::launch_narrow_k(rows, d_in, d_out, A, lda, w, C, d_in, s),
                         "times W^T (narrow)");
    if (d_out <= digest::kTimesWtK && digest::times_wt_lds(d_out, d_in) <= digest::kNarrowNLds)
        return hip_check(digest::launch_times_wt(rows, d_in, d_out, A, lda, w, C, d_in, s),
                         "times W^T (short)");
    digest::GemmArgs h{};
    h.M = rows;
    h.N = d_in;
    h.K = d_out;
    h.A = A;
    h.lda = lda;
    h.B = w;
    h.ldb = d_out;
    h.b_trans = true;
    h.C = C;
    h.ldc = d_in;
    h.splits = 1;
    h.kchunk = d_out;
    h.tile = gemm_tile_for(rows, d_in, d_out, false);
    return hip_check(digest::launch_gemm(h, s), "times W^T");
}

// dw = [h_own; h2]^T G over the n_own owned rows and the n2 rows of a
// second block h2 (the halo rows, or the halo aggregate's boundary rows;
// rows padded_width(d_in) apart), G row-major [n_own + n2][ldg]: split-K
// slices in `part`, summed in slice order.
// Outputs up to kNarrow wide use the narrow MFMA kernel, wider ones the
// GEMM over the owned rows and over the second block's rows.
digest_status weight_grad_rows(digest_partition *p, int32_t layer, const float *h_in,
                               const float *h2, int32_t n2, const float *G, int32_t ldg,
                               float *gpart, float *dw, hipStream_t s, int32_t kind_dw,
                               int32_t kind_reduce)
{
    const int32_t d_in = p->widths[layer - 1], d_out = p->widths[layer];
    const TfPlan t = tf_plan(p->n_own, n2, d_in, d_out);
    {
        Timed tm(p, kind_dw, layer, s);
        if (t.valu) {
            if (digest_status st = hip_check(
                    digest::launch_dw_narrow(p->n_own + n2, p->n_own, d_in, d_out, h_in, h2,
                                             d_in, G, ldg, t.chunk, t.slices, gpart, s,
                                             padded_width(d_in)),
                    "dW narrow"))
                return st;
        } else {
            digest::GemmArgs g{};
            g.M = d_in;
            g.N = d_out;
            g.lda = d_in;
            g.a_trans = true;
            g.ldb = ldg;
            g.ldc = d_out;
            g.K = p->n_own;
            g.A = h_in;
            g.B = G;
            g.splits = t.s_own;
            g.kchunk = t.k_own;
            g.tile = gemm_tile_for(d_in, d_out, g.K, true);
            g.C = gpart;
            if (digest_status st = hip_check(digest::launch_gemm(g, s), "dW gemm"))
                return st;
            if (n2 > 0) {
                g.K = n2;
                g.A = h2;
                g.lda = padded_width(d_in);
                g.B = G + (int64_t)p->n_own * ldg;
                g.splits = t.s_halo;
                g.kchunk = t.k_halo;
                g.tile = gemm_tile_for(d_in, d_out, g.K, true);
                g.C = gpart + (int64_t)t.s_own * d_in * d_out;
                if (digest_status st = hip_check(digest::launch_gemm(g, s), "dW gemm"))
                    return st;
            }
        }
    }
    {
        Timed tm(p, kind_reduce, layer, s);
        if (digest_status st = hip_check(
                digest::launch_splitk_reduce(gpart, t.slices, (int64_t)d_in * d_out, dw, s),
                "dW reduce"))
            return st;
    }
    return DIGEST_OK;
}

// dW = [h_in; S]^T G and dh_in = G_own W^T for a transform-first layer,
// with G = P_s^T D: G_own = P_in^T D over the owned rows, and the boundary
// rows of G are D's rows of the boundary nodes (P_s's halo-aggregate
// entries are ones), the same dW as [h_in; halo]^T P_m^T D.  With dh_halo,
// the halo rows' gradient (P_out^T D) W^T comes from one more aggregation
// over P_out^T, into G's rows past the owned ones before the boundary rows
// take their place.  D = dh_out, or for a ReLU layer dh_out masked by
// h_out > 0, formed once (padded rows) before the transposed aggregations.
digest_status backward_transform_first(digest_partition *p, int32_t layer, const float *h_in,
                                       const float *h_out, const float *dh_out, const float *w,
                                       float *dw, float *dh_in, float *dh_halo, hipStream_t s)
{
    const int32_t d_in = p->widths[layer - 1], d_out = p->widths[layer];
    const float *hs = p->n_bnd > 0 ? p->at<float>(p->lay.hagg[layer - 1]) : nullptr;
    // G's rows are padded like T's, so that the products that read it load
    // whole vectors
    float *G = p->at<float>(p->lay.tbuf);
    const int32_t ldg = padded_width(d_out);
    float *G2 = G + (int64_t)p->n_own * ldg;   // the halo, then the boundary rows
    float *gpart = p->at<float>(p->lay.gemm_part);
    // When the widths allow, the transposed aggregations also write their
    // rows times W^T: dh_in for the owned rows, dh_halo for the halo rows.
    const bool fused_dh = dh_in && p->n_own > 0 && narrow_valu(d_in, d_out) &&
                          digest::spmm_epilogue_ok(d_out, d_in, dh_in) &&
                          (!dh_halo || digest::spmm_epilogue_ok(d_out, d_in, dh_halo));
    const digest::SpmmEpilogue ep{w, p->n_own, d_in, dh_in, nullptr};
    const digest::SpmmEpilogue ep_halo{w, 0, d_in, nullptr, dh_halo};
    // A ReLU layer's D is formed once, rows padded like G's.  Otherwise,
    // without the epilogue (which reads the stored rows back), rows of a
    // width not a multiple of 4 are gathered from a padded copy of dh_out,
    // whole float4 vectors wide; G keeps the padding columns (never read).
    const float *src = dh_out;
    int32_t dg = d_out, lsrc = d_out;   // gathered width, row stride of src
    if (p->act[layer] == DIGEST_ACT_RELU) {
        float *dm = p->at<float>(p->lay.hpad);
        Timed t(p, K_RELU_MASK, layer, s);
        if (digest_status st = hip_check(digest::launch_relu_mask(p->n_own, d_out, dh_out, d_out,
                                                                  h_out, d_out, dm, ldg, s),
                                         "relu mask"))
            return st;
        src = dm;
        lsrc = ldg;
        dg = fused_dh ? d_out : ldg;   // the epilogue contracts exactly d_out columns
    } else if (!fused_dh && ldg != d_out) {
        float *dp = p->at<float>(p->lay.hpad);
        Timed t(p, K_PAD_ROWS, layer, s);
        if (digest_status st = hip_check(digest::launch_copy_rows(nullptr, nullptr, p->n_own,
                                                                  d_out, dh_out, dp, s, d_out,
                                                                  ldg),
                                         "pad rows"))
            return st;
        src = dp;
        dg = lsrc = ldg;
    }
    if (digest_status st = run_spmm(p, Csr::InT, src, nullptr, p->n_own, dg, G, layer, s,
                                    fused_dh ? &ep : nullptr, -1, nullptr, INT32_MAX, nullptr,
                                    false, nullptr, lsrc, ldg, dg))
        return st;
    if (dh_halo) {
        // G_halo = P_out^T D; dh_halo = G_halo W^T (in the same launch when
        // the epilogue applies)
        if (digest_status st = run_spmm(p, Csr::HaloT, src, nullptr, p->n_own, dg, G2, layer, s,
                                        fused_dh ? &ep_halo : nullptr, K_HALO_GRAD, nullptr,
                                        INT32_MAX, nullptr, false, nullptr, lsrc, ldg, dg))
            return st;
        if (!fused_dh) {
            Timed tm(p, K_HALO_GRAD, layer, s);
            if (digest_status st = times_wt(p->n_halo, d_in, d_out, G2, ldg, w, dh_halo, s))
                return st;
        }
    }
    if (p->n_bnd > 0) {
        Timed t(p, K_BND_ROWS, layer, s);
        if (digest_status st = hip_check(
                digest::launch_copy_rows(p->at<int32_t>(p->lay.bnd_local), nullptr, p->n_bnd, dg,
                                         src, G2, s, lsrc, ldg),
                "boundary rows"))
            return st;
    }
    // The weight gradient and the product by W^T both only read G.  A large
    // weight gradient runs on the side stream next to it (neither kind keeps
    // the MFMA units busy alone on these narrow shapes), joined back before
    // the call returns.
    hipStream_t sw = s;
    if (!fused_dh && dh_in && side_pays(2.0 * ((double)p->n_own + p->n_bnd) * d_in * d_out))
        if (digest_status st = fork_side(p, s, &sw))
            return st;
    const digest_status st_all = [&]() -> digest_status {
        if (digest_status st = weight_grad_rows(p, layer, h_in, hs, p->n_bnd, G, ldg, gpart, dw,
                                                sw, K_GEMM_DW, K_REDUCE_DW))
            return st;
        if (fused_dh || !dh_in)
            return DIGEST_OK;
        Timed tm(p, K_GEMM_DH, layer, s);
        return times_wt(p->n_own, d_in, d_out, G, ldg, w, dh_in, s);
    }();
    if (sw != s) {
        const digest_status st = join_side(p, s);
        return st_all ? st_all : st;
    }
    return st_all;
}

}  // namespace

}  // extern "C"

namespace {

// The layer backward of both entry points.  With dh_halo (layer >= 2, dh_in
// given) the halo rows' gradient P_out^T D W^T comes out of the same
// products: aggregating first, the transposed aggregation runs over all of
// P_m^T, its owned rows into dh_in and its halo rows into dh_halo (or into
// the halo scratch that one more product by W^T finishes); transform-first,
// one more aggregation over P_out^T (backward_transform_first).
digest_status layer_backward(digest_partition *p, int32_t layer, const float *h_in,
                             const float *h_out, const float *dh_out, const float *w, float *dw,
                             float *dh_in, float *dh_halo, hipStream_t s)
{
    if (p->n_halo == 0)
        dh_halo = nullptr;
    const int32_t d_in = p->widths[layer - 1], d_out = p->widths[layer];
    if (p->tf[layer] && p->n_own > 0)
        return backward_transform_first(p, layer, h_in, h_out, dh_out, w, dw, dh_in, dh_halo,
                                        s);
    const bool relu = p->act[layer] == DIGEST_ACT_RELU;
    const float *ah = p->at<float>(p->lay.ah[layer]);
    // The fused input gradient: D = dh_out masked by the ReLU derivative is
    // formed once (the weight gradient reads it too), then (P_in^T D) W^T in
    // one pass after a long-row pass.
    const int32_t ldz = padded_width(d_out);
    float *dz = p->at<float>(p->lay.fz);
    float *zpre = dz + (int64_t)p->n_own * ldz;
    const bool fused = dh_in && !dh_halo && relu && p->n_own > 0 &&
                       fuse_backward(*p, layer, false) &&
                       digest::spmm_gemm_ok(d_out, ldz, ldz, dz, nullptr, nullptr, zpre);
    const float *gd = fused ? dz : dh_out;   // the weight gradient's D operand
    const int32_t ldd = fused ? ldz : d_out;

    // dW = AH^T D, D = dh_out (masked by h_out > 0 for ReLU), split over rows,
    // on stream sw.
    auto weight_grad = [&](hipStream_t sw) -> digest_status {
        digest::GemmArgs g{};
        g.M = d_in;
        g.N = d_out;
        g.K = p->n_own;
        g.A = ah;
        g.lda = padded_width(d_in);
        g.a_trans = true;
        g.B = gd;
        g.ldb = ldd;
        g.b_mask = relu && !fused ? h_out : nullptr;
        splitk_plan(d_in, d_out, p->n_own, g.splits, g.kchunk,
                    sw != s ? kSideSplitTarget : kSplitTarget);
        g.tile = gemm_tile_for(d_in, d_out, p->n_own, true);
        float *gpart = p->at<float>(p->lay.gemm_part);
        g.C = g.splits > 1 ? gpart : dw;
        g.ldc = d_out;
        {
            Timed t(p, K_GEMM_DW, layer, sw);
            if (digest_status st = hip_check(digest::launch_gemm(g, sw), "dW gemm"))
                return st;
        }
        if (g.splits <= 1)
            return DIGEST_OK;
        Timed t(p, K_REDUCE_DW, layer, sw);
        return hip_check(
            digest::launch_splitk_reduce(gpart, g.splits, (int64_t)d_in * d_out, dw, sw),
            "dW reduce");
    };
    if (!dh_in || p->n_own == 0) {
        if (digest_status st = weight_grad(s))
            return st;
        if (p->n_own == 0 && dh_halo)
            // no owned row reads a halo row: the halo gradient is zero
            return hip_check(digest::launch_fill_zero(dh_halo, (int64_t)p->n_halo * d_in, s),
                             "zero halo gradient");
        return DIGEST_OK;
    }

    // The input gradient: its transposed aggregation is bound by memory, so
    // a large weight gradient (bound by the MFMA units) runs next to it on the
    // side stream, started right before it and joined at the end of the call.
    hipStream_t sw = s;
    auto start_weight_grad = [&]() -> digest_status {
        if (side_pays(2.0 * p->n_own * d_in * d_out))
            if (digest_status st = fork_side(p, s, &sw))
                return st;
        return weight_grad(sw);
    };
    const digest_status st_all = [&]() -> digest_status {
        if (fused) {
            {
                Timed t(p, K_RELU_MASK, layer, s);
                if (digest_status st = hip_check(digest::launch_relu_mask(p->n_own, d_out, dh_out,
                                                                          d_out, h_out, d_out,
                                                                          dz, ldz, s),
                                                 "relu mask"))
                    return st;
            }
            if (digest_status st = start_weight_grad())
                return st;
            float *wt = p->at<float>(p->lay.wt);
            {
                Timed t(p, K_TRANSPOSE_W, layer, s);
                if (digest_status st =
                        hip_check(digest::launch_transpose(d_in, d_out, w, wt, s), "W^T"))
                    return st;
            }
            const int32_t *trp = p->at<int32_t>(p->lay.t_rowptr);
            const int32_t *tsrc = p->at<int32_t>(p->lay.t_src);
            const float *tval = p->at<float>(p->lay.t_val);
            if (p->long_t > 0) {
                Timed t(p, K_SPMM_BWD, layer, s);
                if (digest_status st = hip_check(
                        digest::launch_spmm(p->at<SpmmBlock>(p->lay.blocks_t), p->long_t,
                                            p->long_t, trp, tsrc, tval, dz, nullptr, p->n_own,
                                            ldz, zpre, s),
                        "transposed spmm long rows"))
                    return st;
            }
            Timed t(p, K_SPMM_GEMM_BWD, layer, s);
            return hip_check(digest::launch_spmm_gemm(p->n_own, trp, tsrc, tval,
                                                      p->at<uint8_t>(p->lay.fuse_order_t), dz,
                                                      nullptr, p->n_own, ldz, d_out, nullptr,
                                                      zpre, ldz, wt, d_in, dh_in, d_in, false, s),
                             "fused input gradient");
        }
        // P_in^T alone, or P_m^T with its halo rows split off
        const Csr tr = dh_halo ? Csr::FullT : Csr::InT;
        const int32_t split = dh_halo ? p->n_own : INT32_MAX;
        float *tmp = p->at<float>(p->lay.tmp);
        if (!relu && d_out < d_in) {
            // Narrower output: aggregate D first (width d_out), then times W^T.
            float *gh = p->at<float>(p->lay.tmp_halo);
            if (digest_status st = start_weight_grad())
                return st;
            if (digest_status st = run_spmm(p, tr, dh_out, nullptr, p->n_own, d_out, tmp, layer,
                                            s, nullptr, -1, dh_halo ? gh : nullptr, split))
                return st;
            {
                Timed t(p, K_GEMM_DH, layer, s);
                if (digest_status st = times_wt(p->n_own, d_in, d_out, tmp, d_out, w, dh_in, s))
                    return st;
            }
            if (!dh_halo)
                return DIGEST_OK;
            Timed t(p, K_HALO_GRAD, layer, s);
            return times_wt(p->n_halo, d_in, d_out, gh, d_out, w, dh_halo, s);
        }
        // Otherwise G = D W^T (mask fused into the operand load), then the
        // transposed aggregation of G.
        digest::GemmArgs h{};
        h.M = p->n_own;
        h.N = d_in;
        h.K = d_out;
        h.B = w;
        h.ldb = d_out;
        h.b_trans = true;
        h.ldc = d_in;
        h.splits = 1;
        h.kchunk = d_out;
        h.tile = gemm_tile_for(p->n_own, d_in, d_out, false);
        h.A = dh_out;
        h.lda = d_out;
        h.a_mask = relu ? h_out : nullptr;
        h.C = tmp;
        {
            Timed t(p, K_GEMM_DH, layer, s);
            if (digest_status st = hip_check(digest::launch_gemm(h, s), "dgrad gemm"))
                return st;
        }
        if (digest_status st = start_weight_grad())
            return st;
        return run_spmm(p, tr, tmp, nullptr, p->n_own, d_in, dh_in, layer, s, nullptr, -1,
                        dh_halo, split);
    }();
    if (sw != s) {
        const digest_status st = join_side(p, s);
        return st_all ? st_all : st;
    }
    return st_all;
}

// Argument and state checks shared by both backward entry points.
digest_status check_backward(const digest_partition *p, int32_t layer, const float *h_in,
                             const float *h_out, const float *dh_out, const float *w,
                             const float *dw)
{
    if (digest_status st = need_bound(p))
        return st;
    if (layer < 1 || layer > p->L)
        return fail(DIGEST_EINVAL, "layer %d outside [1, %d]", layer, p->L);
    if (!dw || !w || (p->n_own > 0 && (!h_in || !h_out || !dh_out)))
        return fail(DIGEST_EINVAL, "NULL h_in, h_out, dh_out, w or dw");
    if (!p->fwd_done[layer])
        return fail(DIGEST_ESTATE, "no forward of layer %d since the workspace was bound",
                    layer);
    if (p->fwd_gen[layer] != p->pull_gen[layer - 1])
        return fail(DIGEST_ESTATE,
                    "level %d was pulled again between the forward and backward of layer %d",
                    layer - 1, layer);
    return DIGEST_OK;
}

}  // namespace

extern "C" {

digest_status digest_layer_backward(digest_partition *p, int32_t layer, const float *h_in,
                                    const float *h_out, const float *dh_out, const float *w,
                                    float *dw, float *dh_in, void *hip_stream)
{
    if (digest_status st = check_backward(p, layer, h_in, h_out, dh_out, w, dw))
        return st;
    return layer_backward(p, layer, h_in, h_out, dh_out, w, dw, dh_in, nullptr,
                          (hipStream_t)hip_stream);
}

digest_status digest_layer_backward_halo(digest_partition *p, int32_t layer, const float *h_in,
                                         const float *h_out, const float *dh_out,
                                         const float *w, float *dw, float *dh_in,
                                         float *dh_halo, void *hip_stream)
{
    if (digest_status st = need_bound(p))
        return st;
    if (layer < 2 || layer > p->L)
        return fail(DIGEST_EINVAL, "halo gradient of layer %d outside [2, %d]", layer, p->L);
    if ((p->n_own > 0 && !dh_in) || (p->n_halo > 0 && !dh_halo))
        return fail(DIGEST_EINVAL, "NULL dh_in or dh_halo");
    if (digest_status st = check_backward(p, layer, h_in, h_out, dh_out, w, dw))
        return st;
    return layer_backward(p, layer, h_in, h_out, dh_out, w, dw, dh_in, dh_halo,
                          (hipStream_t)hip_stream);
}

digest_status digest_softmax_xent(digest_partition *p, const float *logits,
                                  const int32_t *labels, float *dlogits, float *loss,
                                  void *hip_stream)
{
    if (digest_status st = need_bound(p))
        return st;
    if (!loss || (p->n_own > 0 && (!logits || !labels || !dlogits)))
        return fail(DIGEST_EINVAL, "NULL logits, labels, dlogits or loss");
    hipStream_t s = (hipStream_t)hip_stream;
    const int32_t C = p->widths[p->L];
    float *part = p->at<float>(p->lay.loss_part);
    {
        Timed t(p, K_LOSS, p->L, s);
        if (digest_status st = hip_check(
                digest::launch_softmax_xent(logits, labels, p->n_own, C, dlogits, part, s),
                "softmax xent"))
            return st;
    }
    Timed t(p, K_LOSS_MEAN, p->L, s);
    return hip_check(digest::launch_loss_mean(part, p->n_own, C, loss, s), "loss mean");
}

digest_status digest_softmax_xent_static(int64_t n_rows, int32_t n_classes,
                                         const float *logits, const int32_t *labels,
                                         float *dlogits, float *loss, void *hip_stream)
{
    static_assert(DIGEST_STATIC_SCRATCH_FLOATS == digest::kStaticScratchFloats,
                  "the header's scratch size is the library's");
    if (n_rows < 0 || n_rows >= INT32_MAX)
        return fail(DIGEST_EINVAL, "n_rows %lld out of range", (long long)n_rows);
    if (n_classes < 1 || n_classes > kMaxWidth)
        return fail(DIGEST_EINVAL, "n_classes %d outside [1, %d]", n_classes, kMaxWidth);
    if (!loss || (n_rows > 0 && (!logits || !labels || !dlogits)))
        return fail(DIGEST_EINVAL, "NULL logits, labels, dlogits or loss");
    const int64_t blocks = digest::softmax_xent_blocks((int32_t)n_rows, n_classes);
    if (blocks > (int64_t)digest::kStaticScratchFloats)
        return fail(DIGEST_EINVAL,
                    "%lld rows of %d classes need %lld partial sums; the static scratch holds "
                    "%zu (at most %lld rows)",
                    (long long)n_rows, n_classes, (long long)blocks, digest::kStaticScratchFloats,
                    (long long)digest::kStaticScratchFloats *
                        digest::softmax_xent_rows_per_block(n_classes));
    hipStream_t s = (hipStream_t)hip_stream;
    int dev = -1;
    if (digest_status st = hip_check(hipGetDevice(&dev), "current device"))
        return st;
    if (s) {
        hipDevice_t sdev = -1;
        if (digest_status st = hip_check(hipStreamGetDevice(s, &sdev), "stream device"))
            return st;
        if (sdev != dev)
            return fail(DIGEST_EINVAL, "the stream belongs to device %d, the current device is %d",
                        (int)sdev, dev);
    }
    float *part = nullptr;
    if (digest_status st = hip_check(digest::static_scratch(&part), "static scratch"))
        return st;
    if (digest_status st = hip_check(digest::launch_softmax_xent(logits, labels, (int32_t)n_rows,
                                                                 n_classes, dlogits, part, s),
                                     "softmax xent"))
        return st;
    return hip_check(digest::launch_loss_mean(part, (int32_t)n_rows, n_classes, loss, s),
                     "loss mean");
}

digest_status digest_halo_gradient(digest_partition *p, int32_t layer, const float *h_out,
                                   const float *dh_out, const float *w, float *dh_halo,
                                   void *hip_stream)
{
    if (digest_status st = need_bound(p))
        return st;
    if (layer < 2 || layer > p->L)
        return fail(DIGEST_EINVAL, "halo gradient of layer %d outside [2, %d]", layer, p->L);
    if (!w || (p->n_own > 0 && (!h_out || !dh_out)) || (p->n_halo > 0 && !dh_halo))
        return fail(DIGEST_EINVAL, "NULL h_out, dh_out, w or dh_halo");
    if (!p->fwd_done[layer])
        return fail(DIGEST_ESTATE, "no forward of layer %d since the workspace was bound",
                    layer);
    if (p->n_halo == 0)
        return DIGEST_OK;
    hipStream_t s = (hipStream_t)hip_stream;
    const int32_t d_in = p->widths[layer - 1], d_out = p->widths[layer];
    const bool relu = p->act[layer] == DIGEST_ACT_RELU;
    digest::GemmArgs h{};
    h.N = d_in;
    h.K = d_out;
    h.B = w;
    h.ldb = d_out;
    h.b_trans = true;
    h.ldc = d_in;
    h.splits = 1;
    h.kchunk = d_out;
    if (!relu && d_out < d_in) {
        // narrower output: (P_out^T D) W^T, the aggregation at width d_out
        float *gh = p->at<float>(p->lay.tmp_halo);
        if (digest_status st = run_spmm(p, Csr::HaloT, dh_out, nullptr, p->n_own, d_out, gh,
                                        layer, s, nullptr, K_HALO_GRAD))
            return st;
        Timed t(p, K_HALO_GRAD, layer, s);
        return times_wt(p->n_halo, d_in, d_out, gh, d_out, w, dh_halo, s);
    }
    // otherwise P_out^T (D W^T), with the ReLU mask fused into the GEMM
    float *tmp = p->at<float>(p->lay.tmp);
    h.M = p->n_own;
    h.A = dh_out;
    h.lda = d_out;
    h.a_mask = relu ? h_out : nullptr;
    h.C = tmp;
    h.tile = gemm_tile_for(p->n_own, d_in, d_out, false);
    {
        Timed t(p, K_HALO_GRAD, layer, s);
        if (digest_status st = hip_check(digest::launch_gemm(h, s), "halo gradient"))
            return st;
    }
    return run_spmm(p, Csr::HaloT, tmp, nullptr, p->n_own, d_in, dh_halo, layer, s, nullptr,
                    K_HALO_GRAD);
}

digest_status digest_push_add(digest_partition *p, int32_t level, const float *dh_halo,
                              float *gstore, void *hip_stream)
{
    if (digest_status st = need_bound(p))
        return st;
    if (level < 1 || level >= p->L)
        return fail(DIGEST_EINVAL, "gradient level %d outside [1, %d)", level, p->L);
    if (!gstore || (p->n_halo > 0 && !dh_halo))
        return fail(DIGEST_EINVAL, "NULL dh_halo or gradient store");
    if (p->n_halo == 0)
        return DIGEST_OK;
    hipStream_t s = (hipStream_t)hip_stream;
    Timed t(p, K_GRAD_PUSH, level, s);
    return hip_check(digest::launch_add_rows(nullptr, p->at<int32_t>(p->lay.halo_gid),
                                             p->n_halo, p->widths[level], dh_halo, gstore, s),
                     "gradient push");
}

digest_status digest_pull_add(digest_partition *p, int32_t level, float *gstore, float *dh_own,
                              void *hip_stream)
{
    if (digest_status st = need_bound(p))
        return st;
    if (level < 1 || level >= p->L)
        return fail(DIGEST_EINVAL, "gradient level %d outside [1, %d)", level, p->L);
    if (!gstore || (p->n_own > 0 && !dh_own))
        return fail(DIGEST_EINVAL, "NULL gradient store or dh_own");
    if (p->n_own == 0)
        return DIGEST_OK;
    hipStream_t s = (hipStream_t)hip_stream;
    Timed t(p, K_GRAD_PULL, level, s);
    return hip_check(digest::launch_add_clear_rows(p->at<int32_t>(p->lay.owned_gid), nullptr,
                                                   p->n_own, p->widths[level], gstore, dh_own,
                                                   s),
                     "gradient pull");
}

digest_status digest_sgd_average(float *w, const float *const *grads, int32_t n_grads,
                                 int64_t count, float lr, void *hip_stream)
{
    if (n_grads < 1 || n_grads > digest::kMaxAverage)
        return fail(DIGEST_EINVAL, "need 1 <= n_grads <= %d, got %d", digest::kMaxAverage,
                    n_grads);
    if (count < 0)
        return fail(DIGEST_EINVAL, "negative count");
    if (count > 0 && (!w || !grads))
        return fail(DIGEST_EINVAL, "NULL w or grads");
    digest::GradList g{};
    for (int32_t m = 0; m < n_grads && count > 0; ++m) {
        if (!grads[m])
            return fail(DIGEST_EINVAL, "grads[%d] is NULL", m);
        g.g[m] = grads[m];
    }
    return hip_check(digest::launch_sgd_average(w, g, n_grads, count, lr,
                                                (hipStream_t)hip_stream),
                     "sgd average");
}

digest_status digest_gat_query(const digest_partition *p, size_t *workspace_bytes)
{
    if (!p || !workspace_bytes)
        return fail(DIGEST_EINVAL, "NULL handle or output");
    *workspace_bytes = p->glay.total;
    return DIGEST_OK;
}

digest_status digest_gat_bind_workspace(digest_partition *p, void *dev_ptr, size_t bytes,
                                        void *hip_stream)
{
    if (!p || !dev_ptr)
        return fail(DIGEST_EINVAL, "NULL handle or workspace");
    if ((uintptr_t)dev_ptr % kAlign)
        return fail(DIGEST_EINVAL, "workspace must be %zu-byte aligned", kAlign);
    if (bytes < p->glay.total)
        return fail(DIGEST_ENOMEM, "GAT workspace has %zu bytes, needs %zu", bytes,
                    p->glay.total);
    hipStream_t s = (hipStream_t)hip_stream;
    char *ws = (char *)dev_ptr;
    if (p->nnz > 0)
        if (digest_status st = hip_check(
                hipMemcpyAsync(ws + p->glay.t_perm, p->t_perm.data(), sizeof(int32_t) * p->nnz,
                               hipMemcpyHostToDevice, s),
                "GAT upload"))
            return st;
    if (p->n_own > 0) {
        const std::vector<float> ones((size_t)p->n_own, 1.0f);
        if (digest_status st = hip_check(
                hipMemcpyAsync(ws + p->glay.ones, ones.data(), sizeof(float) * p->n_own,
                               hipMemcpyHostToDevice, s),
                "GAT upload"))
            return st;
        // the host vector dies here: wait for the copy
        if (digest_status st = hip_check(hipStreamSynchronize(s), "GAT upload"))
            return st;
    }
    p->gws = ws;
    std::fill(p->gat_done.begin(), p->gat_done.end(), 0);
    return DIGEST_OK;
}

digest_status digest_gat_forward(digest_partition *p, int32_t layer, const float *h_in,
                                 const float *w, const float *att, float negative_slope,
                                 float *h_out, int32_t act, void *hip_stream)
{
    if (digest_status st = need_bound(p))
        return st;
    if (!p->gws)
        return fail(DIGEST_ESTATE, "no GAT workspace bound");
    if (layer < 1 || layer > p->L)
        return fail(DIGEST_EINVAL, "layer %d outside [1, %d]", layer, p->L);
    if (act != DIGEST_ACT_RELU && act != DIGEST_ACT_IDENTITY)
        return fail(DIGEST_EINVAL, "unknown activation %d", act);
    if (!(negative_slope >= 0.f && negative_slope <= 1.f))
        return fail(DIGEST_EINVAL, "negative slope must be in [0, 1]");
    const int32_t d_out = p->widths[layer];
    if (d_out > digest::kGatMaxWidth)
        return fail(DIGEST_EINVAL, "GAT layer width %d above %d", d_out, digest::kGatMaxWidth);
    if (!w || !att || (p->n_own > 0 && (!h_in || !h_out)))
        return fail(DIGEST_EINVAL, "NULL h_in, w, att or h_out");
    if (p->n_halo > 0 && !p->pulled[layer - 1])
        return fail(DIGEST_ESTATE, "level %d was never pulled", layer - 1);
    if (p->n_halo > 0 && p->pull_mode != DIGEST_PULL_ROWS)
        return fail(DIGEST_ESTATE, "the GAT layer reads halo rows, which the pull mode skips");
    hipStream_t s = (hipStream_t)hip_stream;
    const float *halo = p->n_halo > 0 ? p->at<float>(p->lay.halo_buf[layer - 1]) : nullptr;
    const int32_t R = p->n_own + p->n_halo;
    float *Z = p->gat<float>(p->glay.z[layer]);
    float *S = p->gat<float>(p->glay.s[layer]);
    float *alpha = p->gat<float>(p->glay.alpha[layer]);
    {
        Timed t(p, K_GAT_TRANSFORM, layer, s);
        if (digest_status st = transform_rows(p, layer, h_in, halo, p->n_halo, w, Z,
                                              p->widths[layer], s))
            return st;
    }
    {
        // scores: S = Z att, [R][2] (source, target)
        Timed t(p, K_GAT_SCORES, layer, s);
        if (digest_status st = hip_check(
                digest::launch_narrow_n(R, R, d_out, 2, Z, nullptr, d_out, att, S, 2, false, s),
                "GAT scores"))
            return st;
    }
    if (p->n_own > 0) {
        {
            Timed t(p, K_GAT_SOFTMAX, layer, s);
            if (digest_status st = hip_check(
                    digest::launch_gat_softmax(p->n_own, p->at<int32_t>(p->lay.rowptr),
                                               p->at<int32_t>(p->lay.col), S, negative_slope,
                                               alpha, s),
                    "GAT softmax"))
                return st;
        }
        if (digest_status st = run_spmm(p, Csr::Fwd, Z, nullptr, R, d_out, h_out, layer, s,
                                        nullptr, K_GAT_AGG, nullptr, INT32_MAX, alpha,
                                        act == DIGEST_ACT_RELU))
            return st;
    }
    p->gat_done[layer] = 1;
    p->gat_gen[layer] = p->pull_gen[layer - 1];
    p->gat_act[layer] = act;
    p->gat_slope[layer] = negative_slope;
    return DIGEST_OK;
}

digest_status digest_gat_backward(digest_partition *p, int32_t layer, const float *h_in,
                                  const float *h_out, const float *dh_out, const float *w,
                                  const float *att, float *dw, float *datt, float *dh_in,
                                  void *hip_stream)
{
    if (digest_status st = need_bound(p))
        return st;
    if (!p->gws)
        return fail(DIGEST_ESTATE, "no GAT workspace bound");
    if (layer < 1 || layer > p->L)
        return fail(DIGEST_EINVAL, "layer %d outside [1, %d]", layer, p->L);
    if (!w || !att || !dw || !datt || (p->n_own > 0 && (!h_in || !h_out || !dh_out)))
        return fail(DIGEST_EINVAL, "NULL h_in, h_out, dh_out, w, att, dw or datt");
    if (!p->gat_done[layer])
        return fail(DIGEST_ESTATE, "no GAT forward of layer %d since the GAT workspace was bound",
                    layer);
    if (p->gat_gen[layer] != p->pull_gen[layer - 1])
        return fail(DIGEST_ESTATE,
                    "level %d was pulled again between the GAT forward and backward of layer %d",
                    layer - 1, layer);
    if (p->n_halo > 0 && p->pull_mode != DIGEST_PULL_ROWS)
        return fail(DIGEST_ESTATE, "the GAT layer reads halo rows, which the pull mode skips");
    hipStream_t s = (hipStream_t)hip_stream;
    const int32_t d_in = p->widths[layer - 1], d_out = p->widths[layer];
    const int32_t R = p->n_own + p->n_halo;
    const float *halo = p->n_halo > 0 ? p->at<float>(p->lay.halo_buf[layer - 1]) : nullptr;
    const float *Z = p->gat<float>(p->glay.z[layer]);
    const float *S = p->gat<float>(p->glay.s[layer]);
    const float *alpha = p->gat<float>(p->glay.alpha[layer]);
    float *alpha_t = p->gat<float>(p->glay.alpha_t);
    float *dpre = p->gat<float>(p->glay.dpre);
    float *dpre_t = p->gat<float>(p->glay.dpre_t);
    float *dO = p->gat<float>(p->glay.d_o);
    float *dz = p->gat<float>(p->glay.dz);
    float *ds_src = p->gat<float>(p->glay.ds_src);
    float *g2 = p->gat<float>(p->glay.g2);
    float *part = p->gat<float>(p->glay.part);
    {
        // dO, the per-edge score gradients and their row sums (g2[i][1])
        Timed t(p, K_GAT_EDGE_GRAD, layer, s);
        if (digest_status st = hip_check(
                digest::launch_gat_edge_grad(p->at<SpmmBlock>(p->lay.blocks_f),
                                             (int32_t)p->blocks_f.size(), d_out,
                                             p->at<int32_t>(p->lay.rowptr),
                                             p->at<int32_t>(p->lay.col), alpha, S, Z, h_out,
                                             dh_out, p->gat_act[layer] == DIGEST_ACT_RELU,
                                             p->gat_slope[layer], dO, dpre, g2, s),
                "GAT edge gradient"))
            return st;
    }
    {
        Timed t(p, K_GAT_PERM, layer, s);
        if (digest_status st = hip_check(
                digest::launch_gather_perm2(p->nnz, p->gat<int32_t>(p->glay.t_perm), alpha, dpre,
                                            alpha_t, dpre_t, s),
                "GAT transpose"))
            return st;
    }
    // source-score gradients: column sums of dpre
    if (digest_status st = run_spmm(p, Csr::FullT, p->gat<float>(p->glay.ones), nullptr,
                                    p->n_own, 1, ds_src, layer, s, nullptr, K_GAT_SCORE_SUMS,
                                    nullptr, INT32_MAX, dpre_t))
        return st;
    // dz = (alpha-weighted P_m)^T dO over every local row, plus the score
    // terms ds_src[v] att[:,0] + (owned v) g2[v][1] att[:,1] added in its store
    {
        digest::SpmmRank1 r1;
        r1.a = att;
        r1.x = ds_src;
        r1.y = g2;
        r1.ny = p->n_own;
        if (digest_status st = run_spmm(p, Csr::FullT, dO, nullptr, p->n_own, d_out, dz, layer,
                                        s, nullptr, K_GAT_AGG_T, nullptr, INT32_MAX, alpha_t,
                                        false, &r1))
            return st;
    }
    {
        // the datt operand [ds_src, row sums of the owned rows]
        Timed t(p, K_GAT_SCORE_GRAD, layer, s);
        if (digest_status st = hip_check(
                digest::launch_gat_score_cols(R, p->n_own, ds_src, g2, s), "GAT score columns"))
            return st;
    }
    {
        // datt = Z^T g2 ([d_out][2])
        int32_t chunk, slices;
        narrow_rows_plan(R, d_out, chunk, slices);
        Timed t(p, K_GAT_DATT, layer, s);
        if (digest_status st = hip_check(
                digest::launch_dw_narrow(R, R, d_out, 2, Z, nullptr, d_out, g2, 2, chunk, slices,
                                         part, s),
                "GAT datt"))
            return st;
        if (digest_status st = hip_check(
                digest::launch_splitk_reduce(part, slices, (int64_t)d_out * 2, datt, s),
                "GAT datt reduce"))
            return st;
    }
    if (digest_status st = weight_grad_rows(p, layer, h_in, halo, p->n_halo, dz, d_out, part, dw,
                                            s, K_GAT_DW, K_REDUCE_DW))
        return st;
    if (!dh_in || p->n_own == 0)
        return DIGEST_OK;
    Timed t(p, K_GAT_DGRAD, layer, s);
    return times_wt(p->n_own, d_in, d_out, dz, d_out, w, dh_in, s);
}

digest_status digest_sync_period(int32_t K, int64_t iter, int32_t *do_pull, int32_t *do_push)
{
    if (K < 1 || iter < 1 || !do_pull || !do_push)
        return fail(DIGEST_EINVAL, "need K >= 1, iter >= 1 and non-NULL outputs");
    *do_pull = (iter % K) == 0;
    *do_push = ((iter - 1) % K) == 0;
    return DIGEST_OK;
}

digest_status digest_profile_enable(digest_partition *p, int32_t on)
{
    if (!p)
        return fail(DIGEST_EINVAL, "NULL partition handle");
    p->prof = on != 0;
    return DIGEST_OK;
}

digest_status digest_profile_read(digest_partition *p, double *total_ms, int64_t *launches)
{
    if (!p || !total_ms || !launches)
        return fail(DIGEST_EINVAL, "NULL argument");
    const int32_t slots = p->L + 1;
    for (int32_t k = 0; k < K_COUNT * slots; ++k) {
        total_ms[k] = 0.0;
        launches[k] = 0;
    }
    digest_status st = DIGEST_OK;
    for (auto &r : p->recs) {
        if (!st) {
            hipError_t e = hipEventSynchronize(r.b);
            float ms = 0.f;
            if (e == hipSuccess)
                e = hipEventElapsedTime(&ms, r.a, r.b);
            if (e != hipSuccess)
                st = hip_check(e, "profile read");
            total_ms[r.kind * slots + r.layer] += ms;
            launches[r.kind * slots + r.layer] += 1;
        }
        p->pool.push_back(r.a);
        p->pool.push_back(r.b);
    }
    p->recs.clear();
    return st;
}

int32_t digest_profile_kernel_count(void) { return K_COUNT; }

const char *digest_profile_kernel_name(int32_t kind)
{
    return (kind >= 0 && kind < K_COUNT) ? kKindNames[kind] : "";
}

}  // extern "C"

namespace {

// The plan of one layer (see digest_layer_plan).  Device pointers are
// assumed 16-byte aligned, as the layer calls' callers pass them.
digest_layer_plan layer_plan(const digest_partition &p, int32_t layer)
{
    digest_layer_plan pl{};
    const int32_t d_in = p.widths[layer - 1], d_out = p.widths[layer];
    const bool relu = layer < p.L;
    pl.transform_first = p.n_own > 0 && transform_first_cheaper(p, layer, relu);
    pl.forward_narrow = narrow_out(d_in, d_out);
    pl.forward_fused = fuse_forward(p, layer, pl.transform_first);
    pl.backward_fused = fuse_backward(p, layer, pl.transform_first);
    if (pl.transform_first) {
        pl.dw_slices = tf_plan(p.n_own, p.n_bnd, d_in, d_out).slices;
        pl.dgrad_fused = layer > 1 && narrow_valu(d_in, d_out) &&
                         digest::spmm_epilogue_ok(d_out, d_in, nullptr);
    } else {
        int32_t splits = 1, kchunk = 0;
        splitk_plan(d_in, d_out, p.n_own, splits, kchunk);
        pl.dw_slices = splits;
        pl.dgrad_narrow_first = !relu && d_out < d_in;
        if (const TierPlan *t = find_tiers(p, Csr::InH, padded_width(d_in))) {
            pl.tiers_fwd = t->tiers;
            pl.tier_rows_fwd = t->rows_per_tier;
            pl.tier_entries_fwd = t->tier_entries;
        }
        if (layer > 1)
            if (const TierPlan *t =
                    find_tiers(p, Csr::InT, pl.dgrad_narrow_first ? d_out : d_in)) {
                pl.tiers_bwd = t->tiers;
                pl.tier_rows_bwd = t->rows_per_tier;
                pl.tier_entries_bwd = t->tier_entries;
            }
    }
    return pl;
}

}  // namespace

extern "C" {

digest_status digest_partition_plan(const digest_partition *p, int32_t layer,
                                    digest_layer_plan *out)
{
    if (!p || !out)
        return fail(DIGEST_EINVAL, "NULL handle or output");
    if (layer < 1 || layer > p->L)
        return fail(DIGEST_EINVAL, "layer %d outside [1, %d]", layer, p->L);
    *out = layer_plan(*p, layer);
    return DIGEST_OK;
}

digest_status digest_profile_model(const digest_partition *p, int32_t model, double *bytes,
                                   double *flops, int64_t *entries)
{
    if (!p || !bytes || !flops || !entries)
        return fail(DIGEST_EINVAL, "NULL argument");
    if (model != DIGEST_MODEL_GCN && model != DIGEST_MODEL_GAT)
        return fail(DIGEST_EINVAL, "unknown model %d", model);
    const int32_t slots = p->L + 1;
    for (int32_t k = 0; k < K_COUNT * slots; ++k) {
        bytes[k] = 0.0;
        flops[k] = 0.0;
        entries[k] = 0;
    }
    auto put = [&](int32_t kind, int32_t slot, double b, double f = 0.0, int64_t e = 0) {
        bytes[kind * slots + slot] = b;
        flops[kind * slots + slot] = f;
        entries[kind * slots + slot] = e;
    };
    const double n = p->n_own, nh = p->n_halo, nb = p->n_bnd, R = n + nh, Rs = n + nb;
    const double nnz = (double)p->nnz, nnz_in = (double)p->nnz_in, nnz_s = (double)p->nnz_s;
    const int32_t L = p->L;
    for (int32_t l = 1; l <= L; ++l) {
        const double di = p->widths[l - 1], dout = p->widths[l];
        const bool relu = l < L;
        if (model == DIGEST_MODEL_GAT) {
            const TfPlan t = tf_plan(p->n_own, p->n_halo, p->widths[l - 1], p->widths[l]);
            put(K_GAT_TRANSFORM, l, 4 * (R * di + di * dout + R * dout), 2 * R * di * dout);
            put(K_GAT_SCORES, l, 4 * (R * dout + 2 * dout + 2 * R), 4 * R * dout);
            put(K_GAT_SOFTMAX, l, 4 * (n + 1) + 16 * nnz + 4 * n);
            put(K_GAT_AGG, l, 4 * (n + 1) + 8 * nnz + 4 * R * dout + 4 * n * dout, 0.0, p->nnz);
            put(K_GAT_EDGE_GRAD, l,
                4 * (n + 1) + 12 * nnz + 12 * n * dout + 4 * R * dout + 8 * R + 4 * n, 0.0,
                p->nnz);
            put(K_GAT_PERM, l, 20 * nnz);
            put(K_GAT_AGG_T, l,
                4 * (R + 1) + 8 * nnz + 4 * n * dout + 4 * R * dout + 4 * R + 4 * n + 8 * dout,
                0.0, p->nnz);
            put(K_GAT_SCORE_SUMS, l, 4 * (R + 1) + 8 * nnz + 4 * n + 4 * R);
            put(K_GAT_SCORE_GRAD, l, 8 * R + 4 * nh);
            put(K_GAT_DATT, l, 4 * (R * dout + 2 * R + 2 * dout), 4 * R * dout);
            put(K_GAT_DW, l, 4 * (R * di + R * dout + di * dout), 2 * R * di * dout);
            put(K_REDUCE_DW, l, 4 * (t.slices + 1) * di * dout);
            if (l > 1)
                put(K_GAT_DGRAD, l, 4 * (n * dout + di * dout + n * di), 2 * n * di * dout);
            continue;
        }
        const digest_layer_plan pl = layer_plan(*p, l);
        if (pl.transform_first) {
            // over the owned rows and the halo aggregate's boundary rows
            put(K_GEMM_FWD, l, 4 * (Rs * di + di * dout + Rs * dout), 2 * Rs * di * dout);
            put(K_SPMM_FWD, l, 4 * (n + 1) + 8 * nnz_s + 4 * Rs * dout + 4 * n * dout, 0.0,
                p->nnz_s);
            put(K_SPMM_BWD, l,
                4 * (n + 1) + 8 * nnz_in + 8 * n * dout +
                    (pl.dgrad_fused ? 4 * (n * di + di * dout) : 0.0),
                0.0, p->nnz_in);
            if (p->n_bnd > 0)
                put(K_BND_ROWS, l, 8 * nb * dout + 4 * nb);
            if (relu)   // D formed once
                put(K_RELU_MASK, l, 12 * n * dout);
            else if (!pl.dgrad_fused && p->widths[l] % 4)   // the padded copy of dh_out
                put(K_PAD_ROWS, l, 4 * n * (dout + padded_width(p->widths[l])));
            put(K_GEMM_DW, l, 4 * (Rs * di + Rs * dout + di * dout), 2 * Rs * di * dout);
            put(K_REDUCE_DW, l, 4 * (pl.dw_slices + 1) * di * dout);
            if (l > 1 && !pl.dgrad_fused)
                put(K_GEMM_DH, l, 4 * (n * dout + di * dout + n * di), 2 * n * di * dout);
            continue;
        }
        if (pl.forward_fused) {
            // the long-row pass, then the fused pass: the short rows' entries
            // and distinct sources, the long rows read back, AH of the short
            // rows written, W, the output
            const double nl = (double)p->long_rows_f, el = (double)p->long_nnz_f;
            if (p->long_f > 0)
                put(K_SPMM_FWD, l, 4 * 2 * nl + 8 * el + 4 * p->src_long_f * di + 4 * nl * di,
                    0.0, p->long_nnz_f);
            put(K_SPMM_GEMM_FWD, l,
                4 * (n + 1) + 8 * (nnz_s - el) + 4 * p->src_short_f * di + 4 * nl * di +
                    4 * (n - nl) * di + 4 * di * dout + 4 * n * dout,
                2 * n * di * dout, p->nnz_s - p->long_nnz_f);
        } else {
            put(K_SPMM_FWD, l, 4 * (n + 1) + 8 * nnz_s + 4 * Rs * di + 4 * n * di, 0.0,
                p->nnz_s);
            put(K_GEMM_FWD, l, 4 * (n * di + di * dout + n * dout), 2 * n * di * dout);
        }
        if (p->widths[l - 1] % 4)   // the padded copy of h_in
            put(K_PAD_ROWS, l, 4 * n * (di + padded_width(p->widths[l - 1])));
        put(K_GEMM_DW, l, 4 * (n * di + n * dout * (relu && !pl.backward_fused ? 2 : 1) + di * dout),
            2 * n * di * dout);
        if (pl.dw_slices > 1)
            put(K_REDUCE_DW, l, 4 * (pl.dw_slices + 1) * di * dout);
        if (l > 1 && pl.backward_fused) {
            // D formed once; the long rows of P_in^T over D, then the fused
            // pass: the short rows' entries and distinct sources, the long
            // rows read back, W^T, dh_in
            const double nl = (double)p->long_rows_t, el = (double)p->long_nnz_t;
            put(K_RELU_MASK, l, 12 * n * dout);
            put(K_TRANSPOSE_W, l, 8 * di * dout);
            if (p->long_t > 0)
                put(K_SPMM_BWD, l, 4 * 2 * nl + 8 * el + 4 * p->src_long_t * dout + 4 * nl * dout,
                    0.0, p->long_nnz_t);
            put(K_SPMM_GEMM_BWD, l,
                4 * (n + 1) + 8 * (nnz_in - el) + 4 * p->src_short_t * dout + 4 * nl * dout +
                    4 * di * dout + 4 * n * di,
                2 * n * di * dout, p->nnz_in - p->long_nnz_t);
        } else if (l > 1) {
            const double w = pl.dgrad_narrow_first ? dout : di;
            put(K_SPMM_BWD, l, 4 * (n + 1) + 8 * nnz_in + 8 * n * w, 0.0, p->nnz_in);
            put(K_GEMM_DH, l,
                4 * (n * dout * ((pl.dgrad_narrow_first || !relu) ? 1 : 2) + di * dout + n * di),
                2 * n * di * dout);
        }
    }
    const double C = p->widths[L];
    put(K_LOSS, L, 4 * (2 * n * C + n));
    put(K_LOSS_MEAN, L, 4.0 * digest::softmax_xent_blocks(p->n_own, p->widths[L]) + 4);
    const bool rows = p->pull_mode == DIGEST_PULL_ROWS;
    for (int32_t lev = 0; lev < L; ++lev) {
        if (rows)
            put(K_PULL, lev, 8 * nh * p->widths[lev] + 4 * nh);
        // the GCN pull's halo aggregate: P_b's entries, its distinct sources
        // (at most every halo row, from the halo buffer or the store), S
        // written
        if (model == DIGEST_MODEL_GCN && p->n_bnd > 0)
            put(K_HALO_AGG, lev,
                4 * (nb + 1) + 8 * (double)p->nnz_b + 4 * (nh + nb) * p->widths[lev], 0.0,
                p->nnz_b);
    }
    for (int32_t lev = 1; lev < L; ++lev)
        put(K_PUSH, lev, 8 * nb * p->widths[lev] + 8 * nb);
    return DIGEST_OK;
}

}  // extern "C"
