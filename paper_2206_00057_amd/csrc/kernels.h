// Internal interface between the host library (digest_host.cpp) and the
// gfx950 kernels (digest_kernels.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstdint>

namespace digest {

// One block of sparse-aggregation work (kSpmmThreads threads = 8 waves).
//   nrows > 0: the short rows [row, row + nrows), one per wave (nrows <= 8);
//   nrows == 0: the single long row `row`, whose entries [kb, ke) the waves
//               split among themselves.
struct SpmmBlock {
    int32_t row, nrows, kb, ke;
};

constexpr int kSpmmThreads = 512;
// Widest side handled by the narrow kernels.
constexpr int kNarrow = 16;
// Widest row the row-per-lane-group aggregation takes.
constexpr int kNarrowWide = 64;
// Rows with more entries than this get a whole block.
constexpr int32_t kSpmmLongRow = 64;
// Rows with more entries than this get a whole block in a sliced pass.
constexpr int32_t kTierLongRow = 1024;

// dst[didx ? didx[r] : r, :] = src[sidx ? sidx[r] : r, :] for r < n_rows, d
// columns of rows with strides lds and ldd (0: d).
hipError_t launch_copy_rows(const int32_t *sidx, const int32_t *didx, int32_t n_rows,
                            int32_t d, const float *src, float *dst, hipStream_t s,
                            int32_t lds = 0, int32_t ldd = 0);
// The same with dst += src; the listed destination rows must be distinct.
hipError_t launch_add_rows(const int32_t *sidx, const int32_t *didx, int32_t n_rows, int32_t d,
                           const float *src, float *dst, hipStream_t s);
// dst += src, then the source rows are set to zero; the listed source rows
// and the listed destination rows must each be distinct.
hipError_t launch_add_clear_rows(const int32_t *sidx, const int32_t *didx, int32_t n_rows,
                                 int32_t d, float *src, float *dst, hipStream_t s);

// Two-source CSR aggregation out[r] = sum_k val[k] * src(col[k]) over the
// rows named by the blocks.  Column c < n_src0 reads row c of src0,
// otherwise row (c - n_src0) of src1.  Every named row is fully written:
// row r < n_out0 to out0[r], row r >= n_out0 to out1[r - n_out0]; relu
// stores max(x, 0) (not with an epilogue).
// Optional epilogue of a narrow aggregation (d <= kNarrow): rows r < rows
// also get out2[r][n] = sum_k out[r][k] w[n][k] for n < n2, w row-major
// [n2][d] (out times w^T), and with out3 the rows r >= rows get the same
// product in out3[r - rows].  Needs spmm_epilogue_ok(d, n2, out2 and out3).
struct SpmmEpilogue {
    const float *w;
    int32_t rows, n2;
    float *out2;
    float *out3 = nullptr;
};
bool spmm_epilogue_ok(int32_t d, int32_t n2, const float *out2);

// Rank-one terms an aggregation can add to its row r before the store:
// out[r][f] += x[r] a[f][0] + (r < ny ? y[2r + 1] : 0) a[f][1], with a
// row-major [d][2] and y [rows][2] (the GAT backward's score terms).
struct SpmmRank1 {
    const float *a = nullptr;
    const float *x = nullptr;
    const float *y = nullptr;
    int32_t ny = 0;
};

// The first n_long blocks are the long-row blocks (nrows == 0), the rest
// short-row blocks.
// acc: add each row's sum to what out already holds.  Rows are gathered d
// floats wide from sources of row stride lds (0: d) and stored out_w (0: d)
// floats wide, out_w <= d, into outputs of row stride out_ld (0: d); a
// gather padded wider than the output lets rows of odd width load whole
// vectors (the padding columns are summed and not stored).
hipError_t launch_spmm(const SpmmBlock *blocks, int32_t n_blocks, int32_t n_long,
                       const int32_t *rowptr, const int32_t *col, const float *val,
                       const float *src0, const float *src1, int32_t n_src0, int32_t d,
                       float *out0, hipStream_t s, const SpmmEpilogue *ep = nullptr,
                       float *out1 = nullptr, int32_t n_out0 = INT32_MAX, bool relu = false,
                       const SpmmRank1 *r1 = nullptr, bool acc = false, int32_t lds = 0,
                       int32_t out_ld = 0, int32_t out_w = 0);

// The same aggregation (one output, no epilogue) as one pass over column
// slices of kSliceFloats floats, the slices dealt to the 8 XCDs so that each
// XCD gathers only its slices of the source rows (a set of rows whose slices
// fit one L2 stays resident there).  Needs rows of an even width with 8-byte
// aligned sources and output (16-byte for float4 gathers).  acc as above.
constexpr int kSliceFloats = 32;
bool spmm_sliced_ok(int32_t d, const float *src0, const float *src1, const float *out0);
// The rows are 0 .. n_rows-1 of the CSR; blocks lists its work blocks (the
// n_long long-row blocks first); nnz >= 1 entries.
hipError_t launch_spmm_sliced(const SpmmBlock *blocks, int32_t n_blocks, int32_t n_long,
                              const int32_t *rowptr, const int32_t *col, const float *val,
                              int64_t nnz, const float *src0, const float *src1, int32_t n_src0,
                              int32_t n_rows, int32_t d, float *out0, bool acc, hipStream_t s);

// An aggregation and a product in one pass: AH = the aggregation of rows
// 0 .. n_rows-1 (as launch_spmm, sources of row stride lds, d floats
// gathered) is stored to ah (row stride ld_ah, columns d .. ld_ah zero; ah
// may be null) and C = act(AH W) (W row-major [d][N], C of row stride ldc)
// is computed from the tiles of AH in LDS.  Rows with more than kFuseLong
// entries must already be in pre (row stride ld_ah; the long-row blocks of
// launch_spmm over the same CSR, run before on the same stream); the others
// are gathered here.  order holds, per tile of kFuseRows rows, a
// permutation of its row offsets: the order in which the tile's waves take
// the rows.  Needs spmm_gemm_ok(d, lds, ld_ah, src0, src1, ah, pre).
constexpr int kFuseRows = 32;
constexpr int kFuseThreads = 256;
constexpr int kFuseWavesPerSimd = 4;   // workgroups per CU x waves per workgroup / 4
constexpr int32_t kFuseLong = kSpmmLongRow;
constexpr int32_t kFuseMaxWidth = 256;
constexpr int32_t kFuseMinWidth = 65;   // narrower rows go to the narrow kernels
bool spmm_gemm_ok(int32_t d, int32_t lds, int32_t ld_ah, const float *src0, const float *src1,
                  const float *ah, const float *pre);
hipError_t launch_spmm_gemm(int32_t n_rows, const int32_t *rowptr, const int32_t *col,
                            const float *val, const uint8_t *order, const float *src0,
                            const float *src1, int32_t n_src0, int32_t lds, int32_t d,
                            float *ah, const float *pre, int32_t ld_ah, const float *W,
                            int32_t N, float *C, int32_t ldc, bool relu, hipStream_t s);

// out[r][c] = h[r][c] > 0 ? g[r][c] : 0 (the ReLU derivative applied), row
// strides ldg, ldh, ldo.
hipError_t launch_relu_mask(int64_t n, int32_t d, const float *g, int32_t ldg, const float *h,
                            int32_t ldh, float *out, int32_t ldo, hipStream_t s);
// dst (cols x rows) = src^T for a row-major rows x cols src.
hipError_t launch_transpose(int32_t rows, int32_t cols, const float *src, float *dst,
                            hipStream_t s);

// C = op(A) op(B) in fp32 on MFMA, K-range split into `splits`
// slices (each its own grid part) when splits > 1.
//   op(A)(m,k) = a_trans ? A[k*lda + m] : A[m*lda + k]      (M x K)
//   op(B)(k,n) = b_trans ? B[n*ldb + k] : B[k*ldb + n]      (K x N)
//   a_mask / b_mask (optional, same layout as A / B): operand element is
//   zeroed unless the mask element is > 0 (the ReLU derivative).
//   splits > 1: split z writes C + z*M*ldc (a [splits, M, ldc] scratch).
//   relu: epilogue max(x, 0).
struct GemmArgs {
    int32_t M, N, K;
    const float *A;
    int32_t lda;
    bool a_trans;
    const float *a_mask;
    const float *B;
    int32_t ldb;
    bool b_trans;
    const float *b_mask;
    float *C;
    int32_t ldc;
    bool relu;
    int32_t splits;
    int32_t kchunk;
    int32_t tile = 0;   // workgroup tile of C: 0 = 64x64, 1 = 64x128, 2 = 128x64, 3 = 128x128
};

hipError_t launch_gemm(const GemmArgs &a, hipStream_t s);

// out[e] = sum_{z < splits} part[z*count + e], in z order.
hipError_t launch_splitk_reduce(const float *part, int32_t splits, int64_t count, float *out,
                                hipStream_t s);

// Dense products with one narrow side, bound by streaming the wide operand.

// C[r][n] = sum_k A(r)[k] B[k][n], n < N <= kNarrowN, B row-major [K][N];
// A(r) is row r of A0 (leading dim lda) for r < m0, else row r - m0 of A1
// (leading dim lda1, 0: lda);
// relu: epilogue max(x, 0).  B is held in LDS: needs
// narrow_n_lds(K, N) <= kNarrowNLds.
constexpr int kNarrowN = 64;
constexpr size_t kNarrowNLds = 64 * 1024;
size_t narrow_n_lds(int32_t K, int32_t N);
// Row stride (floats) of B^T in LDS: K rounded up to 16, plus 4.
constexpr int32_t narrow_n_stride(int32_t K) { return (K + 15) / 16 * 16 + 4; }
hipError_t launch_narrow_n(int32_t M, int32_t m0, int32_t K, int32_t N, const float *A0,
                           const float *A1, int32_t lda, const float *B, float *C, int32_t ldc,
                           bool relu, hipStream_t s, int32_t lda1 = 0);

// C[r][n] = sum_{k < K} A[r][k] W[n][k] with K <= kNarrow, W row-major [N][K].
hipError_t launch_narrow_k(int32_t M, int32_t N, int32_t K, const float *A, int32_t lda,
                           const float *W, float *C, int32_t ldc, hipStream_t s);

// The same product for kNarrow < K <= kTimesWtK on MFMA with W held in LDS:
// needs times_wt_lds(K, N) <= kNarrowNLds.
constexpr int kTimesWtK = 64;
size_t times_wt_lds(int32_t K, int32_t N);
hipError_t launch_times_wt(int32_t M, int32_t N, int32_t K, const float *A, int32_t lda,
                           const float *W, float *C, int32_t ldc, hipStream_t s);

// part[z][f][n] = sum over rows r in [z*chunk, (z+1)*chunk) of H(r)[f] G[r][n]
// (f < F, n < N <= kNarrow; H(r) from H0 (leading dim ldh) for r < m0 else
// H1 (leading dim ldh1, 0: ldh); G row-major with leading dim ldg).  Sum the
// slices with launch_splitk_reduce.
hipError_t launch_dw_narrow(int32_t R, int32_t m0, int32_t F, int32_t N, const float *H0,
                            const float *H1, int32_t ldh, const float *G, int32_t ldg,
                            int32_t chunk, int32_t splits, float *part, hipStream_t s,
                            int32_t ldh1 = 0);

// Row-wise softmax cross entropy (C >= 1): dlogits and the per-block loss
// sums (softmax_xent_blocks(n, C) floats); launch_loss_mean then writes
// their mean over the n rows.
int32_t softmax_xent_blocks(int32_t n, int32_t C);
int32_t softmax_xent_rows_per_block(int32_t C);
hipError_t launch_softmax_xent(const float *logits, const int32_t *labels, int32_t n,
                               int32_t C, float *dlogits, float *block_loss, hipStream_t s);
hipError_t launch_loss_mean(const float *block_loss, int32_t n, int32_t C, float *loss,
                            hipStream_t s);

// w[e] -= lr * (1/n) * sum_{m < n} g[m][e], the sum in m order, for
// 1 <= n <= kMaxAverage device arrays of count floats.
constexpr int kMaxAverage = 64;
struct GradList {
    const float *g[kMaxAverage];
};
hipError_t launch_sgd_average(float *w, const GradList &g, int32_t n, int64_t count, float lr,
                              hipStream_t s);

// The library's fixed device scratch array (kStaticScratchFloats floats, one
// copy per GPU, 256-byte aligned): its address on the current device,
// looked up on the first call per device.
constexpr size_t kStaticScratchFloats = 256 * 1024;
hipError_t static_scratch(float **ptr);

// p[0 .. count) = 0.
hipError_t launch_fill_zero(float *p, int64_t count, hipStream_t s);

// GAT layer (attention aggregation over stale halo rows).  s is [rows][2]
// (source score, target score); alpha, dpre are in CSR entry order.
constexpr int kGatMaxWidth = 512;
// alpha[k] = softmax over row i's entries of LeakyReLU(s[i][1] + s[col k][0]).
hipError_t launch_gat_softmax(int32_t n_rows, const int32_t *rowptr, const int32_t *col,
                              const float *s, float slope, float *alpha, hipStream_t st);
// dO = dh_out (masked by h_out > 0 with relu), dpre[k] the gradient of the
// k-th pre-activation score, g2[i][1] = sum of row i's dpre; d <= kGatMaxWidth.
hipError_t launch_gat_edge_grad(const SpmmBlock *blocks, int32_t n_blocks, int32_t d,
                                const int32_t *rowptr, const int32_t *col, const float *alpha,
                                const float *s, const float *z, const float *h_out,
                                const float *dh_out, bool relu, float slope, float *dO,
                                float *dpre, float *g2, hipStream_t st);
// a_t[k] = a[perm[k]], b_t[k] = b[perm[k]] for k < n.
hipError_t launch_gather_perm2(int64_t n, const int32_t *perm, const float *a, const float *b,
                               float *a_t, float *b_t, hipStream_t st);
// The score-gradient operand of datt: g2[v][0] = ds_src[v] for v < R and
// g2[v][1] = 0 for n_own <= v < R (the owned rows keep their row sums).
hipError_t launch_gat_score_cols(int64_t R, int32_t n_own, const float *ds_src, float *g2,
                                 hipStream_t st);

// GEMM K step; the smallest workgroup tile of C is kGemmBM x kGemmBN.
constexpr int kGemmBM = 64;
constexpr int kGemmBN = 64;
constexpr int kGemmBK = 32;

}  // namespace digest
