// gfx950 kernels of the DIGEST per-partition GCN layer.
//
//   k_copy_rows    pull (gather halo rows out of the store) and push
//                  (scatter boundary rows into it), Sec. 3.2: one row per
//                  lane group, 16-byte vectors when the width allows.
//   k_spmm         two-source CSR aggregation P_in H_in + P_out H~_out of
//                  Eq. 5 (and P_in^T G of the backward): one wave per work
//                  item of at most a fixed number of entries, lanes split
//                  into groups over entries x feature vectors, entry
//                  indices fetched 64 at a time and broadcast across the
//                  wave, wave-level segmented reduction across groups.
//                  Long rows are split into several items whose partial
//                  sums are added by k_spmm_fixup in a fixed order, so
//                  results are deterministic and no float atomics are used.
//   k_gemm         fp32 MFMA (v_mfma_f32_32x32x2f32) GEMM with optional
//                  transposed operands, ReLU-derivative operand masks, a
//                  ReLU epilogue and split-K over grid.z: the dense
//                  transform AH W, the weight gradient AH^T D and D W^T.
//   k_splitk_reduce  deterministic sum of split-K partial products.
//   k_softmax_xent / k_loss_reduce  the mean cross-entropy loss head.
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace digest {
namespace {

constexpr int kWave = 64;

template <int VEC>
__device__ __forceinline__ void load_vec(const float *p, float (&x)[VEC])
{
    if constexpr (VEC == 4) {
        const float4 v = *reinterpret_cast<const float4 *>(p);
        x[0] = v.x;
        x[1] = v.y;
        x[2] = v.z;
        x[3] = v.w;
    } else if constexpr (VEC == 2) {
        const float2 v = *reinterpret_cast<const float2 *>(p);
        x[0] = v.x;
        x[1] = v.y;
    } else {
        x[0] = *p;
    }
}

template <int VEC>
__device__ __forceinline__ void store_vec(float *p, const float (&x)[VEC])
{
    if constexpr (VEC == 4) {
        *reinterpret_cast<float4 *>(p) = make_float4(x[0], x[1], x[2], x[3]);
    } else if constexpr (VEC == 2) {
        *reinterpret_cast<float2 *>(p) = make_float2(x[0], x[1]);
    } else {
        *p = x[0];
    }
}

__device__ __forceinline__ int readlane_i(int v, int lane)
{
    return __builtin_amdgcn_readlane(v, lane);
}

__device__ __forceinline__ float readlane_f(float v, int lane)
{
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

// ---------------------------------------------------------------------------
// Row copy (pull / push)
// ---------------------------------------------------------------------------

// A wave holds 64/GL groups of GL lanes; each group copies one row, lane j of
// the group moving vectors j, j+GL, ...
template <int VEC, int GL>
__global__ __launch_bounds__(256) void k_copy_rows(const int32_t *__restrict__ sidx,
                                                   const int32_t *__restrict__ didx,
                                                   int32_t n_rows, int32_t d,
                                                   const float *__restrict__ src,
                                                   float *__restrict__ dst)
{
    constexpr int G = kWave / GL;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t r = ((int64_t)blockIdx.x * (blockDim.x / kWave) + (threadIdx.x / kWave)) * G +
                      lane / GL;
    if (r >= n_rows)
        return;
    const int gl = lane % GL;
    const int64_t sr = sidx ? sidx[r] : r;
    const int64_t dr = didx ? didx[r] : r;
    const float *s = src + sr * d;
    float *t = dst + dr * d;
    const int dv = d / VEC;
    for (int c = gl; c < dv; c += GL) {
        float x[VEC];
        load_vec<VEC>(s + c * VEC, x);
        store_vec<VEC>(t + c * VEC, x);
    }
}

// ---------------------------------------------------------------------------
// Sparse aggregation
// ---------------------------------------------------------------------------

template <int VEC, int GL, bool TWO>
__global__ __launch_bounds__(256) void k_spmm(const SpmmItem *__restrict__ items,
                                              int32_t n_items, const int32_t *__restrict__ col,
                                              const float *__restrict__ val,
                                              const float *__restrict__ src0,
                                              const float *__restrict__ src1, int32_t n_src0,
                                              int32_t d, float *__restrict__ out,
                                              float *__restrict__ partial)
{
    constexpr int G = kWave / GL;   // entry groups per wave
    constexpr int U = 4;            // entries in flight per group
    const int lane = threadIdx.x & (kWave - 1);
    const int w = blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
    if (w >= n_items)
        return;   // uniform per wave
    const SpmmItem it = items[w];
    const int g = lane / GL;
    const int gl = lane % GL;
    const int dv = d / VEC;
    float *dst = it.dst >= 0 ? out + (int64_t)it.dst * d
                             : partial + (int64_t)(-(it.dst + 1)) * d;

    for (int c0 = 0; c0 < dv; c0 += GL) {
        const int c = c0 + gl;
        const bool active = c < dv;
        float acc[VEC];
#pragma unroll
        for (int v = 0; v < VEC; ++v)
            acc[v] = 0.f;

        for (int kb = it.kb; kb < it.ke; kb += kWave) {
            const int nb = min(kWave, it.ke - kb);
            int mc = 0;
            float mv = 0.f;
            if (lane < nb) {
                mc = col[kb + lane];
                mv = val[kb + lane];
            }
            const int steps = (nb + G - 1) / G;
            int s = 0;
            for (; s + U <= steps; s += U) {
                int cc[U];
                float aa[U];
                float x[U][VEC];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    if constexpr (G == 1) {
                        cc[u] = readlane_i(mc, s + u);
                        aa[u] = readlane_f(mv, s + u);
                    } else {
                        const int j = (s + u) * G + g;
                        cc[u] = __shfl(mc, j & (kWave - 1));
                        aa[u] = __shfl(mv, j & (kWave - 1));
                        if (j >= nb)
                            aa[u] = 0.f;
                    }
                }
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int j = (s + u) * G + g;
                    if (active && j < nb) {
                        const float *sp = (TWO && cc[u] >= n_src0)
                                              ? src1 + (int64_t)(cc[u] - n_src0) * d
                                              : src0 + (int64_t)cc[u] * d;
                        load_vec<VEC>(sp + c * VEC, x[u]);
                    } else {
#pragma unroll
                        for (int v = 0; v < VEC; ++v)
                            x[u][v] = 0.f;
                    }
                }
#pragma unroll
                for (int u = 0; u < U; ++u)
#pragma unroll
                    for (int v = 0; v < VEC; ++v)
                        acc[v] = fmaf(aa[u], x[u][v], acc[v]);
            }
            for (; s < steps; ++s) {
                int cj;
                float aj;
                const int j = s * G + g;
                if constexpr (G == 1) {
                    cj = readlane_i(mc, s);
                    aj = readlane_f(mv, s);
                } else {
                    cj = __shfl(mc, j & (kWave - 1));
                    aj = __shfl(mv, j & (kWave - 1));
                }
                if (active && j < nb) {
                    const float *sp = (TWO && cj >= n_src0) ? src1 + (int64_t)(cj - n_src0) * d
                                                            : src0 + (int64_t)cj * d;
                    float x[VEC];
                    load_vec<VEC>(sp + c * VEC, x);
#pragma unroll
                    for (int v = 0; v < VEC; ++v)
                        acc[v] = fmaf(aj, x[v], acc[v]);
                }
            }
        }
        if constexpr (G > 1) {
#pragma unroll
            for (int off = GL; off < kWave; off <<= 1)
#pragma unroll
                for (int v = 0; v < VEC; ++v)
                    acc[v] += __shfl_xor(acc[v], off);
        }
        if (g == 0 && active)
            store_vec<VEC>(dst + c * VEC, acc);
    }
}

__global__ __launch_bounds__(256) void k_spmm_fixup(const FixupItem *__restrict__ items,
                                                    int32_t n_items, int32_t d,
                                                    const float *__restrict__ partial,
                                                    float *__restrict__ out)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int w = blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
    if (w >= n_items)
        return;
    const FixupItem it = items[w];
    for (int c = lane; c < d; c += kWave) {
        float acc = 0.f;
        for (int s = 0; s < it.nseg; ++s)
            acc += partial[(int64_t)(it.slot + s) * d + c];
        out[(int64_t)it.row * d + c] = acc;
    }
}

// ---------------------------------------------------------------------------
// fp32 MFMA GEMM
// ---------------------------------------------------------------------------

typedef float floatx16 __attribute__((ext_vector_type(16)));

// 64x64 tile of C per workgroup, 4 waves in a 2x2 arrangement, each wave one
// 32x32 block accumulated with v_mfma_f32_32x32x2f32.  Operand tiles are
// staged through LDS as [k][m] / [k][n] so that the fragment reads (lane l
// takes row l%32 at k = l/32) are contiguous; the next K tile is fetched into
// registers while the current one is multiplied.
template <bool AT, bool BT, bool AMASK, bool BMASK, bool RELU>
__global__ __launch_bounds__(256) void k_gemm(int32_t M, int32_t N, int32_t K, int32_t kchunk,
                                              const float *__restrict__ A, int32_t lda,
                                              const float *__restrict__ Am,
                                              const float *__restrict__ B, int32_t ldb,
                                              const float *__restrict__ Bm,
                                              float *__restrict__ C, int32_t ldc,
                                              int64_t c_split_stride)
{
    constexpr int BM = kGemmBM, BN = kGemmBN, BK = kGemmBK, PAD = 4;
    constexpr int PER = BM * BK / 256;   // elements per thread and operand
    static_assert(BM * BK == BN * BK, "square operand tiles");
    __shared__ float As[BK][BM + PAD];
    __shared__ float Bs[BK][BN + PAD];

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wid = tid / kWave;
    const int m0 = blockIdx.x * BM;
    const int n0 = blockIdx.y * BN;
    const int kb = blockIdx.z * kchunk;
    const int ke = min(K, kb + kchunk);
    const int wm = (wid >> 1) * 32;
    const int wn = (wid & 1) * 32;

    floatx16 acc;
#pragma unroll
    for (int i = 0; i < 16; ++i)
        acc[i] = 0.f;

    float ra[PER], rb[PER];
    auto a_coord = [](int e, int &m, int &k) {
        if (AT) {
            m = e % BM;
            k = e / BM;
        } else {
            k = e % BK;
            m = e / BK;
        }
    };
    auto b_coord = [](int e, int &n, int &k) {
        if (BT) {
            k = e % BK;
            n = e / BK;
        } else {
            n = e % BN;
            k = e / BN;
        }
    };
    auto fetch = [&](int k0) {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int e = tid + i * 256;
            int m, n, k;
            a_coord(e, m, k);
            float v = 0.f;
            if (m0 + m < M && k0 + k < ke) {
                const int64_t idx = AT ? (int64_t)(k0 + k) * lda + (m0 + m)
                                       : (int64_t)(m0 + m) * lda + (k0 + k);
                v = A[idx];
                if (AMASK && !(Am[idx] > 0.f))
                    v = 0.f;
            }
            ra[i] = v;
            b_coord(e, n, k);
            float u = 0.f;
            if (n0 + n < N && k0 + k < ke) {
                const int64_t idx = BT ? (int64_t)(n0 + n) * ldb + (k0 + k)
                                       : (int64_t)(k0 + k) * ldb + (n0 + n);
                u = B[idx];
                if (BMASK && !(Bm[idx] > 0.f))
                    u = 0.f;
            }
            rb[i] = u;
        }
    };
    auto stash = [&]() {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int e = tid + i * 256;
            int m, n, k;
            a_coord(e, m, k);
            As[k][m] = ra[i];
            b_coord(e, n, k);
            Bs[k][n] = rb[i];
        }
    };

    if (kb < ke)
        fetch(kb);
    for (int k0 = kb; k0 < ke; k0 += BK) {
        __syncthreads();
        stash();
        __syncthreads();
        if (k0 + BK < ke)
            fetch(k0 + BK);
#pragma unroll
        for (int kk = 0; kk < BK; kk += 2) {
            const float a = As[kk + (lane >> 5)][wm + (lane & 31)];
            const float b = Bs[kk + (lane >> 5)][wn + (lane & 31)];
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc, 0, 0, 0);
        }
    }

    float *Cz = C + (int64_t)blockIdx.z * c_split_stride;
    const int cn = n0 + wn + (lane & 31);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const int r = m0 + wm + (i >> 2) * 8 + (lane >> 5) * 4 + (i & 3);
        if (r < M && cn < N) {
            float v = acc[i];
            if (RELU)
                v = fmaxf(v, 0.f);
            Cz[(int64_t)r * ldc + cn] = v;
        }
    }
}

__global__ __launch_bounds__(256) void k_splitk_reduce(const float *__restrict__ part,
                                                       int32_t splits, int64_t count,
                                                       float *__restrict__ out)
{
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= count)
        return;
    float acc = 0.f;
    for (int z = 0; z < splits; ++z)
        acc += part[(int64_t)z * count + e];
    out[e] = acc;
}

// ---------------------------------------------------------------------------
// Softmax cross entropy
// ---------------------------------------------------------------------------

constexpr int kLossRowsPerBlock = 4;   // one row per wave

__global__ __launch_bounds__(256) void k_softmax_xent(const float *__restrict__ logits,
                                                      const int32_t *__restrict__ labels,
                                                      int32_t n, int32_t C, float inv_n,
                                                      float *__restrict__ dlogits,
                                                      float *__restrict__ block_loss)
{
    __shared__ float wave_loss[kLossRowsPerBlock];
    const int lane = threadIdx.x & (kWave - 1);
    const int wid = threadIdx.x / kWave;
    const int r = blockIdx.x * kLossRowsPerBlock + wid;
    float row_loss = 0.f;
    if (r < n) {
        const float *z = logits + (int64_t)r * C;
        float *dz = dlogits + (int64_t)r * C;
        const int y = labels[r];
        const bool bad = y < 0 || y >= C;
        float m = -INFINITY;
        for (int c = lane; c < C; c += kWave)
            m = fmaxf(m, z[c]);
        for (int off = kWave / 2; off > 0; off >>= 1)
            m = fmaxf(m, __shfl_xor(m, off));
        float s = 0.f;
        for (int c = lane; c < C; c += kWave)
            s += expf(z[c] - m);
        for (int off = kWave / 2; off > 0; off >>= 1)
            s += __shfl_xor(s, off);
        const float log_s = logf(s);
        for (int c = lane; c < C; c += kWave) {
            const float p = expf(z[c] - m - log_s);
            dz[c] = bad ? 0.f : (p - (c == y ? 1.f : 0.f)) * inv_n;
        }
        const int ys = bad ? 0 : y;   // never index with a bad label
        row_loss = bad ? NAN : -(z[ys] - m - log_s);
    }
    if (lane == 0)
        wave_loss[wid] = row_loss;
    __syncthreads();
    if (threadIdx.x == 0) {
        float t = 0.f;
        for (int i = 0; i < kLossRowsPerBlock; ++i)
            t += wave_loss[i];
        block_loss[blockIdx.x] = t;
    }
}

__global__ __launch_bounds__(256) void k_loss_reduce(const float *__restrict__ block_loss,
                                                     int32_t nb, float inv_n,
                                                     float *__restrict__ loss)
{
    __shared__ float part[256];
    float t = 0.f;
    for (int i = threadIdx.x; i < nb; i += blockDim.x)
        t += block_loss[i];
    part[threadIdx.x] = t;
    __syncthreads();
    for (int off = 128; off > 0; off >>= 1) {
        if ((int)threadIdx.x < off)
            part[threadIdx.x] += part[threadIdx.x + off];
        __syncthreads();
    }
    if (threadIdx.x == 0)
        loss[0] = part[0] * inv_n;
}

// ---------------------------------------------------------------------------
// dispatch helpers
// ---------------------------------------------------------------------------

int pick_vec(int32_t d, const void *a, const void *b)
{
    auto aligned = [](const void *p, uintptr_t n) { return p == nullptr || ((uintptr_t)p % n) == 0; };
    if (d % 4 == 0 && aligned(a, 16) && aligned(b, 16))
        return 4;
    if (d % 2 == 0 && aligned(a, 8) && aligned(b, 8))
        return 2;
    return 1;
}

int pick_group(int32_t dv)
{
    if (dv <= 4)
        return 4;
    if (dv <= 8)
        return 8;
    if (dv <= 16)
        return 16;
    if (dv <= 32)
        return 32;
    return 64;
}

template <int VEC, int GL>
hipError_t copy_rows_t(const int32_t *sidx, const int32_t *didx, int32_t n_rows, int32_t d,
                       const float *src, float *dst, hipStream_t s)
{
    constexpr int rows_per_block = 4 * (kWave / GL);
    const int64_t blocks = ((int64_t)n_rows + rows_per_block - 1) / rows_per_block;
    hipLaunchKernelGGL((k_copy_rows<VEC, GL>), dim3((unsigned)blocks), dim3(256), 0, s, sidx,
                       didx, n_rows, d, src, dst);
    return hipGetLastError();
}

template <int VEC>
hipError_t copy_rows_v(int gl, const int32_t *sidx, const int32_t *didx, int32_t n_rows,
                       int32_t d, const float *src, float *dst, hipStream_t s)
{
    switch (gl) {
    case 4: return copy_rows_t<VEC, 4>(sidx, didx, n_rows, d, src, dst, s);
    case 8: return copy_rows_t<VEC, 8>(sidx, didx, n_rows, d, src, dst, s);
    case 16: return copy_rows_t<VEC, 16>(sidx, didx, n_rows, d, src, dst, s);
    case 32: return copy_rows_t<VEC, 32>(sidx, didx, n_rows, d, src, dst, s);
    default: return copy_rows_t<VEC, 64>(sidx, didx, n_rows, d, src, dst, s);
    }
}

template <int VEC, int GL, bool TWO>
hipError_t spmm_t(const SpmmItem *items, int32_t n_items, const int32_t *col, const float *val,
                  const float *src0, const float *src1, int32_t n_src0, int32_t d, float *out,
                  float *partial, hipStream_t s)
{
    const int64_t blocks = ((int64_t)n_items + 3) / 4;
    hipLaunchKernelGGL((k_spmm<VEC, GL, TWO>), dim3((unsigned)blocks), dim3(256), 0, s, items,
                       n_items, col, val, src0, src1, n_src0, d, out, partial);
    return hipGetLastError();
}

template <int VEC, bool TWO>
hipError_t spmm_g(int gl, const SpmmItem *items, int32_t n_items, const int32_t *col,
                  const float *val, const float *src0, const float *src1, int32_t n_src0,
                  int32_t d, float *out, float *partial, hipStream_t s)
{
    switch (gl) {
    case 4: return spmm_t<VEC, 4, TWO>(items, n_items, col, val, src0, src1, n_src0, d, out, partial, s);
    case 8: return spmm_t<VEC, 8, TWO>(items, n_items, col, val, src0, src1, n_src0, d, out, partial, s);
    case 16: return spmm_t<VEC, 16, TWO>(items, n_items, col, val, src0, src1, n_src0, d, out, partial, s);
    case 32: return spmm_t<VEC, 32, TWO>(items, n_items, col, val, src0, src1, n_src0, d, out, partial, s);
    default: return spmm_t<VEC, 64, TWO>(items, n_items, col, val, src0, src1, n_src0, d, out, partial, s);
    }
}

template <bool TWO>
hipError_t spmm_v(int vec, int gl, const SpmmItem *items, int32_t n_items, const int32_t *col,
                  const float *val, const float *src0, const float *src1, int32_t n_src0,
                  int32_t d, float *out, float *partial, hipStream_t s)
{
    switch (vec) {
    case 4: return spmm_g<4, TWO>(gl, items, n_items, col, val, src0, src1, n_src0, d, out, partial, s);
    case 2: return spmm_g<2, TWO>(gl, items, n_items, col, val, src0, src1, n_src0, d, out, partial, s);
    default: return spmm_g<1, TWO>(gl, items, n_items, col, val, src0, src1, n_src0, d, out, partial, s);
    }
}

template <bool AT, bool BT, bool AMASK, bool BMASK, bool RELU>
hipError_t gemm_t(const GemmArgs &a, hipStream_t s)
{
    const dim3 grid((unsigned)((a.M + kGemmBM - 1) / kGemmBM),
                    (unsigned)((a.N + kGemmBN - 1) / kGemmBN), (unsigned)a.splits);
    const int64_t split_stride = a.splits > 1 ? (int64_t)a.M * a.ldc : 0;
    hipLaunchKernelGGL((k_gemm<AT, BT, AMASK, BMASK, RELU>), grid, dim3(256), 0, s, a.M, a.N,
                       a.K, a.kchunk, a.A, a.lda, a.a_mask, a.B, a.ldb, a.b_mask, a.C, a.ldc,
                       split_stride);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_copy_rows(const int32_t *sidx, const int32_t *didx, int32_t n_rows,
                            int32_t d, const float *src, float *dst, hipStream_t s)
{
    if (n_rows <= 0 || d <= 0)
        return hipSuccess;
    const int vec = pick_vec(d, src, dst);
    const int gl = pick_group(d / vec);
    switch (vec) {
    case 4: return copy_rows_v<4>(gl, sidx, didx, n_rows, d, src, dst, s);
    case 2: return copy_rows_v<2>(gl, sidx, didx, n_rows, d, src, dst, s);
    default: return copy_rows_v<1>(gl, sidx, didx, n_rows, d, src, dst, s);
    }
}

hipError_t launch_spmm(const SpmmItem *items, int32_t n_items, const int32_t *col,
                       const float *val, const float *src0, const float *src1,
                       int32_t n_src0, int32_t d, float *out, float *partial, hipStream_t s)
{
    if (n_items <= 0 || d <= 0)
        return hipSuccess;
    int vec = pick_vec(d, src0, out);
    if (src1 && pick_vec(d, src1, partial) < vec)
        vec = pick_vec(d, src1, partial);
    const int gl = pick_group(d / vec);
    if (src1)
        return spmm_v<true>(vec, gl, items, n_items, col, val, src0, src1, n_src0, d, out,
                            partial, s);
    return spmm_v<false>(vec, gl, items, n_items, col, val, src0, src1, n_src0, d, out, partial,
                         s);
}

hipError_t launch_spmm_fixup(const FixupItem *items, int32_t n_items, int32_t d,
                             const float *partial, float *out, hipStream_t s)
{
    if (n_items <= 0 || d <= 0)
        return hipSuccess;
    const int64_t blocks = ((int64_t)n_items + 3) / 4;
    hipLaunchKernelGGL(k_spmm_fixup, dim3((unsigned)blocks), dim3(256), 0, s, items, n_items, d,
                       partial, out);
    return hipGetLastError();
}

hipError_t launch_gemm(const GemmArgs &a, hipStream_t s)
{
    if (a.M <= 0 || a.N <= 0)
        return hipSuccess;
    const bool am = a.a_mask != nullptr, bm = a.b_mask != nullptr;
    // The instantiations the layer needs:
    //   forward      A.B        (+ReLU epilogue)
    //   dW           A^T.B      (B optionally masked)
    //   D.W^T        A.B^T      (A optionally masked)
    if (!a.a_trans && !a.b_trans && !am && !bm)
        return a.relu ? gemm_t<false, false, false, false, true>(a, s)
                      : gemm_t<false, false, false, false, false>(a, s);
    if (a.a_trans && !a.b_trans && !am && !a.relu)
        return bm ? gemm_t<true, false, false, true, false>(a, s)
                  : gemm_t<true, false, false, false, false>(a, s);
    if (!a.a_trans && a.b_trans && !bm && !a.relu)
        return am ? gemm_t<false, true, true, false, false>(a, s)
                  : gemm_t<false, true, false, false, false>(a, s);
    return hipErrorInvalidValue;
}

hipError_t launch_splitk_reduce(const float *part, int32_t splits, int64_t count, float *out,
                                hipStream_t s)
{
    if (count <= 0)
        return hipSuccess;
    const int64_t blocks = (count + 255) / 256;
    hipLaunchKernelGGL(k_splitk_reduce, dim3((unsigned)blocks), dim3(256), 0, s, part, splits,
                       count, out);
    return hipGetLastError();
}

int32_t softmax_xent_blocks(int32_t n)
{
    return (n + kLossRowsPerBlock - 1) / kLossRowsPerBlock;
}

hipError_t launch_softmax_xent(const float *logits, const int32_t *labels, int32_t n,
                               int32_t C, float *dlogits, float *block_loss, float *loss,
                               hipStream_t s)
{
    const int32_t nb = softmax_xent_blocks(n);
    const float inv_n = n > 0 ? 1.0f / (float)n : 0.f;
    if (nb > 0) {
        hipLaunchKernelGGL(k_softmax_xent, dim3((unsigned)nb), dim3(256), 0, s, logits, labels, n,
                           C, inv_n, dlogits, block_loss);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess)
            return e;
    }
    hipLaunchKernelGGL(k_loss_reduce, dim3(1), dim3(256), 0, s, block_loss, nb, inv_n, loss);
    return hipGetLastError();
}

}  // namespace digest
