// gfx950 kernels of the DIGEST per-partition GCN layer.
//
//   k_copy_rows    pull (gather halo rows out of the store) and push
//                  (scatter boundary rows into it), Sec. 3.2: one row per
//                  lane group, 16-byte vectors when the width allows.
//   k_spmm         two-source CSR aggregation P_in H_in + P_out H~_out of
//                  Eq. 5 (and P_in^T G of the backward).  Short rows take
//                  one wave each; a long row takes a whole 8-wave block
//                  whose waves split its entries and add their sums in LDS
//                  in a fixed order.  Inside a wave, lanes split into groups
//                  over entries x feature vectors, entry indices are fetched
//                  64 at a time and broadcast, many gathers are kept in
//                  flight, and groups are combined by a butterfly.  Results
//                  are deterministic; no float atomics, no global fences.
//   k_gemm         fp32 MFMA (v_mfma_f32_32x32x2f32) GEMM with optional
//                  transposed operands, ReLU-derivative operand masks, a
//                  ReLU epilogue and split-K; tiles are dealt to the XCDs in
//                  contiguous runs (shared operand strips share an L2): the dense
//                  transform AH W, the weight gradient AH^T D and D W^T.
//   k_splitk_reduce  deterministic sum of split-K partial products.
//   k_narrow_n / k_narrow_k / k_times_wt / k_dw_narrow  products with one
//                  narrow side (the transform-first last layer).
//   k_softmax_xent / k_loss_reduce  the mean cross-entropy loss head.
//   k_sgd_average  Algorithm 1's global update: the average of the M
//                  locally updated models, W - lr * mean of the gradients.
//   k_gat_*        the GAT layer over stale halo rows (Eq. 4 with an
//                  attention aggregation): edge softmax, the per-edge
//                  gradient, and the helpers of its backward.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "kernels.h"

// The library's fixed scratch array for callers that cannot allocate
// (digest_softmax_xent_static): every GPU the library runs on holds its own
// copy until the process ends.  On the host this name is only a stand-in
// for the symbol, not a device address; host code uses the address that
// digest::static_scratch() looks up.
static __device__ __align__(256) float scratch[digest::kStaticScratchFloats];

namespace digest {
namespace {

constexpr int kWave = 64;

// The dispatcher deals workgroups to the 8 XCDs (each with its own L2) in
// turn by linear id.  xcd_contiguous maps the linear id p of an n-workgroup
// grid to a logical id such that every XCD receives one contiguous run of
// logical ids, in increasing order; it is a bijection of [0, n).  Kernels
// order their logical work so that neighbours share operand data.
constexpr uint32_t kXcds = 8;

__device__ __forceinline__ uint32_t xcd_contiguous(uint32_t p, uint32_t n)
{
    const uint32_t q = n / kXcds, rem = n % kXcds;
    const uint32_t x = p % kXcds, slot = p / kXcds;
    return (x < rem ? x * (q + 1) : rem * (q + 1) + (x - rem) * q) + slot;
}

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

// Fill an LDS array of `count` floats, value(i) for i < count, with the
// block's threads: loads are issued in batches of 16 per thread before their
// stores, so staging costs one round trip per batch rather than per element.
template <class F>
__device__ __forceinline__ void stage_lds(float *dst, int count, F value)
{
    constexpr int BATCH = 16;
    const int stride = blockDim.x;
    for (int base = threadIdx.x; base < count; base += BATCH * stride) {
        float v[BATCH];
#pragma unroll
        for (int b = 0; b < BATCH; ++b) {
            const int i = base + b * stride;
            v[b] = i < count ? value(i) : 0.f;
        }
#pragma unroll
        for (int b = 0; b < BATCH; ++b) {
            const int i = base + b * stride;
            if (i < count)
                dst[i] = v[b];
        }
    }
}

// ---------------------------------------------------------------------------
// Row copy (pull / push)
// ---------------------------------------------------------------------------

// A wave holds 64/GL groups of GL lanes; each group moves one row, lane j of
// the group handling vectors j, j+GL, ...  MODE: kCopy dst = src, kAdd
// dst += src, kAddClear dst += src then src = 0 (each row of src and of
// dst is touched by one group only, so no two lanes race).
enum RowMode { kCopy = 0, kAdd = 1, kAddClear = 2 };

template <int VEC, int GL, int MODE>
__global__ __launch_bounds__(256) void k_copy_rows(const int32_t *__restrict__ sidx,
                                                   const int32_t *__restrict__ didx,
                                                   int32_t n_rows, int32_t d,
                                                   float *__restrict__ src, int32_t lds,
                                                   float *__restrict__ dst, int32_t ldd)
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
    float *sp = src + sr * lds;
    float *t = dst + dr * ldd;
    const int dv = d / VEC;
    for (int c = gl; c < dv; c += GL) {
        float x[VEC];
        load_vec<VEC>(sp + c * VEC, x);
        if constexpr (MODE != kCopy) {
            float y[VEC];
            load_vec<VEC>(t + c * VEC, y);
#pragma unroll
            for (int v = 0; v < VEC; ++v)
                x[v] += y[v];
        }
        store_vec<VEC>(t + c * VEC, x);
        if constexpr (MODE == kAddClear) {
            float z[VEC];
#pragma unroll
            for (int v = 0; v < VEC; ++v)
                z[v] = 0.f;
            store_vec<VEC>(sp + c * VEC, z);
        }
    }
}

// ---------------------------------------------------------------------------
// Sparse aggregation
// ---------------------------------------------------------------------------

constexpr int kSpmmWaves = kSpmmThreads / kWave;

// Entries in flight per lane group: a register budget of ~48 gathered floats
// when the whole wave shares one entry (scalar addresses), ~32 when every
// group has its own (per-lane 64-bit addresses).
constexpr int spmm_inflight(int groups, int nch, int vec)
{
    const int budget = groups == 1 ? 48 : 32;
    const int cap = groups == 1 ? 12 : 8;
    const int u = budget / (nch * vec);
    return u < 2 ? 2 : (u > cap ? cap : u);
}

// One block of kSpmmWaves waves.  A short-row block gives wave w the row
// b.row + w (w < b.nrows); a long-row block splits the entries [b.kb, b.ke)
// of row b.row into kSpmmWaves contiguous parts, one per wave, and adds the
// per-wave sums in LDS in wave order.  Inside a wave the lanes form 64/GL
// groups: group g takes the entries j = g, g + G, ... of its range, lane gl
// of a group accumulates the feature vectors gl, gl + GL, ... (NCH of them
// per column pass).  Entry ids and weights are fetched 64 at a time (one per
// lane) and broadcast; up to U entries per group are in flight.
// Destination of an aggregation's rows: row r < n0 is out0 + r ld, row
// r >= n0 is out1 + (r - n0) ld.  n0 = INT32_MAX makes one contiguous output;
// a split lets one launch over P_m^T write the owned rows and the halo rows
// to buffers of their own.  With acc the row's sum is added to what the
// output already holds (a later pass over more entries of the same rows).
// Only the first w columns are stored (the gathered rows may be padded
// wider); vst says whether a vector of the gather's width may be stored as
// one (the output's rows are aligned for it), else the columns go one by one.
struct SpmmOut {
    float *out0;
    float *out1;
    int32_t n0;
    bool relu;      // store max(x, 0)
    SpmmRank1 r1;   // rank-one terms added first when r1.a is set
    int32_t ld;     // row stride of out0 and out1 (floats)
    bool acc;       // out = out + sum
    int32_t w;      // stored columns
    bool vst;       // vector stores allowed

    __device__ __forceinline__ float *row(int32_t r) const
    {
        return r < n0 ? out0 + (int64_t)r * ld : out1 + (int64_t)(r - n0) * ld;
    }
    // the stored value of feature f of row r whose sum is v
    __device__ __forceinline__ float fin(int32_t r, int32_t f, float v) const
    {
        if (acc)
            v += row(r)[f];
        if (r1.a) {
            const float xa = r1.x[r];
            const float yb = r < r1.ny ? r1.y[2 * (int64_t)r + 1] : 0.f;
            v += xa * r1.a[2 * f] + yb * r1.a[2 * f + 1];
        }
        return relu ? fmaxf(v, 0.f) : v;
    }
    template <int VEC>
    __device__ __forceinline__ void put(int32_t r, int32_t off, float (&v)[VEC]) const
    {
        float *p = row(r) + off;
        const bool whole = vst && off + VEC <= w;
        if (acc) {
            float prev[VEC];
            if (whole) {
                load_vec<VEC>(p, prev);
            } else {
#pragma unroll
                for (int i = 0; i < VEC; ++i)
                    prev[i] = off + i < w ? p[i] : 0.f;
            }
#pragma unroll
            for (int i = 0; i < VEC; ++i)
                v[i] += prev[i];
        }
        if (relu || r1.a) {
#pragma unroll
            for (int i = 0; i < VEC; ++i) {
                float t = v[i];
                if (r1.a) {
                    const float xa = r1.x[r];
                    const float yb = r < r1.ny ? r1.y[2 * (int64_t)r + 1] : 0.f;
                    t += xa * r1.a[2 * (off + i)] + yb * r1.a[2 * (off + i) + 1];
                }
                v[i] = relu ? fmaxf(t, 0.f) : t;
            }
        }
        if (whole) {
            store_vec<VEC>(p, v);
        } else {
#pragma unroll
            for (int i = 0; i < VEC; ++i)
                if (off + i < w)
                    p[i] = v[i];
        }
    }
};

template <int VEC, int GL, int NCH, bool TWO>
__device__ __forceinline__ void spmm_block(const SpmmBlock b, const int32_t *__restrict__ rowptr,
                                           const int32_t *__restrict__ col,
                                           const float *__restrict__ val,
                                           const float *__restrict__ src0,
                                           const float *__restrict__ src1, int32_t n_src0,
                                           int32_t d, int32_t lds, const SpmmOut out,
                                           float (*red)[NCH * GL * VEC])
{
    constexpr int G = kWave / GL;
    constexpr int U = spmm_inflight(G, NCH, VEC);
    constexpr int SPAN = NCH * GL;   // feature vectors per column pass

    const int wave = threadIdx.x / kWave;
    const int lane = threadIdx.x % kWave;
    const int g = lane / GL;
    const int gl = lane % GL;
    const int dv = d / VEC;
    const bool long_row = b.nrows == 0;   // uniform over the block
    int row, kb, ke;
    if (long_row) {
        row = b.row;
        const int per = (b.ke - b.kb + kSpmmWaves - 1) / kSpmmWaves;
        kb = min(b.ke, b.kb + wave * per);
        ke = min(b.ke, kb + per);
    } else {
        row = b.row + wave;
        if (wave < b.nrows) {
            kb = rowptr[row];
            ke = rowptr[row + 1];
        } else {
            kb = ke = 0;
        }
    }

    for (int c0 = 0; c0 < dv; c0 += SPAN) {
        float acc[NCH][VEC];
#pragma unroll
        for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
            for (int v = 0; v < VEC; ++v)
                acc[ch][v] = 0.f;

        for (int k0 = kb; k0 < ke; k0 += kWave) {
            const int nb = min(kWave, ke - k0);
            int mc = 0;
            float mv = 0.f;
            if (lane < nb) {
                mc = col[k0 + lane];
                mv = val[k0 + lane];
            }
            const int steps = (nb + G - 1) / G;
            for (int s = 0; s < steps; s += U) {
                int cc[U];
                float aa[U];
                bool ok[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int j = (s + u) * G + g;
                    if constexpr (G == 1) {
                        cc[u] = readlane_i(mc, (s + u) & (kWave - 1));
                        aa[u] = readlane_f(mv, (s + u) & (kWave - 1));
                    } else {
                        cc[u] = __shfl(mc, j & (kWave - 1));
                        aa[u] = __shfl(mv, j & (kWave - 1));
                    }
                    ok[u] = j < nb;
                }
                float x[U][NCH][VEC];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const float *sp = (TWO && cc[u] >= n_src0)
                                          ? src1 + (int64_t)(cc[u] - n_src0) * lds
                                          : src0 + (int64_t)cc[u] * lds;
#pragma unroll
                    for (int ch = 0; ch < NCH; ++ch) {
                        const int c = c0 + ch * GL + gl;
                        if (ok[u] && c < dv) {
                            load_vec<VEC>(sp + c * VEC, x[u][ch]);
                        } else {
#pragma unroll
                            for (int v = 0; v < VEC; ++v)
                                x[u][ch][v] = 0.f;
                        }
                    }
                }
#pragma unroll
                for (int u = 0; u < U; ++u)
#pragma unroll
                    for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
                        for (int v = 0; v < VEC; ++v)
                            acc[ch][v] = fmaf(aa[u], x[u][ch][v], acc[ch][v]);
            }
        }
        if constexpr (G > 1) {
#pragma unroll
            for (int off = GL; off < kWave; off <<= 1)
#pragma unroll
                for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
                    for (int v = 0; v < VEC; ++v)
                        acc[ch][v] += __shfl_xor(acc[ch][v], off);
        }
        if (!long_row) {
            if (wave < b.nrows && g == 0) {
#pragma unroll
                for (int ch = 0; ch < NCH; ++ch) {
                    const int c = c0 + ch * GL + gl;
                    if (c < dv)
                        out.put<VEC>(row, c * VEC, acc[ch]);
                }
            }
        } else {
            if (g == 0) {
#pragma unroll
                for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
                    for (int v = 0; v < VEC; ++v)
                        red[wave][(ch * GL + gl) * VEC + v] = acc[ch][v];
            }
            __syncthreads();
            for (int t = threadIdx.x; t < SPAN * VEC; t += kSpmmThreads) {
                const int c = c0 + t / VEC;
                if (c < dv && c * VEC + t % VEC < out.w) {
                    float sum = 0.f;
#pragma unroll
                    for (int w = 0; w < kSpmmWaves; ++w)
                        sum += red[w][t];
                    out.row(row)[(int64_t)c * VEC + t % VEC] = out.fin(row, c * VEC + t % VEC, sum);
                }
            }
            __syncthreads();
        }
    }
}

// out2[4 n4 .. 4 n4 + 3] = sum_{k < d} gk[k] w[k][4 n4 ..], w in LDS as [k][n2].
__device__ __forceinline__ void narrow_ep_store(const float (&gk)[kNarrow], int d,
                                                const float *ws, int n2, int n4, float *out2)
{
    float o[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = 0; k < kNarrow; ++k) {
        if (k < d) {
            const float4 w = *reinterpret_cast<const float4 *>(ws + k * n2 + 4 * n4);
            o[0] = fmaf(gk[k], w.x, o[0]);
            o[1] = fmaf(gk[k], w.y, o[1]);
            o[2] = fmaf(gk[k], w.z, o[2]);
            o[3] = fmaf(gk[k], w.w, o[3]);
        }
    }
    *reinterpret_cast<float4 *>(out2 + 4 * n4) = make_float4(o[0], o[1], o[2], o[3]);
}

template <int VEC, int GL, int NCH, bool TWO>
__global__ __launch_bounds__(kSpmmThreads) void k_spmm(const SpmmBlock *__restrict__ blocks,
                                                       const int32_t *__restrict__ rowptr,
                                                       const int32_t *__restrict__ col,
                                                       const float *__restrict__ val,
                                                       const float *__restrict__ src0,
                                                       const float *__restrict__ src1,
                                                       int32_t n_src0, int32_t d,
                                                       int32_t lds, SpmmOut out)
{
    __shared__ float red[kSpmmWaves][NCH * GL * VEC];
    spmm_block<VEC, GL, NCH, TWO>(blocks[blockIdx.x], rowptr, col, val, src0, src1, n_src0, d,
                                  lds, out, red);
}

// Epilogue destination of row r: out2 for r < rows, out3 (if any) after.
__device__ __forceinline__ float *ep_row(const SpmmEpilogue &ep, int32_t r)
{
    if (r < ep.rows)
        return ep.out2 + (int64_t)r * ep.n2;
    return ep.out3 ? ep.out3 + (int64_t)(r - ep.rows) * ep.n2 : nullptr;
}

// Aggregation for rows of at most kNarrowWide floats, where one row per
// wave would leave most lanes idle: the n_long long-row blocks (first in
// the list) run as in k_spmm, one per workgroup; every wave of the remaining
// workgroups takes one short-row block (up to kSpmmWaves consecutive rows)
// and gives each of its lane groups a row of its own, GL lanes holding NCH
// vectors of VEC floats each (GL * NCH * VEC >= the row width).  A group
// fetches NB * GL entry ids and weights at a time (NB per lane), broadcasts
// them inside the group and keeps all of their gathers in flight, so a row
// of up to that many entries costs one dependent round trip; the entries
// of a row are added in CSR order, so results do not depend on the launch
// shape.  NB is chosen so that a lane holds at most 64 gathered floats.
// With EP (rows of at most kNarrow floats, NCH = 1), rows r < ep.rows also
// get out2[r][n] = sum_k out[r][k] w[n][k] (w row-major [n2][d], staged in
// LDS as [k][n2]); a lane group shares its row by shuffles and writes it out
// in float4 pieces.
// With SL the rows are d floats wide (sources and output, stride d) and
// the launch covers them in column slices of kSliceFloats: workgroup w
// takes slice (w mod 8) + 8 ((w / 8) mod q) of work block w / (8 q), q the
// slices per XCD, so every workgroup of one slice runs on one XCD (the
// dispatcher deals workgroups to the 8 XCDs in turn) and the slice of the
// rows a pass gathers stays in that XCD's L2.
template <int VEC, int GL, int NCH, int NB, bool TWO, bool EP, bool SL = false>
__global__ __launch_bounds__(kSpmmThreads) void k_spmm_narrow(
    const SpmmBlock *__restrict__ blocks, int32_t n_long, int32_t n_blocks,
    const int32_t *__restrict__ rowptr, const int32_t *__restrict__ col,
    const float *__restrict__ val, const float *__restrict__ src0, const float *__restrict__ src1,
    int32_t n_src0, int32_t d, int32_t lds, SpmmOut out, SpmmEpilogue ep)
{
    static_assert(!EP || (NCH == 1 && GL * VEC <= kNarrow), "epilogue rows are kNarrow wide");
    static_assert(!SL || !EP, "no epilogue on a sliced pass");
    __shared__ float red[kSpmmWaves][NCH * GL * VEC];
    int32_t wb = (int32_t)blockIdx.x;   // work block
    if constexpr (SL) {
        const int32_t q = (d + kXcds * kSliceFloats - 1) / (kXcds * kSliceFloats);
        const int32_t off = (wb % kXcds + kXcds * ((wb / kXcds) % q)) * kSliceFloats;
        if (off >= d)
            return;   // the whole workgroup: no slice here
        wb /= kXcds * q;
        src0 += off;
        if (src1)
            src1 += off;
        out.out0 += off;
        if (out.out1)
            out.out1 += off;
        d = min(kSliceFloats, d - off);
        out.w = d;
    }
    extern __shared__ float ws[];   // EP: w as [k][n2]
    if constexpr (EP) {
        stage_lds(ws, d * ep.n2, [&](int i) {
            const int k = i / ep.n2, n = i % ep.n2;
            return ep.w[(int64_t)n * d + k];
        });
        __syncthreads();
    }
    if (wb < n_long) {   // uniform over the block
        const SpmmBlock b = blocks[wb];
        spmm_block<VEC, GL, NCH, TWO>(b, rowptr, col, val, src0, src1, n_src0, d, lds, out, red);
        if constexpr (EP) {
            // the row was written by this block before spmm_block's last barrier
            if (float *o2 = ep_row(ep, b.row)) {
                const float *orow = out.row(b.row);
                float gk[kNarrow];
#pragma unroll
                for (int k = 0; k < kNarrow; ++k)
                    gk[k] = k < d ? orow[k] : 0.f;
                for (int n4 = threadIdx.x; n4 < ep.n2 / 4; n4 += kSpmmThreads)
                    narrow_ep_store(gk, d, ws, ep.n2, n4, o2);
            }
        }
        return;
    }
    constexpr int G = kWave / GL;
    const int wave = threadIdx.x / kWave;
    const int lane = threadIdx.x % kWave;
    const int g = lane / GL;
    const int gl = lane % GL;
    const int bi = n_long + (wb - n_long) * kSpmmWaves + wave;
    if (bi >= n_blocks)
        return;
    const SpmmBlock b = blocks[bi];
    const int dv = d / VEC;
    for (int i = g; i < b.nrows; i += G) {
        const int row = b.row + i;
        const int kb = rowptr[row], ke = rowptr[row + 1];
        float acc[NCH][VEC];
#pragma unroll
        for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
            for (int v = 0; v < VEC; ++v)
                acc[ch][v] = 0.f;
        constexpr int E = NB * GL;   // entries per batch
        for (int k0 = kb; k0 < ke; k0 += E) {
            // Every load is unconditional so that all of a batch's gathers
            // are in flight together: an entry past the row rereads the
            // row's last entry with weight 0 (it adds nothing, and no other
            // row's data can enter), a vector past the width rereads the
            // row's first vector and is not stored.
            int mc[NB];
            float mv[NB];
#pragma unroll
            for (int j = 0; j < NB; ++j) {   // entry k0 + j*GL + gl
                const int k = k0 + j * GL + gl;
                const int kc = k < ke ? k : ke - 1;
                mc[j] = col[kc];
                mv[j] = val[kc] * (k < ke ? 1.f : 0.f);
            }
            int cc[NB][GL];
            float aa[NB][GL];
#pragma unroll
            for (int j = 0; j < NB; ++j)
#pragma unroll
                for (int u = 0; u < GL; ++u) {
                    cc[j][u] = __shfl(mc[j], g * GL + u);
                    aa[j][u] = __shfl(mv[j], g * GL + u);
                }
            float x[NB][GL][NCH][VEC];
#pragma unroll
            for (int j = 0; j < NB; ++j)
#pragma unroll
                for (int u = 0; u < GL; ++u) {
                    const int c = cc[j][u];
                    const float *sp = (TWO && c >= n_src0) ? src1 + (int64_t)(c - n_src0) * lds
                                                           : src0 + (int64_t)c * lds;
#pragma unroll
                    for (int ch = 0; ch < NCH; ++ch) {
                        const int cv = ch * GL + gl;
                        load_vec<VEC>(sp + (cv < dv ? cv : 0) * VEC, x[j][u][ch]);
                    }
                }
#pragma unroll
            for (int j = 0; j < NB; ++j)
#pragma unroll
                for (int u = 0; u < GL; ++u)
#pragma unroll
                    for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
                        for (int v = 0; v < VEC; ++v)
                            acc[ch][v] = fmaf(aa[j][u], x[j][u][ch][v], acc[ch][v]);
        }
#pragma unroll
        for (int ch = 0; ch < NCH; ++ch) {
            const int cv = ch * GL + gl;
            if (cv < dv)
                out.put<VEC>(row, cv * VEC, acc[ch]);
        }
        if constexpr (EP) {
            if (float *o2 = ep_row(ep, row)) {
                float gk[kNarrow];
#pragma unroll
                for (int k = 0; k < kNarrow; ++k) {
                    const float v = __shfl(acc[0][k % VEC], (g * GL + k / VEC) & (kWave - 1));
                    gk[k] = k < d ? v : 0.f;
                }
                for (int n4 = gl; n4 < ep.n2 / 4; n4 += GL)
                    narrow_ep_store(gk, d, ws, ep.n2, n4, o2);
            }
        }
    }
}

// Sliced pass of a tiered aggregation over its rows of at most
// kTierLongRow entries (longer rows are left to the long-row blocks of
// k_spmm_narrow).  Workgroups map to XCDs and column slices as in
// k_spmm_narrow's sliced mode; each wave then walks a strip of rows_per_wave
// consecutive rows with one lane group (GL lanes, one vector each) per row,
// G rows at a time.  A group takes its rows' entries in batches of NB * GL,
// and the loop is software-pipelined so that a batch's gathers are in
// flight together with the index loads of the group's next batch and the
// row pointers of its row after next: a step costs one gather round trip
// (from the L2 that holds this XCD's slices of the tier's rows), not the
// three dependent round trips of index, pointer and gather.  Every load
// is unconditional (padding entries reread entry 0 with weight 0) so that
// the wait counts stay static.  A row's entries are added in CSR order.
constexpr int kTierNB = 2;

template <int VEC, bool TWO>
__global__ __launch_bounds__(256) void k_spmm_tier(
    const int32_t *__restrict__ rowptr, const int32_t *__restrict__ col,
    const float *__restrict__ val, const float *__restrict__ src0,
    const float *__restrict__ src1, int32_t n_src0, int32_t n_rows, int32_t d,
    int32_t rows_per_wave, SpmmOut out)
{
    constexpr int GL = kSliceFloats / VEC;   // lanes per row slice
    constexpr int G = kWave / GL;            // rows in flight per wave
    constexpr int E = kTierNB * GL;          // entries per group batch
    int32_t wb = (int32_t)blockIdx.x;
    const int32_t lds = d;
    {
        const int32_t q = (d + kXcds * kSliceFloats - 1) / (kXcds * kSliceFloats);
        const int32_t off = (wb % kXcds + kXcds * ((wb / kXcds) % q)) * kSliceFloats;
        if (off >= d)
            return;
        wb /= kXcds * q;
        src0 += off;
        if (src1)
            src1 += off;
        out.out0 += off;
        d = min(kSliceFloats, d - off);
        out.w = d;
    }
    const int lane = threadIdx.x & (kWave - 1);
    const int g = lane / GL, gl = lane % GL;
    const int64_t wave = (int64_t)wb * (256 / kWave) + threadIdx.x / kWave;
    const int64_t rb = wave * rows_per_wave;
    if (rb >= n_rows)
        return;   // the whole wave (no barriers in this kernel)
    const int32_t r_begin = (int32_t)rb;
    const int32_t r_end = (int32_t)min<int64_t>(n_rows, rb + rows_per_wave);
    const int dv = d / VEC;
    const int cv = gl < dv ? gl : 0;   // lanes past the slice reread vector 0, store nothing

    // entry range of row rr; rows past the strip and long rows (left to the
    // long-row blocks, `lng` set) read as empty.  The pointer loads are
    // clamped into the strip, so they are unconditional.
    auto bounds = [&](int32_t rr, int32_t &kb, int32_t &ke, bool &lng) {
        const int32_t rc = rr < r_end ? rr : r_end - 1;
        kb = rowptr[rc];
        ke = rowptr[rc + 1];
        lng = ke - kb > kTierLongRow;
        if (rr >= r_end || lng)
            ke = kb;
    };
    int32_t r = r_begin + g;
    int32_t k, ke, nk, nke;
    bool lng, nlng;
    bounds(r, k, ke, lng);
    bounds(r + G, nk, nke, nlng);
    int mc[kTierNB];
    float mv[kTierNB];
    auto fetch = [&](int32_t kk0, int32_t kke, bool live, int (&c)[kTierNB], float (&a)[kTierNB]) {
#pragma unroll
        for (int j = 0; j < kTierNB; ++j) {
            const int32_t kk = kk0 + j * GL + gl;
            const bool in = live && kk < kke;
            c[j] = col[in ? kk : 0];
            a[j] = val[in ? kk : 0] * (in ? 1.f : 0.f);
        }
    };
    fetch(k, ke, r < r_end, mc, mv);
    float acc[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v)
        acc[v] = 0.f;
    while (__any(r < r_end)) {
        float x[kTierNB][GL][VEC];
        float aa[kTierNB][GL];
#pragma unroll
        for (int j = 0; j < kTierNB; ++j)
#pragma unroll
            for (int u = 0; u < GL; ++u) {
                const int c = __shfl(mc[j], g * GL + u);
                aa[j][u] = __shfl(mv[j], g * GL + u);
                const float *sp = (TWO && c >= n_src0) ? src1 + (int64_t)(c - n_src0) * lds
                                                       : src0 + (int64_t)c * lds;
                load_vec<VEC>(sp + cv * VEC, x[j][u]);
            }
        // the next batch: more of this row, or the first of the group's next row
        const bool row_end = k + E >= ke;
        const int32_t k2 = row_end ? nk : k + E;
        const int32_t ke2 = row_end ? nke : ke;
        const int32_t r2 = row_end ? r + G : r;
        int mc2[kTierNB];
        float mv2[kTierNB];
        fetch(k2, ke2, r2 < r_end, mc2, mv2);
        int32_t nnk, nnke;
        bool nnlng;
        bounds(r + 2 * G, nnk, nnke, nnlng);   // used only when this row ends
#pragma unroll
        for (int j = 0; j < kTierNB; ++j)
#pragma unroll
            for (int u = 0; u < GL; ++u)
#pragma unroll
                for (int v = 0; v < VEC; ++v)
                    acc[v] = fmaf(aa[j][u], x[j][u][v], acc[v]);
        if (row_end) {
            if (r < r_end && gl < dv && !lng)
                out.put<VEC>(r, gl * VEC, acc);
#pragma unroll
            for (int v = 0; v < VEC; ++v)
                acc[v] = 0.f;
            r += G;
            k = nk;
            ke = nke;
            lng = nlng;
            nk = nnk;
            nke = nnke;
            nlng = nnlng;
        } else {
            k += E;
        }
#pragma unroll
        for (int j = 0; j < kTierNB; ++j) {
            mc[j] = mc2[j];
            mv[j] = mv2[j];
        }
    }
}

// ---------------------------------------------------------------------------
// fp32 MFMA GEMM
// ---------------------------------------------------------------------------

typedef float floatx16 __attribute__((ext_vector_type(16)));

// One operand quad in flight: 4 consecutive elements of a row-major operand
// (and of its mask) as loaded, plus whether they lie inside the operand.
// The loads are issued unconditionally (an out-of-range quad reads the
// operand's first element instead) so that the number of loads in flight is
// static; the zero fill and the mask are applied only when the quad is
// written to LDS, so no wait on the loads sits between fetch and compute.
// With VEC a quad is one aligned 16-byte load (the row stride is a multiple
// of 4, so a quad that starts inside a row ends inside its stride); its
// elements past the extent are zeroed, so padding columns may hold
// anything, NaN included.
template <bool VEC, bool MASK>
struct Quad {
    float v[4];
    float m[4];
    uint32_t ok;   // bit j: element j is inside the operand

    __device__ __forceinline__ void load(const float *__restrict__ base,
                                         const float *__restrict__ mbase, int64_t off, int pos,
                                         int lim, bool row_ok)
    {
        if constexpr (VEC) {
            const bool in = row_ok && pos < lim;
            const int64_t o = in ? off : 0;
            const float4 a = *reinterpret_cast<const float4 *>(base + o);
            v[0] = a.x;
            v[1] = a.y;
            v[2] = a.z;
            v[3] = a.w;
            if constexpr (MASK) {
                const float4 b = *reinterpret_cast<const float4 *>(mbase + o);
                m[0] = b.x;
                m[1] = b.y;
                m[2] = b.z;
                m[3] = b.w;
            }
            const int left = lim - pos;
            ok = !in ? 0u : left >= 4 ? 0xFu : (1u << left) - 1u;
        } else {
            ok = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const bool in = row_ok && pos + j < lim;
                const int64_t o = in ? off + j : 0;
                v[j] = base[o];
                if constexpr (MASK)
                    m[j] = mbase[o];
                ok |= in ? (1u << j) : 0u;
            }
        }
    }

    __device__ __forceinline__ float get(int j) const
    {
        const bool keep = ((ok >> j) & 1u) && (!MASK || m[j] > 0.f);
        return keep ? v[j] : 0.f;
    }
};

// BM x BN tile of C per workgroup; 4 waves in a 2x2 arrangement, each owning
// (BM/2) x (BN/2) as TM x TN blocks of 32x32 accumulated with
// v_mfma_f32_32x32x2f32 (the A fragment of a k step is shared by the TN
// blocks of a row, the B fragment by the TM blocks of a column).  K advances
// BK = 32 at a time through two LDS buffers ([k][m] and [k][n], so that the
// fragment read of lane l -- row l%32 at k = l/32 -- is contiguous); the two
// following K tiles are in flight in registers while the current one is
// multiplied; one barrier per K step.
template <int BM, int BN, bool AT, bool BT, bool AMASK, bool BMASK, bool RELU, bool VA, bool VB>
__global__ __launch_bounds__(256) void k_gemm(int32_t M, int32_t N, int32_t K, int32_t kchunk,
                                              const float *__restrict__ A, int32_t lda,
                                              const float *__restrict__ Am,
                                              const float *__restrict__ B, int32_t ldb,
                                              const float *__restrict__ Bm,
                                              float *__restrict__ C, int32_t ldc,
                                              int64_t c_split_stride, int32_t gm, int32_t gn)
{
    constexpr int BK = kGemmBK;
    constexpr int TM = BM / 64, TN = BN / 64;     // 32x32 blocks per wave
    constexpr int QA = BM * BK / 4 / 256;         // operand quads per thread
    constexpr int QB = BN * BK / 4 / 256;
    constexpr int PA = AT ? 4 : 1;   // [k][m] rows written as float4 when m is contiguous
    constexpr int PB = BT ? 1 : 4;
    static_assert(BK == 32 && (BM == 64 || BM == 128) && (BN == 64 || BN == 128), "tile");
    __shared__ float As[2][BK][BM + PA];
    __shared__ float Bs[2][BK][BN + PB];

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wid = tid / kWave;
    // Logical tiles: split-major, then M strip, then N tile, so that an XCD
    // holds whole K slices and the N tiles of an M strip (shared operands).
    const uint32_t logical = xcd_contiguous(blockIdx.x, gridDim.x);
    const uint32_t per_split = (uint32_t)gm * (uint32_t)gn;
    const int z = (int)(logical / per_split);
    const uint32_t t = logical % per_split;
    const int m0 = (int)(t / (uint32_t)gn) * BM;
    const int n0 = (int)(t % (uint32_t)gn) * BN;
    const int kb = z * kchunk;
    const int ke = min(K, kb + kchunk);
    const int wm = (wid >> 1) * (BM / 2);
    const int wn = (wid & 1) * (BN / 2);

    floatx16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e)
                acc[i][j][e] = 0.f;

    using QAt = Quad<VA, AMASK>;
    using QBt = Quad<VB, BMASK>;
    QAt qa0[QA], qa1[QA];
    QBt qb0[QB], qb1[QB];
    auto fetch = [&](int k0, QAt (&qa)[QA], QBt (&qb)[QB]) {
#pragma unroll
        for (int i = 0; i < QA; ++i) {
            const int q = tid + 256 * i;
            if (AT) {   // A(m,k) = A[k*lda + m]; quad along m
                const int k = q / (BM / 4), m = (q % (BM / 4)) * 4;
                qa[i].load(A, Am, (int64_t)(k0 + k) * lda + (m0 + m), m0 + m, M, k0 + k < ke);
            } else {    // A(m,k) = A[m*lda + k]; quad along k
                const int m = q / (BK / 4), k = (q % (BK / 4)) * 4;
                qa[i].load(A, Am, (int64_t)(m0 + m) * lda + (k0 + k), k0 + k, ke, m0 + m < M);
            }
        }
#pragma unroll
        for (int i = 0; i < QB; ++i) {
            const int q = tid + 256 * i;
            if (BT) {   // B(k,n) = B[n*ldb + k]; quad along k
                const int n = q / (BK / 4), k = (q % (BK / 4)) * 4;
                qb[i].load(B, Bm, (int64_t)(n0 + n) * ldb + (k0 + k), k0 + k, ke, n0 + n < N);
            } else {    // B(k,n) = B[k*ldb + n]; quad along n
                const int k = q / (BN / 4), n = (q % (BN / 4)) * 4;
                qb[i].load(B, Bm, (int64_t)(k0 + k) * ldb + (n0 + n), n0 + n, N, k0 + k < ke);
            }
        }
    };
    auto stash = [&](int buf, const QAt (&qa)[QA], const QBt (&qb)[QB]) {
#pragma unroll
        for (int i = 0; i < QA; ++i) {
            const int q = tid + 256 * i;
            if (AT) {
                const int k = q / (BM / 4), m = (q % (BM / 4)) * 4;
                *reinterpret_cast<float4 *>(&As[buf][k][m]) =
                    make_float4(qa[i].get(0), qa[i].get(1), qa[i].get(2), qa[i].get(3));
            } else {
                const int m = q / (BK / 4), k = (q % (BK / 4)) * 4;
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    As[buf][k + j][m] = qa[i].get(j);
            }
        }
#pragma unroll
        for (int i = 0; i < QB; ++i) {
            const int q = tid + 256 * i;
            if (BT) {
                const int n = q / (BK / 4), k = (q % (BK / 4)) * 4;
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    Bs[buf][k + j][n] = qb[i].get(j);
            } else {
                const int k = q / (BN / 4), n = (q % (BN / 4)) * 4;
                *reinterpret_cast<float4 *>(&Bs[buf][k][n]) =
                    make_float4(qb[i].get(0), qb[i].get(1), qb[i].get(2), qb[i].get(3));
            }
        }
    };
    auto compute = [&](int buf) {
        float fa[BK / 2][TM], fb[BK / 2][TN];
#pragma unroll
        for (int st = 0; st < BK / 2; ++st) {
#pragma unroll
            for (int i = 0; i < TM; ++i)
                fa[st][i] = As[buf][2 * st + (lane >> 5)][wm + 32 * i + (lane & 31)];
#pragma unroll
            for (int j = 0; j < TN; ++j)
                fb[st][j] = Bs[buf][2 * st + (lane >> 5)][wn + 32 * j + (lane & 31)];
        }
#pragma unroll
        for (int st = 0; st < BK / 2; ++st)
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(fa[st][i], fb[st][j],
                                                                     acc[i][j], 0, 0, 0);
    };

    // Tile t sits in LDS buffer t % 2; tile t+1 is in flight in one register
    // set while tile t+2 is requested into the other.  The loop body is
    // straight-line (tiles past the end load as zeros and add nothing), so
    // the compiler can wait on exactly the older register set.
    const int ntiles = ke > kb ? (ke - kb + BK - 1) / BK : 0;
    if (ntiles > 0) {
        fetch(kb, qa0, qb0);
        stash(0, qa0, qb0);
        fetch(kb + BK, qa1, qb1);
    }
    __syncthreads();
    for (int t = 0; t < ntiles; t += 2) {
        const int k0 = kb + t * BK;
        fetch(k0 + 2 * BK, qa0, qb0);
        compute(0);
        stash(1, qa1, qb1);
        __syncthreads();
        fetch(k0 + 3 * BK, qa1, qb1);
        compute(1);
        stash(0, qa0, qb0);
        __syncthreads();
    }

    float *Cz = C + (int64_t)z * c_split_stride;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int cn = n0 + wn + 32 * j + (lane & 31);
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int r = m0 + wm + 32 * i + (e >> 2) * 8 + (lane >> 5) * 4 + (e & 3);
                if (r < M && cn < N) {
                    float v = acc[i][j][e];
                    if (RELU)
                        v = fmaxf(v, 0.f);
                    Cz[(int64_t)r * ldc + cn] = v;
                }
            }
        }
}

// out[r][c] = h[r][c] > 0 ? g[r][c] : 0 for r < n, c < d (row strides ldg,
// ldh, ldo), VEC floats per thread.
template <int VEC>
__global__ __launch_bounds__(256) void k_relu_mask(int64_t n, int32_t d, const float *__restrict__ g,
                                                   int32_t ldg, const float *__restrict__ h,
                                                   int32_t ldh, float *__restrict__ out,
                                                   int32_t ldo)
{
    const int32_t dv = d / VEC;
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n * dv)
        return;
    const int64_t r = i / dv;
    const int32_t c = (int32_t)(i % dv) * VEC;
    float gv[VEC], hv[VEC];
    load_vec<VEC>(g + r * ldg + c, gv);
    load_vec<VEC>(h + r * ldh + c, hv);
#pragma unroll
    for (int v = 0; v < VEC; ++v)
        gv[v] = hv[v] > 0.f ? gv[v] : 0.f;
    store_vec<VEC>(out + r * ldo + c, gv);
}

// dst[c][r] = src[r][c] for a rows x cols row-major src: 32x32 tiles through LDS.
__global__ __launch_bounds__(256) void k_transpose(int32_t rows, int32_t cols,
                                                   const float *__restrict__ src,
                                                   float *__restrict__ dst)
{
    __shared__ float t[32][33];
    const int32_t r0 = blockIdx.y * 32, c0 = blockIdx.x * 32;
    const int tx = threadIdx.x % 32, ty = threadIdx.x / 32;   // 8 rows of 32
    for (int y = ty; y < 32; y += 8)
        if (r0 + y < rows && c0 + tx < cols)
            t[y][tx] = src[(int64_t)(r0 + y) * cols + c0 + tx];
    __syncthreads();
    for (int y = ty; y < 32; y += 8)
        if (c0 + y < cols && r0 + tx < rows)
            dst[(int64_t)(c0 + y) * rows + r0 + tx] = t[tx][y];
}

// ---------------------------------------------------------------------------
// An aggregation and a product in one pass
// ---------------------------------------------------------------------------

// An aggregation and a product in one pass, over tiles of kFuseRows
// consecutive rows (the forward of an aggregate-first layer, AH and act(AH
// W); or the input gradient (P_in^T D) W^T).  The 4 waves of a workgroup
// aggregate the tile's rows into LDS (one wave per row, the rows dealt to
// the waves in the order `order` gives, longest first, so that the waves'
// shares are even; a row's entries added in CSR order as in k_spmm),
// storing each row to ah as well when ah is given (the forward keeps AH for
// the weight gradient); then the tile is multiplied by W on MFMA and
// act(tile W) is stored to C.  A CU holds four such workgroups: while one
// multiplies, the others gather, so the product runs in the shadow of the
// memory-bound aggregation instead of as a second pass that reads the
// aggregate back.  Rows of more than kFuseLong entries are aggregated
// beforehand (the long-row blocks of the ordinary kernel write them to pre)
// and read back.  A row is gathered by G groups of 64 / G lanes, which
// split its entries and add their sums at the end (as in k_spmm); a lane
// gathers VEC floats (d <= (64 / G) VEC, sources of row stride lds, ah and
// pre of row stride ld_ah, all multiples of VEC);
// columns d .. ld_ah of ah are stored as zeros.  In the product, each wave
// owns 256 / WAVES columns of every 256-column pass of C (32-column blocks,
// one v_mfma_f32_32x32x2f32 accumulator chain each, over the tile's 32
// rows).  It reads its columns of W, row-major [d][N], straight from global
// memory (W stays in L2), one chunk of KS k-steps ahead, in two register
// sets used in turn.
template <int VEC, int G, bool TWO>
__global__ __launch_bounds__(kFuseThreads) __attribute__((amdgpu_waves_per_eu(kFuseWavesPerSimd))) void
k_spmm_gemm(int32_t n_rows, const int32_t *__restrict__ rowptr, const int32_t *__restrict__ col,
            const float *__restrict__ val, const uint8_t *__restrict__ order,
            const float *__restrict__ src0,
            const float *__restrict__ src1, int32_t n_src0, int32_t lds, int32_t d,
            float *__restrict__ ah, const float *__restrict__ pre, int32_t ld_ah,
            const float *__restrict__ W, int32_t N, float *__restrict__ C, int32_t ldc,
            bool relu)
{
    constexpr int GL = kWave / G;   // lanes per group; the G groups split a row's entries
    constexpr int DMAX = GL * VEC;
    constexpr int LS = DMAX + 1;   // odd row stride: a column of the tile spans all banks
    constexpr int U = 16;          // entries in flight per group
    constexpr int KS = 8;                   // k-steps (of 2) per W chunk
    constexpr int WAVES = kFuseThreads / kWave;
    __shared__ float tile[kFuseRows * LS];

    const int lane = threadIdx.x % kWave;
    const int wave = threadIdx.x / kWave;
    const int64_t r0 = (int64_t)blockIdx.x * kFuseRows;
    const int nr = (int)min<int64_t>(kFuseRows, n_rows - r0);
    const int g = lane / GL, gl = lane % GL;
    const bool lane_cols = gl * VEC < d;

    // Wave w takes the tile positions w, w + WAVES, ... of `order` (rows
    // dealt longest first).  Lane j looks up the pointers of the wave's j-th
    // row, then the entry ids and weights of all the wave's rows are fetched
    // at once (a gathered row has at most kFuseLong <= 64 entries, one per
    // lane), so that no fetch waits between the rows' gathers.
    constexpr int RPW = kFuseRows / WAVES;
    static_assert(kFuseLong <= kWave && RPW <= kWave, "one fetch per row");
    int my_lr = 0, my_kb = 0, my_ke = 0;
    if (lane < RPW) {
        const int p = wave + WAVES * lane;
        my_lr = p < nr ? (int)order[r0 + p] : p;
        if (p < nr) {
            my_kb = rowptr[r0 + my_lr];
            my_ke = rowptr[r0 + my_lr + 1];
        }
    }
    int mcs[RPW];
    float mvs[RPW];
#pragma unroll
    for (int j = 0; j < RPW; ++j) {
        const int kb = readlane_i(my_kb, j), len = readlane_i(my_ke, j) - kb;
        mcs[j] = 0;
        mvs[j] = 0.f;
        if (len <= kFuseLong && lane < len) {
            mcs[j] = col[kb + lane];
            mvs[j] = val[kb + lane];
        }
    }
#pragma unroll
    for (int j = 0; j < RPW; ++j) {
        const int mcA = mcs[j];
        const float mvA = mvs[j];
        const int lrA = readlane_i(my_lr, j);
        const int kbA = readlane_i(my_kb, j), keA = readlane_i(my_ke, j);
        float acc[VEC];
#pragma unroll
        for (int v = 0; v < VEC; ++v)
            acc[v] = 0.f;
        const int len = keA - kbA;
        const int64_t r = r0 + lrA;
        if (len > kFuseLong) {   // aggregated by the long-row pass
            if (g == 0 && lane_cols)
                load_vec<VEC>(pre + r * ld_ah + gl * VEC, acc);
        } else if (len > 0) {
            // group g takes the entries g, g + G, ... (slot t: entry G t + g)
            for (int s0 = 0; s0 * G < len; s0 += U) {
                float x[U][VEC];
                float a[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int e = G * (s0 + u) + g;
                    int c;
                    if constexpr (G == 1) {
                        c = readlane_i(mcA, e & (kWave - 1));
                        a[u] = readlane_f(mvA, e & (kWave - 1));
                    } else {
                        c = __shfl(mcA, e & (kWave - 1));
                        a[u] = __shfl(mvA, e & (kWave - 1));
                    }
                    const float *sp = (TWO && c >= n_src0) ? src1 + (int64_t)(c - n_src0) * lds
                                                           : src0 + (int64_t)c * lds;
                    if (e < len && lane_cols) {
                        load_vec<VEC>(sp + gl * VEC, x[u]);
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
                        acc[v] = fmaf(a[u], x[u][v], acc[v]);
            }
            if constexpr (G > 1) {
#pragma unroll
                for (int off = GL; off < kWave; off <<= 1)
#pragma unroll
                    for (int v = 0; v < VEC; ++v)
                        acc[v] += __shfl_xor(acc[v], off);
            }
        }
        if (ah && g == 0 && len <= kFuseLong && lrA < nr && gl * VEC < ld_ah) {
            float o[VEC];
#pragma unroll
            for (int v = 0; v < VEC; ++v)
                o[v] = gl * VEC + v < d ? acc[v] : 0.f;
            store_vec<VEC>(ah + r * ld_ah + gl * VEC, o);
        }
        if (g == 0) {
#pragma unroll
            for (int v = 0; v < VEC; ++v)
                tile[lrA * LS + gl * VEC + v] = (lrA < nr && gl * VEC + v < d) ? acc[v] : 0.f;
        }
    }
    __syncthreads();

    const int half = lane >> 5, l32 = lane & 31;
    static_assert(kFuseRows == 32, "one 32-row block per tile");
    constexpr int NB = 256 / 32 / WAVES;   // 32-column blocks per wave and pass
    static_assert(NB >= 1 && NB * 32 * WAVES == 256, "256 columns per pass");
    const int n_chunks = (d + 2 * KS - 1) / (2 * KS);   // chunks of 2 KS k
    for (int n0 = 32 * NB * wave; n0 < N; n0 += 256) {
        int nc[NB];
        bool nok[NB];
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            const int n = n0 + 32 * j + l32;
            nok[j] = n < N;
            nc[j] = min(n, N - 1);
        }
        floatx16 acc[NB];
#pragma unroll
        for (int j = 0; j < NB; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e)
                acc[j][e] = 0.f;
        // W fragments of chunk c (rows k = 2 KS c + 2 st + half, the NB
        // column blocks), loaded from clamped addresses; entries past d or
        // N are zeroed where they are used
        auto load_w = [&](int c, float (&b)[KS][NB]) {
#pragma unroll
            for (int st = 0; st < KS; ++st) {
                const int64_t row = (int64_t)min(2 * KS * c + 2 * st + half, d - 1) * N;
#pragma unroll
                for (int j = 0; j < NB; ++j)
                    b[st][j] = W[row + nc[j]];
            }
        };
        auto mul = [&](int c, const float (&b)[KS][NB]) {
            float a[KS];
#pragma unroll
            for (int st = 0; st < KS; ++st)   // k < DMAX: 2 KS c <= DMAX - 2 KS
                a[st] = tile[l32 * LS + 2 * KS * c + 2 * st + half];
#pragma unroll
            for (int st = 0; st < KS; ++st) {
                const bool kok = 2 * KS * c + 2 * st + half < d;
#pragma unroll
                for (int j = 0; j < NB; ++j) {
                    const float bv = (kok && nok[j]) ? b[st][j] : 0.f;
                    acc[j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[st], bv, acc[j], 0, 0, 0);
                }
            }
        };
        // chunk c in set c % 2; the loads of chunk c + 1 are in flight while
        // chunk c is multiplied (chunks past the end load row d - 1 again)
        float b0[KS][NB], b1[KS][NB];
        load_w(0, b0);
        for (int c = 0; c < n_chunks; c += 2) {
            load_w(c + 1, b1);
            mul(c, b0);
            load_w(c + 2, b0);
            if (c + 1 < n_chunks)
                mul(c + 1, b1);
        }
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            if (!nok[j])
                continue;
            const int n = n0 + 32 * j + l32;
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int m = (e >> 2) * 8 + half * 4 + (e & 3);
                const float v = relu ? fmaxf(acc[j][e], 0.f) : acc[j][e];
                if (m < nr)
                    C[(r0 + m) * ldc + n] = v;
            }
        }
    }
}

// out[e] = sum over z of part[z][e], z ascending: one element per thread,
// eight slices in flight (many elements, few slices).
__global__ __launch_bounds__(256) void k_splitk_reduce(const float *__restrict__ part,
                                                       int32_t splits, int64_t count,
                                                       float *__restrict__ out)
{
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= count)
        return;
    float acc = 0.f;
    int z = 0;
    for (; z + 8 <= splits; z += 8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            v[u] = part[(int64_t)(z + u) * count + e];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            acc += v[u];
    }
    for (; z < splits; ++z)
        acc += part[(int64_t)z * count + e];
    out[e] = acc;
}

// The same sum for few elements and many slices: a block takes 8 consecutive
// elements; its 32 slice lanes per element sum the slices z = lane,
// lane + 32, ... in order and the 32 partial sums are added in a fixed tree
// in LDS.
__global__ __launch_bounds__(256) void k_splitk_reduce_wide(const float *__restrict__ part,
                                                            int32_t splits, int64_t count,
                                                            float *__restrict__ out)
{
    constexpr int EPB = 8, SL = 32;   // elements per block, slice lanes
    __shared__ float red[SL][EPB + 1];
    const int el = threadIdx.x % EPB, sl = threadIdx.x / EPB;
    const int64_t e = (int64_t)blockIdx.x * EPB + el;
    float acc = 0.f;
    if (e < count) {
#pragma unroll 4
        for (int z = sl; z < splits; z += SL)
            acc += part[(int64_t)z * count + e];
    }
    red[sl][el] = acc;
    __syncthreads();
    for (int off = SL / 2; off > 0; off >>= 1) {
        if (sl < off)
            red[sl][el] += red[sl + off][el];
        __syncthreads();
    }
    if (sl == 0 && e < count)
        out[e] = red[0][el];
}

// ---------------------------------------------------------------------------
// Narrow dense products (one side <= kNarrow = 16)
// ---------------------------------------------------------------------------

typedef float floatx4 __attribute__((ext_vector_type(4)));

// C[r][n] = sum_k A(r)[k] B[k][n] for n < N <= 16 NB, on v_mfma_f32_16x16x4f32.
// Row r of A is row r of A0 (r < m0) or row r - m0 of A1 (leading dim lda).
// B is staged once per block in LDS transposed, as [n][k] for the 16 NB
// columns (zero-padded in n and in k up to a multiple of 16), its rows
// narrow_n_stride(K) floats apart (4 mod 16, so that the 16 rows one read
// touches start in different bank quads).  The grid is sized to the chip and
// each wave takes 16-row tiles in turn, so the staging is paid once per
// block, not per tile.  The contraction order is permuted so that a lane
// feeds its own 16-byte loads: in MFMA step (j, v) lane group h = lane/16
// contributes k = 16 j + 4 h + v for row lane%16 (A) and column lane%16 of
// each column block (B), and every k is covered once; a lane's four k of a
// step are one 16-byte read of A and one of B per column block.  All A loads
// of a K chunk are issued before its MFMAs, and the NB column blocks share
// them.
template <bool VEC, int NB>
__global__ __launch_bounds__(256) void k_narrow_n(int32_t M, int32_t m0, int32_t K, int32_t N,
                                                  const float *__restrict__ A0,
                                                  const float *__restrict__ A1, int32_t lda,
                                                  int32_t lda1,
                                                  const float *__restrict__ B,
                                                  float *__restrict__ C, int32_t ldc, bool relu)
{
    constexpr int KC = 256;          // k per chunk
    constexpr int J = KC / 16;       // 16-k steps per chunk
    const int BS = narrow_n_stride(K);   // LDS row stride of B^T
    extern __shared__ float Bs[];    // [16 NB][BS]
    stage_lds(Bs, 16 * NB * BS, [&](int i) {
        const int n = i / BS, k = i % BS;
        return n < N && k < K ? B[(int64_t)k * N + n] : 0.f;
    });
    __syncthreads();
    const int lane = threadIdx.x & (kWave - 1);
    const int m = lane & 15, h = lane >> 4;
    const int64_t tiles = ((int64_t)M + 15) / 16;
    const int64_t waves = (int64_t)gridDim.x * (blockDim.x / kWave);
    for (int64_t t = blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave; t < tiles;
         t += waves) {
        const int64_t row0 = t * 16;
        const int64_t r = row0 + m;
        const bool row_ok = r < M;   // a lane past M loads the first element, stores nothing
        const float *a =
            !row_ok ? A0 : (r < m0 ? A0 + r * lda : A1 + (r - m0) * (int64_t)lda1);
        floatx4 acc[NB];
#pragma unroll
        for (int b = 0; b < NB; ++b)
            acc[b] = floatx4{0.f, 0.f, 0.f, 0.f};
        float av[J][4];
        for (int kc = 0; kc < K; kc += KC) {
#pragma unroll
            for (int j = 0; j < J; ++j) {
                const int k = kc + 16 * j + 4 * h;
                if (VEC) {
                    const bool ok = row_ok && k < K;   // K % 4 == 0: quads all in or all out
                    const float4 q = *reinterpret_cast<const float4 *>(ok ? a + k : A0);
                    av[j][0] = ok ? q.x : 0.f;
                    av[j][1] = ok ? q.y : 0.f;
                    av[j][2] = ok ? q.z : 0.f;
                    av[j][3] = ok ? q.w : 0.f;
                } else {
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const bool ok = row_ok && k + v < K;
                        const float q = *(ok ? a + k + v : A0);
                        av[j][v] = ok ? q : 0.f;
                    }
                }
            }
#pragma unroll
            for (int j = 0; j < J; ++j) {
                // B^T rows 16 b + m, k = kc + 16 j + 4 h .. + 3 (zeros past K,
                // and the chunk past the padded K reads row 0 and adds zeros)
                const int k = kc + 16 * j + 4 * h;
                const int kk = k < BS - 4 ? k : 0;
                const float4 *Bs4 = reinterpret_cast<const float4 *>(Bs);   // BS % 4 == 0
                float4 bq[NB];
#pragma unroll
                for (int b = 0; b < NB; ++b)
                    bq[b] = Bs4[(16 * b + m) * (BS / 4) + kk / 4];
#pragma unroll
                for (int v = 0; v < 4; ++v)
#pragma unroll
                    for (int b = 0; b < NB; ++b) {
                        const float bv = k < BS - 4 ? bq[b][v] : 0.f;
                        acc[b] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[j][v], bv, acc[b], 0, 0,
                                                                      0);
                    }
            }
        }
        // lane holds C[row0 + 4h + i][16 b + m] for i < 4
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            const int n = 16 * b + m;
            if (n < N) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int64_t rr = row0 + 4 * h + i;
                    if (rr < M)
                        C[rr * ldc + n] = relu ? fmaxf(acc[b][i], 0.f) : acc[b][i];
                }
            }
        }
    }
}

// C[r][n] = sum_{k < K} A[r][k] W[n][k] (A W^T, W row-major [N][K]) for
// 16 < K <= 4 KS <= 64, on v_mfma_f32_16x16x4f32: a product whose cost is
// writing C.  W is staged once per block in LDS as [k][n] (k zero-padded to
// 4 KS, rows bs floats apart with bs = 16 mod 64, so that the four k rows
// of an MFMA step fall in different banks).  The grid is sized to the chip
// and each wave takes 16-row tiles in turn: lane (m, h) = (lane % 16,
// lane / 16) loads A[row m][4 j + h] for MFMA step j once per tile, and the
// column blocks of C reuse them two at a time.
template <int KS>
__global__ __launch_bounds__(256) void k_times_wt(int32_t M, int32_t N, int32_t K,
                                                  const float *__restrict__ A, int32_t lda,
                                                  const float *__restrict__ W,
                                                  float *__restrict__ C, int32_t ldc, int32_t bs)
{
    extern __shared__ float Ws[];   // [4 KS][bs]
    stage_lds(Ws, 4 * KS * bs, [&](int i) {
        const int k = i / bs, n = i % bs;
        return (k < K && n < N) ? W[(int64_t)n * K + k] : 0.f;
    });
    __syncthreads();
    const int lane = threadIdx.x & (kWave - 1);
    const int m = lane & 15, h = lane >> 4;
    const int nb = (N + 15) / 16;
    const int64_t tiles = ((int64_t)M + 15) / 16;
    const int64_t waves = (int64_t)gridDim.x * (blockDim.x / kWave);
    for (int64_t t = blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave; t < tiles;
         t += waves) {
        const int64_t row0 = t * 16;
        const int64_t r = row0 + m;
        const float *ar = A + (r < M ? r : 0) * (int64_t)lda;
        float a[KS];
#pragma unroll
        for (int j = 0; j < KS; ++j) {
            const int k = 4 * j + h;
            a[j] = (r < M && k < K) ? ar[k] : 0.f;
        }
        for (int b = 0; b < nb; b += 2) {
            // the second block of an odd last pair reads a valid column, stores nothing
            const int c0 = 16 * b + m, c1 = min(16 * (b + 1) + m, bs - 1);
            floatx4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int j = 0; j < KS; ++j) {
                const float *wr = Ws + (4 * j + h) * bs;
                acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(a[j], wr[c0], acc0, 0, 0, 0);
                acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(a[j], wr[c1], acc1, 0, 0, 0);
            }
            // lane holds C[row0 + 4h + i][16 b + m] (acc0) and [16 (b+1) + m] (acc1)
            const int n0 = 16 * b + m, n1 = n0 + 16;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int64_t rr = row0 + 4 * h + i;
                if (rr < M) {
                    if (n0 < N)
                        C[rr * ldc + n0] = acc0[i];
                    if (n1 < N)
                        C[rr * ldc + n1] = acc1[i];
                }
            }
        }
    }
}

// C[r][n] = sum_{k < K} A[r][k] W[n][k] (W row-major [N][K], i.e. A W^T) for
// K <= KK.  A wave owns a slice of 256 columns, four per lane, and keeps
// that slice of W in registers for the whole launch; it then strides over
// the rows, RU at a time: the K inputs of a row are read at a wave-uniform
// address (scalar loads) and every lane writes its four outputs.
constexpr int kNarrowKRows = 4;

template <int KK>
__global__ __launch_bounds__(256) void k_narrow_k(int32_t M, int32_t N, int32_t K,
                                                  const float *__restrict__ A, int32_t lda,
                                                  const float *__restrict__ W,
                                                  float *__restrict__ C, int32_t ldc,
                                                  bool vec_out, int32_t slices)
{
    constexpr int RU = kNarrowKRows;
    const int lane = threadIdx.x & (kWave - 1);
    const int gw = __builtin_amdgcn_readfirstlane(
        (int)(blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave));
    const int nw = (int)(gridDim.x * (blockDim.x / kWave)) / slices;   // waves per slice
    const int slice = gw % slices;
    const int first = gw / slices;
    if (first >= nw)
        return;   // surplus waves (the launcher makes none)
    const int n0 = slice * 256 + lane * 4;
    float w[KK][4];
#pragma unroll
    for (int k = 0; k < KK; ++k)
#pragma unroll
        for (int j = 0; j < 4; ++j)
            w[k][j] = (k < K && n0 + j < N) ? W[(int64_t)(n0 + j) * K + k] : 0.f;
    for (int r0 = first * RU; r0 < M; r0 += nw * RU) {
        float a[RU][KK];
#pragma unroll
        for (int u = 0; u < RU; ++u) {
            const int r = min(r0 + u, M - 1);   // rows past M recompute row M-1, not stored
            const float *ar = A + (int64_t)r * lda;
#pragma unroll
            for (int k = 0; k < KK; ++k)
                a[u][k] = k < K ? ar[k] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < RU; ++u) {
            const int r = r0 + u;
            if (r >= M)
                break;
            float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int k = 0; k < KK; ++k)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[j] = fmaf(a[u][k], w[k][j], acc[j]);
            float *cr = C + (int64_t)r * ldc + n0;
            if (vec_out) {
                if (n0 < N)
                    *reinterpret_cast<float4 *>(cr) = make_float4(acc[0], acc[1], acc[2], acc[3]);
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (n0 + j < N)
                        cr[j] = acc[j];
            }
        }
    }
}

// Split-K partial of dW = H^T G for N <= 16, on v_mfma_f32_16x16x4f32:
//   part[z][f][n] = sum over the rows r of slice z of H(r)[f] G[r][n],
// row r of H from H0 (r < m0) or H1 (leading dim ldh); G row-major [R][N].
// A wave owns 64 features (four 16-feature MFMA blocks sharing every G
// load) and one slice of rows; in MFMA step s lane group h contributes row
// rb + 4 s + h.  The 4 waves of a block take 4 consecutive slices.
__global__ __launch_bounds__(256) void k_dw_narrow(int32_t R, int32_t m0, int32_t F, int32_t N,
                                                   const float *__restrict__ H0,
                                                   const float *__restrict__ H1, int32_t ldh,
                                                   int32_t ldh1, const float *__restrict__ G,
                                                   int32_t ldg,
                                                   int32_t chunk, int32_t splits,
                                                   float *__restrict__ part)
{
    constexpr int SB = 8;   // MFMA steps (32 rows) per batch of loads
    const int lane = threadIdx.x & (kWave - 1);
    const int z = blockIdx.y * (blockDim.x / kWave) + threadIdx.x / kWave;
    if (z >= splits)
        return;   // uniform per wave
    const int f0 = blockIdx.x * 64;
    const int rb = z * chunk;
    const int re = min(R, rb + chunk);
    const int m = lane & 15, h = lane >> 4;
    floatx4 acc[4];
#pragma unroll
    for (int q = 0; q < 4; ++q)
        acc[q] = floatx4{0.f, 0.f, 0.f, 0.f};
    for (int r0 = rb; r0 < re; r0 += 4 * SB) {
        float av[SB][4], bv[SB];
#pragma unroll
        for (int s = 0; s < SB; ++s) {
            const int r = r0 + 4 * s + h;
            const bool ok = r < re;
            const float *hp = r < m0 ? H0 + (int64_t)r * ldh : H1 + (int64_t)(r - m0) * ldh1;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int f = f0 + 16 * q + m;
                const bool okf = ok && f < F;
                const float v = *(okf ? hp + f : H0);
                av[s][q] = okf ? v : 0.f;
            }
            const bool okg = ok && m < N;
            const float g = *(okg ? G + (int64_t)r * ldg + m : G);
            bv[s] = okg ? g : 0.f;
        }
#pragma unroll
        for (int s = 0; s < SB; ++s)
#pragma unroll
            for (int q = 0; q < 4; ++q)
                acc[q] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[s][q], bv[s], acc[q], 0, 0, 0);
    }
    // acc[q] lane holds D[f0 + 16 q + 4 h + i][m]
    if (m < N) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int f = f0 + 16 * q + 4 * h + i;
                if (f < F)
                    part[((int64_t)z * F + f) * N + m] = acc[q][i];
            }
    }
}

// ---------------------------------------------------------------------------
// Softmax cross entropy
// ---------------------------------------------------------------------------

constexpr int kLossThreads = 256;

// Block sum of the rows' losses into block_loss[blockIdx.x]: a butterfly
// inside each wave, then the waves in order (a fixed order).
__device__ __forceinline__ void loss_block_sum(float row_loss, float *__restrict__ block_loss)
{
    __shared__ float part[kLossThreads / kWave];
    const int lane = threadIdx.x & (kWave - 1);
    const int wid = threadIdx.x / kWave;
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1)
        row_loss += __shfl_xor(row_loss, off);
    if (lane == 0)
        part[wid] = row_loss;
    __syncthreads();
    if (threadIdx.x == 0) {
        float t = 0.f;
        for (int i = 0; i < kLossThreads / kWave; ++i)
            t += part[i];
        block_loss[blockIdx.x] = t;
    }
}

// loss = inv_n * sum of the block sums, in a fixed order: thread j of one
// kLossReduceThreads block adds the block sums j, j + T, ... (loaded eight at
// a time), then the threads' sums are added by a butterfly inside each wave
// and the waves' in wave order.
constexpr int kLossReduceThreads = 1024;

__global__ __launch_bounds__(kLossReduceThreads) void k_loss_reduce(
    const float *__restrict__ block_loss, int32_t nb, float inv_n, float *__restrict__ loss)
{
    constexpr int U = 8, T = kLossReduceThreads;
    __shared__ float part[T / kWave];
    float t = 0.f;
    for (int i0 = threadIdx.x; i0 < nb; i0 += U * T) {
        float v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = i0 + u * T;
            v[u] = i < nb ? block_loss[i] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
            t += v[u];
    }
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1)
        t += __shfl_xor(t, off);
    if ((threadIdx.x & (kWave - 1)) == 0)
        part[threadIdx.x / kWave] = t;
    __syncthreads();
    if (threadIdx.x == 0) {
        float sum = 0.f;
        for (int w = 0; w < T / kWave; ++w)
            sum += part[w];
        loss[0] = sum * inv_n;
    }
}

// Row-wise softmax cross entropy.  A row belongs to a group of GL lanes;
// lane gl of the group holds the classes gl, gl + GL, ... (NJ of them) in
// registers, so each logit is read once; a wave holds 64/GL rows.
template <int GL, int NJ>
__global__ __launch_bounds__(kLossThreads) void k_softmax_xent(
    const float *__restrict__ logits, const int32_t *__restrict__ labels, int32_t n, int32_t C,
    float inv_n, float *__restrict__ dlogits, float *__restrict__ block_loss)
{
    constexpr int G = kWave / GL;
    const int lane = threadIdx.x & (kWave - 1);
    const int g = lane / GL, gl = lane % GL;
    const int r = (blockIdx.x * (kLossThreads / kWave) + threadIdx.x / kWave) * G + g;
    float row_loss = 0.f;
    if (r < n) {
        const float *z = logits + (int64_t)r * C;
        float *dz = dlogits + (int64_t)r * C;
        const int y = labels[r];
        const bool bad = y < 0 || y >= C;
        float v[NJ];
        float m = -INFINITY;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int c = gl + j * GL;
            v[j] = c < C ? z[c] : -INFINITY;
            m = fmaxf(m, v[j]);
        }
#pragma unroll
        for (int off = GL / 2; off > 0; off >>= 1)
            m = fmaxf(m, __shfl_xor(m, off));
        float sum = 0.f;
#pragma unroll
        for (int j = 0; j < NJ; ++j)
            if (gl + j * GL < C)
                sum += expf(v[j] - m);
#pragma unroll
        for (int off = GL / 2; off > 0; off >>= 1)
            sum += __shfl_xor(sum, off);
        const float log_s = logf(sum);
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int c = gl + j * GL;
            if (c < C) {
                const float lp = v[j] - m - log_s;
                dz[c] = bad ? 0.f : (expf(lp) - (c == y ? 1.f : 0.f)) * inv_n;
                if (c == y)
                    row_loss = -lp;
            }
        }
        if (bad && gl == 0)
            row_loss = NAN;
    }
    loss_block_sum(row_loss, block_loss);
}

// The same loss for any class count: a wave per row, lane c holding the
// classes c, c + 64, ... read from memory in three passes.
__global__ __launch_bounds__(kLossThreads) void k_softmax_xent_wide(
    const float *__restrict__ logits, const int32_t *__restrict__ labels, int32_t n, int32_t C,
    float inv_n, float *__restrict__ dlogits, float *__restrict__ block_loss)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int r = blockIdx.x * (kLossThreads / kWave) + threadIdx.x / kWave;
    float row_loss = 0.f;
    if (r < n) {
        const float *z = logits + (int64_t)r * C;
        float *dz = dlogits + (int64_t)r * C;
        const int y = labels[r];
        const bool bad = y < 0 || y >= C;
        float m = -INFINITY;
        for (int c = lane; c < C; c += kWave)
            m = fmaxf(m, z[c]);
#pragma unroll
        for (int off = kWave / 2; off > 0; off >>= 1)
            m = fmaxf(m, __shfl_xor(m, off));
        float sum = 0.f;
        for (int c = lane; c < C; c += kWave)
            sum += expf(z[c] - m);
#pragma unroll
        for (int off = kWave / 2; off > 0; off >>= 1)
            sum += __shfl_xor(sum, off);
        const float log_s = logf(sum);
        for (int c = lane; c < C; c += kWave) {
            const float lp = z[c] - m - log_s;
            dz[c] = bad ? 0.f : (expf(lp) - (c == y ? 1.f : 0.f)) * inv_n;
            if (c == y)
                row_loss = -lp;
        }
        if (bad && lane == 0)
            row_loss = NAN;
    }
    loss_block_sum(row_loss, block_loss);
}

// ---------------------------------------------------------------------------
// GAT layer
// ---------------------------------------------------------------------------

constexpr int kGatCache = 4;    // scores a lane keeps between the passes

__device__ __forceinline__ float leaky(float x, float slope) { return x > 0.f ? x : slope * x; }

// alpha[k] = softmax over the entries k of row i of
// LeakyReLU(s[i][1] + s[col[k]][0]), s [rows][2] (source, target score).
// A wave takes a row and strides over its entries three times (the
// maximum, the sum of exponentials, the weights), combining its lanes by a
// fixed butterfly, so results are deterministic.  Each lane keeps its first
// kGatCache scores in registers (rows up to 256 entries are read once);
// beyond them the passes recompute the scores kGatCache entries at a time,
// their loads all issued before use.
__global__ __launch_bounds__(256) void k_gat_softmax(int32_t n_rows,
                                                     const int32_t *__restrict__ rowptr,
                                                     const int32_t *__restrict__ col,
                                                     const float *__restrict__ s, float slope,
                                                     float *__restrict__ alpha)
{
    constexpr int U = kGatCache;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t row = (int64_t)blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
    if (row >= n_rows)
        return;   // uniform per wave
    const int kb = rowptr[row], ke = rowptr[row + 1];
    if (ke <= kb)
        return;   // an empty row has no weights
    const float t = s[2 * row + 1];
    // scores of entries k0 + lane + u * 64, u < U (-inf past the row); the
    // loads are unconditional (an entry past the row reads its last one)
    auto scores = [&](int k0, float (&e)[U]) {
        int c[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int k = k0 + lane + u * kWave;
            c[u] = col[k < ke ? k : ke - 1];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const float v = leaky(t + s[2 * (int64_t)c[u]], slope);
            e[u] = k0 + lane + u * kWave < ke ? v : -INFINITY;
        }
    };
    constexpr int SPAN = U * kWave;
    float ec[U];
    scores(kb, ec);
    float m = -INFINITY;
#pragma unroll
    for (int u = 0; u < U; ++u)
        m = fmaxf(m, ec[u]);
    for (int k0 = kb + SPAN; k0 < ke; k0 += SPAN) {
        float e[U];
        scores(k0, e);
#pragma unroll
        for (int u = 0; u < U; ++u)
            m = fmaxf(m, e[u]);
    }
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1)
        m = fmaxf(m, __shfl_xor(m, off));
    float l = 0.f;
#pragma unroll
    for (int u = 0; u < U; ++u)
        l += kb + lane + u * kWave < ke ? expf(ec[u] - m) : 0.f;
    for (int k0 = kb + SPAN; k0 < ke; k0 += SPAN) {
        float e[U];
        scores(k0, e);
#pragma unroll
        for (int u = 0; u < U; ++u)
            l += k0 + lane + u * kWave < ke ? expf(e[u] - m) : 0.f;
    }
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1)
        l += __shfl_xor(l, off);
    const float inv = 1.f / l;
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int k = kb + lane + u * kWave;
        if (k < ke)
            alpha[k] = expf(ec[u] - m) * inv;
    }
    for (int k0 = kb + SPAN; k0 < ke; k0 += SPAN) {
        float e[U];
        scores(k0, e);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int k = k0 + lane + u * kWave;
            if (k < ke)
                alpha[k] = expf(e[u] - m) * inv;
        }
    }
}

// Per-edge gradient of the GAT layer over the owned rows i:
//   D_i     = dh_out_i * 1[h_out_i > 0] (relu) or dh_out_i    -> dO_i
//   c_i     = D_i . h_out_i  (= D_i . o_i: the mask zeroes D where o <= 0)
//   dpre[k] = alpha[k] (D_i . z_{col k} - c_i) * LeakyReLU'(t_i + s_{col k})
//   g2[i][1] = sum_k dpre[k]
// Work follows the aggregation's block plan: a short-row block gives wave w
// the row b.row + w; a long-row block splits the entries of row b.row into
// kSpmmWaves contiguous parts, one per wave, and adds the waves' row sums
// in LDS in wave order (so a row of thousands of entries is not one wave's
// serial loop).  Inside a wave the G = 64 / GL lane groups split the
// entries, U per group in flight at once; inside a group GL lanes hold D_i
// as NCH vectors of VEC features and gather the matching features of z; the
// U dot products of a group go through one butterfly together.  All sums
// have a fixed order.  At most four waves per SIMD: left to maximise
// occupancy the compiler reuses one register quad for every gather and
// waits on each, which serialises the step.
template <int VEC, int GL, int NCH, int U>
__global__ __launch_bounds__(kSpmmThreads) __attribute__((amdgpu_waves_per_eu(1, 4))) void
k_gat_edge_grad(const SpmmBlock *__restrict__ blocks, int32_t d,
                const int32_t *__restrict__ rowptr, const int32_t *__restrict__ col,
                const float *__restrict__ alpha, const float *__restrict__ s,
                const float *__restrict__ z, const float *__restrict__ h_out,
                const float *__restrict__ dh_out, bool relu, float slope, float *__restrict__ dO,
                float *__restrict__ dpre, float *__restrict__ g2)
{
    constexpr int G = kWave / GL;
    __shared__ float red[kSpmmWaves];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int g = lane / GL, gl = lane % GL;
    const SpmmBlock b = blocks[blockIdx.x];
    const bool long_row = b.nrows == 0;   // uniform over the block
    int64_t row;
    int kb, ke;
    if (long_row) {
        row = b.row;
        const int per = (b.ke - b.kb + kSpmmWaves - 1) / kSpmmWaves;
        kb = min(b.ke, b.kb + wave * per);
        ke = min(b.ke, kb + per);
    } else {
        if (wave >= b.nrows)
            return;   // uniform per wave; short-row blocks have no barrier
        row = b.row + wave;
        kb = rowptr[row];
        ke = rowptr[row + 1];
    }
    const bool writer = !long_row || wave == 0;   // stores dO and g2
    const int dv = d / VEC;
    float D[NCH][VEC];
    float c = 0.f;
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
        const int cv = ch * GL + gl;
        if (cv < dv) {
            float dh[VEC], h[VEC];
            load_vec<VEC>(dh_out + row * d + cv * VEC, dh);
            load_vec<VEC>(h_out + row * d + cv * VEC, h);
#pragma unroll
            for (int v = 0; v < VEC; ++v) {
                D[ch][v] = (!relu || h[v] > 0.f) ? dh[v] : 0.f;
                c = fmaf(D[ch][v], h[v], c);
            }
            if (writer && g == 0)
                store_vec<VEC>(dO + row * d + cv * VEC, D[ch]);
        } else {
#pragma unroll
            for (int v = 0; v < VEC; ++v)
                D[ch][v] = 0.f;
        }
    }
#pragma unroll
    for (int off = GL / 2; off > 0; off >>= 1)
        c += __shfl_xor(c, off);
    const float t = s[2 * row + 1];
    float rowsum = 0.f;
    // Every load below is issued unconditionally from a valid address (an
    // entry past the part reads the part's last entry, a vector past the
    // width its first vector) and its result is ignored or multiplied by a
    // zero of D, so all U x NCH gathers of a step are in flight together.
    for (int k0 = kb; k0 < ke; k0 += G * U) {
        int kk[U];
        bool ok[U];
        int64_t jj[U];
        float al[U], sj[U], dot[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            kk[u] = k0 + u * G + g;
            ok[u] = kk[u] < ke;
            kk[u] = ok[u] ? kk[u] : ke - 1;
            jj[u] = col[kk[u]];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            al[u] = alpha[kk[u]];
            sj[u] = s[2 * jj[u]];
            dot[u] = 0.f;
        }
        float zv[U][NCH][VEC];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int ch = 0; ch < NCH; ++ch) {
                const int cv = ch * GL + gl < dv ? ch * GL + gl : 0;
                load_vec<VEC>(z + jj[u] * d + cv * VEC, zv[u][ch]);
            }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
                for (int v = 0; v < VEC; ++v)
                    dot[u] = fmaf(D[ch][v], zv[u][ch][v], dot[u]);
#pragma unroll
        for (int off = GL / 2; off > 0; off >>= 1)
#pragma unroll
            for (int u = 0; u < U; ++u)
                dot[u] += __shfl_xor(dot[u], off);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (ok[u]) {
                const float pre = t + sj[u];
                const float dp = al[u] * (dot[u] - c) * (pre > 0.f ? 1.f : slope);
                if (gl == 0) {
                    dpre[kk[u]] = dp;
                    rowsum += dp;
                }
            }
        }
    }
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1)
        rowsum += __shfl_xor(rowsum, off);
    if (long_row) {
        if (lane == 0)
            red[wave] = rowsum;
        __syncthreads();
        if (threadIdx.x == 0) {
            float r = 0.f;
#pragma unroll
            for (int w = 0; w < kSpmmWaves; ++w)
                r += red[w];
            g2[2 * row + 1] = r;
        }
    } else if (lane == 0) {
        g2[2 * row + 1] = rowsum;
    }
}

// a_t[k] = a[perm[k]], b_t[k] = b[perm[k]]: edge values into the entry order
// of the transposed CSR.
__global__ __launch_bounds__(256) void k_gather_perm2(int64_t n, const int32_t *__restrict__ perm,
                                                      const float *__restrict__ a,
                                                      const float *__restrict__ b,
                                                      float *__restrict__ a_t,
                                                      float *__restrict__ b_t)
{
    const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (k < n) {
        const int32_t p = perm[k];
        a_t[k] = a[p];
        b_t[k] = b[p];
    }
}

// Score terms of the GAT backward over the local rows v < R:
//   dz[v] += ds_src[v] att[:,0] + (v < n_own ? g2[v][1] att[:,1] : 0)
//   g2[v][0] = ds_src[v];  g2[v][1] = 0 for the halo rows
// (g2 then holds the gradient of the scores, [R][2]).  A thread per element
// of dz; the thread of column 0 writes g2.
__global__ __launch_bounds__(256) void k_gat_score_cols(int64_t R, int32_t n_own,
                                                        const float *__restrict__ ds_src,
                                                        float *__restrict__ g2)
{
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v >= R)
        return;
    g2[2 * v] = ds_src[v];
    if (v >= n_own)
        g2[2 * v + 1] = 0.f;
}

// ---------------------------------------------------------------------------
// Global parameter update
// ---------------------------------------------------------------------------

// w[e] -= lr * (1/n) * sum over m of g.g[m][e], m ascending; a thread per
// element.
__global__ __launch_bounds__(256) void k_sgd_average(float *__restrict__ w, GradList g,
                                                     int32_t n, int64_t count, float lr)
{
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= count)
        return;
    float sum = 0.f;
    for (int m = 0; m < n; ++m)
        sum += g.g[m][e];
    w[e] = w[e] - lr * (sum / (float)n);
}

// p[e] = 0 for e < count, a thread per element (a kernel rather than a
// memset, so that it records as a kernel node under graph capture).
__global__ __launch_bounds__(256) void k_fill_zero(float *__restrict__ p, int64_t count)
{
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e < count)
        p[e] = 0.f;
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
hipError_t copy_rows_t(int mode, const int32_t *sidx, const int32_t *didx, int32_t n_rows,
                       int32_t d, float *src, int32_t lds, float *dst, int32_t ldd,
                       hipStream_t s)
{
    constexpr int rows_per_block = 4 * (kWave / GL);
    const int64_t blocks = ((int64_t)n_rows + rows_per_block - 1) / rows_per_block;
    const dim3 grid((unsigned)blocks), block(256);
    if (mode == kAdd)
        hipLaunchKernelGGL((k_copy_rows<VEC, GL, kAdd>), grid, block, 0, s, sidx, didx, n_rows, d,
                           src, lds, dst, ldd);
    else if (mode == kAddClear)
        hipLaunchKernelGGL((k_copy_rows<VEC, GL, kAddClear>), grid, block, 0, s, sidx, didx,
                           n_rows, d, src, lds, dst, ldd);
    else
        hipLaunchKernelGGL((k_copy_rows<VEC, GL, kCopy>), grid, block, 0, s, sidx, didx, n_rows,
                           d, src, lds, dst, ldd);
    return hipGetLastError();
}

template <int VEC>
hipError_t copy_rows_v(int gl, int mode, const int32_t *sidx, const int32_t *didx,
                       int32_t n_rows, int32_t d, float *src, int32_t lds, float *dst,
                       int32_t ldd, hipStream_t s)
{
    switch (gl) {
    case 4: return copy_rows_t<VEC, 4>(mode, sidx, didx, n_rows, d, src, lds, dst, ldd, s);
    case 8: return copy_rows_t<VEC, 8>(mode, sidx, didx, n_rows, d, src, lds, dst, ldd, s);
    case 16: return copy_rows_t<VEC, 16>(mode, sidx, didx, n_rows, d, src, lds, dst, ldd, s);
    case 32: return copy_rows_t<VEC, 32>(mode, sidx, didx, n_rows, d, src, lds, dst, ldd, s);
    default: return copy_rows_t<VEC, 64>(mode, sidx, didx, n_rows, d, src, lds, dst, ldd, s);
    }
}

// Gathered floats one lane of the narrow kernel holds per batch.
constexpr int kNarrowLaneFloats = 64;
constexpr int narrow_nb(int gl, int nch, int vec)
{
    const int nb = kNarrowLaneFloats / (gl * nch * vec);
    return nb < 1 ? 1 : (nb > 4 ? 4 : nb);
}

template <int VEC, int GL, int NCH, bool TWO>
hipError_t spmm_narrow_t(const SpmmBlock *blocks, int32_t n_long, int32_t n_blocks,
                         const int32_t *rowptr, const int32_t *col, const float *val,
                         const float *src0, const float *src1, int32_t n_src0, int32_t d,
                         int32_t lds, SpmmOut out, const SpmmEpilogue *ep, hipStream_t s)
{
    constexpr int NB = narrow_nb(GL, NCH, VEC);
    const int64_t grid = n_long + ((int64_t)(n_blocks - n_long) + kSpmmWaves - 1) / kSpmmWaves;
    if (grid > 0x7fffffff)
        return hipErrorInvalidConfiguration;
    if constexpr (NCH == 1 && GL * VEC <= kNarrow) {
        if (ep) {
            const size_t lds_bytes = sizeof(float) * (size_t)d * ep->n2;
            hipLaunchKernelGGL((k_spmm_narrow<VEC, GL, NCH, NB, TWO, true>), dim3((unsigned)grid),
                               dim3(kSpmmThreads), lds_bytes, s, blocks, n_long, n_blocks, rowptr,
                               col, val, src0, src1, n_src0, d, lds, out, *ep);
            return hipGetLastError();
        }
    } else {
        if (ep)
            return hipErrorInvalidValue;
    }
    hipLaunchKernelGGL((k_spmm_narrow<VEC, GL, NCH, NB, TWO, false>), dim3((unsigned)grid),
                       dim3(kSpmmThreads), 0, s, blocks, n_long, n_blocks, rowptr, col, val, src0,
                       src1, n_src0, d, lds, out, SpmmEpilogue{});
    return hipGetLastError();
}

template <int VEC, int GL, int NCH, bool TWO>
hipError_t spmm_t(const SpmmBlock *blocks, int32_t n_blocks, const int32_t *rowptr,
                  const int32_t *col, const float *val, const float *src0, const float *src1,
                  int32_t n_src0, int32_t d, int32_t lds, SpmmOut out, hipStream_t s)
{
    hipLaunchKernelGGL((k_spmm<VEC, GL, NCH, TWO>), dim3((unsigned)n_blocks), dim3(kSpmmThreads),
                       0, s, blocks, rowptr, col, val, src0, src1, n_src0, d, lds, out);
    return hipGetLastError();
}

// A sliced pass (kSliceFloats-column slices dealt to the XCDs) of the narrow
// kernel over rows of d floats.
template <int VEC, bool TWO>
hipError_t spmm_sliced_t(const SpmmBlock *blocks, int32_t n_long, int32_t n_blocks,
                         const int32_t *rowptr, const int32_t *col, const float *val,
                         const float *src0, const float *src1, int32_t n_src0, int32_t d,
                         SpmmOut out, hipStream_t s)
{
    constexpr int GL = kSliceFloats / VEC;
    constexpr int NB = narrow_nb(GL, 1, VEC);
    const int64_t work = n_long + ((int64_t)(n_blocks - n_long) + kSpmmWaves - 1) / kSpmmWaves;
    const int64_t q = (d + kXcds * kSliceFloats - 1) / (kXcds * kSliceFloats);
    const int64_t grid = work * kXcds * q;
    if (grid > 0x7fffffff)
        return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((k_spmm_narrow<VEC, GL, 1, NB, TWO, false, true>), dim3((unsigned)grid),
                       dim3(kSpmmThreads), 0, s, blocks, n_long, n_blocks, rowptr, col, val, src0,
                       src1, n_src0, d, d, out, SpmmEpilogue{});
    return hipGetLastError();
}

#define DIGEST_SPMM_ARGS blocks, n_blocks, rowptr, col, val, src0, src1, n_src0, d, lds, out, s

template <int VEC, bool TWO>
hipError_t spmm_g(int gl, int nch, const SpmmBlock *blocks, int32_t n_blocks,
                  const int32_t *rowptr, const int32_t *col, const float *val, const float *src0,
                  const float *src1, int32_t n_src0, int32_t d, int32_t lds, SpmmOut out,
                  hipStream_t s)
{
    switch (gl) {
    case 4: return spmm_t<VEC, 4, 1, TWO>(DIGEST_SPMM_ARGS);
    case 8: return spmm_t<VEC, 8, 1, TWO>(DIGEST_SPMM_ARGS);
    case 16: return spmm_t<VEC, 16, 1, TWO>(DIGEST_SPMM_ARGS);
    case 32: return spmm_t<VEC, 32, 1, TWO>(DIGEST_SPMM_ARGS);
    default: break;
    }
    if constexpr (VEC == 4) {
        switch (nch) {
        case 1: return spmm_t<4, 64, 1, TWO>(DIGEST_SPMM_ARGS);
        case 2: return spmm_t<4, 64, 2, TWO>(DIGEST_SPMM_ARGS);
        default: return spmm_t<4, 64, 3, TWO>(DIGEST_SPMM_ARGS);
        }
    } else if constexpr (VEC == 2) {
        switch (nch) {
        case 1: return spmm_t<2, 64, 1, TWO>(DIGEST_SPMM_ARGS);
        case 2: return spmm_t<2, 64, 2, TWO>(DIGEST_SPMM_ARGS);
        case 3: return spmm_t<2, 64, 3, TWO>(DIGEST_SPMM_ARGS);
        case 4: return spmm_t<2, 64, 4, TWO>(DIGEST_SPMM_ARGS);
        default: return spmm_t<2, 64, 5, TWO>(DIGEST_SPMM_ARGS);
        }
    } else {
        switch (nch) {
        case 1: return spmm_t<1, 64, 1, TWO>(DIGEST_SPMM_ARGS);
        case 2: return spmm_t<1, 64, 2, TWO>(DIGEST_SPMM_ARGS);
        default: return spmm_t<1, 64, 4, TWO>(DIGEST_SPMM_ARGS);
        }
    }
}

template <bool TWO>
hipError_t spmm_v(int vec, int gl, int nch, const SpmmBlock *blocks, int32_t n_blocks,
                  const int32_t *rowptr, const int32_t *col, const float *val, const float *src0,
                  const float *src1, int32_t n_src0, int32_t d, int32_t lds, SpmmOut out,
                  hipStream_t s)
{
    switch (vec) {
    case 4: return spmm_g<4, TWO>(gl, nch, DIGEST_SPMM_ARGS);
    case 2: return spmm_g<2, TWO>(gl, nch, DIGEST_SPMM_ARGS);
    default: return spmm_g<1, TWO>(gl, nch, DIGEST_SPMM_ARGS);
    }
}

template <int BM, int BN, bool AT, bool BT, bool AMASK, bool BMASK, bool RELU, bool VA, bool VB>
hipError_t gemm_t(const GemmArgs &a, hipStream_t s)
{
    const int64_t gm = (a.M + BM - 1) / BM, gn = (a.N + BN - 1) / BN;
    const int64_t grid = gm * gn * a.splits;
    if (grid > 0x7fffffff)
        return hipErrorInvalidConfiguration;
    const int64_t split_stride = a.splits > 1 ? (int64_t)a.M * a.ldc : 0;
    hipLaunchKernelGGL((k_gemm<BM, BN, AT, BT, AMASK, BMASK, RELU, VA, VB>), dim3((unsigned)grid),
                       dim3(256), 0, s, a.M, a.N, a.K, a.kchunk, a.A, a.lda, a.a_mask, a.B, a.ldb,
                       a.b_mask, a.C, a.ldc, split_stride, (int32_t)gm, (int32_t)gn);
    return hipGetLastError();
}

template <bool AT, bool BT, bool AMASK, bool BMASK, bool RELU, bool VA, bool VB>
hipError_t gemm_tile(const GemmArgs &a, hipStream_t s)
{
    switch (a.tile) {
    case 1: return gemm_t<64, 128, AT, BT, AMASK, BMASK, RELU, VA, VB>(a, s);
    case 2: return gemm_t<128, 64, AT, BT, AMASK, BMASK, RELU, VA, VB>(a, s);
    case 3: return gemm_t<128, 128, AT, BT, AMASK, BMASK, RELU, VA, VB>(a, s);
    default: return gemm_t<64, 64, AT, BT, AMASK, BMASK, RELU, VA, VB>(a, s);
    }
}

// 16-byte operand loads need a 16-byte aligned base (and mask) and a leading
// dimension that keeps every row 16-byte aligned.
bool quad_ok(const float *p, const float *mask, int32_t ld)
{
    auto al = [](const float *q) { return q == nullptr || ((uintptr_t)q % 16) == 0; };
    return al(p) && al(mask) && ld % 4 == 0;
}

template <bool AT, bool BT, bool AMASK, bool BMASK, bool RELU>
hipError_t gemm_q(const GemmArgs &a, hipStream_t s)
{
    const bool va = quad_ok(a.A, a.a_mask, a.lda), vb = quad_ok(a.B, a.b_mask, a.ldb);
    if (va && vb)
        return gemm_tile<AT, BT, AMASK, BMASK, RELU, true, true>(a, s);
    if (va)
        return gemm_tile<AT, BT, AMASK, BMASK, RELU, true, false>(a, s);
    if (vb)
        return gemm_tile<AT, BT, AMASK, BMASK, RELU, false, true>(a, s);
    return gemm_tile<AT, BT, AMASK, BMASK, RELU, false, false>(a, s);
}

}  // namespace

namespace {

hipError_t move_rows(int mode, const int32_t *sidx, const int32_t *didx, int32_t n_rows,
                     int32_t d, float *src, float *dst, hipStream_t s, int32_t lds = 0,
                     int32_t ldd = 0)
{
    if (n_rows <= 0 || d <= 0)
        return hipSuccess;
    lds = lds > 0 ? lds : d;
    ldd = ldd > 0 ? ldd : d;
    if (lds < d || ldd < d)
        return hipErrorInvalidValue;
    // the widest vector that the width, both strides and both bases allow
    int vec = pick_vec(d, src, dst);
    while (vec > 1 && (lds % vec || ldd % vec))
        vec /= 2;
    const int gl = pick_group(d / vec);
    switch (vec) {
    case 4: return copy_rows_v<4>(gl, mode, sidx, didx, n_rows, d, src, lds, dst, ldd, s);
    case 2: return copy_rows_v<2>(gl, mode, sidx, didx, n_rows, d, src, lds, dst, ldd, s);
    default: return copy_rows_v<1>(gl, mode, sidx, didx, n_rows, d, src, lds, dst, ldd, s);
    }
}

}  // namespace

hipError_t launch_copy_rows(const int32_t *sidx, const int32_t *didx, int32_t n_rows,
                            int32_t d, const float *src, float *dst, hipStream_t s,
                            int32_t lds, int32_t ldd)
{
    return move_rows(kCopy, sidx, didx, n_rows, d, const_cast<float *>(src), dst, s, lds, ldd);
}

hipError_t launch_add_rows(const int32_t *sidx, const int32_t *didx, int32_t n_rows, int32_t d,
                           const float *src, float *dst, hipStream_t s)
{
    return move_rows(kAdd, sidx, didx, n_rows, d, const_cast<float *>(src), dst, s);
}

hipError_t launch_add_clear_rows(const int32_t *sidx, const int32_t *didx, int32_t n_rows,
                                 int32_t d, float *src, float *dst, hipStream_t s)
{
    return move_rows(kAddClear, sidx, didx, n_rows, d, src, dst, s);
}

bool spmm_epilogue_ok(int32_t d, int32_t n2, const float *out2)
{
    return d >= 1 && d <= kNarrow && n2 >= 4 && n2 % 4 == 0 &&
           (size_t)d * n2 * sizeof(float) <= 64 * 1024 && ((uintptr_t)out2 % 16) == 0;
}

bool spmm_sliced_ok(int32_t d, const float *src0, const float *src1, const float *out0)
{
    return d > 0 && pick_vec(d, src0, out0) >= 2 && (!src1 || pick_vec(d, src1, nullptr) >= 2);
}

namespace {

template <int VEC, bool TWO>
hipError_t spmm_tier_t(const SpmmBlock *blocks, int32_t n_long, const int32_t *rowptr,
                       const int32_t *col, const float *val, const float *src0,
                       const float *src1, int32_t n_src0, int32_t n_rows, int32_t d,
                       SpmmOut out, hipStream_t s)
{
    // the long rows: whole workgroups, as in the unsliced kernel's plan
    if (n_long > 0)
        if (hipError_t e = spmm_sliced_t<VEC, TWO>(blocks, n_long, n_long, rowptr, col, val,
                                                   src0, src1, n_src0, d, out, s))
            return e;
    // the short rows: strips of rows per wave, about four rounds of waves
    // of the whole chip (256 CUs x 16 waves)
    constexpr int G = kWave / (kSliceFloats / VEC);
    const int64_t q = (d + kXcds * kSliceFloats - 1) / (kXcds * kSliceFloats);
    int64_t rpw = kXcds * q * (int64_t)n_rows / (256 * 16 * 4);
    rpw = std::min<int64_t>(256, std::max<int64_t>(G, (rpw + G - 1) / G * G));
    const int64_t waves = (n_rows + rpw - 1) / rpw;
    const int64_t grid = (waves + 3) / 4 * kXcds * q;
    if (grid > 0x7fffffff)
        return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((k_spmm_tier<VEC, TWO>), dim3((unsigned)grid), dim3(256), 0, s, rowptr,
                       col, val, src0, src1, n_src0, n_rows, d, (int32_t)rpw, out);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_spmm_sliced(const SpmmBlock *blocks, int32_t n_blocks, int32_t n_long,
                              const int32_t *rowptr, const int32_t *col, const float *val,
                              int64_t nnz, const float *src0, const float *src1, int32_t n_src0,
                              int32_t n_rows, int32_t d, float *out0, bool acc, hipStream_t s)
{
    if (n_rows <= 0 || d <= 0)
        return hipSuccess;
    if (n_long < 0 || n_long > n_blocks || nnz < 1)
        return hipErrorInvalidValue;   // padding entries reread entry 0
    const SpmmOut out{out0, nullptr, INT32_MAX, false, SpmmRank1{}, d, acc, d, true};
    // every slice starts on a multiple of kSliceFloats, so the vector width
    // of the whole row is the slices' too
    int vec = pick_vec(d, src0, out0);
    if (src1 && pick_vec(d, src1, nullptr) < vec)
        vec = pick_vec(d, src1, nullptr);
#define DIGEST_TIER(V, T)                                                                       \
    return spmm_tier_t<V, T>(blocks, n_long, rowptr, col, val, src0, src1, n_src0, n_rows, d,   \
                             out, s)
    if (vec == 4) {
        if (src1)
            DIGEST_TIER(4, true);
        DIGEST_TIER(4, false);
    }
    if (vec == 2) {
        if (src1)
            DIGEST_TIER(2, true);
        DIGEST_TIER(2, false);
    }
#undef DIGEST_TIER
    return hipErrorInvalidValue;   // rows of odd width take the unsliced kernel
}

hipError_t launch_spmm(const SpmmBlock *blocks, int32_t n_blocks, int32_t n_long,
                       const int32_t *rowptr, const int32_t *col, const float *val,
                       const float *src0, const float *src1, int32_t n_src0, int32_t d,
                       float *out0, hipStream_t s, const SpmmEpilogue *ep, float *out1,
                       int32_t n_out0, bool relu, const SpmmRank1 *r1, bool acc, int32_t lds,
                       int32_t out_ld, int32_t out_w)
{
    lds = lds > 0 ? lds : d;
    out_ld = out_ld > 0 ? out_ld : d;
    out_w = out_w > 0 ? out_w : d;
    if (lds < d || out_w > d || out_ld < out_w)
        return hipErrorInvalidValue;
    if (ep && (!spmm_epilogue_ok(d, ep->n2, ep->out2) ||
               (ep->out3 && !spmm_epilogue_ok(d, ep->n2, ep->out3))))
        return hipErrorInvalidValue;
    if (n_out0 < 0 || (n_out0 != INT32_MAX && !out1))
        return hipErrorInvalidValue;
    if (n_blocks <= 0 || d <= 0)
        return hipSuccess;
    if ((relu || (r1 && r1->a)) && ep)
        return hipErrorInvalidValue;   // the epilogue reads the stored row back
    if (r1 && r1->a && (!r1->x || (r1->ny > 0 && !r1->y)))
        return hipErrorInvalidValue;
    // the gather's vector width follows the sources (width, stride and
    // alignment); the stores use it where the output's rows allow, else go
    // column by column
    int vec = pick_vec(d, src0, nullptr);
    if (lds % vec)
        vec = lds % 2 ? 1 : std::min(vec, 2);
    if (src1 && pick_vec(d, src1, nullptr) < vec)
        vec = pick_vec(d, src1, nullptr);
    const bool vst = out_ld % vec == 0 && pick_vec(vec, out0, out1) >= vec;
    const SpmmOut out{out0, out1, n_out0, relu, r1 ? *r1 : SpmmRank1{}, out_ld, acc, out_w, vst};
    const int dv = d / vec;
    const int gl = pick_group(dv);
    // rows of at most kNarrowWide floats: the row-per-lane-group kernel, in
    // groups of at most 16 lanes holding NCH vectors each; wider rows: the
    // row-per-wave kernel
    const bool narrow = d <= kNarrowWide;
    if (ep && d > kNarrow)
        return hipErrorInvalidValue;
    if (narrow) {   // narrow rows: a row per lane group
        if (n_long < 0 || n_long > n_blocks)
            return hipErrorInvalidValue;
        const int ngl = gl > 16 ? 16 : gl;
        const int nnch = (dv + ngl - 1) / ngl;
#define DIGEST_NARROW(V, L, C)                                                                   \
    return src1 ? spmm_narrow_t<V, L, C, true>(blocks, n_long, n_blocks, rowptr, col, val,      \
                                               src0, src1, n_src0, d, lds, out, ep, s)         \
                : spmm_narrow_t<V, L, C, false>(blocks, n_long, n_blocks, rowptr, col, val,     \
                                                src0, src1, n_src0, d, lds, out, ep, s)
        if (vec == 4) {   // dv <= 16
            if (ngl == 4) DIGEST_NARROW(4, 4, 1);
            if (ngl == 8) DIGEST_NARROW(4, 8, 1);
            DIGEST_NARROW(4, 16, 1);
        } else if (vec == 2) {   // dv <= 32
            if (ngl == 4) DIGEST_NARROW(2, 4, 1);
            if (ngl == 8) DIGEST_NARROW(2, 8, 1);
            if (nnch <= 1) DIGEST_NARROW(2, 16, 1);
            DIGEST_NARROW(2, 16, 2);
        } else {   // dv <= 64
            if (ngl == 4) DIGEST_NARROW(1, 4, 1);
            if (ngl == 8) DIGEST_NARROW(1, 8, 1);
            if (nnch <= 1) DIGEST_NARROW(1, 16, 1);
            if (nnch <= 2) DIGEST_NARROW(1, 16, 2);
            if (nnch <= 3) DIGEST_NARROW(1, 16, 3);
            DIGEST_NARROW(1, 16, 4);
        }
#undef DIGEST_NARROW
    }
    const int max_nch = vec == 4 ? 3 : (vec == 2 ? 5 : 4);
    int nch = (dv + kWave - 1) / kWave;
    if (vec == 1 && nch == 3)
        nch = 4;
    nch = nch < 1 ? 1 : (nch > max_nch ? max_nch : nch);
    if (src1)
        return spmm_v<true>(vec, gl, nch, DIGEST_SPMM_ARGS);
    return spmm_v<false>(vec, gl, nch, DIGEST_SPMM_ARGS);
}

hipError_t launch_gemm(const GemmArgs &a, hipStream_t s)
{
    if (a.M <= 0 || a.N <= 0)
        return hipSuccess;
    if (a.tile < 0 || a.tile > 3)
        return hipErrorInvalidValue;
    if (a.splits > 1 && a.kchunk % kGemmBK != 0)
        return hipErrorInvalidValue;   // split starts must stay quad aligned
    const bool am = a.a_mask != nullptr, bm = a.b_mask != nullptr;
    // The instantiations the layer needs:
    //   forward      A.B        (+ReLU epilogue)
    //   dW           A^T.B      (B optionally masked)
    //   D.W^T        A.B^T      (A optionally masked)
    if (!a.a_trans && !a.b_trans && !am && !bm)
        return a.relu ? gemm_q<false, false, false, false, true>(a, s)
                      : gemm_q<false, false, false, false, false>(a, s);
    if (a.a_trans && !a.b_trans && !am && !a.relu)
        return bm ? gemm_q<true, false, false, true, false>(a, s)
                  : gemm_q<true, false, false, false, false>(a, s);
    if (!a.a_trans && a.b_trans && !bm && !a.relu)
        return am ? gemm_q<false, true, true, false, false>(a, s)
                  : gemm_q<false, true, false, false, false>(a, s);
    return hipErrorInvalidValue;
}

hipError_t launch_relu_mask(int64_t n, int32_t d, const float *g, int32_t ldg, const float *h,
                            int32_t ldh, float *out, int32_t ldo, hipStream_t s)
{
    if (n <= 0 || d <= 0)
        return hipSuccess;
    auto al = [](const void *q) { return ((uintptr_t)q % 16) == 0; };
    const bool v4 = d % 4 == 0 && ldg % 4 == 0 && ldh % 4 == 0 && ldo % 4 == 0 && al(g) &&
                    al(h) && al(out);
    const int64_t items = n * (v4 ? d / 4 : d);
    const int64_t grid = (items + 255) / 256;
    if (grid > 0x7fffffff)
        return hipErrorInvalidConfiguration;
    if (v4)
        hipLaunchKernelGGL((k_relu_mask<4>), dim3((unsigned)grid), dim3(256), 0, s, n, d, g, ldg,
                           h, ldh, out, ldo);
    else
        hipLaunchKernelGGL((k_relu_mask<1>), dim3((unsigned)grid), dim3(256), 0, s, n, d, g, ldg,
                           h, ldh, out, ldo);
    return hipGetLastError();
}

hipError_t launch_transpose(int32_t rows, int32_t cols, const float *src, float *dst,
                            hipStream_t s)
{
    if (rows <= 0 || cols <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(k_transpose,
                       dim3((unsigned)((cols + 31) / 32), (unsigned)((rows + 31) / 32)),
                       dim3(256), 0, s, rows, cols, src, dst);
    return hipGetLastError();
}

bool spmm_gemm_ok(int32_t d, int32_t lds, int32_t ld_ah, const float *src0, const float *src1,
                  const float *ah, const float *pre)
{
    constexpr int vec = 4;
    auto al = [&](const float *q) { return q == nullptr || ((uintptr_t)q % (4 * vec)) == 0; };
    return d >= kFuseMinWidth && d <= kFuseMaxWidth && lds >= d && ld_ah >= d &&
           lds % vec == 0 &&
           ld_ah % vec == 0 && al(src0) && al(src1) && al(ah) && al(pre);
}

hipError_t launch_spmm_gemm(int32_t n_rows, const int32_t *rowptr, const int32_t *col,
                            const float *val, const uint8_t *order, const float *src0,
                            const float *src1, int32_t n_src0, int32_t lds, int32_t d,
                            float *ah, const float *pre, int32_t ld_ah, const float *W,
                            int32_t N, float *C, int32_t ldc, bool relu, hipStream_t s)
{
    if (n_rows <= 0 || N <= 0)
        return hipSuccess;
    if (!pre || !spmm_gemm_ok(d, lds, ld_ah, src0, src1, ah, pre) || ldc < N)
        return hipErrorInvalidValue;
    const bool two = src1 != nullptr;
    const unsigned grid = (unsigned)((n_rows + kFuseRows - 1) / kFuseRows);
#define DIGEST_FUSE_ARGS                                                                      \
    dim3(grid), dim3(kFuseThreads), 0, s, n_rows, rowptr, col, val, order, src0, src1, n_src0, \
        lds, d, ah, pre, ld_ah, W, N, C, ldc, relu
    if (d <= 2 * kWave) {   // two lane groups of 32, float4 each, split each row
        if (two)
            hipLaunchKernelGGL((k_spmm_gemm<4, 2, true>), DIGEST_FUSE_ARGS);
        else
            hipLaunchKernelGGL((k_spmm_gemm<4, 2, false>), DIGEST_FUSE_ARGS);
    } else {
        if (two)
            hipLaunchKernelGGL((k_spmm_gemm<4, 1, true>), DIGEST_FUSE_ARGS);
        else
            hipLaunchKernelGGL((k_spmm_gemm<4, 1, false>), DIGEST_FUSE_ARGS);
    }
#undef DIGEST_FUSE_ARGS
    return hipGetLastError();
}

hipError_t launch_splitk_reduce(const float *part, int32_t splits, int64_t count, float *out,
                                hipStream_t s)
{
    if (count <= 0)
        return hipSuccess;
    if (splits >= 64 && count < 64 * 1024) {
        const int64_t blocks = (count + 7) / 8;
        hipLaunchKernelGGL(k_splitk_reduce_wide, dim3((unsigned)blocks), dim3(256), 0, s, part,
                           splits, count, out);
    } else {
        const int64_t blocks = (count + 255) / 256;
        hipLaunchKernelGGL(k_splitk_reduce, dim3((unsigned)blocks), dim3(256), 0, s, part, splits,
                           count, out);
    }
    return hipGetLastError();
}

// Lanes per row of the loss head and class slots per lane: up to 128
// classes every logit of a row sits in a register of its group; wider rows
// take a wave each.
int loss_group(int32_t C) { return C <= 8 ? 8 : (C <= 64 ? 16 : (C <= 128 ? 32 : 64)); }
int loss_slots(int32_t C) { return (C + loss_group(C) - 1) / loss_group(C); }

int32_t softmax_xent_rows_per_block(int32_t C)
{
    return (kLossThreads / kWave) * (kWave / loss_group(C));
}

int32_t softmax_xent_blocks(int32_t n, int32_t C)
{
    const int32_t rows_per_block = softmax_xent_rows_per_block(C);
    return std::max<int32_t>(1, (n + rows_per_block - 1) / rows_per_block);
}

hipError_t launch_softmax_xent(const float *logits, const int32_t *labels, int32_t n,
                               int32_t C, float *dlogits, float *block_loss, hipStream_t s)
{
    if (C <= 0)
        return hipErrorInvalidValue;
    const int32_t nb = softmax_xent_blocks(n, C);
    const float inv_n = n > 0 ? 1.0f / (float)n : 0.f;
#define DIGEST_LOSS(GL, NJ)                                                                     \
    hipLaunchKernelGGL((k_softmax_xent<GL, NJ>), dim3((unsigned)nb), dim3(kLossThreads), 0, s,  \
                       logits, labels, n, C, inv_n, dlogits, block_loss)
    const int gl = loss_group(C), nj = loss_slots(C);
    if (gl == 8)
        DIGEST_LOSS(8, 1);
    else if (gl == 16 && nj == 1)
        DIGEST_LOSS(16, 1);
    else if (gl == 16 && nj == 2)
        DIGEST_LOSS(16, 2);
    else if (gl == 16 && nj == 3)
        DIGEST_LOSS(16, 3);
    else if (gl == 16)
        DIGEST_LOSS(16, 4);
    else if (gl == 32 && nj == 3)
        DIGEST_LOSS(32, 3);
    else if (gl == 32)
        DIGEST_LOSS(32, 4);
    else
        hipLaunchKernelGGL(k_softmax_xent_wide, dim3((unsigned)nb), dim3(kLossThreads), 0, s,
                           logits, labels, n, C, inv_n, dlogits, block_loss);
#undef DIGEST_LOSS
    return hipGetLastError();
}

hipError_t launch_loss_mean(const float *block_loss, int32_t n, int32_t C, float *loss,
                            hipStream_t s)
{
    if (C <= 0)
        return hipErrorInvalidValue;
    const int32_t nb = softmax_xent_blocks(n, C);
    const float inv_n = n > 0 ? 1.0f / (float)n : 0.f;
    hipLaunchKernelGGL(k_loss_reduce, dim3(1), dim3(kLossReduceThreads), 0, s, block_loss, nb,
                       inv_n, loss);
    return hipGetLastError();
}


namespace {

// Blocks of a persistent launch: enough for every tile, at most what the
// chip holds at once given the block's LDS (256 CUs, 160 KB each, at most 8
// blocks per CU).
int64_t persistent_blocks(int64_t tiles_per_block_work, size_t lds)
{
    const int64_t per_cu = std::max<int64_t>(1, std::min<int64_t>(8, (160 * 1024) / std::max<size_t>(lds, 1)));
    return std::max<int64_t>(1, std::min<int64_t>(tiles_per_block_work, 256 * per_cu));
}

}  // namespace

size_t narrow_n_lds(int32_t K, int32_t N)
{
    const int nb = (N + 15) / 16;
    return sizeof(float) * (size_t)16 * nb * narrow_n_stride(K);
}

hipError_t launch_narrow_n(int32_t M, int32_t m0, int32_t K, int32_t N, const float *A0,
                           const float *A1, int32_t lda, const float *B, float *C, int32_t ldc,
                           bool relu, hipStream_t s, int32_t lda1)
{
    if (M <= 0 || N <= 0)
        return hipSuccess;
    if (N > kNarrowN || K <= 0 || narrow_n_lds(K, N) > kNarrowNLds)
        return hipErrorInvalidValue;
    lda1 = lda1 > 0 ? lda1 : lda;
    const bool v4 = K % 4 == 0 && lda % 4 == 0 && lda1 % 4 == 0 && ((uintptr_t)A0 % 16) == 0 &&
                    (A1 == nullptr || ((uintptr_t)A1 % 16) == 0);
    const size_t lds = narrow_n_lds(K, N);
    const int64_t blocks = persistent_blocks((((int64_t)M + 15) / 16 + 3) / 4, lds);
    const int nb = (N + 15) / 16;
#define DIGEST_NN(V, NB)                                                                       \
    hipLaunchKernelGGL((k_narrow_n<V, NB>), dim3((unsigned)blocks), dim3(256), lds, s, M, m0, K, \
                       N, A0, A1, lda, lda1, B, C, ldc, relu)
    if (v4) {
        switch (nb) {
        case 1: DIGEST_NN(true, 1); break;
        case 2: DIGEST_NN(true, 2); break;
        case 3: DIGEST_NN(true, 3); break;
        default: DIGEST_NN(true, 4); break;
        }
    } else {
        switch (nb) {
        case 1: DIGEST_NN(false, 1); break;
        case 2: DIGEST_NN(false, 2); break;
        case 3: DIGEST_NN(false, 3); break;
        default: DIGEST_NN(false, 4); break;
        }
    }
#undef DIGEST_NN
    return hipGetLastError();
}

namespace {

// LDS row stride of W^T in k_times_wt (at least N, = 16 mod 64) and its MFMA
// k-steps.
int32_t times_wt_stride(int32_t N)
{
    int32_t bs = (N + 15) / 16 * 16;
    while (bs % 64 != 16)
        bs += 16;
    return bs;
}

int times_wt_steps(int32_t K) { return K <= 32 ? 8 : (K <= 48 ? 12 : 16); }

}  // namespace

size_t times_wt_lds(int32_t K, int32_t N)
{
    return sizeof(float) * (size_t)(4 * times_wt_steps(K)) * times_wt_stride(N);
}

hipError_t launch_times_wt(int32_t M, int32_t N, int32_t K, const float *A, int32_t lda,
                           const float *W, float *C, int32_t ldc, hipStream_t s)
{
    if (M <= 0 || N <= 0)
        return hipSuccess;
    if (K <= kNarrow || K > kTimesWtK || times_wt_lds(K, N) > kNarrowNLds)
        return hipErrorInvalidValue;
    const int32_t bs = times_wt_stride(N);
    const int ks = times_wt_steps(K);
    const size_t lds = times_wt_lds(K, N);
    const int64_t blocks = persistent_blocks((((int64_t)M + 15) / 16 + 3) / 4, lds);
    if (ks == 8)
        hipLaunchKernelGGL((k_times_wt<8>), dim3((unsigned)blocks), dim3(256), lds, s, M, N, K, A,
                           lda, W, C, ldc, bs);
    else if (ks == 12)
        hipLaunchKernelGGL((k_times_wt<12>), dim3((unsigned)blocks), dim3(256), lds, s, M, N, K,
                           A, lda, W, C, ldc, bs);
    else
        hipLaunchKernelGGL((k_times_wt<16>), dim3((unsigned)blocks), dim3(256), lds, s, M, N, K,
                           A, lda, W, C, ldc, bs);
    return hipGetLastError();
}

hipError_t launch_narrow_k(int32_t M, int32_t N, int32_t K, const float *A, int32_t lda,
                           const float *W, float *C, int32_t ldc, hipStream_t s)
{
    if (M <= 0 || N <= 0)
        return hipSuccess;
    if (K <= 0 || K > kNarrow)
        return hipErrorInvalidValue;
    // per column slice: enough waves to give each at least kNarrowKRows
    // rows, at most 4096 in all
    const int64_t slices = (N + 255) / 256;
    const int64_t row_groups = ((int64_t)M + kNarrowKRows - 1) / kNarrowKRows;
    const int64_t per_slice = std::min<int64_t>(row_groups, std::max<int64_t>(1, 4096 / slices));
    const int64_t blocks = (per_slice * slices + 3) / 4;   // the kernel idles any surplus wave
    if (blocks * 4 * 64 > INT32_MAX)
        return hipErrorInvalidValue;
    const bool vec_out = N % 4 == 0 && ldc % 4 == 0 && ((uintptr_t)C % 16) == 0;
    if (K <= 8)
        hipLaunchKernelGGL((k_narrow_k<8>), dim3((unsigned)blocks), dim3(256), 0, s, M, N, K, A,
                           lda, W, C, ldc, vec_out, (int32_t)slices);
    else
        hipLaunchKernelGGL((k_narrow_k<16>), dim3((unsigned)blocks), dim3(256), 0, s, M, N, K, A,
                           lda, W, C, ldc, vec_out, (int32_t)slices);
    return hipGetLastError();
}

hipError_t launch_dw_narrow(int32_t R, int32_t m0, int32_t F, int32_t N, const float *H0,
                            const float *H1, int32_t ldh, const float *G, int32_t ldg,
                            int32_t chunk, int32_t splits, float *part, hipStream_t s,
                            int32_t ldh1)
{
    ldh1 = ldh1 > 0 ? ldh1 : ldh;
    if (F <= 0 || N <= 0)
        return hipSuccess;
    if (N > kNarrow || splits < 1 || chunk < 1)
        return hipErrorInvalidValue;
    const dim3 grid((unsigned)((F + 63) / 64), (unsigned)((splits + 3) / 4));
    hipLaunchKernelGGL(k_dw_narrow, grid, dim3(256), 0, s, R, m0, F, N, H0, H1, ldh, ldh1, G, ldg,
                       chunk,
                       splits, part);
    return hipGetLastError();
}

hipError_t launch_sgd_average(float *w, const GradList &g, int32_t n, int64_t count, float lr,
                              hipStream_t s)
{
    if (n < 1 || n > kMaxAverage || count < 0)
        return hipErrorInvalidValue;
    if (count == 0)
        return hipSuccess;
    const int64_t blocks = (count + 255) / 256;
    if (blocks > 0x7fffffff)
        return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(k_sgd_average, dim3((unsigned)blocks), dim3(256), 0, s, w, g, n, count, lr);
    return hipGetLastError();
}

hipError_t static_scratch(float **ptr)
{
    // device address of `scratch` per device, looked up once per device with
    // that device current (the caller's current device)
    static std::mutex mu;
    static std::vector<float *> addr;
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return e;
    if (dev < 0)
        return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if ((size_t)dev >= addr.size())
        addr.resize((size_t)dev + 1, nullptr);
    if (!addr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess)
            return e;
        if (!p)
            return hipErrorInvalidSymbol;
        addr[dev] = static_cast<float *>(p);
    }
    *ptr = addr[dev];
    return hipSuccess;
}

hipError_t launch_fill_zero(float *p, int64_t count, hipStream_t s)
{
    if (count <= 0)
        return hipSuccess;
    const int64_t blocks = (count + 255) / 256;
    if (blocks > 0x7fffffff)
        return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(k_fill_zero, dim3((unsigned)blocks), dim3(256), 0, s, p, count);
    return hipGetLastError();
}

hipError_t launch_gat_softmax(int32_t n_rows, const int32_t *rowptr, const int32_t *col,
                              const float *s, float slope, float *alpha, hipStream_t st)
{
    if (n_rows <= 0)
        return hipSuccess;
    const int64_t blocks = ((int64_t)n_rows + 3) / 4;   // a wave per row
    if (blocks > 0x7fffffff)
        return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(k_gat_softmax, dim3((unsigned)blocks), dim3(256), 0, st, n_rows, rowptr,
                       col, s, slope, alpha);
    return hipGetLastError();
}

namespace {

template <int VEC, int GL, int NCH, int U = 2>
hipError_t gat_edge_grad_t(const SpmmBlock *blocks, int32_t n_blocks, int32_t d,
                           const int32_t *rowptr, const int32_t *col, const float *alpha,
                           const float *s, const float *z, const float *h_out,
                           const float *dh_out, bool relu, float slope, float *dO, float *dpre,
                           float *g2, hipStream_t st)
{
    hipLaunchKernelGGL((k_gat_edge_grad<VEC, GL, NCH, U>), dim3((unsigned)n_blocks),
                       dim3(kSpmmThreads), 0, st, blocks, d, rowptr, col, alpha, s, z, h_out,
                       dh_out, relu, slope, dO, dpre, g2);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gat_edge_grad(const SpmmBlock *blocks, int32_t n_blocks, int32_t d,
                                const int32_t *rowptr, const int32_t *col, const float *alpha,
                                const float *s, const float *z, const float *h_out,
                                const float *dh_out, bool relu, float slope, float *dO,
                                float *dpre, float *g2, hipStream_t st)
{
    if (n_blocks <= 0)
        return hipSuccess;
    if (d < 1 || d > kGatMaxWidth)
        return hipErrorInvalidValue;
    // vectors of 4/2/1 floats as width and alignment allow; groups of at
    // most 16 lanes (at least four entries per wave step) up to 128 vectors
    // per row, whole-wave groups beyond; up to 8 vectors per lane
    int vec = 1;
    auto al = [](const void *q, uintptr_t n) { return ((uintptr_t)q % n) == 0; };
    if (d % 4 == 0 && al(z, 16) && al(h_out, 16) && al(dh_out, 16) && al(dO, 16))
        vec = 4;
    else if (d % 2 == 0 && al(z, 8) && al(h_out, 8) && al(dh_out, 8) && al(dO, 8))
        vec = 2;
    const int dv = d / vec;
    const int gl = dv <= 4 ? 4 : (dv <= 8 ? 8 : (dv <= 128 ? 16 : 64));
    const int nch = (dv + gl - 1) / gl;
#define DIGEST_GEG(V, L, C)                                                                     \
    return gat_edge_grad_t<V, L, C>(blocks, n_blocks, d, rowptr, col, alpha, s, z, h_out,       \
                                    dh_out, relu, slope, dO, dpre, g2, st)
#define DIGEST_GEG_V(V)                                                                         \
    do {                                                                                        \
        if (gl == 4) DIGEST_GEG(V, 4, 1);                                                       \
        if (gl == 8) DIGEST_GEG(V, 8, 1);                                                       \
        if (gl == 16) {                                                                         \
            if (nch <= 1) DIGEST_GEG(V, 16, 1);                                                 \
            if (nch <= 2) DIGEST_GEG(V, 16, 2);                                                 \
            if (nch <= 4) DIGEST_GEG(V, 16, 4);                                                 \
            DIGEST_GEG(V, 16, 8);                                                               \
        }                                                                                       \
        if (nch <= 4) DIGEST_GEG(V, 64, 4);                                                     \
        DIGEST_GEG(V, 64, 8);                                                                   \
    } while (0)
    if (vec == 4)
        DIGEST_GEG_V(4);
    if (vec == 2)
        DIGEST_GEG_V(2);
    DIGEST_GEG_V(1);
#undef DIGEST_GEG_V
#undef DIGEST_GEG
}

hipError_t launch_gather_perm2(int64_t n, const int32_t *perm, const float *a, const float *b,
                               float *a_t, float *b_t, hipStream_t st)
{
    if (n <= 0)
        return hipSuccess;
    const int64_t blocks = (n + 255) / 256;
    if (blocks > 0x7fffffff)
        return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(k_gather_perm2, dim3((unsigned)blocks), dim3(256), 0, st, n, perm, a, b,
                       a_t, b_t);
    return hipGetLastError();
}

hipError_t launch_gat_score_cols(int64_t R, int32_t n_own, const float *ds_src, float *g2,
                                 hipStream_t st)
{
    if (R <= 0)
        return hipSuccess;
    const int64_t blocks = (R + 255) / 256;
    if (blocks > 0x7fffffff)
        return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(k_gat_score_cols, dim3((unsigned)blocks), dim3(256), 0, st, R, n_own,
                       ds_src, g2);
    return hipGetLastError();
}

}  // namespace digest
