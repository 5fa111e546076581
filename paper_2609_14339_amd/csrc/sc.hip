// Spectral corrector for gfx950 (paper Sec. 3.2; Alg. 1; App. E).
//
// sc_build_prior: anchor EMA, then the top-r SVD of the EMA by randomised
// block subspace iteration (MFMA tall-skinny passes over M, CholeskyQR2 with an
// fp64 Gram and an fp64 Cholesky in LDS), Rayleigh-Ritz by one-sided Jacobi in
// LDS, and the soft filter.
// sc_correct: T = G V (MFMA, split-K), X = U^T T, X_f = d X d, P = U X_f, then
// one fused pass G_proj = alpha G + (1 - alpha) P V^T.
#include "common.h"

#include <cstdlib>
#include <cstring>
#include "sc_pass.h"
#include "sc_blend.h"
#include "sc_chol.h"
#include "sc_orth.h"

#include <algorithm>
#include <utility>
#include <vector>

namespace acsc {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(short)))) short bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef float nf4 __attribute__((ext_vector_type(4)));
typedef unsigned int nu4 __attribute__((ext_vector_type(4)));

constexpr int kKMax = SC_KMAX;
constexpr int kBM = 64;   // rows of the output per workgroup in the tall GEMM
constexpr int kBK = 32;   // depth of one K step
constexpr int kNTMax = kKMax / 16;
// Singular values of the prior at or below this fraction of the largest are
// returned as zero (numerical rank of an fp32 subspace iteration).
constexpr double kRankCutoff = 1e-5;
// Largest k whose Rayleigh-Ritz Jacobi runs in fp64 (beyond it: fp32, whose
// columns take half the LDS)
constexpr int kJacobiF64MaxK = 128;

__host__ __device__ inline int64_t round_up(int64_t a, int64_t b) { return (a + b - 1) / b * b; }

// A launch works on up to kMaxBatch matrices: blockIdx.z selects the job,
// whose pointers and sizes travel by value in the kernel arguments.
constexpr int kMaxBatch = 16;
template <class Job>
struct Batch {
    int count;
    Job j[kMaxBatch];
};
__host__ __device__ inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// ---------------------------------------------------------------------------
// Element conversion helpers.  "CT" is the compute element type of the matrix
// cores: uint16_t (bf16 bits) or float.
// ---------------------------------------------------------------------------
template <typename T>
__device__ __forceinline__ float to_f32(T v);
template <>
__device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <>
__device__ __forceinline__ float to_f32<uint16_t>(uint16_t v) { return bf16_to_f32(v); }

template <typename T>
__device__ __forceinline__ T from_f32(float v);
template <>
__device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <>
__device__ __forceinline__ uint16_t from_f32<uint16_t>(float v) { return f32_to_bf16(v); }

template <typename T>
__device__ __forceinline__ T cvt_ct(float v) { return from_f32<T>(v); }

// ---------------------------------------------------------------------------
// Tall-skinny GEMM with split-K:
//   C[s][i, c] = sum_{k in split s} opA[i, k] * B[k, c]
// opA = A (A is [M, K] row-major) or A^T (A is stored [K, M] row-major).
// B is fp32 [K, ldb]; columns >= nvalid read as zero.  C gets `nwrite`
// columns.  With one split the result goes straight to C (which may then be
// A itself for a square right factor: each workgroup reads all of its rows
// before it writes them).
// A of type float runs on v_mfma_f32_16x16x4f32, bf16 on
// v_mfma_f32_16x16x32_bf16; B is converted to A's type in LDS.
// ---------------------------------------------------------------------------
template <typename TA>
struct GemmLds;
template <>
struct GemmLds<uint16_t> {
    static constexpr int APITCH = kBK + 8;   // 80-byte rows keep 16-byte alignment
    static constexpr int BPITCH = kBK + 8;
};
template <>
struct GemmLds<float> {
    static constexpr int APITCH = kBK + 1;
    static constexpr int BPITCH = kBK + 1;
};

template <typename TA, typename TO>
struct GemmJob {
    const TA *A;
    int64_t lda;
    const float *B;
    int64_t ldb;
    TO *C;
    int64_t ldc, split_stride;
    int M, K, nvalid, nwrite, kchunk, splits;
    uint16_t *Ct16;
    int64_t ldct;
};

template <typename TA, bool TRANS, typename TO>
__global__ __launch_bounds__(256) void gemm_tall_kernel(const Batch<GemmJob<TA, TO>> jb)
{
    const GemmJob<TA, TO> &J = jb.j[blockIdx.z];
    if (static_cast<int>(blockIdx.y) >= J.splits || static_cast<int>(blockIdx.x) * kBM >= J.M)
        return;
    const TA *A = J.A;
    const int64_t lda = J.lda;
    const float *B = J.B;
    const int64_t ldb = J.ldb;
    TO *C = J.C;
    const int64_t ldc = J.ldc, split_stride = J.split_stride;
    const int M = J.M, K = J.K, nvalid = J.nvalid, nwrite = J.nwrite, kchunk = J.kchunk;
    uint16_t *Ct16 = J.Ct16;
    const int64_t ldct = J.ldct;
    using L = GemmLds<TA>;
    __shared__ __attribute__((aligned(16))) TA As[kBM * L::APITCH];
    __shared__ __attribute__((aligned(16))) TA Bs[kKMax * L::BPITCH];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int row0 = blockIdx.x * kBM;
    const int kbeg = blockIdx.y * kchunk;
    const int kend = min(K, kbeg + kchunk);
    const int NP = static_cast<int>(round_up(nwrite, 16));
    const int NT = NP / 16;

    f32x4 acc[kNTMax];
#pragma unroll
    for (int t = 0; t < kNTMax; ++t)
        acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int k0 = kbeg; k0 < kend; k0 += kBK) {
        __syncthreads();
        // A tile -> As[i][kk]
        if (!TRANS) {
            const int i = tid >> 2;
            const int c0 = (tid & 3) * 8;
            const int gi = row0 + i;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int gk = k0 + c0 + e;
                TA v = 0;
                if (gi < M && gk < kend)
                    v = A[static_cast<int64_t>(gi) * lda + gk];
                As[i * L::APITCH + c0 + e] = v;
            }
        } else {
            const int kk = tid >> 3;
            const int i0 = (tid & 7) * 8;
            const int gk = k0 + kk;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int gi = row0 + i0 + e;
                TA v = 0;
                if (gi < M && gk < kend)
                    v = A[static_cast<int64_t>(gk) * lda + gi];
                As[(i0 + e) * L::APITCH + kk] = v;
            }
        }
        // B tile -> Bs[c][kk]
        for (int idx = tid; idx < kBK * NP; idx += 256) {
            const int kk = idx / NP;
            const int c = idx - kk * NP;
            const int gk = k0 + kk;
            float v = 0.f;
            if (gk < kend && c < nvalid)
                v = B[static_cast<int64_t>(gk) * ldb + c];
            Bs[c * L::BPITCH + kk] = cvt_ct<TA>(v);
        }
        __syncthreads();
        const int ar = wave * 16 + (lane & 15);
        if constexpr (sizeof(TA) == 2) {
            const bf16x8 a = *reinterpret_cast<const bf16x8 *>(&As[ar * L::APITCH + (lane >> 4) * 8]);
#pragma unroll
            for (int t = 0; t < kNTMax; ++t) {
                if (t < NT) {
                    const bf16x8 b = *reinterpret_cast<const bf16x8 *>(
                        &Bs[(t * 16 + (lane & 15)) * L::BPITCH + (lane >> 4) * 8]);
                    acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[t], 0, 0, 0);
                }
            }
        } else {
#pragma unroll
            for (int s4 = 0; s4 < kBK / 4; ++s4) {
                const float a = As[ar * L::APITCH + s4 * 4 + (lane >> 4)];
#pragma unroll
                for (int t = 0; t < kNTMax; ++t) {
                    if (t < NT) {
                        const float b = Bs[(t * 16 + (lane & 15)) * L::BPITCH + s4 * 4 + (lane >> 4)];
                        acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc[t], 0, 0, 0);
                    }
                }
            }
        }
    }
    TO *Cs = C + static_cast<int64_t>(blockIdx.y) * split_stride;
#pragma unroll
    for (int t = 0; t < kNTMax; ++t) {
        if (t < NT) {
            const int col = t * 16 + (lane & 15);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int row = row0 + wave * 16 + (lane >> 4) * 4 + e;
                if (row < M && col < nwrite) {
                    Cs[static_cast<int64_t>(row) * ldc + col] = from_f32<TO>(acc[t][e]);
                    if (Ct16)
                        Ct16[static_cast<int64_t>(col) * ldct + row] = f32_to_bf16(acc[t][e]);
                }
            }
        }
    }
}

// Anchor EMA with a bf16 shadow for the streaming passes (one thread per 8
// consecutive elements of a row; 16-byte accesses when rows are aligned):
//   M <- beta * M + (1 - beta) * G;  M16 <- bf16(M).   With G == NULL only the
// shadow is written.  The shadow is stored in 64 x 64 tiles (ntc tiles per
// tile row; see sc_pass.h).
template <typename GT>
struct EmaJob {
    float *M;
    const GT *G;
    int m, n, vec;
    uint16_t *M16;
    int64_t ntc;
};

__device__ __forceinline__ int64_t tile_at(int64_t i, int64_t j, int64_t ntc)
{
    return ((i >> 6) * ntc + (j >> 6)) * 4096 + (i & 63) * 64 + (j & 63);
}

template <typename GT>
__global__ __launch_bounds__(256) void ema_shadow_kernel(const Batch<EmaJob<GT>> jb, float beta, float omb)
{
    const EmaJob<GT> &J = jb.j[blockIdx.z];
    float *M = J.M;
    const GT *G = J.G;
    const int m = J.m, n = J.n;
    const bool VEC = J.vec != 0;
    uint16_t *M16 = J.M16;
    const int64_t ntc = J.ntc;
    const int nch = (n + 7) / 8;
    const int64_t total = static_cast<int64_t>(m) * nch;
    for (int64_t q = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; q < total;
         q += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t i = q / nch;
        const int j0 = static_cast<int>(q - i * nch) * 8;
        float *mr = M + i * n + j0;
        const GT *gr = G ? G + i * n + j0 : nullptr;
        float v[8];
        if (VEC && j0 + 8 <= n) {
            const nf4 m0 = __builtin_nontemporal_load(reinterpret_cast<const nf4 *>(mr));
            const nf4 m1 = __builtin_nontemporal_load(reinterpret_cast<const nf4 *>(mr + 4));
            v[0] = m0.x; v[1] = m0.y; v[2] = m0.z; v[3] = m0.w;
            v[4] = m1.x; v[5] = m1.y; v[6] = m1.z; v[7] = m1.w;
            if (gr) {
                float g[8];
                if constexpr (sizeof(GT) == 2) {
                    const nu4 gb = __builtin_nontemporal_load(reinterpret_cast<const nu4 *>(gr));
                    const uint32_t w4[4] = {gb.x, gb.y, gb.z, gb.w};
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        g[2 * e] = __uint_as_float(w4[e] << 16);
                        g[2 * e + 1] = __uint_as_float(w4[e] & 0xFFFF0000u);
                    }
                } else {
                    const float4 g0 = *reinterpret_cast<const float4 *>(gr);
                    const float4 g1 = *reinterpret_cast<const float4 *>(gr + 4);
                    g[0] = g0.x; g[1] = g0.y; g[2] = g0.z; g[3] = g0.w;
                    g[4] = g1.x; g[5] = g1.y; g[6] = g1.z; g[7] = g1.w;
                }
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    v[e] = ema_step(v[e], g[e], beta, omb);
                __builtin_nontemporal_store(nf4{v[0], v[1], v[2], v[3]}, reinterpret_cast<nf4 *>(mr));
                __builtin_nontemporal_store(nf4{v[4], v[5], v[6], v[7]}, reinterpret_cast<nf4 *>(mr + 4));
            }
            uint16_t h[8];
#pragma unroll
            for (int e = 0; e < 8; ++e)
                h[e] = f32_to_bf16(v[e]);
            *reinterpret_cast<uint4 *>(M16 + tile_at(i, j0, ntc)) = *reinterpret_cast<const uint4 *>(h);
        } else {
            for (int e = 0; e < 8 && j0 + e < n; ++e) {
                float x = mr[e];
                if (gr) {
                    x = ema_step(x, to_f32<GT>(gr[e]), beta, omb);
                    mr[e] = x;
                }
                M16[tile_at(i, j0 + e, ntc)] = f32_to_bf16(x);
            }
        }
    }
}

// C[i, c] = sum_s P[s][i, c] for c < nwrite (P has row stride ldp).
template <typename TO>
struct ReduceJob {
    const float *P;
    int64_t ldp, split_stride;
    int splits, M, nwrite;
    TO *C;
    int64_t ldc;
};

template <typename TO>
__global__ __launch_bounds__(256) void reduce_splits_kernel(const Batch<ReduceJob<TO>> jb)
{
    const ReduceJob<TO> &J = jb.j[blockIdx.z];
    const float *P = J.P;
    const int64_t ldp = J.ldp, split_stride = J.split_stride, ldc = J.ldc;
    const int splits = J.splits, M = J.M, nwrite = J.nwrite;
    TO *C = J.C;
    if constexpr (sizeof(TO) == 4) {
        // four columns per thread when every row is 16-byte aligned
        if ((nwrite & 3) == 0 && (ldp & 3) == 0 && (ldc & 3) == 0 && (split_stride & 3) == 0 &&
            (reinterpret_cast<uintptr_t>(P) & 15) == 0 && (reinterpret_cast<uintptr_t>(C) & 15) == 0) {
            const int nq = nwrite >> 2;
            const int64_t total = static_cast<int64_t>(M) * nq;
            for (int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; idx < total;
                 idx += static_cast<int64_t>(gridDim.x) * blockDim.x) {
                const int64_t i = idx / nq;
                const int c = static_cast<int>(idx - i * nq) * 4;
                float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
                for (int p = 0; p < splits; ++p) {
                    const float4 v = *reinterpret_cast<const float4 *>(P + p * split_stride + i * ldp + c);
                    acc.x += v.x;
                    acc.y += v.y;
                    acc.z += v.z;
                    acc.w += v.w;
                }
                *reinterpret_cast<float4 *>(C + i * ldc + c) = acc;
            }
            return;
        }
    }
    const int64_t total = static_cast<int64_t>(M) * nwrite;
    for (int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; idx < total;
         idx += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t i = idx / nwrite;
        const int c = static_cast<int>(idx - i * nwrite);
        float s = 0.f;
        for (int p = 0; p < splits; ++p)
            s += P[p * split_stride + i * ldp + c];
        C[i * ldc + c] = from_f32<TO>(s);
    }
}

// ---------------------------------------------------------------------------
// fp64 Gram matrix of the first KP columns of A (rows x lda, fp32), on
// v_mfma_f64_16x16x4_f64: one workgroup per block of rows computes every
// upper 16 x 16 tile (ti <= tj) of that block's partial Gram; the partials
// are summed by gram_reduce_kernel, which also mirrors the lower triangle.
// The rows pass through LDS in 32-row chunks, converted to fp64 once and
// double-buffered (one barrier per chunk).  Operands (one fp64 per lane):
// A[i][k] in lane i + 16 k, B[k][j] in lane j + 16 k, so both come from the
// same read of a chunk row group: lane l takes row k0 + l / 16, column
// 16 b + l % 16, and every wave reads the KP / 16 column blocks once per
// 4-row step.  The result D[i][j] sits in lane j + 16 (i % 4), element i / 4.
// ---------------------------------------------------------------------------
constexpr int kGT = 16;
constexpr int kGRows = 32;
constexpr int kGWaves = 8;                         // waves per Gram workgroup
typedef double v4d __attribute__((ext_vector_type(4)));

struct GramJob {
    const float *A;
    int64_t lda;
    int rows, rows_per_block, blocks;
    double *part;
};

// Staged row pitch in doubles: an odd multiple of 128 bytes, so that the two
// rows of a 32-lane half of an operand read fall in different bank halves.
__host__ __device__ constexpr int gram_pitch(int NB) { return NB * kGT + ((NB & 1) ? 0 : kGT); }

// Upper tiles in row-major order: tile t of an NB x NB block grid.
__host__ __device__ constexpr int gram_tile_row(int t, int NB)
{
    int ti = 0;
    while (t >= NB - ti) {
        t -= NB - ti;
        ++ti;
    }
    return ti;
}
__host__ __device__ constexpr int gram_tile_col(int t, int NB)
{
    int ti = 0;
    while (t >= NB - ti) {
        t -= NB - ti;
        ++ti;
    }
    return ti + t;
}

// One 4-row step of wave W's tiles: tile T = W + kGWaves U takes block rows
// ti(T) and tj(T) of the step's operands (indices fixed at compile time).
template <int NB, int T>
__device__ __forceinline__ v4d gram_mfma(const double (&op)[NB], v4d acc)
{
    constexpr int ti = gram_tile_row(T, NB), tj = gram_tile_col(T, NB);
    return __builtin_amdgcn_mfma_f64_16x16x4f64(op[ti], op[tj], acc, 0, 0, 0);
}
template <int NB, int W, int... U>
__device__ __forceinline__ void gram_mfmas(v4d *acc, const double (&op)[NB], std::integer_sequence<int, U...>)
{
    ((acc[U] = gram_mfma<NB, W + kGWaves * U>(op, acc[U])), ...);
}

// Wave W's share of the upper tiles: t = W, W + kGWaves, ...  (compile-time, so
// that the operand registers are indexed by constants).
template <int NB, int W>
__device__ __forceinline__ void gram_wave(double *Ys0, double *Ys1, int lane, int nchunks,
                                          const float *A, int64_t lda, int r0, int r1, int KP, double *pb, int tid)
{
    constexpr int NTILES = NB * (NB + 1) / 2;
    constexpr int TPW = NTILES > W ? (NTILES - W + kGWaves - 1) / kGWaves : 0;
    constexpr int NTH = 64 * kGWaves;              // threads
    constexpr int PITCH = gram_pitch(NB);          // doubles per staged row
    constexpr int q4 = NB * kGT / 4;               // float4 per staged row
    constexpr int PF = (kGRows * q4 + NTH - 1) / NTH;  // float4 per thread and chunk
    v4d acc[TPW > 0 ? TPW : 1];
#pragma unroll
    for (int u = 0; u < TPW; ++u)
        acc[u] = v4d{0.0, 0.0, 0.0, 0.0};
    float4 pf[PF];
    auto load = [&](int rb) {
#pragma unroll
        for (int u = 0; u < PF; ++u) {
            const int idx = tid + NTH * u;
            const int rr = idx / q4, c4 = (idx % q4) * 4;
            const int gr = rb + rr;
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (idx < kGRows * q4 && gr < r1 && c4 < KP)
                v = *reinterpret_cast<const float4 *>(A + static_cast<int64_t>(gr) * lda + c4);
            pf[u] = v;
        }
    };
    load(r0);
    for (int c = 0; c < nchunks; ++c) {
        double *Ys = (c & 1) ? Ys1 : Ys0;
        // stage this chunk (loaded during the previous one) as fp64; the
        // buffer was last read two chunks ago, before the previous barrier
#pragma unroll
        for (int u = 0; u < PF; ++u) {
            const int idx = tid + NTH * u;
            if (idx < kGRows * q4) {
                double *d = Ys + (idx / q4) * PITCH + (idx % q4) * 4;
                *reinterpret_cast<double2 *>(d) = make_double2(pf[u].x, pf[u].y);
                *reinterpret_cast<double2 *>(d + 2) = make_double2(pf[u].z, pf[u].w);
            }
        }
        __syncthreads();
        if (c + 1 < nchunks)
            load(r0 + (c + 1) * kGRows);
        if constexpr (TPW > 0) {
            // the next step's operands are read before this step's products
            // are issued, so their latency hides under the MFMAs
            const double *yr = Ys + (lane >> 4) * PITCH + (lane & 15);
            double opA[NB], opB[NB];
            auto read = [&](double (&o)[NB], int k0) {
#pragma unroll
                for (int b = 0; b < NB; ++b)
                    o[b] = yr[k0 * PITCH + b * kGT];
            };
            // (scheduling barriers keep each read ahead of the products before
            // it: left alone, the compiler sinks the reads to just before
            // their use and waits for them there)
            read(opA, 0);
#pragma unroll
            for (int k0 = 0; k0 < kGRows; k0 += 8) {
                read(opB, k0 + 4);
                __builtin_amdgcn_sched_barrier(0);
                gram_mfmas<NB, W>(acc, opA, std::make_integer_sequence<int, TPW>{});
                __builtin_amdgcn_sched_barrier(0);
                if (k0 + 8 < kGRows)
                    read(opA, k0 + 8);
                __builtin_amdgcn_sched_barrier(0);
                gram_mfmas<NB, W>(acc, opB, std::make_integer_sequence<int, TPW>{});
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    }
#pragma unroll
    for (int u = 0; u < TPW; ++u) {
        const int t = W + kGWaves * u;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int i = gram_tile_row(t, NB) * kGT + (lane >> 4) + 4 * e;
            const int j = gram_tile_col(t, NB) * kGT + (lane & 15);
            if (i < KP && j < KP)
                pb[static_cast<int64_t>(i) * KP + j] = acc[u][e];
        }
    }
}

template <int NB>
__global__ __launch_bounds__(64 * kGWaves) void gram_partial_kernel(const Batch<GramJob> jb, int KP)
{
    const GramJob &J = jb.j[blockIdx.z];
    if (static_cast<int>(blockIdx.x) >= J.blocks)
        return;
    constexpr int PITCH = gram_pitch(NB);
    __shared__ __attribute__((aligned(16))) double Ys[2][kGRows * PITCH];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r0 = blockIdx.x * J.rows_per_block;
    const int r1 = min(J.rows, r0 + J.rows_per_block);
    const int nchunks = (r1 - r0 + kGRows - 1) / kGRows;
    double *pb = J.part + static_cast<int64_t>(blockIdx.x) * KP * KP;
    switch (wave) {
    case 0: gram_wave<NB, 0>(Ys[0], Ys[1], lane, nchunks, J.A, J.lda, r0, r1, KP, pb, tid); break;
    case 1: gram_wave<NB, 1>(Ys[0], Ys[1], lane, nchunks, J.A, J.lda, r0, r1, KP, pb, tid); break;
    case 2: gram_wave<NB, 2>(Ys[0], Ys[1], lane, nchunks, J.A, J.lda, r0, r1, KP, pb, tid); break;
    case 3: gram_wave<NB, 3>(Ys[0], Ys[1], lane, nchunks, J.A, J.lda, r0, r1, KP, pb, tid); break;
    case 4: gram_wave<NB, 4>(Ys[0], Ys[1], lane, nchunks, J.A, J.lda, r0, r1, KP, pb, tid); break;
    case 5: gram_wave<NB, 5>(Ys[0], Ys[1], lane, nchunks, J.A, J.lda, r0, r1, KP, pb, tid); break;
    case 6: gram_wave<NB, 6>(Ys[0], Ys[1], lane, nchunks, J.A, J.lda, r0, r1, KP, pb, tid); break;
    default: gram_wave<NB, 7>(Ys[0], Ys[1], lane, nchunks, J.A, J.lda, r0, r1, KP, pb, tid); break;
    }
}

struct GramRedJob {
    const double *part;
    int blocks;
    double *G;
};

__global__ __launch_bounds__(256) void gram_reduce_kernel(const Batch<GramRedJob> jb, int KP)
{
    // 32 consecutive elements x 8 groups of blocks per workgroup; only the
    // upper tiles are read (coalesced) and each is also written mirrored
    const GramRedJob &J = jb.j[blockIdx.z];
    __shared__ double red[8][32];
    const int e = threadIdx.x & 31, g = threadIdx.x >> 5;
    const int idx = blockIdx.x * 32 + e;
    const int i = idx / KP, j = idx - (idx / KP) * KP;
    const bool live = idx < KP * KP && i / kGT <= j / kGT;
    double s = 0.0;
    if (live) {
        const int64_t stride = static_cast<int64_t>(KP) * KP;
        const double *p = J.part + idx;
        double s0 = 0.0, s1 = 0.0;
        int b = g;
        for (; b + 8 < J.blocks; b += 16) {
            s0 += p[b * stride];
            s1 += p[(b + 8) * stride];
        }
        if (b < J.blocks)
            s0 += p[b * stride];
        s = s0 + s1;
    }
    red[g][e] = s;
    __syncthreads();
    if (g == 0 && live) {
        double t = 0.0;
#pragma unroll
        for (int q = 0; q < 8; ++q)
            t += red[q][e];
        J.G[idx] = t;
        if (i / kGT < j / kGT)
            J.G[static_cast<int64_t>(j) * KP + i] = t;
    }
}

// Sum over each group of 8 lanes with DPP lane permutes (VALU, no LDS):
// quad_perm [1,0,3,2] and [2,3,0,1] (xor 1, xor 2), then row_half_mirror
// (pairs the two quads of each 8-lane half row); every lane of the group ends
// with the group's sum.
__device__ __forceinline__ float group8_sum(float x)
{
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, false));
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x4E, 0xF, 0xF, false));
    x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x141, 0xF, 0xF, false));
    return x;
}

__device__ __forceinline__ double group8_sum(double x)
{
#define ACSC_DPP64(CTRL)                                                                          \
    {                                                                                             \
        const int lo = __double2loint(x), hi = __double2hiint(x);                                 \
        const int plo = __builtin_amdgcn_update_dpp(0, lo, CTRL, 0xF, 0xF, false);                \
        const int phi = __builtin_amdgcn_update_dpp(0, hi, CTRL, 0xF, 0xF, false);                \
        x += __hiloint2double(phi, plo);                                                          \
    }
    ACSC_DPP64(0xB1)
    ACSC_DPP64(0x4E)
    ACSC_DPP64(0x141)
#undef ACSC_DPP64
    return x;
}

// Reciprocal and reciprocal square root of the rotation formulas: the fp32
// path takes the hardware approximations (about 1 ulp; a rotation only has to
// be orthogonal, and the next sweep corrects its angle).  fp64 refines the
// hardware estimates (v_rsq_f64, v_rcp_f64) by two Newton steps each, to
// within a few ulp: much shorter dependent chains than the correctly rounded
// square root and division, which sit on every round's critical path, and c
// and s = c t stay orthogonal to working precision.  The arguments are
// positive and finite (the caller skips pairs with a zero norm or product).
__device__ __forceinline__ float jac_rsqrt(float x) { return __builtin_amdgcn_rsqf(x); }
__device__ __forceinline__ double jac_rsqrt(double x)
{
    double y = __builtin_amdgcn_rsq(x);
    const double hx = 0.5 * x;
    y = __builtin_fma(y, __builtin_fma(-hx * y, y, 0.5), y);   // y + y (1 - x y^2) / 2
    y = __builtin_fma(y, __builtin_fma(-hx * y, y, 0.5), y);
    return y;
}
__device__ __forceinline__ float jac_rcp(float x) { return __builtin_amdgcn_rcpf(x); }
__device__ __forceinline__ double jac_rcp(double x)
{
    double y = __builtin_amdgcn_rcp(x);
    y = __builtin_fma(y, __builtin_fma(-x, y, 1.0), y);        // y + y (1 - x y)
    y = __builtin_fma(y, __builtin_fma(-x, y, 1.0), y);
    return y;
}

// ---------------------------------------------------------------------------
// One-sided (Hestenes) Jacobi SVD of the k x k factor L in LDS, one
// workgroup: rotate column pairs (round-robin tournament, every pair of a round
// at once on 8 lanes) until every pair is orthogonal to `tol`.  Then sigma_c = ||a_c||,
// u_c = a_c / sigma_c, sorted descending, and the right factors of the final
// products are written:  Bu[:, t] = u_(t), Bv[:, t] = u_(t) / sigma_(t),
// s[t] = sigma_(t), d[t] = s / (s + tau) for t < r.
// ---------------------------------------------------------------------------
struct JacJob {
    const double *Lf;
    float *Bu, *Bv, *s_out, *d_out;
    int *info;
};

// Status words at the head of a build workspace: the Jacobi sweeps used, the
// last sweep's largest off-diagonal ratio and the tolerance (float bits), a
// status (bit 0: the sweep cap was reached above the tolerance; bit 1: the
// Rayleigh-Ritz phase found no stamp of a subspace phase), and the stamp the
// subspace phase leaves for the Rayleigh-Ritz phase, which clears it.
constexpr int kInfoSweeps = 0, kInfoResidual = 1, kInfoTol = 2, kInfoStatus = 3, kInfoStamp = 4, kInfoStall = 5;
constexpr int kStatusNoConv = 1, kStatusNoSubspace = 2, kStatusStalled = 4;
// The stamp a subspace phase leaves for its Rayleigh-Ritz phase: the plain
// one, or the one that also says its fused EMA pass gave up a wait.
constexpr int kSubspaceStamp = 0x5B5D7A11, kSubspaceStalledStamp = 0x5B5D7A13;
constexpr int kJacobiMaxSweeps = 40;

// End of a subspace phase: fold the EMA pass's stall word into the stamp and
// clear it for the next phase.
__global__ __launch_bounds__(64) void stamp_kernel(const Batch<JacJob> jb)
{
    if (threadIdx.x == 0) {
        int *info = jb.j[blockIdx.z].info;
        const bool stalled = info[kInfoStall] == pass::kEmaStallMark;
        info[kInfoStall] = 0;
        info[kInfoStamp] = stalled ? kSubspaceStalledStamp : kSubspaceStamp;
    }
}

template <typename T, int RC>
__global__ __launch_bounds__(1024) void jacobi_kernel(const Batch<JacJob> jb, int k, int KP, int r,
                                                      int RP, float tau, T tol, int max_sweeps)
{
    const JacJob &J = jb.j[blockIdx.z];
    const double *Lf = J.Lf;
    float *Bu = J.Bu, *Bv = J.Bv, *s_out = J.s_out, *d_out = J.d_out;
    int *info = J.info;
    extern __shared__ __attribute__((aligned(16))) unsigned char jsm[];
    // column c at A[c * kp]; kp = k rounded up to 8 V (= 8 RC; 32 rows in
    // fp32, 16 in fp64), rows k..kp-1 are zero.  Lane gl of a pair's 8 lanes
    // holds the R = kp / 8 consecutive rows gl R .. gl R + R - 1 of both
    // columns (R a multiple of V: 16-byte LDS accesses).  Every round reads
    // and writes whole columns, so the padding is kept to what the 16-byte
    // accesses need.
    constexpr int V = 16 / sizeof(T);   // elements per 16-byte access
    T *A = reinterpret_cast<T *>(jsm);
    const int kp = (k + 8 * V - 1) / (8 * V) * (8 * V);
    T *nrm = A + static_cast<size_t>(k) * kp;   // squared column norms
    __shared__ unsigned int sh_off;
    __shared__ double sh_cut;
    __shared__ double sig[kKMax];
    __shared__ int rank_of[kKMax];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nwave = blockDim.x >> 6;
    for (int idx = tid; idx < k * kp; idx += blockDim.x) {
        const int c = idx / kp, i = idx % kp;
        A[c * kp + i] = i < k ? static_cast<T>(Lf[static_cast<int64_t>(i) * KP + c]) : T(0);
    }
    const int n2 = k + (k & 1);
    const int npairs = n2 / 2;
    // eight column pairs per wave, 8 lanes each
    const int grp = lane >> 3, gl = lane & 7;
    const int slots = nwave * 8;
    constexpr int R = RC;
    constexpr int RMAX = RC;
    static_assert(R % V == 0, "rows per lane");
    int sweeps_used = 0;
    float last_off = 0.f;
    // the subspace phase that produced Lf stamps the workspace (read before
    // this kernel clears the stamp, by the same thread)
    const int stamp = (tid == 0 && info) ? info[kInfoStamp] : 0;
    __syncthreads();
    for (int sweep = 0; sweep < max_sweeps; ++sweep) {
        // exact squared norms at the start of every sweep (the rotations
        // update them incrementally within it)
        for (int c = wave * 8 + grp; c < k; c += slots) {
            const T *ac = A + c * kp + gl * R;
            T ss = 0;
#pragma unroll
            for (int e = 0; e < RMAX; ++e)
                if (e < R)
                    ss += ac[e] * ac[e];
            ss = group8_sum(ss);
            if (gl == 0)
                nrm[c] = ss;
        }
        if (tid == 0)
            sh_off = 0u;
        __syncthreads();
        float wmax = 0.f;
        for (int round = 0; round < n2 - 1; ++round) {
            for (int p = wave * 8 + grp; p < npairs; p += slots) {
                auto pos = [&](int x) {
                    if (x == 0)
                        return 0;
                    int t = x - 1 + round;
                    if (t >= n2 - 1)
                        t -= n2 - 1;
                    return t + 1;
                };
                int cp = pos(p), cq = pos(n2 - 1 - p);
                if (cp >= k || cq >= k)
                    continue;
                if (cp > cq) {
                    const int t = cp;
                    cp = cq;
                    cq = t;
                }
                T *ap = A + cp * kp + gl * R;
                T *aq = A + cq * kp + gl * R;
                T xv[RMAX], yv[RMAX];
#pragma unroll
                for (int e = 0; e < RMAX; e += V) {
                    uint4 ux = make_uint4(0u, 0u, 0u, 0u), uy = ux;
                    if (e < R) {
                        ux = *reinterpret_cast<const uint4 *>(ap + e);
                        uy = *reinterpret_cast<const uint4 *>(aq + e);
                    }
                    __builtin_memcpy(&xv[e], &ux, 16);
                    __builtin_memcpy(&yv[e], &uy, 16);
                }
                const T al = nrm[cp], be = nrm[cq];
                T gp[4] = {0, 0, 0, 0};
#pragma unroll
                for (int e = 0; e < RMAX; ++e)
                    gp[e & 3] += xv[e] * yv[e];
                const T ga = group8_sum((gp[0] + gp[1]) + (gp[2] + gp[3]));
                const T prod = al * be;
                if (ga == T(0) || prod == T(0))
                    continue;
                const T ratio = fabs(ga) * jac_rsqrt(prod);
                wmax = fmaxf(wmax, static_cast<float>(ratio));
                if (ratio <= tol)
                    continue;
                const T zeta = (be - al) * jac_rcp(T(2) * ga);
                const T z2 = T(1) + zeta * zeta;
                const T t = (zeta >= T(0) ? T(1) : T(-1)) * jac_rcp(fabs(zeta) + z2 * jac_rsqrt(z2));
                const T c = jac_rsqrt(T(1) + t * t);
                const T sn = c * t;
#pragma unroll
                for (int e = 0; e < RMAX; e += V) {
                    if (e < R) {
                        T xo[V], yo[V];
#pragma unroll
                        for (int v = 0; v < V; ++v) {
                            xo[v] = c * xv[e + v] - sn * yv[e + v];
                            yo[v] = sn * xv[e + v] + c * yv[e + v];
                        }
                        uint4 ux, uy;
                        __builtin_memcpy(&ux, xo, 16);
                        __builtin_memcpy(&uy, yo, 16);
                        *reinterpret_cast<uint4 *>(ap + e) = ux;
                        *reinterpret_cast<uint4 *>(aq + e) = uy;
                    }
                }
                // the rotation zeroes the pair's inner product: the norms move by t gamma
                if (gl == 0) {
                    nrm[cp] = al - t * ga;
                    nrm[cq] = be + t * ga;
                }
            }
            __syncthreads();
        }
        // reduce the sweep's largest off-diagonal ratio over the workgroup
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1)
            wmax = fmaxf(wmax, __shfl_xor(wmax, off, 64));
        if (lane == 0)
            atomicMax(&sh_off, __float_as_uint(wmax));
        __syncthreads();
        const float off = __uint_as_float(sh_off);
        __syncthreads();
        sweeps_used = sweep + 1;
        last_off = off;
        if (off <= static_cast<float>(tol))
            break;
    }
    if (tid == 0 && info) {
        info[kInfoSweeps] = sweeps_used;
        info[kInfoResidual] = __float_as_int(last_off);
        info[kInfoTol] = __float_as_int(static_cast<float>(tol));
        info[kInfoStatus] = (last_off > static_cast<float>(tol) ? kStatusNoConv : 0) |
                            (stamp != kSubspaceStamp && stamp != kSubspaceStalledStamp ? kStatusNoSubspace : 0) |
                            (stamp == kSubspaceStalledStamp ? kStatusStalled : 0);
        info[kInfoStamp] = 0;
    }
    // norms (one wave per column)
    for (int c = wave; c < k; c += nwave) {
        double ss = 0.0;
        for (int i = lane; i < k; i += 64) {
            const double x = A[c * kp + i];
            ss += x * x;
        }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1)
            ss += __shfl_xor(ss, off, 64);
        if (lane == 0)
            sig[c] = sqrt(ss);
    }
    __syncthreads();
    for (int c = tid; c < k; c += blockDim.x) {
        int rk = 0;
        for (int c2 = 0; c2 < k; ++c2)
            rk += (sig[c2] > sig[c]) || (sig[c2] == sig[c] && c2 < c);
        rank_of[c] = rk;
    }
    __syncthreads();
    // numerical rank: singular values at the fp32 rounding floor of the
    // largest one are zero (their vectors are noise, and 1/sigma would blow up)
    if (tid == 0) {
        double mx = 0.0;
        for (int c = 0; c < k; ++c)
            mx = fmax(mx, sig[c]);
        sh_cut = kRankCutoff * mx;
    }
    __syncthreads();
    for (int c = tid; c < k; c += blockDim.x)
        if (sig[c] <= sh_cut)
            sig[c] = 0.0;
    __syncthreads();
    for (int idx = tid; idx < KP * RP; idx += blockDim.x) {
        Bu[idx] = 0.f;
        Bv[idx] = 0.f;
    }
    __syncthreads();
    for (int idx = tid; idx < k * k; idx += blockDim.x) {
        const int c = idx / k, i = idx % k;
        const int t = rank_of[c];
        if (t < r) {
            const double sg = sig[c];
            const double u = sg > 0.0 ? static_cast<double>(A[c * kp + i]) / sg : 0.0;
            Bu[i * RP + t] = static_cast<float>(u);
            Bv[i * RP + t] = sg > 0.0 ? static_cast<float>(u / sg) : 0.f;
        }
    }
    for (int c = tid; c < k; c += blockDim.x) {
        const int t = rank_of[c];
        if (t < r) {
            const float sg = static_cast<float>(sig[c]);
            s_out[t] = sg;
            const float den = sg + tau;
            d_out[t] = den != 0.f ? sg / den : 0.f;
        }
    }
}

// ---------------------------------------------------------------------------
// Elementwise kernels.
// ---------------------------------------------------------------------------
// M <- beta * M + (1 - beta) * G  (fp32 state)
template <typename GT>
struct Ema32Job {
    float *M;
    const GT *G;
    int64_t count;
};

template <typename GT>
__global__ __launch_bounds__(256) void ema_kernel(const Batch<Ema32Job<GT>> jb, float beta, float omb)
{
    float *M = jb.j[blockIdx.z].M;
    const GT *G = jb.j[blockIdx.z].G;
    const int64_t count = jb.j[blockIdx.z].count;
    if (!G)
        return;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x * 4;
    for (int64_t i = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) * 4; i < count;
         i += stride) {
        if (i + 4 <= count) {
            float4 m = *reinterpret_cast<const float4 *>(M + i);
            float g0, g1, g2, g3;
            if constexpr (sizeof(GT) == 2) {
                const uint2 gb = *reinterpret_cast<const uint2 *>(G + i);
                g0 = __uint_as_float(gb.x << 16);
                g1 = __uint_as_float(gb.x & 0xFFFF0000u);
                g2 = __uint_as_float(gb.y << 16);
                g3 = __uint_as_float(gb.y & 0xFFFF0000u);
            } else {
                const float4 gv = *reinterpret_cast<const float4 *>(G + i);
                g0 = gv.x;
                g1 = gv.y;
                g2 = gv.z;
                g3 = gv.w;
            }
            m.x = ema_step(m.x, g0, beta, omb);
            m.y = ema_step(m.y, g1, beta, omb);
            m.z = ema_step(m.z, g2, beta, omb);
            m.w = ema_step(m.w, g3, beta, omb);
            *reinterpret_cast<float4 *>(M + i) = m;
        } else {
            for (int64_t j = i; j < count; ++j)
                M[j] = ema_step(M[j], to_f32<GT>(G[j]), beta, omb);
        }
    }
}

// Starting block Z0 [n, KP]: V_warm columns first (if given), then uniform
// random values in [-1, 1) from a counter-based hash of (seed, i, c); zero
// beyond k.
// Entry (i, c) of the seeded starting block: the low 32 bits of the seed
// added to a Weyl combination of row and column, then C. Wellons's lowbias32
// integer hash (two 32-bit multiplies), the top 24 bits mapped to [-1, 1).
// The subspace iteration only needs a seeded block of full rank with no
// preferred direction; a 64-bit mixer here made the start block the most
// expensive step of a cold build after the passes.
__device__ __forceinline__ float start_uniform(uint64_t seed, int64_t i, int c)
{
    uint32_t h = static_cast<uint32_t>(i) * 0x9E3779B1u + static_cast<uint32_t>(c) * 0x632BE5ABu +
                 static_cast<uint32_t>(seed) + static_cast<uint32_t>(seed >> 32) * 0x85EBCA6Bu;
    h ^= h >> 16;
    h *= 0x7FEB352Du;
    h ^= h >> 15;
    h *= 0x846CA68Bu;
    h ^= h >> 16;
    return static_cast<float>(h >> 8) * (2.0f / 16777216.0f) - 1.0f;
}

struct InitJob {
    float *Z;
    int n;
    const float *Vw;
    uint64_t seed;
};

__global__ __launch_bounds__(256) void init_block_kernel(const Batch<InitJob> jb, int k, int KP, int r)
{
    float *Z = jb.j[blockIdx.z].Z;
    const int n = jb.j[blockIdx.z].n;
    const float *Vw = jb.j[blockIdx.z].Vw;
    const int rw = Vw ? r : 0;
    const uint64_t seed = jb.j[blockIdx.z].seed;
    const int64_t total = static_cast<int64_t>(n) * KP;
    for (int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; idx < total;
         idx += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t i = idx / KP;
        const int c = static_cast<int>(idx - i * KP);
        float v = 0.f;
        if (c < k) {
            if (Vw && c < rw)
                v = Vw[i * rw + c];
            else
                v = start_uniform(seed, i, c);
        }
        Z[idx] = v;
    }
}

// 64-row tiles of a thin fp32 block [rows, cols] to bf16, zero-padded to CP
// columns, through LDS: the transposed copy Xt[c][i] (row stride ldt, 16-byte
// stores along i) and/or the row-major copy Xc[i][c] (row stride CP).  With
// X == nullptr the block is the starting block of the subspace iteration
// (V_warm columns, then seeded uniform draws, for c < cols).
struct TileJob {
    const float *X;
    int64_t ldx;
    int rows, cols, CP;
    uint16_t *Xt;
    int64_t ldt;
    uint16_t *Xc;
    const float *Vw;
    int rw;
    uint64_t seed;
    int blk0;   // first workgroup of this job in the launch (set by launch_tiles)
};

constexpr int kTileRows = 64;

__global__ __launch_bounds__(256) void tile_bf16_kernel(const Batch<TileJob> jb)
{
    // one workgroup per 64-row tile of every job of the batch, jobs one after
    // another along x
    int ji = 0;
    while (ji + 1 < jb.count && static_cast<int>(blockIdx.x) >= jb.j[ji + 1].blk0)
        ++ji;
    const TileJob &J = jb.j[ji];
    const int row0 = (static_cast<int>(blockIdx.x) - J.blk0) * kTileRows;
    if (row0 >= J.rows)
        return;
    // The tile is staged already rounded to bf16 (both copies take bf16 of the
    // same values): 25 KiB, six workgroups per CU.  Staged rows are 97 words
    // apart, so the eight rows a transposed 16-byte store gathers sit in
    // distinct banks.
    constexpr int kPitch = kKMax + 2;
    __shared__ __attribute__((aligned(16))) uint16_t Ts[kTileRows * kPitch];
    const int CP = J.CP;
    // wave w fills rows w, w + 4, ..., its lanes 64 consecutive columns
    const int cl = threadIdx.x & 63, rg = threadIdx.x >> 6;
    for (int r = rg; r < kTileRows; r += 4) {
        const int64_t i = row0 + r;
        for (int c = cl; c < CP; c += 64) {
            float v = 0.f;
            if (i < J.rows && c < J.cols) {
                if (J.X)
                    v = J.X[i * J.ldx + c];
                else if (J.Vw && c < J.rw)
                    v = J.Vw[i * J.rw + c];
                else
                    v = start_uniform(J.seed, i, c);
            }
            Ts[r * kPitch + c] = f32_to_bf16(v);
        }
    }
    __syncthreads();
    if (J.Xc) {
        // 32 lanes per row, lane q copies the 16-byte chunk q of the row (CP / 8 <= 24 chunks)
        const int q = threadIdx.x & 31;
        if (q < CP / 8)
            for (int r = threadIdx.x >> 5; r < kTileRows && row0 + r < J.rows; r += 8) {
                const uint32_t *src = reinterpret_cast<const uint32_t *>(&Ts[r * kPitch + 8 * q]);
                *reinterpret_cast<uint4 *>(J.Xc + static_cast<int64_t>(row0 + r) * CP + 8 * q) =
                    make_uint4(src[0], src[1], src[2], src[3]);
            }
    }
    if (J.Xt) {
        for (int idx = threadIdx.x; idx < CP * (kTileRows / 8); idx += 256) {
            const int c = idx / (kTileRows / 8), r8 = (idx % (kTileRows / 8)) * 8;
            if (row0 + r8 >= J.rows)
                continue;
            uint32_t w[4];
#pragma unroll
            for (int e = 0; e < 4; ++e)
                w[e] = static_cast<uint32_t>(Ts[(r8 + 2 * e) * kPitch + c]) |
                       (static_cast<uint32_t>(Ts[(r8 + 2 * e + 1) * kPitch + c]) << 16);
            *reinterpret_cast<uint4 *>(J.Xt + static_cast<int64_t>(c) * J.ldt + row0 + r8) = make_uint4(w[0], w[1], w[2], w[3]);
        }
    }
}

// Xf[i][j] = d_i * X[i][j] * d_j for i, j < r; zero elsewhere (RP x RP).
struct FilterJob {
    const float *X;
    const float *d;
    float *Xf;
};

__global__ __launch_bounds__(256) void filter_x_kernel(const Batch<FilterJob> jb, int r, int RP)
{
    const float *X = jb.j[blockIdx.z].X;
    const float *d = jb.j[blockIdx.z].d;
    float *Xf = jb.j[blockIdx.z].Xf;
    const int64_t ldx = RP;
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= RP * RP)
        return;
    const int i = idx / RP, j = idx % RP;
    Xf[idx] = (i < r && j < r) ? d[i] * X[static_cast<int64_t>(i) * ldx + j] * d[j] : 0.f;
}

// ---------------------------------------------------------------------------
// Global-norm clipping of the corrected AdamW step without a pass over
// G_proj: with U and V orthonormal, X = U^T G V and X_f = d X d,
//   ||alpha G + (1 - alpha) U X_f V^T||^2
//     = alpha^2 ||G||^2 + 2 alpha (1 - alpha) <X, X_f> + (1 - alpha)^2 ||X_f||^2.
// ||G||^2 is summed by sumsq_kernel (kSumBlocks fp64 partials per matrix, a
// grid and order that never depend on the device), the rest by
// clip_norm_kernel in one workgroup, matrix by matrix in call order.
// ---------------------------------------------------------------------------
constexpr int kSumBlocks = 512;

struct SumJob {
    const void *G;
    int64_t count;    // elements of G (contiguous)
    int vec;          // 16-byte aligned G and count % 8 == 0: 16-byte loads
    double *part;     // [kSumBlocks]
};

__device__ __forceinline__ double block_sum(double v, double *red)
{
    red[threadIdx.x] = v;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if (static_cast<int>(threadIdx.x) < w)
            red[threadIdx.x] += red[threadIdx.x + w];
        __syncthreads();
    }
    const double t = red[0];
    __syncthreads();
    return t;
}

template <typename GT>
__global__ __launch_bounds__(256) void sumsq_kernel(const Batch<SumJob> jb)
{
    __shared__ double red[256];
    const SumJob &J = jb.j[blockIdx.z];
    const GT *G = static_cast<const GT *>(J.G);
    double acc = 0.0;
    constexpr int V = 16 / sizeof(GT);
    const int64_t stride = static_cast<int64_t>(kSumBlocks) * 256;
    const int64_t start = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (J.vec) {
        // squares of bf16 are exact in fp32; the V of one chunk are added in fp32
        for (int64_t c = start; c < J.count / V; c += stride) {
            const uint4 raw = reinterpret_cast<const uint4 *>(G)[c];
            const GT *e = reinterpret_cast<const GT *>(&raw);
            float s = 0.f;
#pragma unroll
            for (int i = 0; i < V; ++i) {
                const float g = to_f32<GT>(e[i]);
                s += g * g;
            }
            acc += s;
        }
    } else {
        for (int64_t i = start; i < J.count; i += stride) {
            const double g = to_f32<GT>(G[i]);
            acc += g * g;
        }
    }
    const double t = block_sum(acc, red);
    if (threadIdx.x == 0)
        J.part[blockIdx.x] = t;
}

constexpr int kTermBlocks = 16;   // partial terms per matrix
static_assert(kSumBlocks % kTermBlocks == 0, "term slices");

struct NormJob {
    const double *part;   // ||G||^2 partials [kSumBlocks]
    const float *X;       // [r, RP]
    const float *Xf;      // [RP, RP] (rows >= r are zero)
    int r, RP;
    double *terms;        // [kTermBlocks]
};

// Block b of matrix z: its share of alpha^2 ||G||^2 + 2 alpha (1 - alpha)
// <X, X_f> + (1 - alpha)^2 ||X_f||^2, from fixed slices (grid kTermBlocks).
__global__ __launch_bounds__(256) void norm_terms_kernel(const Batch<NormJob> jb, float alpha)
{
    __shared__ double red[256];
    const NormJob &J = jb.j[blockIdx.z];
    const int b = blockIdx.x;
    const double a = alpha, c = 1.0 - static_cast<double>(alpha);
    double gg = 0.0, xx = 0.0, ff = 0.0;
    constexpr int PB = kSumBlocks / kTermBlocks;
    for (int p = threadIdx.x; p < PB; p += 256)
        gg += J.part[b * PB + p];
    const int n = J.r * J.RP;
    const int per = (n + kTermBlocks - 1) / kTermBlocks;
    const int q0 = b * per, q1 = min(n, q0 + per);
    for (int q = q0 + static_cast<int>(threadIdx.x); q < q1; q += 256) {
        const double x = J.X[q], f = J.Xf[q];
        xx += x * f;
        ff += f * f;
    }
    const double t = block_sum(a * a * gg + 2.0 * a * c * xx + c * c * ff, red);
    if (threadIdx.x == 0)
        J.terms[b] = t;
}

// One workgroup.  acc (fp64) carries the squared norm over the launches of
// one call (first: start at zero; last: write the clip coefficient and the
// norm).  Terms are added matrix by matrix in call order.
__global__ __launch_bounds__(64) void clip_norm_kernel(const Batch<NormJob> jb, float max_norm, double *acc,
                                                       float *coef, float *norm_out, int first, int last)
{
    if (threadIdx.x != 0)
        return;
    double total = first ? 0.0 : *acc;
    for (int i = 0; i < jb.count; ++i)
        for (int b = 0; b < kTermBlocks; ++b)
            total += jb.j[i].terms[b];
    *acc = total;
    if (last) {
        const double N = sqrt(total > 0.0 ? total : 0.0);
        float c = 1.0f;
        if (max_norm > 0.f) {
            const double q = static_cast<double>(max_norm) / (N + 1e-6);
            if (q < 1.0)
                c = static_cast<float>(q);
        }
        *coef = c;
        if (norm_out)
            *norm_out = static_cast<float>(N);
    }
}

// Vc[i][c] = V[i][c] for c < r, zero up to RP, converted to the compute type.
template <typename CT>
struct PadJob {
    const float *V;
    int n;
    CT *Vc;
};

template <typename CT>
__global__ __launch_bounds__(256) void pad_convert_kernel(const Batch<PadJob<CT>> jb, int r, int RP)
{
    const float *V = jb.j[blockIdx.z].V;
    const int n = jb.j[blockIdx.z].n;
    CT *Vc = jb.j[blockIdx.z].Vc;
    const int64_t total = static_cast<int64_t>(n) * RP;
    for (int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; idx < total;
         idx += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t i = idx / RP;
        const int c = static_cast<int>(idx - i * RP);
        Vc[idx] = from_f32<CT>(c < r ? V[i * r + c] : 0.f);
    }
}

// ---------------------------------------------------------------------------
// Fused correction pass: out = alpha * G + (1 - alpha) * P V^T for a 64 x 64
// tile, with P [m, RP] and Vc [n, RP] in the compute type (RP a multiple of
// 32, zero padded).  Four waves, each a 32 x 32 quarter of the tile.
// ---------------------------------------------------------------------------
template <typename GT>
struct BlendJob {
    const GT *G;
    GT *out;
    int m, n;
    const GT *P, *Vc;
    float *W, *m1, *m2;   // corrected AdamW: fp32 weights and moments, in place
    float *E;             // error feedback: fp32 memory (holds M), takes M - out
};

// Element (row, col) of G_proj = gp: stored, or (ADAM) the gradient of the
// AdamW step of the same element of W (scaled by the call's clip coefficient).
template <bool ADAM, typename GT>
__device__ __forceinline__ void blend_out(const BlendJob<GT> &J, int64_t o, float gp, float cf,
                                          const blend::AdamArgs &ad)
{
    if constexpr (ADAM) {
        float w = J.W[o], m1 = J.m1[o], m2 = J.m2[o];
        blend::adamw_elem(cf * gp, w, m1, m2, ad);
        J.W[o] = w;
        J.m1[o] = m1;
        J.m2[o] = m2;
    } else {
        J.out[o] = from_f32<GT>(gp);
    }
}

template <typename GT, int MODE>
__global__ __launch_bounds__(256) void blend_kernel(const Batch<BlendJob<GT>> jb, int RP, float alpha,
                                                    const blend::AdamArgs ad)
{
    constexpr bool ADAM = MODE == blend::kAdam;
    const BlendJob<GT> &J = jb.j[blockIdx.z];
    const GT *G = J.G;
    const int m = J.m, n = J.n;
    const GT *P = J.P, *Vc = J.Vc;
    if (static_cast<int>(blockIdx.x) * 64 >= n || static_cast<int>(blockIdx.y) * 64 >= m)
        return;
    extern __shared__ __attribute__((aligned(16))) unsigned char bsm[];
    constexpr int PAD = sizeof(GT) == 2 ? 8 : 1;
    const int pitch = RP + PAD;
    GT *Ps = reinterpret_cast<GT *>(bsm);
    GT *Vs = Ps + kBM * pitch;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int col0 = blockIdx.x * 64, row0 = blockIdx.y * 64;
    for (int idx = tid; idx < 64 * RP; idx += 256) {
        const int rr = idx / RP, c = idx % RP;
        const int gi = row0 + rr, gj = col0 + rr;
        Ps[rr * pitch + c] = gi < m ? P[static_cast<int64_t>(gi) * RP + c] : GT(0);
        Vs[rr * pitch + c] = gj < n ? Vc[static_cast<int64_t>(gj) * RP + c] : GT(0);
    }
    __syncthreads();
    const int wr = wave >> 1, wc = wave & 1;
    f32x4 acc[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
            acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};
    if constexpr (sizeof(GT) == 2) {
        for (int k0 = 0; k0 < RP; k0 += 32) {
            bf16x8 af[2], bfr[2];
#pragma unroll
            for (int a = 0; a < 2; ++a) {
                af[a] = *reinterpret_cast<const bf16x8 *>(
                    &Ps[(wr * 32 + a * 16 + (lane & 15)) * pitch + k0 + (lane >> 4) * 8]);
                bfr[a] = *reinterpret_cast<const bf16x8 *>(
                    &Vs[(wc * 32 + a * 16 + (lane & 15)) * pitch + k0 + (lane >> 4) * 8]);
            }
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int b = 0; b < 2; ++b)
                    acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[a], bfr[b], acc[a][b], 0, 0, 0);
        }
    } else {
        for (int k0 = 0; k0 < RP; k0 += 4) {
            float af[2], bfr[2];
#pragma unroll
            for (int a = 0; a < 2; ++a) {
                af[a] = Ps[(wr * 32 + a * 16 + (lane & 15)) * pitch + k0 + (lane >> 4)];
                bfr[a] = Vs[(wc * 32 + a * 16 + (lane & 15)) * pitch + k0 + (lane >> 4)];
            }
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int b = 0; b < 2; ++b)
                    acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[a], bfr[b], acc[a][b], 0, 0, 0);
        }
    }
    const float oma = 1.0f - alpha;
    const float cf = ADAM ? *ad.coef : 1.0f;
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            const int col = col0 + wc * 32 + b * 16 + (lane & 15);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int row = row0 + wr * 32 + a * 16 + (lane >> 4) * 4 + e;
                if (row < m && col < n) {
                    const int64_t o = static_cast<int64_t>(row) * n + col;
                    if constexpr (MODE == blend::kFeedback) {
                        // out = P V^T as stored; the memory takes M - out
                        const GT ov = from_f32<GT>(acc[a][b][e]);
                        J.out[o] = ov;
                        J.E[o] = J.E[o] - to_f32<GT>(ov);
                    } else {
                        const float g = to_f32<GT>(G[o]);
                        blend_out<ADAM>(J, o, blend_step(g, acc[a][b][e], alpha, oma), cf, ad);
                    }
                }
            }
        }
}

// ---------------------------------------------------------------------------
// Fused correction pass for bf16 G, 128 x 128 output tiles:
//   out = alpha * G + (1 - alpha) * P V^T,  P [m, RP], Vc [n, RP] (bf16, RP a
// multiple of 32, zero padded).
// The G tile is staged in LDS with 16-byte coalesced loads issued before the
// products, blended in place in LDS, and written back with 16-byte coalesced
// stores.  P and V stream through LDS in 32-deep slices.  Four waves, each a
// 64 x 64 quarter (4 x 4 MFMA tiles).  Tile order: block b runs on XCD b % 8,
// and XCD x takes the row blocks congruent to x, walking their column blocks,
// so a row block's slice of P stays in one L2.
// ---------------------------------------------------------------------------
constexpr int kBT = 128;              // tile edge
constexpr int kGPitch = kBT + 8;      // bf16 elements per staged G row (272 bytes)
constexpr int kKPitch = 32 + 8;       // P / V slice rows (80 bytes)

template <bool VEC, bool ADAM>
__global__ __launch_bounds__(256) void blend16_kernel(const Batch<BlendJob<uint16_t>> jb, int RP, float alpha,
                                                      int col_blocks_max, const blend::AdamArgs ad)
{
    const BlendJob<uint16_t> &J = jb.j[blockIdx.z];
    const int m = J.m, n = J.n;
    const int rb_n = (m + kBT - 1) / kBT, cb_n = (n + kBT - 1) / kBT;
    // XCD-aware tile order
    const int b = blockIdx.x;
    const int xcd = b & 7, t = b >> 3;
    const int rb = xcd + 8 * (t / cb_n);
    const int cb = t % cb_n;
    (void)col_blocks_max;
    if (rb >= rb_n)
        return;
    const int row0 = rb * kBT, col0 = cb * kBT;
    // one LDS region: P / V slices during the products, then the G tile
    __shared__ __attribute__((aligned(16))) uint16_t sm[kBT * kGPitch];
    uint16_t *Ps = sm;
    uint16_t *Vs = sm + kBT * kKPitch;
    uint16_t *Gs = sm;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint16_t *G = J.G;
    uint16_t *out = J.out;
    // G tile into registers now (128 rows x 16 chunks; 8 chunks per thread),
    // so its latency overlaps the products
    uint4 gr[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        const int q = tid + 256 * u;
        const int rr = q >> 4, c8 = (q & 15) * 8;
        const int gi = row0 + rr, gj = col0 + c8;
        uint4 v = make_uint4(0u, 0u, 0u, 0u);
        if (gi < m) {
            const uint16_t *src = G + static_cast<int64_t>(gi) * n + gj;
            if (VEC && gj + 8 <= n) {
                v = *reinterpret_cast<const uint4 *>(src);
            } else {
                uint16_t e8[8];
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    e8[e] = (gj + e < n) ? src[e] : uint16_t(0);
                v = *reinterpret_cast<const uint4 *>(e8);
            }
        }
        gr[u] = v;
    }
    // P / V slices: 2 x 128 rows x 4 chunks; 4 chunks per thread, prefetched
    uint4 pv[4];
    auto load_slice = [&](int k0) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int q = tid + 256 * u;
            const bool isV = q >= kBT * 4;
            const int qq = isV ? q - kBT * 4 : q;
            const int rr = qq >> 2, c8 = (qq & 3) * 8;
            const int g = (isV ? col0 : row0) + rr;
            const int lim = isV ? n : m;
            uint4 v = make_uint4(0u, 0u, 0u, 0u);
            if (g < lim)
                v = *reinterpret_cast<const uint4 *>((isV ? J.Vc : J.P) + static_cast<int64_t>(g) * RP + k0 + c8);
            pv[u] = v;
        }
    };
    const int wr = wave >> 1, wc = wave & 1;
    f32x4 acc[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int c = 0; c < 4; ++c)
            acc[a][c] = f32x4{0.f, 0.f, 0.f, 0.f};
    load_slice(0);
    for (int k0 = 0; k0 < RP; k0 += 32) {
        __syncthreads();
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int q = tid + 256 * u;
            const bool isV = q >= kBT * 4;
            const int qq = isV ? q - kBT * 4 : q;
            const int rr = qq >> 2, c8 = (qq & 3) * 8;
            *reinterpret_cast<uint4 *>(&(isV ? Vs : Ps)[rr * kKPitch + c8]) = pv[u];
        }
        __syncthreads();
        if (k0 + 32 < RP)
            load_slice(k0 + 32);
        bf16x8 af[4], bfr[4];
#pragma unroll
        for (int a = 0; a < 4; ++a) {
            af[a] = *reinterpret_cast<const bf16x8 *>(&Ps[(wr * 64 + a * 16 + (lane & 15)) * kKPitch + (lane >> 4) * 8]);
            bfr[a] = *reinterpret_cast<const bf16x8 *>(&Vs[(wc * 64 + a * 16 + (lane & 15)) * kKPitch + (lane >> 4) * 8]);
        }
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int c = 0; c < 4; ++c)
                acc[a][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[a], bfr[c], acc[a][c], 0, 0, 0);
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        const int q = tid + 256 * u;
        const int rr = q >> 4, c8 = (q & 15) * 8;
        *reinterpret_cast<uint4 *>(&Gs[rr * kGPitch + c8]) = gr[u];
    }
    __syncthreads();
    // blend in place in the staged tile
    const float oma = 1.0f - alpha;
    if constexpr (ADAM) {
        // the blended values are the AdamW gradient, never stored
        const float cf = *ad.coef;
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int cc = wc * 64 + c * 16 + (lane & 15);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int rr = wr * 64 + a * 16 + (lane >> 4) * 4 + e;
                    const int gi = row0 + rr, gj = col0 + cc;
                    if (gi < m && gj < n)
                        blend_out<true>(J, static_cast<int64_t>(gi) * n + gj,
                                        blend_step(bf16_to_f32(Gs[rr * kGPitch + cc]), acc[a][c][e], alpha, oma), cf, ad);
                }
            }
        return;
    }
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int cc = wc * 64 + c * 16 + (lane & 15);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int rr = wr * 64 + a * 16 + (lane >> 4) * 4 + e;
                uint16_t &gv = Gs[rr * kGPitch + cc];
                gv = f32_to_bf16(blend_step(bf16_to_f32(gv), acc[a][c][e], alpha, oma));
            }
        }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        const int q = tid + 256 * u;
        const int rr = q >> 4, c8 = (q & 15) * 8;
        const int gi = row0 + rr, gj = col0 + c8;
        if (gi >= m)
            continue;
        uint16_t *dst = out + static_cast<int64_t>(gi) * n + gj;
        const uint4 v = *reinterpret_cast<const uint4 *>(&Gs[rr * kGPitch + c8]);
        if (VEC && gj + 8 <= n) {
            *reinterpret_cast<uint4 *>(dst) = v;
        } else {
            const uint16_t *e8 = reinterpret_cast<const uint16_t *>(&v);
            for (int e = 0; e < 8 && gj + e < n; ++e)
                dst[e] = e8[e];
        }
    }
}

// ---------------------------------------------------------------------------
// Host side.
// ---------------------------------------------------------------------------
struct Carve {
    char *base;
    size_t off = 0;
    explicit Carve(void *b) : base(static_cast<char *>(b)) {}
    template <typename T>
    T *take(size_t count)
    {
        off = static_cast<size_t>(round_up(static_cast<int64_t>(off), 256));
        T *p = base ? reinterpret_cast<T *>(base + off) : nullptr;
        off += count * sizeof(T);
        return p;
    }
};

int split_count(int64_t Mdim, int64_t Kdim)
{
    const int64_t mb = cdiv(Mdim, kBM);
    int64_t s = cdiv(512, mb);
    s = std::min<int64_t>(s, std::max<int64_t>(1, Kdim / 256));
    return static_cast<int>(std::max<int64_t>(1, s));
}

int64_t split_chunk(int64_t Kdim, int splits) { return round_up(cdiv(Kdim, splits), kBK); }

// Most Gram partial blocks a matrix of this many rows may be split into.
int gram_blocks_max(int64_t rows) { return static_cast<int>(std::min<int64_t>(128, cdiv(rows, kGRows))); }

struct Dims {
    int m, n, r, k, KP, RP;
};

Dims dims_of(int m, int n, int r, int oversample)
{
    Dims d;
    d.m = m;
    d.n = n;
    d.r = r;
    d.k = std::min(std::min(r + oversample, std::min(m, n)), kKMax);
    d.KP = static_cast<int>(round_up(d.k, 16));
    d.RP = static_cast<int>(round_up(r, 32));
    return d;
}

// Buffers of sc_build_prior (carved in this order).
struct PriorWs {
    int *info;   // status words (kInfo*): Jacobi sweeps, residual, tolerance, status, phase stamp
    float *Y, *Z, *part, *T, *Bu, *Bv;
    double *gpart, *gram;
    uint16_t *M16, *Yt16, *Zt16;   // bf16 path: shadow of M (64 x 64 tiles), transposed thin factors
    int64_t ntc16, ldy16, ldz16;
};

size_t carve_prior(const Dims &d, bool use16, void *base, PriorWs *w)
{
    Carve c(base);
    const int64_t mx = std::max(d.m, d.n);
    int64_t s1 = split_count(d.m, d.n), s2 = split_count(d.n, d.m);
    if (use16) {
        s1 = std::max<int64_t>(s1, pass::max_splits(d.m, d.n));
        s2 = std::max<int64_t>(s2, pass::max_splits(d.n, d.m));
    }
    const int64_t part = std::max<int64_t>(s1 * d.m, s2 * d.n) * d.KP;
    PriorWs t;
    t.info = c.take<int>(64);
    t.ntc16 = pass::tiles_per_row(d.n);
    t.ldy16 = round_up(d.m, 8);
    t.ldz16 = round_up(d.n, 8);
    t.M16 = use16 ? c.take<uint16_t>(static_cast<size_t>(pass::tiled_elems(d.m, d.n))) : nullptr;
    t.Yt16 = use16 ? c.take<uint16_t>(static_cast<size_t>(d.KP) * t.ldy16) : nullptr;
    t.Zt16 = use16 ? c.take<uint16_t>(static_cast<size_t>(d.KP) * t.ldz16) : nullptr;
    t.Y = c.take<float>(static_cast<size_t>(d.m) * d.KP);
    t.Z = c.take<float>(static_cast<size_t>(d.n) * d.KP);
    t.part = c.take<float>(static_cast<size_t>(part));
    t.T = c.take<float>(static_cast<size_t>(d.KP) * d.KP);
    t.Bu = c.take<float>(static_cast<size_t>(d.KP) * d.RP);
    t.Bv = c.take<float>(static_cast<size_t>(d.KP) * d.RP);
    t.gpart = c.take<double>(static_cast<size_t>(gram_blocks_max(mx)) * d.KP * d.KP);
    t.gram = c.take<double>(static_cast<size_t>(d.KP) * d.KP);
    if (w)
        *w = t;
    return c.off;
}

// Buffers of sc_correct.
struct CorrWs {
    float *Tm, *part, *xpart, *X, *Xf;
    void *Pc, *Vc;
    uint16_t *Vt16;
    int64_t ldv16;
    double *sq, *terms, *acc;
    float *coef;
};

size_t carve_correct(const Dims &d, size_t esize, void *base, CorrWs *w)
{
    Carve c(base);
    const int s1 = std::max(split_count(d.m, d.n), esize == 2 ? pass::max_splits(d.m, d.n) : 1);
    const int s2 = split_count(d.r, d.m);
    CorrWs t;
    t.ldv16 = round_up(d.n, 8);
    t.Vt16 = esize == 2 ? c.take<uint16_t>(static_cast<size_t>(d.RP) * t.ldv16) : nullptr;
    t.Tm = c.take<float>(static_cast<size_t>(d.m) * d.RP);
    t.part = c.take<float>(static_cast<size_t>(s1) * d.m * d.RP);
    t.xpart = c.take<float>(static_cast<size_t>(s2) * d.r * d.RP);
    t.X = c.take<float>(static_cast<size_t>(d.r) * d.RP);
    t.Xf = c.take<float>(static_cast<size_t>(d.RP) * d.RP);
    t.Pc = c.take<unsigned char>(static_cast<size_t>(d.m) * d.RP * esize);
    t.Vc = c.take<unsigned char>(static_cast<size_t>(d.n) * d.RP * esize);
    // corrected AdamW: ||G||^2 partials, the norm accumulator, the clip coefficient
    t.sq = c.take<double>(kSumBlocks);
    t.terms = c.take<double>(kTermBlocks);
    t.acc = c.take<double>(1);
    t.coef = c.take<float>(1);
    if (w)
        *w = t;
    return c.off;
}

unsigned grid1d(int64_t total, int per = 256)
{
    return static_cast<unsigned>(std::max<int64_t>(1, std::min<int64_t>(cdiv(total, per), 65536)));
}

// Enqueue `kernel` over `jobs`, kMaxBatch jobs per launch (grid.z = job).
template <class Job, class K, class... Args>
void launch_jobs(const char *tag, K kernel, const std::vector<Job> &jobs, dim3 grid, dim3 block, size_t lds,
                 hipStream_t st, Args... args)
{
    for (size_t c0 = 0; c0 < jobs.size(); c0 += kMaxBatch) {
        Batch<Job> b{};
        b.count = static_cast<int>(std::min<size_t>(kMaxBatch, jobs.size() - c0));
        for (int i = 0; i < b.count; ++i)
            b.j[i] = jobs[c0 + i];
        ACSC_LAUNCH(tag, kernel, dim3(grid.x, grid.y, b.count), block, lds, st, b, args...);
    }
}

// tile_bf16_kernel over a list of jobs: each launch takes up to kMaxBatch jobs
// and exactly as many workgroups as they have 64-row tiles.
void launch_tiles(const char *tag, std::vector<TileJob> jobs, hipStream_t st)
{
    for (size_t c0 = 0; c0 < jobs.size(); c0 += kMaxBatch) {
        Batch<TileJob> b{};
        b.count = static_cast<int>(std::min<size_t>(kMaxBatch, jobs.size() - c0));
        int blocks = 0;
        for (int i = 0; i < b.count; ++i) {
            b.j[i] = jobs[c0 + i];
            b.j[i].blk0 = blocks;
            blocks += static_cast<int>(cdiv(b.j[i].rows, kTileRows));
        }
        if (blocks > 0)
            ACSC_LAUNCH(tag, tile_bf16_kernel, dim3(blocks), dim3(256), 0, st, b);
    }
}

// The Jacobi kernel for order k, by rows per lane (k rounded up to 32, over 8).
template <typename T>
using JacobiFn = void (*)(const Batch<JacJob>, int, int, int, int, float, T, int);

// rows per lane: k rounded up to 8 V, divided by 8 (fp64: k <= 128)
template <typename T>
JacobiFn<T> jacobi_fn(int k)
{
    switch (((k + 15) & ~15) / 8) {
    case 2: return jacobi_kernel<T, 2>;
    case 4: return jacobi_kernel<T, 4>;
    case 6: return jacobi_kernel<T, 6>;
    case 8: return jacobi_kernel<T, 8>;
    case 10: return jacobi_kernel<T, 10>;
    case 12: return jacobi_kernel<T, 12>;
    case 14: return jacobi_kernel<T, 14>;
    default: return jacobi_kernel<T, 16>;
    }
}
template <>
JacobiFn<float> jacobi_fn<float>(int k)
{
    switch (((k + 31) & ~31) / 8) {
    case 4: return jacobi_kernel<float, 4>;
    case 8: return jacobi_kernel<float, 8>;
    case 12: return jacobi_kernel<float, 12>;
    case 16: return jacobi_kernel<float, 16>;
    case 20: return jacobi_kernel<float, 20>;
    default: return jacobi_kernel<float, 24>;
    }
}

// one 8-lane group per column pair of a round, at least 4 and at most 16 waves
unsigned jacobi_threads(int k)
{
    const int npairs = (k + (k & 1)) / 2;
    return 64u * static_cast<unsigned>(std::min<int64_t>(16, std::max<int64_t>(4, cdiv(npairs, 8))));
}

// columns padded to a multiple of 8 V rows (32 in fp32, 16 in fp64), plus the squared norms
size_t jacobi_lds(int k, size_t es) { return (static_cast<size_t>(k) * round_up(k, es == 8 ? 16 : 32) + k) * es; }

// One tall-skinny product per job (opA * B), split-K through the job's
// partial buffer `part` (nullptr: one split, straight into C).
template <typename TA, typename TO>
struct GemmReq {
    const TA *A;
    int64_t lda;
    const float *B;
    int64_t ldb;
    TO *C;
    int64_t ldc;
    int M, K, nvalid, nwrite;
    float *part;
    uint16_t *Ct16;
    int64_t ldct;
};

template <typename TA, bool TRANS, typename TO>
void tall_gemm(const char *tag, const std::vector<GemmReq<TA, TO>> &reqs, hipStream_t st)
{
    std::vector<GemmJob<TA, TO>> direct;
    std::vector<GemmJob<TA, float>> split;
    std::vector<ReduceJob<TO>> red;
    int gx = 1, gy = 1, sx = 1, sy = 1;
    int64_t rtot = 1;
    for (const auto &q : reqs) {
        const int NP = static_cast<int>(round_up(q.nwrite, 16));
        int splits = q.part ? split_count(q.M, q.K) : 1;
        const int64_t chunk = split_chunk(q.K, splits);
        splits = static_cast<int>(cdiv(q.K, chunk));
        const int mb = static_cast<int>(cdiv(q.M, kBM));
        if (splits == 1) {
            direct.push_back(GemmJob<TA, TO>{q.A, q.lda, q.B, q.ldb, q.C, q.ldc, 0, q.M, q.K, q.nvalid, q.nwrite,
                                             static_cast<int>(chunk), 1, q.Ct16, q.ldct});
            gx = std::max(gx, mb);
        } else {
            const int64_t ss = static_cast<int64_t>(q.M) * NP;
            split.push_back(GemmJob<TA, float>{q.A, q.lda, q.B, q.ldb, q.part, NP, ss, q.M, q.K, q.nvalid, NP,
                                               static_cast<int>(chunk), splits, nullptr, 0});
            red.push_back(ReduceJob<TO>{q.part, NP, ss, splits, q.M, q.nwrite, q.C, q.ldc});
            sx = std::max(sx, mb);
            sy = std::max(sy, splits);
            rtot = std::max<int64_t>(rtot, static_cast<int64_t>(q.M) * q.nwrite);
        }
    }
    if (!direct.empty())
        launch_jobs(tag, gemm_tall_kernel<TA, TRANS, TO>, direct, dim3(gx, gy), dim3(256), 0, st);
    if (!split.empty()) {
        launch_jobs(tag, gemm_tall_kernel<TA, TRANS, float>, split, dim3(sx, sy), dim3(256), 0, st);
        launch_jobs("sc_split_reduce", reduce_splits_kernel<TO>, red, dim3(grid1d(rtot)), dim3(256), 0, st);
    }
}

// Per-matrix state of a batched call.
struct Mat {
    const sc_matrix *in;
    Dims D;
    PriorWs pw;
    CorrWs cw;
    uint64_t seed;
    const sc_adamw_state *ad = nullptr;   // corrected AdamW: this matrix's optimiser state
};

// Corrected AdamW: the epilogue constants and the call's norm accumulator.
struct AdamCtx {
    blend::AdamArgs args;   // args.coef: the clip coefficient (workspace of the call's first matrix)
    double *acc;            // squared-norm accumulator (same workspace)
    float max_norm;
    float *norm_out;        // device or NULL
};

// Gram matrices (fp64) of the first KP columns of one block per matrix.
void gram(const std::vector<Mat> &ms, const std::vector<const float *> &A, const std::vector<int> &rows,
          hipStream_t st)
{
    const int KP = ms[0].D.KP;
    const int nt = static_cast<int>(cdiv(KP, kGT));
    std::vector<GramJob> gj;
    std::vector<GramRedJob> rj;
    int gy = 1;
    // one row count per block across the batch, so that the blocks of all
    // matrices (one workgroup each) come to at most two per CU
    int64_t total = 0;
    for (int r : rows)
        total += r;
    auto rpb_of = [&](size_t i, int64_t rpb_batch) {
        return std::max<int64_t>(rpb_batch, round_up(cdiv(rows[i], gram_blocks_max(rows[i])), kGRows));
    };
    int64_t rpb_batch = round_up(std::max<int64_t>(1, cdiv(total, 512)), kGRows);
    for (;;) {
        int64_t nb = 0;
        for (size_t i = 0; i < ms.size(); ++i)
            nb += cdiv(rows[i], rpb_of(i, rpb_batch));
        if (nb <= 512 || rpb_batch >= total)
            break;
        rpb_batch += kGRows;
    }
    for (size_t i = 0; i < ms.size(); ++i) {
        const int rpb = static_cast<int>(rpb_of(i, rpb_batch));
        const int gb = static_cast<int>(cdiv(rows[i], rpb));
        gj.push_back(GramJob{A[i], KP, rows[i], rpb, gb, ms[i].pw.gpart});
        rj.push_back(GramRedJob{ms[i].pw.gpart, gb, ms[i].pw.gram});
        gy = std::max(gy, gb);
    }
    switch (nt) {
    case 1: launch_jobs("sc_gram", gram_partial_kernel<1>, gj, dim3(gy), dim3(64 * kGWaves), 0, st, KP); break;
    case 2: launch_jobs("sc_gram", gram_partial_kernel<2>, gj, dim3(gy), dim3(64 * kGWaves), 0, st, KP); break;
    case 3: launch_jobs("sc_gram", gram_partial_kernel<3>, gj, dim3(gy), dim3(64 * kGWaves), 0, st, KP); break;
    case 4: launch_jobs("sc_gram", gram_partial_kernel<4>, gj, dim3(gy), dim3(64 * kGWaves), 0, st, KP); break;
    case 5: launch_jobs("sc_gram", gram_partial_kernel<5>, gj, dim3(gy), dim3(64 * kGWaves), 0, st, KP); break;
    case 6: launch_jobs("sc_gram", gram_partial_kernel<6>, gj, dim3(gy), dim3(64 * kGWaves), 0, st, KP); break;
    case 7: launch_jobs("sc_gram", gram_partial_kernel<7>, gj, dim3(gy), dim3(64 * kGWaves), 0, st, KP); break;
    case 8: launch_jobs("sc_gram", gram_partial_kernel<8>, gj, dim3(gy), dim3(64 * kGWaves), 0, st, KP); break;
    case 9: launch_jobs("sc_gram", gram_partial_kernel<9>, gj, dim3(gy), dim3(64 * kGWaves), 0, st, KP); break;
    case 10: launch_jobs("sc_gram", gram_partial_kernel<10>, gj, dim3(gy), dim3(64 * kGWaves), 0, st, KP); break;
    case 11: launch_jobs("sc_gram", gram_partial_kernel<11>, gj, dim3(gy), dim3(64 * kGWaves), 0, st, KP); break;
    default: launch_jobs("sc_gram", gram_partial_kernel<12>, gj, dim3(gy), dim3(64 * kGWaves), 0, st, KP); break;
    }
    launch_jobs("sc_gram_reduce", gram_reduce_kernel, rj, dim3(static_cast<unsigned>(cdiv(int64_t(KP) * KP, 32))),
                dim3(256), 0, st, KP);
}

// Q <- Y L^{-T}, `passes` times (CholeskyQR; two passes = CholeskyQR2), for
// one block Y [rows, KP] per matrix (first k columns live; `which` selects
// the Y or the Z block).  The Gram matrix is accumulated in fp64 from the
// fp32 block, so one pass already leaves the columns orthonormal to about
// 1e-7 * cond(Y); the iteration only needs a well-conditioned basis, and the
// final basis gets the second pass.  The last pass also writes the bf16
// transposed copy that the next streaming pass reads.
int orthonormalise(std::vector<Mat> &ms, bool onY, int passes, bool use16, hipStream_t st)
{
    const Dims &d0 = ms[0].D;
    std::vector<const float *> A;
    std::vector<int> rows;
    for (auto &m : ms) {
        A.push_back(onY ? m.pw.Y : m.pw.Z);
        rows.push_back(onY ? m.D.m : m.D.n);
    }
    for (int pass = 0; pass < passes; ++pass) {
        gram(ms, A, rows, st);
        std::vector<chol::Req> cj;
        for (auto &m : ms)
            cj.push_back(chol::Req{m.pw.gram, m.pw.T});
        if (int rc = chol::run("sc_chol_inv", cj, d0.k, d0.KP, true, st))
            return rc;
        // fp32 Q is read by the second Gram of CholeskyQR2 and by the final
        // basis; otherwise (bf16 passes) only its bf16 transposed copy is
        std::vector<orth::Req> g;
        for (size_t i = 0; i < ms.size(); ++i) {
            float *Y = const_cast<float *>(A[i]);
            uint16_t *t16 = (use16 && pass + 1 == passes) ? (onY ? ms[i].pw.Yt16 : ms[i].pw.Zt16) : nullptr;
            const int64_t ldt = onY ? ms[i].pw.ldy16 : ms[i].pw.ldz16;
            g.push_back(orth::Req{Y, rows[i], ms[i].pw.T, t16, ldt, !use16 || passes == 2});
        }
        if (int rc = orth::run("sc_orth_apply", g, d0.KP, st))
            return rc;
    }
    return ACSC_OK;
}

// EMA + top-r SVD + filter for a group of matrices with the same k.
// Phases of the build: the subspace iteration (EMA, power passes, the final
// Z = M^T Q) and the Rayleigh-Ritz step on Z (Gram, Cholesky, Jacobi, basis,
// filter).  The second reads only what the first left in the workspace.
constexpr int kPhaseSubspace = 1, kPhaseRitz = 2;

int build_group(std::vector<Mat> &ms, acsc_dtype dt, float beta, int r, int power_iters, float tau,
                int phases, hipStream_t st)
{
    const Dims &d0 = ms[0].D;
    const int k = d0.k, KP = d0.KP, RP = d0.RP;
    const bool use16 = dt == ACSC_BF16;
    const float omb = 1.0f - beta;
    // with a bf16 shadow and a large enough batch, the EMA runs fused with the
    // first pass Y = M16 Z (after the starting block exists)
    std::vector<pass::EmaReq> er;
    for (auto &m : ms)
        er.push_back(pass::EmaReq{m.in->M, static_cast<const uint16_t *>(m.in->G), m.pw.M16, m.pw.Zt16, m.pw.ldz16,
                                  m.pw.Y, KP, m.D.m, m.D.n, KP, m.pw.part, m.pw.info + kInfoStall});
    const bool fused = use16 && pass::ema_fusable(er);
    if ((phases & kPhaseSubspace) && !fused) {
        if (use16) {
            std::vector<EmaJob<uint16_t>> j;
            int64_t tot = 1;
            for (auto &m : ms) {
                j.push_back(EmaJob<uint16_t>{m.in->M, static_cast<const uint16_t *>(m.in->G), m.D.m, m.D.n,
                                             (m.D.n % 8) == 0 ? 1 : 0, m.pw.M16, m.pw.ntc16});
                tot = std::max<int64_t>(tot, static_cast<int64_t>(m.D.m) * cdiv(m.D.n, 8));
            }
            launch_jobs("sc_ema", ema_shadow_kernel<uint16_t>, j, dim3(grid1d(tot)), dim3(256), 0, st, beta, omb);
        } else {
            std::vector<Ema32Job<float>> j;
            int64_t tot = 1;
            for (auto &m : ms) {
                const int64_t c = static_cast<int64_t>(m.D.m) * m.D.n;
                j.push_back(Ema32Job<float>{m.in->M, static_cast<const float *>(m.in->G), c});
                tot = std::max(tot, cdiv(c, 4));
            }
            bool any = false;
            for (auto &m : ms)
                any = any || m.in->G;
            if (any)
                launch_jobs("sc_ema", ema_kernel<float>, j, dim3(grid1d(tot)), dim3(256), 0, st, beta, omb);
        }
    }
    if (phases & kPhaseSubspace) {
        std::vector<InitJob> j;
        int64_t tot = 1;
        for (auto &m : ms) {
            j.push_back(InitJob{m.pw.Z, m.D.n, m.in->V_warm, m.seed});
            tot = std::max<int64_t>(tot, static_cast<int64_t>(m.D.n) * KP);
        }
        if (use16) {
            // the bf16 passes read only the transposed copy of the starting block
            std::vector<TileJob> tj;
            for (auto &m : ms)
                tj.push_back(TileJob{nullptr, 0, m.D.n, k, KP, m.pw.Zt16, m.pw.ldz16, nullptr, m.in->V_warm,
                                     m.in->V_warm ? r : 0, m.seed});
            launch_tiles("sc_init", tj, st);
        } else {
            launch_jobs("sc_init", init_block_kernel, j, dim3(grid1d(tot)), dim3(256), 0, st, k, KP, r);
        }
    }
    // one pass Y = M Z  /  Z = M^T Y over every EMA (bf16 shadow on matrix cores, or fp32)
    auto pass = [&](bool mz) {
        if (use16) {
            std::vector<pass::Req> q;
            for (auto &m : ms) {
                if (mz)
                    q.push_back(pass::Req{m.pw.M16, 0, true, m.pw.Zt16, m.pw.ldz16, m.pw.Y, KP, m.D.m, m.D.n,
                                        KP, m.pw.part, static_cast<int>(m.pw.ntc16)});
                else
                    q.push_back(pass::Req{m.pw.M16, 0, true, m.pw.Yt16, m.pw.ldy16, m.pw.Z, KP, m.D.n, m.D.m,
                                        KP, m.pw.part, static_cast<int>(m.pw.ntc16)});
            }
            return mz ? pass::run("sc_pass_mz", false, q, st) : pass::run("sc_pass_mtq", true, q, st);
        } else {
            std::vector<GemmReq<float, float>> q;
            for (auto &m : ms) {
                if (mz)
                    q.push_back(GemmReq<float, float>{m.in->M, m.D.n, m.pw.Z, KP, m.pw.Y, KP, m.D.m, m.D.n, k, KP,
                                                      m.pw.part, nullptr, 0});
                else
                    q.push_back(GemmReq<float, float>{m.in->M, m.D.n, m.pw.Y, KP, m.pw.Z, KP, m.D.n, m.D.m, k, KP,
                                                      m.pw.part, nullptr, 0});
            }
            if (mz)
                tall_gemm<float, false, float>("sc_pass_mz", q, st);
            else
                tall_gemm<float, true, float>("sc_pass_mtq", q, st);
            return ACSC_OK;
        }
    };
    int rc = ACSC_OK;
    if (phases & kPhaseSubspace) {
        rc = fused ? pass::ema_run("sc_ema", er, beta, omb, st) : pass(true);
        if (rc)
            return rc;
        if ((rc = orthonormalise(ms, true, power_iters == 0 ? 2 : 1, use16, st)))
            return rc;
        for (int it = 0; it < power_iters; ++it) {
            if ((rc = pass(false)))
                return rc;
            if ((rc = orthonormalise(ms, false, 1, use16, st)))
                return rc;
            if ((rc = pass(true)))
                return rc;
            if ((rc = orthonormalise(ms, true, it + 1 == power_iters ? 2 : 1, use16, st)))
                return rc;
        }
        // Z = M^T Q (= B^T) for the Rayleigh-Ritz step: B B^T = Z^T Z = L L^T, SVD of L by Jacobi.
        if ((rc = pass(false)))
            return rc;
        std::vector<JacJob> sj;
        for (auto &m : ms)
            sj.push_back(JacJob{nullptr, nullptr, nullptr, nullptr, nullptr, m.pw.info});
        launch_jobs("sc_stamp", stamp_kernel, sj, dim3(1), dim3(64), 0, st);
    }
    if (!(phases & kPhaseRitz))
        return ACSC_OK;
    {
        std::vector<const float *> A;
        std::vector<int> rows;
        std::vector<chol::Req> cj;
        std::vector<JacJob> jj;
        for (auto &m : ms) {
            A.push_back(m.pw.Z);
            rows.push_back(m.D.n);
            cj.push_back(chol::Req{m.pw.gram, nullptr});
            jj.push_back(JacJob{m.pw.gram, m.pw.Bu, m.pw.Bv, m.in->s, m.in->d, m.pw.info});
        }
        gram(ms, A, rows, st);
        if ((rc = chol::run("sc_chol", cj, k, KP, false, st)))
            return rc;
        // the sweep cap can be lowered (not raised) through the environment, so
        // that the non-convergence report can be exercised
        int max_sweeps = kJacobiMaxSweeps;
        if (const char *e = std::getenv("ACSC_JACOBI_MAX_SWEEPS"))
            max_sweeps = std::max(1, std::min(kJacobiMaxSweeps, std::atoi(e)));
        if (k <= kJacobiF64MaxK)
            launch_jobs("sc_jacobi", jacobi_fn<double>(k), jj, dim3(1), dim3(jacobi_threads(k)),
                        jacobi_lds(k, sizeof(double)), st,
                        k, KP, r, RP, tau, 1e-13, max_sweeps);
        else
            launch_jobs("sc_jacobi", jacobi_fn<float>(k), jj, dim3(1), dim3(jacobi_threads(k)),
                        jacobi_lds(k, sizeof(float)), st,
                        k, KP, r, RP, tau, 1e-5f, max_sweeps);
    }
    // U = Q Bu, V = Z Bv (first r columns)
    std::vector<orth::GemmReq> og;
    for (auto &m : ms) {
        og.push_back(orth::GemmReq{m.pw.Y, KP, m.D.m, KP, m.pw.Bu, RP, RP, m.in->U, nullptr, r, r});
        og.push_back(orth::GemmReq{m.pw.Z, KP, m.D.n, KP, m.pw.Bv, RP, RP, m.in->V, nullptr, r, r});
    }
    bool fast = true;
    for (const auto &q : og)
        fast = fast && orth::gemm_supported(q);
    if (fast)
        return orth::gemm("sc_basis", og, st);
    std::vector<GemmReq<float, float>> g;
    for (auto &m : ms) {
        g.push_back(GemmReq<float, float>{m.pw.Y, KP, m.pw.Bu, RP, m.in->U, r, m.D.m, KP, r, r, nullptr, nullptr, 0});
        g.push_back(GemmReq<float, float>{m.pw.Z, KP, m.pw.Bv, RP, m.in->V, r, m.D.n, KP, r, r, nullptr, nullptr, 0});
    }
    tall_gemm<float, false, float>("sc_basis", g, st);
    return ACSC_OK;
}

// Squared global norm of the call's G_proj and the clip coefficient (see
// clip_norm_kernel), from ||G||^2 and the filtered projections X, X_f.
template <typename GT>
void clip_norm(const std::vector<Mat> &ms, int r, float alpha, const AdamCtx &ad, hipStream_t st)
{
    std::vector<SumJob> sj;
    for (const Mat &m : ms) {
        const int64_t cnt = static_cast<int64_t>(m.D.m) * m.D.n;
        const bool vec = aligned(m.in->G, 16) && cnt % (16 / sizeof(GT)) == 0;
        sj.push_back(SumJob{m.in->G, cnt, vec ? 1 : 0, m.cw.sq});
    }
    launch_jobs("sc_sumsq", sumsq_kernel<GT>, sj, dim3(kSumBlocks), dim3(256), 0, st);
    for (size_t c0 = 0; c0 < ms.size(); c0 += kMaxBatch) {
        Batch<NormJob> b{};
        b.count = static_cast<int>(std::min<size_t>(kMaxBatch, ms.size() - c0));
        for (int i = 0; i < b.count; ++i) {
            const Mat &m = ms[c0 + i];
            b.j[i] = NormJob{m.cw.sq, m.cw.X, m.cw.Xf, r, m.D.RP, m.cw.terms};
        }
        const int first = c0 == 0, last = c0 + b.count == ms.size();
        ACSC_LAUNCH("sc_norm_terms", norm_terms_kernel, dim3(kTermBlocks, 1, b.count), dim3(256), 0, st, b, alpha);
        ACSC_LAUNCH("sc_clip_norm", clip_norm_kernel, dim3(1), dim3(64), 0, st, b, ad.max_norm, ad.acc,
                    const_cast<float *>(ad.args.coef), ad.norm_out, first, last);
    }
}

// X = U^T G V, X_f = d X d, P = U X_f, then G_proj = alpha G + (1 - alpha) P V^T,
// stored, or (adam) taken as the gradient of the AdamW step of each matrix.
template <typename GT>
int correct_group(std::vector<Mat> &ms, int r, float alpha, hipStream_t st, const AdamCtx *adam = nullptr)
{
    const int RP = ms[0].D.RP;
    const bool b16 = sizeof(GT) == 2;
    // T = G V   [m, RP]
    if (b16) {
        // V to bf16 once: transposed for T = G V, row-major for the blend
        std::vector<TileJob> t;
        std::vector<pass::Req> q;
        for (auto &m : ms) {
            t.push_back(TileJob{m.in->V, r, m.D.n, r, RP, m.cw.Vt16, m.cw.ldv16, static_cast<uint16_t *>(m.cw.Vc),
                                nullptr, 0, 0});
            const bool avec = aligned(m.in->G, 16) && (m.D.n % 8) == 0;
            q.push_back(pass::Req{static_cast<const uint16_t *>(m.in->G), m.D.n, avec, m.cw.Vt16, m.cw.ldv16, m.cw.Tm,
                                RP, m.D.m, m.D.n, RP, m.cw.part});
        }
        launch_tiles("sc_vconvert", t, st);
        const int rc = pass::run("sc_gv", false, q, st);
        if (rc)
            return rc;
    } else {
        std::vector<GemmReq<float, float>> q;
        for (auto &m : ms)
            q.push_back(GemmReq<float, float>{static_cast<const float *>(m.in->G), m.D.n, m.in->V, r, m.cw.Tm, RP,
                                              m.D.m, m.D.n, r, RP, m.cw.part, nullptr, 0});
        tall_gemm<float, false, float>("sc_gv", q, st);
    }
    // X = U^T T   [r, RP]
    {
        std::vector<orth::InnerReq> iq;
        bool fast = true;
        for (auto &m : ms) {
            iq.push_back(orth::InnerReq{m.in->U, r, m.cw.Tm, RP, m.D.m, r, RP, m.cw.X, RP, m.cw.xpart,
                                        split_count(m.D.r, m.D.m)});
            fast = fast && orth::inner_supported(iq.back());
        }
        if (fast) {
            if (int rc = orth::inner("sc_utt", iq, st))
                return rc;
        } else {
            std::vector<GemmReq<float, float>> q;
            for (auto &m : ms)
                q.push_back(GemmReq<float, float>{m.in->U, r, m.cw.Tm, RP, m.cw.X, RP, r, m.D.m, RP, RP, m.cw.xpart,
                                                  nullptr, 0});
            tall_gemm<float, true, float>("sc_utt", q, st);
        }
    }
    {
        std::vector<FilterJob> f;
        for (auto &m : ms)
            f.push_back(FilterJob{m.cw.X, m.in->d, m.cw.Xf});
        launch_jobs("sc_filter", filter_x_kernel, f, dim3(grid1d(int64_t(RP) * RP)), dim3(256), 0, st, r, RP);
    }
    // P = U X_f  [m, RP] in the compute type; V in the compute type [n, RP]
    {
        std::vector<GemmReq<float, GT>> q;
        std::vector<PadJob<GT>> pj;
        int64_t tot = 1;
        for (auto &m : ms) {
            q.push_back(GemmReq<float, GT>{m.in->U, r, m.cw.Xf, RP, static_cast<GT *>(m.cw.Pc), RP, m.D.m, r, RP, RP,
                                           nullptr, nullptr, 0});
            pj.push_back(PadJob<GT>{m.in->V, m.D.n, static_cast<GT *>(m.cw.Vc)});
            tot = std::max<int64_t>(tot, static_cast<int64_t>(m.D.n) * RP);
        }
        std::vector<orth::GemmReq> og;
        bool fast = true;
        for (auto &m : ms) {
            og.push_back(orth::GemmReq{m.in->U, r, m.D.m, r, m.cw.Xf, RP, RP,
                                       b16 ? nullptr : static_cast<float *>(m.cw.Pc),
                                       b16 ? static_cast<uint16_t *>(m.cw.Pc) : nullptr, RP, RP});
            fast = fast && orth::gemm_supported(og.back());
        }
        if (fast) {
            if (int rc = orth::gemm("sc_ux", og, st))
                return rc;
        } else {
            tall_gemm<float, false, GT>("sc_ux", q, st);
        }
        if (!b16)   // the bf16 copy was made with the transposed one
            launch_jobs("sc_vconvert", pad_convert_kernel<GT>, pj, dim3(grid1d(tot)), dim3(256), 0, st, r, RP);
    }
    if (adam)
        clip_norm<GT>(ms, r, alpha, *adam, st);
    const blend::AdamArgs ad = adam ? adam->args : blend::AdamArgs{};
    const char *btag = adam ? "sc_blend_adamw" : "sc_blend";
    {
        std::vector<BlendJob<GT>> bj;
        int gx = 1, gy = 1;
        for (auto &m : ms) {
            bj.push_back(BlendJob<GT>{static_cast<const GT *>(m.in->G), static_cast<GT *>(m.in->G_proj), m.D.m, m.D.n,
                                      static_cast<const GT *>(m.cw.Pc), static_cast<const GT *>(m.cw.Vc),
                                      m.ad ? m.ad->W : nullptr, m.ad ? m.ad->m1 : nullptr,
                                      m.ad ? m.ad->m2 : nullptr, nullptr});
            gx = std::max<int>(gx, static_cast<int>(cdiv(m.D.n, 64)));
            gy = std::max<int>(gy, static_cast<int>(cdiv(m.D.m, 64)));
        }
        if constexpr (sizeof(GT) == 2) {
            if (blend::supported(RP)) {
                std::vector<blend::Req> q;
                for (auto &m : ms)
                    q.push_back(blend::Req{static_cast<const uint16_t *>(m.in->G), static_cast<uint16_t *>(m.in->G_proj),
                                           m.D.m, m.D.n, static_cast<const uint16_t *>(m.cw.Pc),
                                           static_cast<const uint16_t *>(m.cw.Vc), m.ad ? m.ad->W : nullptr,
                                           m.ad ? m.ad->m1 : nullptr, m.ad ? m.ad->m2 : nullptr, nullptr});
                return blend::run(btag, q, RP, alpha, st, adam ? &ad : nullptr);
            }
            // 128 x 128 tiles, XCD-aware order (see blend16_kernel)
            int tiles = 1, cbm = 1;
            bool vec = true;
            for (auto &m : ms) {
                const int rbn = static_cast<int>(cdiv(m.D.m, kBT)), cbn = static_cast<int>(cdiv(m.D.n, kBT));
                tiles = std::max(tiles, static_cast<int>(round_up(rbn, 8)) * cbn);
                cbm = std::max(cbm, cbn);
                vec = vec && (m.D.n % 8) == 0 && aligned(m.in->G, 16) && (adam || aligned(m.in->G_proj, 16));
            }
            if (adam) {
                if (vec)
                    launch_jobs(btag, blend16_kernel<true, true>, bj, dim3(tiles), dim3(256), 0, st, RP, alpha, cbm, ad);
                else
                    launch_jobs(btag, blend16_kernel<false, true>, bj, dim3(tiles), dim3(256), 0, st, RP, alpha, cbm, ad);
            } else {
                if (vec)
                    launch_jobs(btag, blend16_kernel<true, false>, bj, dim3(tiles), dim3(256), 0, st, RP, alpha, cbm, ad);
                else
                    launch_jobs(btag, blend16_kernel<false, false>, bj, dim3(tiles), dim3(256), 0, st, RP, alpha, cbm, ad);
            }
        } else {
            const size_t pitch = RP + 1;
            const size_t blds = 2 * 64 * pitch * sizeof(GT);
            if (adam)
                launch_jobs(btag, blend_kernel<GT, blend::kAdam>, bj, dim3(gx, gy), dim3(256), blds, st, RP, alpha, ad);
            else
                launch_jobs(btag, blend_kernel<GT, blend::kPlain>, bj, dim3(gx, gy), dim3(256), blds, st, RP, alpha, ad);
        }
    }
    return ACSC_OK;
}

int check_matrix(const sc_matrix &a, int r, int oversample, acsc_dtype dt, bool build, size_t *need,
                 bool need_gproj = true)
{
    ACSC_CHECK_ARG(a.m >= 1 && a.n >= 1, ACSC_EINVAL, "m=%d, n=%d must be >= 1", a.m, a.n);
    ACSC_CHECK_ARG(r >= 1 && r <= std::min(std::min(a.m, a.n), kKMax), ACSC_EINVAL,
                   "r=%d outside [1, min(m, n, %d)] for a %d x %d matrix", r, kKMax, a.m, a.n);
    const Dims d = dims_of(a.m, a.n, r, oversample);
    *need = build ? carve_prior(d, dt == ACSC_BF16, nullptr, nullptr) : carve_correct(d, dtype_size(dt), nullptr, nullptr);
    ACSC_CHECK_ARG(a.ws != nullptr && a.U && a.s && a.V && a.d, ACSC_EINVAL, "null pointer argument");
    ACSC_CHECK_ARG(a.ws_bytes >= *need, ACSC_ENOSPC, "workspace %zu bytes < %zu needed", a.ws_bytes, *need);
    ACSC_CHECK_ARG(aligned(a.ws, 256), ACSC_EALIGN, "workspace must be 256-byte aligned");
    ACSC_CHECK_ARG(aligned(a.U, 4) && aligned(a.V, 4) && aligned(a.s, 4) && aligned(a.d, 4), ACSC_EALIGN,
                   "U, s, V, d must be 4-byte aligned");
    const size_t es = dtype_size(dt);
    if (build) {
        ACSC_CHECK_ARG(a.M != nullptr, ACSC_EINVAL, "M is NULL");
        ACSC_CHECK_ARG(aligned(a.M, 16), ACSC_EALIGN, "M must be 16-byte aligned");
        ACSC_CHECK_ARG(!a.G || aligned(a.G, 16), ACSC_EALIGN, "G_anc must be 16-byte aligned");
    } else {
        ACSC_CHECK_ARG(a.G && (a.G_proj || !need_gproj), ACSC_EINVAL, "G or G_proj is NULL");
        ACSC_CHECK_ARG(aligned(a.G, es) && (!need_gproj || aligned(a.G_proj, es)), ACSC_EALIGN,
                       "G, G_proj must be element-aligned");
    }
    return ACSC_OK;
}

// ---------------------------------------------------------------------------
// PowerSGD compressor with error feedback (the data-parallel compressor the
// method is paired with; rank-r step of Vogels et al. 2019):
//   project:        M = G + E (into E) and P = M Q, one sweep over M (the
//                   fused EMA pass with coefficients 1, 1, which also writes
//                   the bf16 copy of M the second projection reads)
//   orthogonalize:  P_hat = CholeskyQR2(P), Q' = M^T P_hat
//   decompress:     out = P_hat Q'^T and E = M - out, one sweep over E (the
//                   streamed-tile product with the feedback epilogue)
// The phases meet through the caller's P [m, r] and Q [n, r], so that a
// data-parallel caller can average them between the phases.
// ---------------------------------------------------------------------------

// dst [rows, cols] (row stride cols) = the first cols columns of src (row stride lds).
struct CropJob {
    const float *src;
    int64_t lds;
    float *dst;
    int rows, cols;
};

__global__ __launch_bounds__(256) void crop_kernel(const Batch<CropJob> jb)
{
    const CropJob &J = jb.j[blockIdx.z];
    const int64_t total = static_cast<int64_t>(J.rows) * J.cols;
    for (int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; idx < total;
         idx += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t i = idx / J.cols;
        const int c = static_cast<int>(idx - i * J.cols);
        J.dst[idx] = J.src[i * J.lds + c];
    }
}

// Padded rank of the decompression: the streamed-tile widths for bf16.
int psgd_rp(int r, bool use16)
{
    if (!use16)
        return static_cast<int>(round_up(r, 32));
    return r <= 64 ? 64 : (r <= 128 ? 128 : 192);
}

struct PsgdWs {
    PriorWs pw;     // M16, Zt16 (Q^T bf16), Y (P, P_hat), Yt16 (P_hat^T bf16), Z (Q'), part, T, gram
    void *Pc, *Vc;  // decompression factors [m, RPd], [n, RPd] in the compute type
    int RPd;
};

size_t carve_psgd(const Dims &d, acsc_dtype dt, void *base, PsgdWs *w)
{
    const bool use16 = dt == ACSC_BF16;
    PsgdWs t;
    Carve c(base);
    c.off = carve_prior(d, use16, base, &t.pw);
    t.RPd = psgd_rp(d.r, use16);
    const size_t es = dtype_size(dt);
    t.Pc = c.take<unsigned char>(static_cast<size_t>(d.m) * t.RPd * es);
    t.Vc = c.take<unsigned char>(static_cast<size_t>(d.n) * t.RPd * es);
    if (w)
        *w = t;
    return c.off;
}

struct PsgdItem {
    const psgd_matrix *in;
    Mat mat;   // dims and the CholeskyQR2 buffers (mat.pw == w.pw)
    PsgdWs w;
};

void crop(const char *tag, const std::vector<CropJob> &jobs, hipStream_t st)
{
    int64_t tot = 1;
    for (const CropJob &j : jobs)
        tot = std::max<int64_t>(tot, static_cast<int64_t>(j.rows) * j.cols);
    launch_jobs(tag, crop_kernel, jobs, dim3(grid1d(tot)), dim3(256), 0, st);
}

int psgd_project_phase(std::vector<PsgdItem> &it, bool use16, int r, hipStream_t st)
{
    const int KP = it[0].mat.D.KP;
    if (use16) {
        // Q^T in bf16, rows r .. KP-1 zero: the thin factor of the pass
        std::vector<TileJob> tj;
        for (auto &x : it)
            tj.push_back(TileJob{x.in->Q, r, x.in->n, r, KP, x.w.pw.Zt16, x.w.pw.ldz16, nullptr, nullptr, 0, 0});
        launch_tiles("psgd_qconvert", tj, st);
        std::vector<pass::EmaReq> er;
        for (auto &x : it)
            er.push_back(pass::EmaReq{x.in->E, static_cast<const uint16_t *>(x.in->G), x.w.pw.M16, x.w.pw.Zt16,
                                      x.w.pw.ldz16, x.w.pw.Y, KP, x.in->m, x.in->n, KP, x.w.pw.part});
        if (pass::ema_fusable(er)) {
            if (int rc = pass::ema_run("psgd_feedback_mq", er, 1.0f, 1.0f, st))
                return rc;
        } else {
            std::vector<EmaJob<uint16_t>> j;
            std::vector<pass::Req> q;
            int64_t tot = 1;
            for (auto &x : it) {
                j.push_back(EmaJob<uint16_t>{x.in->E, static_cast<const uint16_t *>(x.in->G), x.in->m, x.in->n,
                                             (x.in->n % 8) == 0 ? 1 : 0, x.w.pw.M16, x.w.pw.ntc16});
                tot = std::max<int64_t>(tot, static_cast<int64_t>(x.in->m) * cdiv(x.in->n, 8));
                q.push_back(pass::Req{x.w.pw.M16, 0, true, x.w.pw.Zt16, x.w.pw.ldz16, x.w.pw.Y, KP,
                                      x.in->m, x.in->n, KP, x.w.pw.part, static_cast<int>(x.w.pw.ntc16)});
            }
            launch_jobs("psgd_feedback", ema_shadow_kernel<uint16_t>, j, dim3(grid1d(tot)), dim3(256), 0, st, 1.0f,
                        1.0f);
            if (int rc = pass::run("psgd_pass_mq", false, q, st))
                return rc;
        }
    } else {
        std::vector<PadJob<float>> pj;
        std::vector<Ema32Job<float>> ej;
        std::vector<GemmReq<float, float>> q;
        int64_t tp = 1, te = 1;
        for (auto &x : it) {
            pj.push_back(PadJob<float>{x.in->Q, x.in->n, x.w.pw.Z});
            tp = std::max<int64_t>(tp, static_cast<int64_t>(x.in->n) * KP);
            const int64_t c = static_cast<int64_t>(x.in->m) * x.in->n;
            ej.push_back(Ema32Job<float>{x.in->E, static_cast<const float *>(x.in->G), c});
            te = std::max(te, cdiv(c, 4));
            q.push_back(GemmReq<float, float>{x.in->E, x.in->n, x.w.pw.Z, KP, x.w.pw.Y, KP, x.in->m, x.in->n, r, KP,
                                              x.w.pw.part, nullptr, 0});
        }
        launch_jobs("psgd_qconvert", pad_convert_kernel<float>, pj, dim3(grid1d(tp)), dim3(256), 0, st, r, KP);
        launch_jobs("psgd_feedback", ema_kernel<float>, ej, dim3(grid1d(te)), dim3(256), 0, st, 1.0f, 1.0f);
        tall_gemm<float, false, float>("psgd_pass_mq", q, st);
    }
    std::vector<CropJob> cj;
    for (auto &x : it)
        cj.push_back(CropJob{x.w.pw.Y, KP, x.in->P, x.in->m, r});
    crop("psgd_crop", cj, st);
    return ACSC_OK;
}

int psgd_orthogonalize_phase(std::vector<PsgdItem> &it, bool use16, int r, hipStream_t st)
{
    const int KP = it[0].mat.D.KP;
    {
        std::vector<PadJob<float>> pj;
        int64_t tp = 1;
        for (auto &x : it) {
            pj.push_back(PadJob<float>{x.in->P, x.in->m, x.w.pw.Y});
            tp = std::max<int64_t>(tp, static_cast<int64_t>(x.in->m) * KP);
        }
        launch_jobs("psgd_pconvert", pad_convert_kernel<float>, pj, dim3(grid1d(tp)), dim3(256), 0, st, r, KP);
    }
    std::vector<Mat> ms;
    for (auto &x : it)
        ms.push_back(x.mat);
    // CholeskyQR2: Y <- P_hat (fp32), and its bf16 transposed copy for the pass
    if (int rc = orthonormalise(ms, true, 2, use16, st))
        return rc;
    std::vector<CropJob> cj;
    for (auto &x : it)
        cj.push_back(CropJob{x.w.pw.Y, KP, x.in->P, x.in->m, r});
    crop("psgd_crop", cj, st);
    if (use16) {
        std::vector<pass::Req> q;
        for (auto &x : it)
            q.push_back(pass::Req{x.w.pw.M16, 0, true, x.w.pw.Yt16, x.w.pw.ldy16, x.w.pw.Z, KP, x.in->n,
                                  x.in->m, KP, x.w.pw.part, static_cast<int>(x.w.pw.ntc16)});
        if (int rc = pass::run("psgd_pass_mtp", true, q, st))
            return rc;
    } else {
        std::vector<GemmReq<float, float>> q;
        for (auto &x : it)
            q.push_back(GemmReq<float, float>{x.in->E, x.in->n, x.w.pw.Y, KP, x.w.pw.Z, KP, x.in->n, x.in->m, r, KP,
                                              x.w.pw.part, nullptr, 0});
        tall_gemm<float, true, float>("psgd_pass_mtp", q, st);
    }
    cj.clear();
    for (auto &x : it)
        cj.push_back(CropJob{x.w.pw.Z, KP, x.in->Q, x.in->n, r});
    crop("psgd_crop", cj, st);
    return ACSC_OK;
}

int psgd_decompress_phase(std::vector<PsgdItem> &it, bool use16, int r, hipStream_t st)
{
    const int RPd = it[0].w.RPd;
    if (use16) {
        std::vector<TileJob> tj;
        std::vector<blend::Req> q;
        for (auto &x : it) {
            tj.push_back(TileJob{x.in->P, r, x.in->m, r, RPd, nullptr, 0, static_cast<uint16_t *>(x.w.Pc), nullptr, 0,
                                 0});
            tj.push_back(TileJob{x.in->Q, r, x.in->n, r, RPd, nullptr, 0, static_cast<uint16_t *>(x.w.Vc), nullptr, 0,
                                 0});
            q.push_back(blend::Req{nullptr, static_cast<uint16_t *>(x.in->out), x.in->m, x.in->n,
                                   static_cast<const uint16_t *>(x.w.Pc), static_cast<const uint16_t *>(x.w.Vc),
                                   nullptr, nullptr, nullptr, x.in->E});
        }
        launch_tiles("psgd_fconvert", tj, st);
        return blend::run_feedback("psgd_decompress", q, RPd, st);
    }
    std::vector<PadJob<float>> pj;
    std::vector<BlendJob<float>> bj;
    int64_t tp = 1;
    int gx = 1, gy = 1;
    for (auto &x : it) {
        pj.push_back(PadJob<float>{x.in->P, x.in->m, static_cast<float *>(x.w.Pc)});
        pj.push_back(PadJob<float>{x.in->Q, x.in->n, static_cast<float *>(x.w.Vc)});
        tp = std::max<int64_t>(tp, static_cast<int64_t>(std::max(x.in->m, x.in->n)) * RPd);
        bj.push_back(BlendJob<float>{nullptr, static_cast<float *>(x.in->out), x.in->m, x.in->n,
                                     static_cast<const float *>(x.w.Pc), static_cast<const float *>(x.w.Vc), nullptr,
                                     nullptr, nullptr, x.in->E});
        gx = std::max<int>(gx, static_cast<int>(cdiv(x.in->n, 64)));
        gy = std::max<int>(gy, static_cast<int>(cdiv(x.in->m, 64)));
    }
    launch_jobs("psgd_fconvert", pad_convert_kernel<float>, pj, dim3(grid1d(tp)), dim3(256), 0, st, r, RPd);
    const size_t blds = 2 * 64 * static_cast<size_t>(RPd + 1) * sizeof(float);
    launch_jobs("psgd_decompress", blend_kernel<float, blend::kFeedback>, bj, dim3(gx, gy), dim3(256), blds, st, RPd,
                0.0f, blend::AdamArgs{});
    return ACSC_OK;
}

int check_psgd(const psgd_matrix &a, int i, int r, acsc_dtype dt, int phase)
{
    ACSC_CHECK_ARG(a.m >= 1 && a.n >= 1, ACSC_EINVAL, "matrix %d: m=%d, n=%d must be >= 1", i, a.m, a.n);
    ACSC_CHECK_ARG(r >= 1 && r <= std::min(std::min(a.m, a.n), kKMax), ACSC_EINVAL,
                   "matrix %d: r=%d outside [1, min(m, n, %d)] for a %d x %d matrix", i, r, kKMax, a.m, a.n);
    const Dims d = dims_of(a.m, a.n, r, 0);
    const size_t need = carve_psgd(d, dt, nullptr, nullptr);
    ACSC_CHECK_ARG(a.ws != nullptr && a.E && a.P && a.Q, ACSC_EINVAL, "matrix %d: null ws, E, P or Q", i);
    ACSC_CHECK_ARG(a.ws_bytes >= need, ACSC_ENOSPC, "matrix %d: workspace %zu bytes < %zu needed", i, a.ws_bytes,
                   need);
    ACSC_CHECK_ARG(aligned(a.ws, 256), ACSC_EALIGN, "matrix %d: workspace must be 256-byte aligned", i);
    ACSC_CHECK_ARG(aligned(a.E, 16), ACSC_EALIGN, "matrix %d: E must be 16-byte aligned", i);
    ACSC_CHECK_ARG(aligned(a.P, 4) && aligned(a.Q, 4), ACSC_EALIGN, "matrix %d: P, Q must be 4-byte aligned", i);
    if (phase == 0 || phase == 3) {
        ACSC_CHECK_ARG(a.G != nullptr, ACSC_EINVAL, "matrix %d: G is NULL", i);
        ACSC_CHECK_ARG(aligned(a.G, 16), ACSC_EALIGN, "matrix %d: G must be 16-byte aligned", i);
    }
    if (phase == 2 || phase == 3) {
        ACSC_CHECK_ARG(a.out != nullptr, ACSC_EINVAL, "matrix %d: out is NULL", i);
        ACSC_CHECK_ARG(aligned(a.out, dtype_size(dt)), ACSC_EALIGN, "matrix %d: out must be element-aligned", i);
    }
    return ACSC_OK;
}

// phase 0 project, 1 orthogonalize, 2 decompress, 3 all three
int psgd_run(int count, const psgd_matrix *mats, acsc_dtype dt, int r, int phase, hipStream_t st)
{
    clear_error();
    ACSC_CHECK_ARG(count >= 0, ACSC_EINVAL, "count=%d < 0", count);
    ACSC_CHECK_ARG(count == 0 || mats != nullptr, ACSC_EINVAL, "mats is NULL");
    ACSC_CHECK_ARG(dt == ACSC_F32 || dt == ACSC_BF16, ACSC_EDTYPE, "unknown dtype %d", (int)dt);
    std::vector<PsgdItem> it;
    for (int i = 0; i < count; ++i) {
        if (int rc = check_psgd(mats[i], i, r, dt, phase))
            return rc;
        PsgdItem x;
        x.in = &mats[i];
        x.mat.in = nullptr;
        x.mat.D = dims_of(mats[i].m, mats[i].n, r, 0);
        carve_psgd(x.mat.D, dt, mats[i].ws, &x.w);
        x.mat.pw = x.w.pw;
        x.mat.seed = 0;
        it.push_back(x);
    }
    if (it.empty())
        return ACSC_OK;
    const bool use16 = dt == ACSC_BF16;
    if (int rc = chol::prepare(it[0].mat.D.KP))
        return rc;
    if (!use16) {
        const size_t blds = 2 * 64 * static_cast<size_t>(it[0].w.RPd + 1) * sizeof(float);
        if (int rc = allow_lds(blend_kernel<float, blend::kFeedback>, blds))
            return rc;
    }
    int rc = ACSC_OK;
    if (phase == 0 || phase == 3)
        rc = psgd_project_phase(it, use16, r, st);
    if (!rc && (phase == 1 || phase == 3))
        rc = psgd_orthogonalize_phase(it, use16, r, st);
    if (!rc && (phase == 2 || phase == 3))
        rc = psgd_decompress_phase(it, use16, r, st);
    if (rc)
        return rc;
    return check_launch("psgd");
}

}  // namespace
}  // namespace acsc

using namespace acsc;

extern "C" int sc_workspace_size(int m, int n, int r, int oversample, acsc_dtype dt, size_t *bytes)
{
    clear_error();
    ACSC_CHECK_ARG(bytes != nullptr, ACSC_EINVAL, "bytes is NULL");
    ACSC_CHECK_ARG(dt == ACSC_F32 || dt == ACSC_BF16, ACSC_EDTYPE, "unknown dtype %d", (int)dt);
    ACSC_CHECK_ARG(m >= 1 && n >= 1, ACSC_EINVAL, "m=%d, n=%d must be >= 1", m, n);
    ACSC_CHECK_ARG(r >= 1 && r <= std::min(std::min(m, n), kKMax), ACSC_EINVAL,
                   "r=%d outside [1, min(m, n, %d)]", r, kKMax);
    ACSC_CHECK_ARG(oversample >= 0, ACSC_EINVAL, "oversample=%d < 0", oversample);
    const Dims d = dims_of(m, n, r, oversample);
    *bytes = std::max(carve_prior(d, dt == ACSC_BF16, nullptr, nullptr),
                      carve_correct(d, dtype_size(dt), nullptr, nullptr));
    return ACSC_OK;
}

namespace {

int build_batched(int count, const sc_matrix *mats, acsc_dtype dt, float beta, int r, int oversample,
                  int power_iters, float tau, uint64_t seed, int phases, hipStream_t stream)
{
    clear_error();
    ACSC_CHECK_ARG(count >= 0, ACSC_EINVAL, "count=%d < 0", count);
    ACSC_CHECK_ARG(count == 0 || mats != nullptr, ACSC_EINVAL, "mats is NULL");
    ACSC_CHECK_ARG(dt == ACSC_F32 || dt == ACSC_BF16, ACSC_EDTYPE, "unknown dtype %d", (int)dt);
    ACSC_CHECK_ARG(beta >= 0.f && beta <= 1.f, ACSC_EINVAL, "beta=%g outside [0, 1]", beta);
    ACSC_CHECK_ARG(tau >= 0.f && std::isfinite(tau), ACSC_EINVAL, "tau=%g must be finite, >= 0", tau);
    ACSC_CHECK_ARG(power_iters >= 0 && power_iters <= 64, ACSC_EINVAL, "power_iters=%d outside [0, 64]",
                   power_iters);
    ACSC_CHECK_ARG(oversample >= 0, ACSC_EINVAL, "oversample=%d < 0", oversample);
    std::vector<Mat> all;
    for (int i = 0; i < count; ++i) {
        size_t need = 0;
        int rc = check_matrix(mats[i], r, oversample, dt, true, &need);
        if (rc)
            return rc;
        Mat m;
        m.in = &mats[i];
        m.D = dims_of(mats[i].m, mats[i].n, r, oversample);
        carve_prior(m.D, dt == ACSC_BF16, mats[i].ws, &m.pw);
        m.seed = seed + static_cast<uint64_t>(i);
        all.push_back(m);
    }
    if (all.empty())
        return ACSC_OK;
    // LDS of the one-workgroup kernels, for every k in the batch
    for (const Mat &m : all) {
        int rc = chol::prepare(m.D.KP);
        if (!rc)
            rc = m.D.k <= kJacobiF64MaxK ? allow_lds(jacobi_fn<double>(m.D.k), jacobi_lds(m.D.k, sizeof(double)))
                                         : allow_lds(jacobi_fn<float>(m.D.k), jacobi_lds(m.D.k, sizeof(float)));
        if (rc)
            return rc;
    }
    // matrices with the same k (= min(r + oversample, m, n)) share every launch
    std::vector<bool> done(all.size(), false);
    for (size_t i = 0; i < all.size(); ++i) {
        if (done[i])
            continue;
        std::vector<Mat> group;
        for (size_t j = i; j < all.size(); ++j)
            if (!done[j] && all[j].D.k == all[i].D.k) {
                group.push_back(all[j]);
                done[j] = true;
            }
        const int rc = build_group(group, dt, beta, r, power_iters, tau, phases, stream);
        if (rc)
            return rc;
    }
    return check_launch("sc_build_prior");
}

}  // namespace

extern "C" int sc_build_prior_batched(int count, const sc_matrix *mats, acsc_dtype dt, float beta, int r,
                                      int oversample, int power_iters, float tau, uint64_t seed,
                                      hipStream_t stream)
{
    return build_batched(count, mats, dt, beta, r, oversample, power_iters, tau, seed,
                         kPhaseSubspace | kPhaseRitz, stream);
}

extern "C" int sc_build_subspace_batched(int count, const sc_matrix *mats, acsc_dtype dt, float beta, int r,
                                         int oversample, int power_iters, float tau, uint64_t seed,
                                         hipStream_t stream)
{
    return build_batched(count, mats, dt, beta, r, oversample, power_iters, tau, seed, kPhaseSubspace, stream);
}

extern "C" int sc_build_ritz_batched(int count, const sc_matrix *mats, acsc_dtype dt, float beta, int r,
                                     int oversample, int power_iters, float tau, uint64_t seed,
                                     hipStream_t stream)
{
    return build_batched(count, mats, dt, beta, r, oversample, power_iters, tau, seed, kPhaseRitz, stream);
}

extern "C" int sc_build_status(int count, const sc_matrix *mats, int *sweeps, float *residual, hipStream_t stream)
{
    clear_error();
    ACSC_CHECK_ARG(count >= 0, ACSC_EINVAL, "count=%d < 0", count);
    ACSC_CHECK_ARG(count == 0 || mats != nullptr, ACSC_EINVAL, "mats is NULL");
    for (int i = 0; i < count; ++i) {
        ACSC_CHECK_ARG(mats[i].ws != nullptr, ACSC_EINVAL, "matrix %d: workspace is NULL", i);
        ACSC_CHECK_ARG(aligned(mats[i].ws, 256), ACSC_EALIGN, "matrix %d: workspace must be 256-byte aligned", i);
        ACSC_CHECK_ARG(mats[i].ws_bytes >= 5 * sizeof(int), ACSC_ENOSPC, "matrix %d: workspace too small", i);
    }
    std::vector<int> words(static_cast<size_t>(count) * 5, 0);
    for (int i = 0; i < count; ++i) {
        const hipError_t e = hipMemcpyAsync(words.data() + 5 * i, mats[i].ws, 5 * sizeof(int), hipMemcpyDeviceToHost,
                                            stream);
        if (e != hipSuccess)
            return set_error(ACSC_EHIP, "reading the status of matrix %d: %s", i, hipGetErrorString(e));
    }
    const hipError_t e = hipStreamSynchronize(stream);
    if (e != hipSuccess)
        return set_error(ACSC_EHIP, "hipStreamSynchronize: %s", hipGetErrorString(e));
    int rc = ACSC_OK;
    for (int i = 0; i < count; ++i) {
        const int *w = words.data() + 5 * i;
        float res, tol;
        std::memcpy(&res, &w[kInfoResidual], sizeof(float));
        std::memcpy(&tol, &w[kInfoTol], sizeof(float));
        if (sweeps)
            sweeps[i] = w[kInfoSweeps];
        if (residual)
            residual[i] = res;
        if (rc)
            continue;   // report the first failing matrix
        if (w[kInfoStatus] & kStatusNoSubspace)
            rc = set_error(ACSC_ENOCONV, "matrix %d: the Rayleigh-Ritz phase ran without a subspace phase on its "
                                         "workspace before it", i);
        else if (w[kInfoStatus] & kStatusStalled)
            rc = set_error(ACSC_ENOCONV, "matrix %d: a wait of the fused EMA pass ran out of polls (its "
                                         "subspace and prior are not to be trusted)", i);
        else if (w[kInfoStatus] & kStatusNoConv)
            rc = set_error(ACSC_ENOCONV, "matrix %d: the Rayleigh-Ritz Jacobi stopped after %d sweeps with an "
                                         "off-diagonal ratio %g above its tolerance %g", i, w[kInfoSweeps], res, tol);
        else if (w[kInfoStatus] != 0)
            rc = set_error(ACSC_ENOCONV, "matrix %d: no status of a build (word %d)", i, w[kInfoStatus]);
    }
    return rc;
}

extern "C" int sc_correct_batched(int count, const sc_matrix *mats, acsc_dtype dt, int r, float alpha,
                                  hipStream_t stream)
{
    clear_error();
    ACSC_CHECK_ARG(count >= 0, ACSC_EINVAL, "count=%d < 0", count);
    ACSC_CHECK_ARG(count == 0 || mats != nullptr, ACSC_EINVAL, "mats is NULL");
    ACSC_CHECK_ARG(dt == ACSC_F32 || dt == ACSC_BF16, ACSC_EDTYPE, "unknown dtype %d", (int)dt);
    ACSC_CHECK_ARG(std::isfinite(alpha), ACSC_EINVAL, "alpha must be finite");
    std::vector<Mat> all;
    for (int i = 0; i < count; ++i) {
        size_t need = 0;
        int rc = check_matrix(mats[i], r, 0, dt, false, &need);
        if (rc)
            return rc;
        Mat m;
        m.in = &mats[i];
        m.D = dims_of(mats[i].m, mats[i].n, r, 0);
        carve_correct(m.D, dtype_size(dt), mats[i].ws, &m.cw);
        m.seed = 0;
        all.push_back(m);
    }
    if (all.empty())
        return ACSC_OK;
    const size_t es = dtype_size(dt);
    const size_t blds = 2 * 64 * (all[0].D.RP + (dt == ACSC_BF16 ? 8 : 1)) * es;
    int rc = dt == ACSC_BF16 ? allow_lds(blend_kernel<uint16_t, blend::kPlain>, blds) : allow_lds(blend_kernel<float, blend::kPlain>, blds);
    if (rc)
        return rc;
    if (dt == ACSC_BF16)
        rc = correct_group<uint16_t>(all, r, alpha, stream);
    else
        rc = correct_group<float>(all, r, alpha, stream);
    if (rc)
        return rc;
    return check_launch("sc_correct");
}

extern "C" int sc_adamw_workspace_size(int m, int n, int r, acsc_dtype dt, size_t *bytes)
{
    clear_error();
    ACSC_CHECK_ARG(bytes != nullptr, ACSC_EINVAL, "bytes is NULL");
    ACSC_CHECK_ARG(dt == ACSC_F32 || dt == ACSC_BF16, ACSC_EDTYPE, "unknown dtype %d", (int)dt);
    ACSC_CHECK_ARG(m >= 1 && n >= 1, ACSC_EINVAL, "m=%d, n=%d must be >= 1", m, n);
    ACSC_CHECK_ARG(r >= 1 && r <= std::min(std::min(m, n), kKMax), ACSC_EINVAL,
                   "r=%d outside [1, min(m, n, %d)]", r, kKMax);
    *bytes = carve_correct(dims_of(m, n, r, 0), dtype_size(dt), nullptr, nullptr);
    return ACSC_OK;
}

extern "C" int sc_correct_adamw_batched(int count, const sc_matrix *mats, const sc_adamw_state *states,
                                        acsc_dtype dt, int r, float alpha, const sc_adamw_hparams *hp,
                                        float *norm_out, hipStream_t stream)
{
    clear_error();
    ACSC_CHECK_ARG(count >= 0, ACSC_EINVAL, "count=%d < 0", count);
    ACSC_CHECK_ARG(count == 0 || (mats != nullptr && states != nullptr), ACSC_EINVAL, "mats or states is NULL");
    ACSC_CHECK_ARG(hp != nullptr, ACSC_EINVAL, "hp is NULL");
    ACSC_CHECK_ARG(dt == ACSC_F32 || dt == ACSC_BF16, ACSC_EDTYPE, "unknown dtype %d", (int)dt);
    ACSC_CHECK_ARG(std::isfinite(alpha), ACSC_EINVAL, "alpha must be finite");
    ACSC_CHECK_ARG(std::isfinite(hp->lr) && hp->lr >= 0.f, ACSC_EINVAL, "lr=%g must be finite, >= 0", hp->lr);
    ACSC_CHECK_ARG(hp->beta1 >= 0.f && hp->beta1 < 1.f && hp->beta2 >= 0.f && hp->beta2 < 1.f, ACSC_EINVAL,
                   "betas (%g, %g) must lie in [0, 1)", hp->beta1, hp->beta2);
    ACSC_CHECK_ARG(std::isfinite(hp->eps) && hp->eps > 0.f, ACSC_EINVAL, "eps=%g must be finite, > 0", hp->eps);
    ACSC_CHECK_ARG(std::isfinite(hp->weight_decay) && hp->weight_decay >= 0.f, ACSC_EINVAL,
                   "weight_decay=%g must be finite, >= 0", hp->weight_decay);
    ACSC_CHECK_ARG(hp->step >= 1, ACSC_EINVAL, "step=%lld must be >= 1", (long long)hp->step);
    ACSC_CHECK_ARG(std::isfinite(hp->max_norm), ACSC_EINVAL, "max_norm must be finite");
    ACSC_CHECK_ARG(!norm_out || aligned(norm_out, 4), ACSC_EALIGN, "norm_out must be 4-byte aligned");
    std::vector<Mat> all;
    for (int i = 0; i < count; ++i) {
        size_t need = 0;
        int rc = check_matrix(mats[i], r, 0, dt, false, &need, false);
        if (rc)
            return rc;
        const sc_adamw_state &a = states[i];
        ACSC_CHECK_ARG(a.W && a.m1 && a.m2, ACSC_EINVAL, "state %d: W, m1 or m2 is NULL", i);
        ACSC_CHECK_ARG(aligned(a.W, 4) && aligned(a.m1, 4) && aligned(a.m2, 4), ACSC_EALIGN,
                       "state %d: W, m1, m2 must be 4-byte aligned", i);
        Mat m;
        m.in = &mats[i];
        m.D = dims_of(mats[i].m, mats[i].n, r, 0);
        carve_correct(m.D, dtype_size(dt), mats[i].ws, &m.cw);
        m.seed = 0;
        m.ad = &a;
        all.push_back(m);
    }
    if (all.empty())
        return ACSC_OK;
    const size_t es = dtype_size(dt);
    const size_t blds = 2 * 64 * (all[0].D.RP + (dt == ACSC_BF16 ? 8 : 1)) * es;
    int rc = dt == ACSC_BF16 ? allow_lds(blend_kernel<uint16_t, blend::kAdam>, blds) : allow_lds(blend_kernel<float, blend::kAdam>, blds);
    if (rc)
        return rc;
    // bias corrections and the step size in double on the host, then fp32
    const double t = static_cast<double>(hp->step);
    const double bc1 = 1.0 - std::pow(static_cast<double>(hp->beta1), t);
    const double bc2 = 1.0 - std::pow(static_cast<double>(hp->beta2), t);
    AdamCtx ctx{};
    ctx.args.beta1 = hp->beta1;
    ctx.args.beta2 = hp->beta2;
    ctx.args.omb1 = static_cast<float>(1.0 - hp->beta1);
    ctx.args.omb2 = static_cast<float>(1.0 - hp->beta2);
    ctx.args.wdf = static_cast<float>(1.0 - static_cast<double>(hp->lr) * hp->weight_decay);
    ctx.args.step = static_cast<float>(hp->lr / bc1);
    ctx.args.isbc2 = static_cast<float>(1.0 / std::sqrt(bc2));
    ctx.args.eps = hp->eps;
    ctx.args.coef = all[0].cw.coef;
    ctx.acc = all[0].cw.acc;
    ctx.max_norm = hp->max_norm;
    ctx.norm_out = norm_out;
    if (dt == ACSC_BF16)
        rc = correct_group<uint16_t>(all, r, alpha, stream, &ctx);
    else
        rc = correct_group<float>(all, r, alpha, stream, &ctx);
    if (rc)
        return rc;
    return check_launch("sc_correct_adamw");
}

extern "C" int sc_build_prior(const void *G_anc, acsc_dtype dt, float *M, int m, int n, float beta, int r,
                              int oversample, int power_iters, float tau, const float *V_warm, uint64_t seed,
                              float *U, float *s, float *V, float *d, void *ws, size_t ws_bytes,
                              hipStream_t stream)
{
    sc_matrix a{};
    a.G = G_anc;
    a.M = M;
    a.m = m;
    a.n = n;
    a.U = U;
    a.s = s;
    a.V = V;
    a.d = d;
    a.V_warm = V_warm;
    a.ws = ws;
    a.ws_bytes = ws_bytes;
    return sc_build_prior_batched(1, &a, dt, beta, r, oversample, power_iters, tau, seed, stream);
}

extern "C" int sc_correct(const void *G, acsc_dtype dt, int m, int n, const float *U, const float *d,
                          const float *V, int r, float alpha, void *G_proj, void *ws, size_t ws_bytes,
                          hipStream_t stream)
{
    sc_matrix a{};
    a.G = G;
    a.m = m;
    a.n = n;
    a.U = const_cast<float *>(U);
    a.s = const_cast<float *>(d);   // unused by the correction; only checked non-null
    a.V = const_cast<float *>(V);
    a.d = const_cast<float *>(d);
    a.G_proj = G_proj;
    a.ws = ws;
    a.ws_bytes = ws_bytes;
    return sc_correct_batched(1, &a, dt, r, alpha, stream);
}

extern "C" int psgd_workspace_size(int m, int n, int r, acsc_dtype dt, size_t *bytes)
{
    clear_error();
    ACSC_CHECK_ARG(bytes != nullptr, ACSC_EINVAL, "bytes is NULL");
    ACSC_CHECK_ARG(dt == ACSC_F32 || dt == ACSC_BF16, ACSC_EDTYPE, "unknown dtype %d", (int)dt);
    ACSC_CHECK_ARG(m >= 1 && n >= 1, ACSC_EINVAL, "m=%d, n=%d must be >= 1", m, n);
    ACSC_CHECK_ARG(r >= 1 && r <= std::min(std::min(m, n), kKMax), ACSC_EINVAL,
                   "r=%d outside [1, min(m, n, %d)]", r, kKMax);
    *bytes = carve_psgd(dims_of(m, n, r, 0), dt, nullptr, nullptr);
    return ACSC_OK;
}

extern "C" int psgd_project(int count, const psgd_matrix *mats, acsc_dtype dt, int r, hipStream_t stream)
{
    return psgd_run(count, mats, dt, r, 0, stream);
}

extern "C" int psgd_orthogonalize(int count, const psgd_matrix *mats, acsc_dtype dt, int r, hipStream_t stream)
{
    return psgd_run(count, mats, dt, r, 1, stream);
}

extern "C" int psgd_decompress(int count, const psgd_matrix *mats, acsc_dtype dt, int r, hipStream_t stream)
{
    return psgd_run(count, mats, dt, r, 2, stream);
}

extern "C" int psgd_step(int count, const psgd_matrix *mats, acsc_dtype dt, int r, hipStream_t stream)
{
    return psgd_run(count, mats, dt, r, 3, stream);
}
