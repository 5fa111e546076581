// Spectral corrector for gfx950 (paper Sec. 3.2; Alg. 1; App. D).
//
// sc_build_prior: anchor EMA, then the top-r SVD of the EMA by randomised
// block subspace iteration (MFMA tall-skinny passes over M, CholeskyQR2 with an
// fp64 Gram and an fp64 Cholesky in LDS), Rayleigh-Ritz by one-sided Jacobi in
// LDS, and the soft filter.
// sc_correct: T = G V (MFMA, split-K), X = U^T T, X_f = d X d, P = U X_f, then
// one fused pass G_proj = alpha G + (1 - alpha) P V^T.
#include "common.h"

#include <algorithm>

namespace acsc {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(short)))) short bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;

constexpr int kKMax = SC_KMAX;
constexpr int kBM = 64;   // rows of the output per workgroup in the tall GEMM
constexpr int kBK = 32;   // depth of one K step
constexpr int kNTMax = kKMax / 16;
// Singular values of the prior at or below this fraction of the largest are
// returned as zero (numerical rank of an fp32 subspace iteration).
constexpr double kRankCutoff = 1e-5;

__host__ __device__ inline int64_t round_up(int64_t a, int64_t b) { return (a + b - 1) / b * b; }
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

template <typename TA, bool TRANS, typename TO>
__global__ __launch_bounds__(256) void gemm_tall_kernel(const TA *A, int64_t lda, const float *B,
                                                        int64_t ldb, TO *C, int64_t ldc,
                                                        int64_t split_stride, int M, int K,
                                                        int nvalid, int nwrite, int kchunk)
{
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
                if (row < M && col < nwrite)
                    Cs[static_cast<int64_t>(row) * ldc + col] = from_f32<TO>(acc[t][e]);
            }
        }
    }
}

// C[i, c] = sum_s P[s][i, c] for c < nwrite (P has row stride ldp).
template <typename TO>
__global__ __launch_bounds__(256) void reduce_splits_kernel(const float *P, int64_t ldp,
                                                            int64_t split_stride, int splits,
                                                            int M, int nwrite, TO *C, int64_t ldc)
{
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
// fp64 Gram matrix of the first KP columns of A (rows x lda, fp32):
// upper 64x64 tiles per workgroup, rows split across grid.y, partials summed
// by gram_reduce_kernel, which also mirrors the lower triangle.
// ---------------------------------------------------------------------------
constexpr int kGT = 64;
constexpr int kGRows = 32;

__global__ __launch_bounds__(256) void gram_partial_kernel(const float *A, int64_t lda, int rows,
                                                           int KP, int rows_per_block,
                                                           double *part)
{
    __shared__ float Ai[kGRows][kGT + 1];
    __shared__ float Aj[kGRows][kGT + 1];
    const int nt = static_cast<int>(cdiv(KP, kGT));
    // map blockIdx.x to an upper tile (ti <= tj)
    int t = blockIdx.x, ti = 0;
    while (t >= nt - ti) {
        t -= nt - ti;
        ++ti;
    }
    const int tj = ti + t;
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    const int r0 = blockIdx.y * rows_per_block;
    const int r1 = min(rows, r0 + rows_per_block);
    double acc[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b)
            acc[a][b] = 0.0;
    for (int rb = r0; rb < r1; rb += kGRows) {
        __syncthreads();
        for (int idx = threadIdx.x; idx < kGRows * kGT; idx += 256) {
            const int rr = idx / kGT, c = idx % kGT;
            const int gr = rb + rr;
            const int ci = ti * kGT + c, cj = tj * kGT + c;
            Ai[rr][c] = (gr < r1 && ci < KP) ? A[static_cast<int64_t>(gr) * lda + ci] : 0.f;
            Aj[rr][c] = (gr < r1 && cj < KP) ? A[static_cast<int64_t>(gr) * lda + cj] : 0.f;
        }
        __syncthreads();
#pragma unroll 4
        for (int rr = 0; rr < kGRows; ++rr) {
            double ai[4], aj[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                ai[e] = static_cast<double>(Ai[rr][ty * 4 + e]);
                aj[e] = static_cast<double>(Aj[rr][tx * 4 + e]);
            }
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
                for (int b = 0; b < 4; ++b)
                    acc[a][b] = __builtin_fma(ai[a], aj[b], acc[a][b]);
        }
    }
    double *pb = part + static_cast<int64_t>(blockIdx.y) * KP * KP;
#pragma unroll
    for (int a = 0; a < 4; ++a) {
        const int i = ti * kGT + ty * 4 + a;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const int j = tj * kGT + tx * 4 + b;
            if (i < KP && j < KP)
                pb[static_cast<int64_t>(i) * KP + j] = acc[a][b];
        }
    }
}

__global__ __launch_bounds__(256) void gram_reduce_kernel(const double *part, int blocks, int KP,
                                                          double *G)
{
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= KP * KP)
        return;
    int i = idx / KP, j = idx % KP;
    if (i / kGT > j / kGT) {   // lower tiles were not computed: use the mirror
        const int t = i;
        i = j;
        j = t;
    }
    double s = 0.0;
    for (int b = 0; b < blocks; ++b)
        s += part[static_cast<int64_t>(b) * KP * KP + static_cast<int64_t>(i) * KP + j];
    G[idx] = s;
}

// ---------------------------------------------------------------------------
// Cholesky G = L L^T of a k x k Gram matrix in LDS (fp64, packed lower
// triangle), one workgroup.  Pivots below tiny * max(diag) are taken as zero
// (the column of L becomes zero: a rank-deficient block).
//   INVERT: write T = L^{-T} (k x k, fp32, zero-padded to KP x KP) so that
//           Q = Y T has orthonormal columns (CholeskyQR).
//   else:   write L itself (fp64, KP x KP, zero upper part).
// ---------------------------------------------------------------------------
__device__ __forceinline__ int tri(int i) { return i * (i + 1) / 2; }

template <bool INVERT>
__global__ __launch_bounds__(1024) void chol_kernel(double *G, int k, int KP, float *Tout)
{
    extern __shared__ double Lp[];
    double *tmp = Lp + tri(k);
    __shared__ double sh_max;
    const int tid = threadIdx.x;
    const int nth = blockDim.x;
    for (int idx = tid; idx < k * k; idx += nth) {
        const int i = idx / k, j = idx % k;
        if (j <= i)
            Lp[tri(i) + j] = G[static_cast<int64_t>(i) * KP + j];
    }
    __syncthreads();
    if (tid == 0) {
        double mx = 0.0;
        for (int i = 0; i < k; ++i)
            mx = fmax(mx, Lp[tri(i) + i]);
        sh_max = mx;
    }
    __syncthreads();
    const double thresh = 1e-15 * sh_max * k;
    for (int j = 0; j < k; ++j) {
        if (tid == 0) {
            const double dj = Lp[tri(j) + j];
            Lp[tri(j) + j] = (dj > thresh) ? sqrt(dj) : 0.0;
        }
        __syncthreads();
        const double piv = Lp[tri(j) + j];
        const double inv = piv > 0.0 ? 1.0 / piv : 0.0;
        for (int i = j + 1 + tid; i < k; i += nth)
            Lp[tri(i) + j] *= inv;
        __syncthreads();
        const int w = k - j - 1;
        for (int p = tid; p < w * w; p += nth) {
            const int i = j + 1 + p / w;
            const int c = j + 1 + p % w;
            if (c <= i)
                Lp[tri(i) + c] -= Lp[tri(i) + j] * Lp[tri(c) + j];
        }
        __syncthreads();
    }
    if (INVERT) {
        // in-place inverse of the lower-triangular factor, last column first
        for (int j = k - 1; j >= 0; --j) {
            const double ljj = Lp[tri(j) + j];
            const double ij = ljj > 0.0 ? 1.0 / ljj : 0.0;
            for (int i = j + 1 + tid; i < k; i += nth)
                tmp[i] = Lp[tri(i) + j];
            __syncthreads();
            for (int i = j + 1 + tid; i < k; i += nth) {
                double s = 0.0;
                for (int c = j + 1; c <= i; ++c)
                    s += Lp[tri(i) + c] * tmp[c];
                Lp[tri(i) + j] = -ij * s;
            }
            __syncthreads();
            if (tid == 0)
                Lp[tri(j) + j] = ij;
            __syncthreads();
        }
        // T[c][i] = Linv[i][c]
        for (int idx = tid; idx < KP * KP; idx += nth) {
            const int c = idx / KP, i = idx % KP;
            float v = 0.f;
            if (i < k && c < k && c <= i)
                v = static_cast<float>(Lp[tri(i) + c]);
            Tout[idx] = v;
        }
    } else {
        for (int idx = tid; idx < KP * KP; idx += nth) {
            const int i = idx / KP, c = idx % KP;
            G[idx] = (i < k && c < k && c <= i) ? Lp[tri(i) + c] : 0.0;
        }
    }
}

// ---------------------------------------------------------------------------
// One-sided (Hestenes) Jacobi SVD of the k x k factor L in LDS, one
// workgroup: rotate column pairs (round-robin tournament, one pair per wave at
// a time) until every pair is orthogonal to `tol`.  Then sigma_c = ||a_c||,
// u_c = a_c / sigma_c, sorted descending, and the right factors of the final
// products are written:  Bu[:, t] = u_(t), Bv[:, t] = u_(t) / sigma_(t),
// s[t] = sigma_(t), d[t] = s / (s + tau) for t < r.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(1024) void jacobi_kernel(const double *Lf, int k, int KP, int r,
                                                      int RP, float tau, T tol, int max_sweeps,
                                                      float *Bu, float *Bv, float *s_out,
                                                      float *d_out)
{
    extern __shared__ __attribute__((aligned(16))) unsigned char jsm[];
    T *A = reinterpret_cast<T *>(jsm);   // column c at A[c * k]
    __shared__ unsigned int sh_off;
    __shared__ double sh_cut;
    __shared__ double sig[kKMax];
    __shared__ int rank_of[kKMax];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nwave = blockDim.x >> 6;
    for (int idx = tid; idx < k * k; idx += blockDim.x) {
        const int c = idx / k, i = idx % k;
        A[c * k + i] = static_cast<T>(Lf[static_cast<int64_t>(i) * KP + c]);
    }
    const int n2 = k + (k & 1);
    const int npairs = n2 / 2;
    for (int sweep = 0; sweep < max_sweeps; ++sweep) {
        if (tid == 0)
            sh_off = 0u;
        __syncthreads();
        float wmax = 0.f;
        for (int round = 0; round < n2 - 1; ++round) {
            for (int p = wave; p < npairs; p += nwave) {
                auto pos = [&](int x) { return x == 0 ? 0 : ((x - 1 + round) % (n2 - 1)) + 1; };
                int cp = pos(p), cq = pos(n2 - 1 - p);
                if (cp >= k || cq >= k)
                    continue;
                if (cp > cq) {
                    const int t = cp;
                    cp = cq;
                    cq = t;
                }
                T *ap = A + cp * k;
                T *aq = A + cq * k;
                double al = 0.0, be = 0.0, ga = 0.0;
                for (int i = lane; i < k; i += 64) {
                    const double x = ap[i], y = aq[i];
                    al += x * x;
                    be += y * y;
                    ga += x * y;
                }
#pragma unroll
                for (int off = 32; off >= 1; off >>= 1) {
                    al += __shfl_xor(al, off, 64);
                    be += __shfl_xor(be, off, 64);
                    ga += __shfl_xor(ga, off, 64);
                }
                const double nrm = sqrt(al * be);
                if (ga == 0.0 || nrm == 0.0)
                    continue;
                const double ratio = fabs(ga) / nrm;
                wmax = fmaxf(wmax, static_cast<float>(ratio));
                if (ratio <= static_cast<double>(tol))
                    continue;
                const double zeta = (be - al) / (2.0 * ga);
                const double t = (zeta >= 0.0 ? 1.0 : -1.0) / (fabs(zeta) + sqrt(1.0 + zeta * zeta));
                const double c = 1.0 / sqrt(1.0 + t * t);
                const double sn = c * t;
                for (int i = lane; i < k; i += 64) {
                    const double x = ap[i], y = aq[i];
                    ap[i] = static_cast<T>(c * x - sn * y);
                    aq[i] = static_cast<T>(sn * x + c * y);
                }
            }
            __syncthreads();
        }
        if (lane == 0)
            atomicMax(&sh_off, __float_as_uint(wmax));
        __syncthreads();
        const float off = __uint_as_float(sh_off);
        __syncthreads();
        if (off <= static_cast<float>(tol))
            break;
    }
    // norms (one wave per column)
    for (int c = wave; c < k; c += nwave) {
        double ss = 0.0;
        for (int i = lane; i < k; i += 64) {
            const double x = A[c * k + i];
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
            const double u = sg > 0.0 ? static_cast<double>(A[c * k + i]) / sg : 0.0;
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
__global__ __launch_bounds__(256) void ema_kernel(float *M, const GT *G, int64_t count, float beta,
                                                  float omb)
{
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
            m.x = beta * m.x + omb * g0;
            m.y = beta * m.y + omb * g1;
            m.z = beta * m.z + omb * g2;
            m.w = beta * m.w + omb * g3;
            *reinterpret_cast<float4 *>(M + i) = m;
        } else {
            for (int64_t j = i; j < count; ++j)
                M[j] = beta * M[j] + omb * to_f32<GT>(G[j]);
        }
    }
}

// Starting block Z0 [n, KP]: V_warm columns first (if given), then uniform
// random values in [-1, 1) from a counter-based hash of (seed, i, c); zero
// beyond k.
__global__ __launch_bounds__(256) void init_block_kernel(float *Z, int n, int k, int KP,
                                                         const float *Vw, int rw, uint64_t seed)
{
    const int64_t total = static_cast<int64_t>(n) * KP;
    for (int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; idx < total;
         idx += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t i = idx / KP;
        const int c = static_cast<int>(idx - i * KP);
        float v = 0.f;
        if (c < k) {
            if (Vw && c < rw) {
                v = Vw[i * rw + c];
            } else {
                uint64_t z = seed ^ (static_cast<uint64_t>(i) * 0x100000001B3ull + c);
                z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
                z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
                z ^= z >> 31;
                v = static_cast<float>(z >> 40) * (2.0f / 16777216.0f) - 1.0f;
            }
        }
        Z[idx] = v;
    }
}

// Xf[i][j] = d_i * X[i][j] * d_j for i, j < r; zero elsewhere (RP x RP).
__global__ __launch_bounds__(256) void filter_x_kernel(const float *X, int64_t ldx, const float *d,
                                                       int r, int RP, float *Xf)
{
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= RP * RP)
        return;
    const int i = idx / RP, j = idx % RP;
    Xf[idx] = (i < r && j < r) ? d[i] * X[static_cast<int64_t>(i) * ldx + j] * d[j] : 0.f;
}

// Vc[i][c] = V[i][c] for c < r, zero up to RP, converted to the compute type.
template <typename CT>
__global__ __launch_bounds__(256) void pad_convert_kernel(const float *V, int n, int r, int RP,
                                                          CT *Vc)
{
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
__global__ __launch_bounds__(256) void blend_kernel(const GT *G, GT *out, int m, int n, const GT *P,
                                                    const GT *Vc, int RP, float alpha)
{
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
                    const float g = to_f32<GT>(G[o]);
                    out[o] = from_f32<GT>(alpha * g + oma * acc[a][b][e]);
                }
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

int gram_blocks(int64_t rows) { return static_cast<int>(std::min<int64_t>(64, cdiv(rows, 512))); }

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
    float *Y, *Z, *part, *T, *Bu, *Bv;
    double *gpart, *gram;
};

size_t carve_prior(const Dims &d, void *base, PriorWs *w)
{
    Carve c(base);
    const int64_t mx = std::max(d.m, d.n);
    const int s1 = split_count(d.m, d.n), s2 = split_count(d.n, d.m);
    const int64_t part = std::max<int64_t>(static_cast<int64_t>(s1) * d.m, static_cast<int64_t>(s2) * d.n) * d.KP;
    PriorWs t;
    t.Y = c.take<float>(static_cast<size_t>(d.m) * d.KP);
    t.Z = c.take<float>(static_cast<size_t>(d.n) * d.KP);
    t.part = c.take<float>(static_cast<size_t>(part));
    t.T = c.take<float>(static_cast<size_t>(d.KP) * d.KP);
    t.Bu = c.take<float>(static_cast<size_t>(d.KP) * d.RP);
    t.Bv = c.take<float>(static_cast<size_t>(d.KP) * d.RP);
    t.gpart = c.take<double>(static_cast<size_t>(gram_blocks(mx)) * d.KP * d.KP);
    t.gram = c.take<double>(static_cast<size_t>(d.KP) * d.KP);
    if (w)
        *w = t;
    return c.off;
}

// Buffers of sc_correct.
struct CorrWs {
    float *Tm, *part, *xpart, *X, *Xf;
    void *Pc, *Vc;
};

size_t carve_correct(const Dims &d, size_t esize, void *base, CorrWs *w)
{
    Carve c(base);
    const int s1 = split_count(d.m, d.n);
    const int s2 = split_count(d.r, d.m);
    CorrWs t;
    t.Tm = c.take<float>(static_cast<size_t>(d.m) * d.RP);
    t.part = c.take<float>(static_cast<size_t>(s1) * d.m * d.RP);
    t.xpart = c.take<float>(static_cast<size_t>(s2) * d.r * d.RP);
    t.X = c.take<float>(static_cast<size_t>(d.r) * d.RP);
    t.Xf = c.take<float>(static_cast<size_t>(d.RP) * d.RP);
    t.Pc = c.take<unsigned char>(static_cast<size_t>(d.m) * d.RP * esize);
    t.Vc = c.take<unsigned char>(static_cast<size_t>(d.n) * d.RP * esize);
    if (w)
        *w = t;
    return c.off;
}

unsigned grid1d(int64_t total, int per = 256)
{
    return static_cast<unsigned>(std::max<int64_t>(1, std::min<int64_t>(cdiv(total, per), 65536)));
}

// C = opA * B with split-K through `part` when more than one split pays off.
template <typename TA, bool TRANS, typename TO>
void tall_gemm(const char *tag, const TA *A, int64_t lda, const float *B, int64_t ldb, TO *C,
               int64_t ldc, int M, int K, int nvalid, int nwrite, float *part, int splits,
               hipStream_t st)
{
    const int NP = static_cast<int>(round_up(nwrite, 16));
    const int64_t chunk = split_chunk(K, splits);
    splits = static_cast<int>(cdiv(K, chunk));
    const dim3 grid(static_cast<unsigned>(cdiv(M, kBM)), static_cast<unsigned>(splits));
    if (splits == 1) {
        ACSC_LAUNCH(tag, (gemm_tall_kernel<TA, TRANS, TO>), grid, dim3(256), 0, st, A, lda, B,
                           ldb, C, ldc, int64_t(0), M, K, nvalid, nwrite, static_cast<int>(chunk));
        return;
    }
    const int64_t ss = static_cast<int64_t>(M) * NP;
    ACSC_LAUNCH(tag, (gemm_tall_kernel<TA, TRANS, float>), grid, dim3(256), 0, st, A, lda, B, ldb,
                       part, int64_t(NP), ss, M, K, nvalid, NP, static_cast<int>(chunk));
    ACSC_LAUNCH("sc_split_reduce", (reduce_splits_kernel<TO>), dim3(grid1d(static_cast<int64_t>(M) * nwrite)),
                       dim3(256), 0, st, part, int64_t(NP), ss, splits, M, nwrite, C, ldc);
}

// Raise a kernel's dynamic-LDS limit (needed above the default 64 KiB).
template <typename F>
int allow_lds(F kernel, size_t bytes)
{
    if (bytes <= 64 * 1024)
        return ACSC_OK;
    int dev = 0, lim = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&lim, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
        return set_error(ACSC_EHIP, "cannot query the LDS size of the device");
    if (static_cast<size_t>(lim) < bytes)
        return set_error(ACSC_EINVAL, "needs %zu bytes of LDS per workgroup, device has %d", bytes, lim);
    if (hipFuncSetAttribute(reinterpret_cast<const void *>(kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(bytes)) != hipSuccess)
        return set_error(ACSC_EHIP, "hipFuncSetAttribute failed");
    return ACSC_OK;
}

size_t chol_lds(int k) { return (static_cast<size_t>(k) * (k + 1) / 2 + k) * sizeof(double); }

// Q <- Y L^{-T} twice (CholeskyQR2) for Y [rows, KP] (first k columns live).
void orthonormalise(float *Y, int rows, const Dims &d, PriorWs &w, hipStream_t st)
{
    const int gb = gram_blocks(rows);
    const int rpb = static_cast<int>(round_up(cdiv(rows, gb), kGRows));
    const int nt = static_cast<int>(cdiv(d.KP, kGT));
    for (int pass = 0; pass < 2; ++pass) {
        ACSC_LAUNCH("sc_gram", gram_partial_kernel, dim3(nt * (nt + 1) / 2, gb), dim3(256), 0, st, Y,
                           int64_t(d.KP), rows, d.KP, rpb, w.gpart);
        ACSC_LAUNCH("sc_gram_reduce", gram_reduce_kernel, dim3(grid1d(int64_t(d.KP) * d.KP)), dim3(256), 0, st,
                           w.gpart, gb, d.KP, w.gram);
        ACSC_LAUNCH("sc_chol_inv", (chol_kernel<true>), dim3(1), dim3(1024), chol_lds(d.k), st, w.gram, d.k,
                           d.KP, w.T);
        tall_gemm<float, false, float>("sc_orth_apply", Y, d.KP, w.T, d.KP, Y, d.KP, rows, d.KP, d.KP, d.KP, nullptr,
                                       1, st);
    }
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
    *bytes = std::max(carve_prior(d, nullptr, nullptr), carve_correct(d, dtype_size(dt), nullptr, nullptr));
    return ACSC_OK;
}

extern "C" int sc_build_prior(const void *G_anc, acsc_dtype dt, float *M, int m, int n, float beta,
                              int r, int oversample, int power_iters, float tau,
                              const float *V_warm, uint64_t seed, float *U, float *s, float *V,
                              float *d, void *ws, size_t ws_bytes, hipStream_t stream)
{
    size_t need = 0;
    int rc = sc_workspace_size(m, n, r, oversample, dt, &need);
    if (rc)
        return rc;
    ACSC_CHECK_ARG(M && U && s && V && d && ws, ACSC_EINVAL, "null pointer argument");
    ACSC_CHECK_ARG(beta >= 0.f && beta <= 1.f, ACSC_EINVAL, "beta=%g outside [0, 1]", beta);
    ACSC_CHECK_ARG(tau >= 0.f && std::isfinite(tau), ACSC_EINVAL, "tau=%g must be finite, >= 0", tau);
    ACSC_CHECK_ARG(power_iters >= 0 && power_iters <= 64, ACSC_EINVAL, "power_iters=%d outside [0, 64]",
                   power_iters);
    ACSC_CHECK_ARG(ws_bytes >= need, ACSC_ENOSPC, "workspace %zu bytes < %zu needed", ws_bytes, need);
    ACSC_CHECK_ARG(aligned(ws, 256), ACSC_EALIGN, "workspace must be 256-byte aligned");
    ACSC_CHECK_ARG(aligned(M, 16), ACSC_EALIGN, "M must be 16-byte aligned");
    ACSC_CHECK_ARG(!G_anc || aligned(G_anc, 16), ACSC_EALIGN, "G_anc must be 16-byte aligned");
    const Dims D = dims_of(m, n, r, oversample);
    rc = allow_lds(chol_kernel<true>, chol_lds(D.k));
    if (!rc)
        rc = allow_lds(chol_kernel<false>, chol_lds(D.k));
    if (!rc)
        rc = D.k <= 128 ? allow_lds(jacobi_kernel<double>, static_cast<size_t>(D.k) * D.k * sizeof(double))
                        : allow_lds(jacobi_kernel<float>, static_cast<size_t>(D.k) * D.k * sizeof(float));
    if (rc)
        return rc;
    PriorWs w;
    carve_prior(D, ws, &w);
    hipStream_t st = stream;
    const int64_t count = static_cast<int64_t>(m) * n;
    if (G_anc) {
        if (dt == ACSC_BF16)
            ACSC_LAUNCH("sc_ema", (ema_kernel<uint16_t>), dim3(grid1d(cdiv(count, 4))), dim3(256), 0, st, M,
                               static_cast<const uint16_t *>(G_anc), count, beta, 1.0f - beta);
        else
            ACSC_LAUNCH("sc_ema", (ema_kernel<float>), dim3(grid1d(cdiv(count, 4))), dim3(256), 0, st, M,
                               static_cast<const float *>(G_anc), count, beta, 1.0f - beta);
    }
    ACSC_LAUNCH("sc_init", init_block_kernel, dim3(grid1d(int64_t(n) * D.KP)), dim3(256), 0, st, w.Z, n, D.k,
                       D.KP, V_warm, V_warm ? r : 0, seed);
    const int sY = split_count(m, n), sZ = split_count(n, m);
    // Y = M Z0
    tall_gemm<float, false, float>("sc_pass_mz", M, n, w.Z, D.KP, w.Y, D.KP, m, n, D.k, D.KP, w.part, sY, st);
    orthonormalise(w.Y, m, D, w, st);
    for (int it = 0; it < power_iters; ++it) {
        tall_gemm<float, true, float>("sc_pass_mtq", M, n, w.Y, D.KP, w.Z, D.KP, n, m, D.k, D.KP, w.part, sZ, st);
        orthonormalise(w.Z, n, D, w, st);
        tall_gemm<float, false, float>("sc_pass_mz", M, n, w.Z, D.KP, w.Y, D.KP, m, n, D.k, D.KP, w.part, sY, st);
        orthonormalise(w.Y, m, D, w, st);
    }
    // Rayleigh-Ritz: Z = M^T Q (= B^T), B B^T = Z^T Z = L L^T, SVD of L by Jacobi.
    tall_gemm<float, true, float>("sc_pass_mtq", M, n, w.Y, D.KP, w.Z, D.KP, n, m, D.k, D.KP, w.part, sZ, st);
    {
        const int gb = gram_blocks(n);
        const int rpb = static_cast<int>(round_up(cdiv(n, gb), kGRows));
        const int nt = static_cast<int>(cdiv(D.KP, kGT));
        ACSC_LAUNCH("sc_gram", gram_partial_kernel, dim3(nt * (nt + 1) / 2, gb), dim3(256), 0, st, w.Z,
                           int64_t(D.KP), n, D.KP, rpb, w.gpart);
        ACSC_LAUNCH("sc_gram_reduce", gram_reduce_kernel, dim3(grid1d(int64_t(D.KP) * D.KP)), dim3(256), 0, st,
                           w.gpart, gb, D.KP, w.gram);
        ACSC_LAUNCH("sc_chol", (chol_kernel<false>), dim3(1), dim3(1024), chol_lds(D.k), st, w.gram, D.k,
                           D.KP, static_cast<float *>(nullptr));
    }
    if (D.k <= 128)
        ACSC_LAUNCH("sc_jacobi", (jacobi_kernel<double>), dim3(1), dim3(1024),
                           static_cast<size_t>(D.k) * D.k * sizeof(double), st, w.gram, D.k, D.KP, r,
                           D.RP, tau, 1e-13, 60, w.Bu, w.Bv, s, d);
    else
        ACSC_LAUNCH("sc_jacobi", (jacobi_kernel<float>), dim3(1), dim3(1024),
                           static_cast<size_t>(D.k) * D.k * sizeof(float), st, w.gram, D.k, D.KP, r,
                           D.RP, tau, 2e-6f, 60, w.Bu, w.Bv, s, d);
    // U = Q Bu, V = Z Bv (first r columns)
    tall_gemm<float, false, float>("sc_basis", w.Y, D.KP, w.Bu, D.RP, U, r, m, D.KP, r, r, nullptr, 1, st);
    tall_gemm<float, false, float>("sc_basis", w.Z, D.KP, w.Bv, D.RP, V, r, n, D.KP, r, r, nullptr, 1, st);
    return check_launch("sc_build_prior");
}

extern "C" int sc_correct(const void *G, acsc_dtype dt, int m, int n, const float *U, const float *d,
                          const float *V, int r, float alpha, void *G_proj, void *ws, size_t ws_bytes,
                          hipStream_t stream)
{
    size_t need = 0;
    int rc = sc_workspace_size(m, n, r, 0, dt, &need);
    if (rc)
        return rc;
    ACSC_CHECK_ARG(G && U && d && V && G_proj && ws, ACSC_EINVAL, "null pointer argument");
    ACSC_CHECK_ARG(std::isfinite(alpha), ACSC_EINVAL, "alpha must be finite");
    ACSC_CHECK_ARG(ws_bytes >= need, ACSC_ENOSPC, "workspace %zu bytes < %zu needed", ws_bytes, need);
    ACSC_CHECK_ARG(aligned(ws, 256), ACSC_EALIGN, "workspace must be 256-byte aligned");
    const size_t es = dtype_size(dt);
    ACSC_CHECK_ARG(aligned(G, es) && aligned(G_proj, es) && aligned(U, 4) && aligned(V, 4) && aligned(d, 4),
                   ACSC_EALIGN, "G, G_proj, U, d, V must be aligned to their element size");
    const Dims D = dims_of(m, n, r, 0);
    {
        const size_t pitch = D.RP + (dt == ACSC_BF16 ? 8 : 1);
        const size_t blds = 2 * 64 * pitch * es;
        rc = dt == ACSC_BF16 ? allow_lds(blend_kernel<uint16_t>, blds) : allow_lds(blend_kernel<float>, blds);
        if (rc)
            return rc;
    }
    CorrWs w;
    carve_correct(D, es, ws, &w);
    hipStream_t st = stream;
    const int s1 = split_count(m, n), s2 = split_count(r, m);
    // T = G V   [m, RP]
    if (dt == ACSC_BF16)
        tall_gemm<uint16_t, false, float>("sc_gv", static_cast<const uint16_t *>(G), n, V, r, w.Tm, D.RP, m, n, r,
                                          D.RP, w.part, s1, st);
    else
        tall_gemm<float, false, float>("sc_gv", static_cast<const float *>(G), n, V, r, w.Tm, D.RP, m, n, r, D.RP,
                                       w.part, s1, st);
    // X = U^T T   [r, RP]
    tall_gemm<float, true, float>("sc_utt", U, r, w.Tm, D.RP, w.X, D.RP, r, m, D.RP, D.RP, w.xpart, s2, st);
    ACSC_LAUNCH("sc_filter", filter_x_kernel, dim3(grid1d(int64_t(D.RP) * D.RP)), dim3(256), 0, st, w.X,
                       int64_t(D.RP), d, r, D.RP, w.Xf);
    const dim3 bgrid(static_cast<unsigned>(cdiv(n, 64)), static_cast<unsigned>(cdiv(m, 64)));
    const size_t pitch = D.RP + (dt == ACSC_BF16 ? 8 : 1);
    const size_t blds = 2 * 64 * pitch * es;
    if (dt == ACSC_BF16) {
        uint16_t *Pc = static_cast<uint16_t *>(w.Pc), *Vc = static_cast<uint16_t *>(w.Vc);
        // P = U X_f  [m, RP] in bf16
        tall_gemm<float, false, uint16_t>("sc_ux", U, r, w.Xf, D.RP, Pc, D.RP, m, r, D.RP, D.RP, nullptr, 1, st);
        ACSC_LAUNCH("sc_vconvert", (pad_convert_kernel<uint16_t>), dim3(grid1d(int64_t(n) * D.RP)), dim3(256), 0,
                           st, V, n, r, D.RP, Vc);
        ACSC_LAUNCH("sc_blend", (blend_kernel<uint16_t>), bgrid, dim3(256), blds, st,
                           static_cast<const uint16_t *>(G), static_cast<uint16_t *>(G_proj), m, n, Pc,
                           Vc, D.RP, alpha);
    } else {
        float *Pc = static_cast<float *>(w.Pc), *Vc = static_cast<float *>(w.Vc);
        tall_gemm<float, false, float>("sc_ux", U, r, w.Xf, D.RP, Pc, D.RP, m, r, D.RP, D.RP, nullptr, 1, st);
        ACSC_LAUNCH("sc_vconvert", (pad_convert_kernel<float>), dim3(grid1d(int64_t(n) * D.RP)), dim3(256), 0, st,
                           V, n, r, D.RP, Vc);
        ACSC_LAUNCH("sc_blend", (blend_kernel<float>), bgrid, dim3(256), blds, st,
                           static_cast<const float *>(G), static_cast<float *>(G_proj), m, n, Pc, Vc,
                           D.RP, alpha);
    }
    return check_launch("sc_correct");
}
