// Blocked Cholesky factor and triangular inverse for gfx950 (see sc_chol.h).
//
// One workgroup of 16 waves per matrix.  The lower triangle of G lives in LDS
// as 16 x 16 fp64 blocks; all of SC_KMAX = 192 fits (78 blocks, 156 KiB).
// Right-looking blocked factorisation, per block column p:
//   - the diagonal block is factored and inverted by one wave in registers:
//     symmetric elimination on [A_pp | I] (16 steps; the pivot row travels
//     by DPP row broadcast, the pivot column by one lane permute), and
//     X_pp = L_pp^{-1} replaces A_pp in LDS;
//   - the panel L_ip = A_ip X_pp^T and the trailing update
//     A_ij -= L_ip L_jp^T run on v_mfma_f64_16x16x4f64, one block per wave.
//   Wave 0 updates and factors the next diagonal block while the other waves
//   finish the trailing update (look-ahead), so the serial chain is the
//   16-step eliminations plus two barriers per block column.
// Inverse: U_ij = X_ii L_ij below the diagonal, then block rows in order,
//   X_ip = -sum_{j = p}^{i-1} U_ij X_jp   (from L X = I).
#include "common.h"
#include "sc_chol.h"

#include <algorithm>

namespace acsc {
namespace chol {
namespace {

typedef double v4d __attribute__((ext_vector_type(4)));

constexpr int kNB = 16;             // block edge
constexpr int kBlk = kNB * kNB;     // doubles per block
constexpr int kMaxJobs = 16;

struct Job {
    double *G;
    float *T;
};
struct Batch {
    int count;
    Job j[kMaxJobs];
};

// block (i, j), j <= i, in row-major order of the lower block triangle
__device__ __forceinline__ int bidx(int i, int j) { return i * (i + 1) / 2 + j; }
// element (r, c) of a block: rows of 16 doubles, columns XOR-swizzled by r / 2
// so that a column read by 16 lanes touches 16 different bank pairs
__device__ __forceinline__ int eoff(int r, int c) { return r * kNB + (c ^ ((r >> 1) & 7)); }

__device__ __forceinline__ double readlane64(double v, int lane)
{
    const int lo = __builtin_amdgcn_readlane(__double2loint(v), lane);
    const int hi = __builtin_amdgcn_readlane(__double2hiint(v), lane);
    return __hiloint2double(hi, lo);
}

__device__ __forceinline__ double bpermute64(double v, int src)
{
    const int lo = __builtin_amdgcn_ds_bpermute(src << 2, __double2loint(v));
    const int hi = __builtin_amdgcn_ds_bpermute(src << 2, __double2hiint(v));
    return __hiloint2double(hi, lo);
}

// DPP row_newbcast:J -- every lane of each 16-lane row takes lane J of its row
template <int J>
__device__ __forceinline__ double row_bcast(double v)
{
    const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(v), 0x150 + J, 0xF, 0xF, false);
    const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(v), 0x150 + J, 0xF, 0xF, false);
    return __hiloint2double(hi, lo);
}

// 1 / sqrt(d) for d > 0 from the hardware estimate and two Newton steps
// (y <- y + y (1 - d y^2) / 2; each step about doubles the correct bits), so
// that a pivot costs a few dependent multiply-adds rather than a correctly
// rounded square root and division; within an ulp or two of 1.0 / sqrt(d).
__device__ __forceinline__ double rsqrt_refined(double d)
{
    double y = __builtin_amdgcn_rsq(d);
    const double hd = 0.5 * d;
    y = fma(y, fma(-hd * y, y, 0.5), y);
    y = fma(y, fma(-hd * y, y, 0.5), y);
    return y;
}

// One elimination step on the diagonal block.  Lane (i, h) = (lane % 16,
// lane / 16) holds A[i][4h .. 4h+3] in a[] and X[i][4h .. 4h+3] in x[].
// Rows below the pivot lose their multiple f_i = A[i][J] / d_J of pivot row
// J (trailing columns of A, all of X); column J keeps A[i][J] (= L_unit[i][J]
// d_J).  dsc[J] = 1 / sqrt(d_J), or 0 for a pivot at or below the threshold.
template <int J>
__device__ __forceinline__ void elim_step(double (&a)[4], double (&x)[4], double (&dsc)[kNB], int i, int h,
                                          double thresh)
{
    constexpr int HJ = J >> 2, EJ = J & 3;
    const double d = readlane64(a[EJ], J + 16 * HJ);
    const double rs = d > thresh ? rsqrt_refined(d) : 0.0;
    dsc[J] = rs;
    const double cij = bpermute64(a[EJ], i + 16 * HJ);
    const double f = i > J ? cij * (rs * rs) : 0.0;
    double ra[4], rx[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        ra[e] = row_bcast<J>(a[e]);
        rx[e] = row_bcast<J>(x[e]);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        a[e] = 4 * h + e > J ? fma(-f, ra[e], a[e]) : a[e];
        x[e] = fma(-f, rx[e], x[e]);
    }
}

template <int J>
struct Elim {
    static __device__ __forceinline__ void run(double (&a)[4], double (&x)[4], double (&dsc)[kNB], int i, int h,
                                               double thresh)
    {
        elim_step<J>(a, x, dsc, i, h, thresh);
        Elim<J + 1>::run(a, x, dsc, i, h, thresh);
    }
};
template <>
struct Elim<kNB> {
    static __device__ __forceinline__ void run(double (&)[4], double (&)[4], double (&)[kNB], int, int, double) {}
};

// Factor the diagonal block `blk` (one wave): X_pp = L_pp^{-1} over it, and
// L_pp itself to Lg (row stride ldg) when Lg is given.
__device__ __forceinline__ void factor_diag(double *blk, double thresh, double *Lg, int ldg)
{
    const int l = threadIdx.x & 63, i = l & 15, h = l >> 4;
    double a[4], x[4], dsc[kNB];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        a[e] = blk[eoff(i, 4 * h + e)];
        x[e] = 4 * h + e == i ? 1.0 : 0.0;
    }
    Elim<0>::run(a, x, dsc, i, h, thresh);
    // X = D^{-1/2} L_unit^{-1}
    double si = 0.0;
#pragma unroll
    for (int t = 0; t < kNB; ++t)
        si = i == t ? dsc[t] : si;
#pragma unroll
    for (int e = 0; e < 4; ++e)
        blk[eoff(i, 4 * h + e)] = x[e] * si;
    if (Lg) {
        // L = L_unit D^{1/2}: below the diagonal A[i][c] / sqrt(d_c)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int c = 4 * h + e;
            const double sc = h == 0 ? dsc[e] : h == 1 ? dsc[4 + e] : h == 2 ? dsc[8 + e] : dsc[12 + e];
            const double v = c < i ? a[e] * sc : c == i ? (sc > 0.0 ? 1.0 / sc : 0.0) : 0.0;
            Lg[static_cast<int64_t>(i) * ldg + c] = v;
        }
    }
}

// MFMA operands from a block (16x16x4 f64: A[i][k] in lane i + 16 k, B[k][j]
// in lane j + 16 k, D[i][j] in lane j + 16 (i % 4), element i / 4).
__device__ __forceinline__ double ld_ik(const double *b, int s, int l) { return b[eoff(l & 15, 4 * s + (l >> 4))]; }
__device__ __forceinline__ double ld_kj(const double *b, int s, int l) { return b[eoff(4 * s + (l >> 4), l & 15)]; }

__device__ __forceinline__ v4d ld_d(const double *b, int l)
{
    v4d v;
#pragma unroll
    for (int e = 0; e < 4; ++e)
        v[e] = b[eoff(4 * e + (l >> 4), l & 15)];
    return v;
}

__device__ __forceinline__ void st_d(double *b, v4d v, int l)
{
#pragma unroll
    for (int e = 0; e < 4; ++e)
        b[eoff(4 * e + (l >> 4), l & 15)] = v[e];
}

__device__ __forceinline__ v4d mfma64(double a, double b, v4d c)
{
    return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
}

// A_ij -= L_ip L_jp^T
__device__ __forceinline__ void trail_update(double *S, int bi, int bj, int p, int l)
{
    double *A = S + bidx(bi, bj) * kBlk;
    const double *Li = S + bidx(bi, p) * kBlk, *Lj = S + bidx(bj, p) * kBlk;
    v4d acc = ld_d(A, l);
#pragma unroll
    for (int s = 0; s < 4; ++s)
        acc = mfma64(-ld_ik(Li, s, l), ld_ik(Lj, s, l), acc);
    st_d(A, acc, l);
}

template <bool INVERT>
__global__ __launch_bounds__(1024) void chol_blocked_kernel(const Batch jb, int k, int KP)
{
    extern __shared__ double S[];
    __shared__ double sh_thresh;
    const Job &J = jb.j[blockIdx.z];
    double *G = J.G;
    const int NB = KP / kNB;
    const int tid = threadIdx.x, l = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    // the lower blocks of G (zero outside the leading k x k)
    for (int idx = tid; idx < KP * KP; idx += 1024) {
        const int i = idx / KP, c = idx - i * KP;
        if ((c >> 4) <= (i >> 4))
            S[bidx(i >> 4, c >> 4) * kBlk + eoff(i & 15, c & 15)] = (i < k && c < k) ? G[idx] : 0.0;
    }
    if (w == 0) {
        double mx = 0.0;
        for (int i = l; i < k; i += 64)
            mx = fmax(mx, G[static_cast<int64_t>(i) * KP + i]);
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1)
            mx = fmax(mx, __shfl_xor(mx, off, 64));
        if (l == 0)
            sh_thresh = 1e-15 * k * mx;
    }
    __syncthreads();
    const double thresh = sh_thresh;
    double *Lg = INVERT ? nullptr : G;
    if (w == 0)
        factor_diag(S, thresh, Lg, KP);
    __syncthreads();
    for (int p = 0; p < NB; ++p) {
        // panel: L_ip = A_ip X_pp^T, one block per wave
        const int bi = p + 1 + w;
        if (bi < NB) {
            double *A = S + bidx(bi, p) * kBlk;
            const double *X = S + bidx(p, p) * kBlk;
            v4d acc = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
            for (int s = 0; s < 4; ++s)
                acc = mfma64(ld_ik(A, s, l), ld_ik(X, s, l), acc);
            st_d(A, acc, l);
        }
        __syncthreads();
        if (p + 1 == NB)
            break;
        // trailing update of blocks (p+1+ri, p+1+rj), rj <= ri, numbered
        // row-major from 0; wave 0 takes block 0 = (p+1, p+1) and factors it
        const int n = NB - 1 - p;
        const int ntot = n * (n + 1) / 2;
        if (w == 0) {
            trail_update(S, p + 1, p + 1, p, l);
            factor_diag(S + bidx(p + 1, p + 1) * kBlk, thresh,
                        Lg ? Lg + static_cast<int64_t>(kNB * (p + 1)) * KP + kNB * (p + 1) : nullptr, KP);
        } else {
            for (int t = w; t < ntot; t += 15) {
                int ri = 0;
                while ((ri + 1) * (ri + 2) / 2 <= t)
                    ++ri;
                const int rj = t - ri * (ri + 1) / 2;
                trail_update(S, p + 1 + ri, p + 1 + rj, p, l);
            }
        }
        __syncthreads();
    }
    if (INVERT) {
        // U_ij = X_ii L_ij below the diagonal (block t: row bi holds bi blocks)
        const int noff = NB * (NB - 1) / 2;
        for (int t = w; t < noff; t += 16) {
            int bi = 1, rem = t;
            while (rem >= bi) {
                rem -= bi;
                ++bi;
            }
            double *Lb = S + bidx(bi, rem) * kBlk;
            const double *X = S + bidx(bi, bi) * kBlk;
            v4d acc = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
            for (int s = 0; s < 4; ++s)
                acc = mfma64(ld_ik(X, s, l), ld_kj(Lb, s, l), acc);
            st_d(Lb, acc, l);
        }
        __syncthreads();
        // block rows of X in order; wave p computes X_ip
        for (int bi = 1; bi < NB; ++bi) {
            v4d acc = {0.0, 0.0, 0.0, 0.0};
            const int p = w;
            if (p < bi) {
                for (int j = p; j < bi; ++j) {
                    const double *U = S + bidx(bi, j) * kBlk, *X = S + bidx(j, p) * kBlk;
#pragma unroll
                    for (int s = 0; s < 4; ++s)
                        acc = mfma64(-ld_ik(U, s, l), ld_kj(X, s, l), acc);
                }
            }
            __syncthreads();   // every read of row bi's U blocks is done
            if (p < bi)
                st_d(S + bidx(bi, p) * kBlk, acc, l);
            __syncthreads();
        }
        // T[c][i] = X[i][c]
        float *T = J.T;
        for (int idx = tid; idx < KP * KP; idx += 1024) {
            const int c = idx / KP, i = idx - c * KP;
            T[idx] = c <= i ? static_cast<float>(S[bidx(i >> 4, c >> 4) * kBlk + eoff(i & 15, c & 15)]) : 0.f;
        }
    } else {
        // blocks below the diagonal, and the zero upper part (the diagonal
        // blocks were written as they were factored)
        for (int idx = tid; idx < KP * KP; idx += 1024) {
            const int i = idx / KP, c = idx - i * KP;
            if ((c >> 4) < (i >> 4))
                G[idx] = S[bidx(i >> 4, c >> 4) * kBlk + eoff(i & 15, c & 15)];
            else if ((c >> 4) > (i >> 4))
                G[idx] = 0.0;
        }
    }
}

}  // namespace

bool supported(int KP) { return KP >= kNB && KP % kNB == 0 && KP <= SC_KMAX; }

size_t lds_bytes(int KP)
{
    const size_t nb = static_cast<size_t>(KP / kNB);
    return nb * (nb + 1) / 2 * kBlk * sizeof(double);
}

int prepare(int KP)
{
    if (!supported(KP))
        return set_error(ACSC_EINVAL, "chol: padded order %d not handled", KP);
    int rc = allow_lds(chol_blocked_kernel<true>, lds_bytes(KP));
    if (rc)
        return rc;
    return allow_lds(chol_blocked_kernel<false>, lds_bytes(KP));
}

int run(const char *tag, const std::vector<Req> &reqs, int k, int KP, bool invert, hipStream_t st)
{
    if (!supported(KP) || k < 1 || k > KP)
        return set_error(ACSC_EINVAL, "chol: order %d (padded %d) not handled", k, KP);
    for (size_t c0 = 0; c0 < reqs.size(); c0 += kMaxJobs) {
        Batch b{};
        b.count = static_cast<int>(std::min<size_t>(kMaxJobs, reqs.size() - c0));
        for (int i = 0; i < b.count; ++i)
            b.j[i] = Job{reqs[c0 + i].G, reqs[c0 + i].T};
        if (invert)
            ACSC_LAUNCH(tag, chol_blocked_kernel<true>, dim3(1, 1, b.count), dim3(1024), lds_bytes(KP), st, b, k, KP);
        else
            ACSC_LAUNCH(tag, chol_blocked_kernel<false>, dim3(1, 1, b.count), dim3(1024), lds_bytes(KP), st, b, k,
                        KP);
    }
    return ACSC_OK;
}

}  // namespace chol
}  // namespace acsc
