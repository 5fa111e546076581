// Cholesky factor and triangular inverse of the small fp64 Gram matrices of
// the spectral corrector (internal; not part of the ABI).
//
// For G = Y^T Y (k x k, symmetric positive semi-definite, stored full as
// KP x KP fp64, KP = k rounded up to 16):  G = L L^T with L lower triangular.
// A pivot at or below 1e-15 * k * max_i G[i][i] is taken as zero: that
// column of L (and that row of L^{-1}) is zero, which is how a rank-deficient
// block is handled.  Rows and columns k .. KP-1 are zero on output.
//   invert: T = (L^{-1})^T in fp32 (KP x KP, upper triangular), so that
//           Q = Y T has orthonormal columns (CholeskyQR, Sec. 3.2 basis
//           construction);
//   else:   L itself over G (fp64, zero upper part), the input of the
//           Rayleigh-Ritz step.
#pragma once

#include <hip/hip_runtime.h>

#include <vector>

namespace acsc {
namespace chol {

struct Req {
    double *G;   // [KP, KP] fp64, row stride KP
    float *T;    // [KP, KP] fp32 (invert) or unused
};

// KP = padded order this kernel handles (a multiple of 16, at most SC_KMAX).
bool supported(int KP);

// Dynamic LDS bytes per workgroup for order KP (the caller raises the limit).
size_t lds_bytes(int KP);

// Raise the dynamic-LDS limit of the kernels for order KP.
int prepare(int KP);

// Enqueue one factorisation per request on `st` (all share k and KP).
int run(const char *tag, const std::vector<Req> &reqs, int k, int KP, bool invert, hipStream_t st);

}  // namespace chol
}  // namespace acsc
