// Tall-times-small products of the spectral corrector (internal; not part of
// the ABI), on fp32 matrix cores:
//   C = A B,  A [rows, K] fp32 (a tall block),  B [K, N] fp32 (K, N <= SC_KMAX).
// Uses (Sec. 3.2): the CholeskyQR step Q = Y T with T = (L^{-1})^T upper
// triangular, in place, optionally with the bf16 transposed copy Q^T that the
// next streaming pass reads; the basis U = Q Bu, V = Z Bv; and P = U X_f.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <vector>

namespace acsc {
namespace orth {

struct Req {
    float *Y;            // [rows, KP] fp32, row stride KP; overwritten by Q when write32
    int rows;
    const float *T;      // [KP, KP] fp32, zero below the diagonal
    uint16_t *Qt16;      // [KP, ldq] bf16 (Q^T), or nullptr
    int64_t ldq;         // a multiple of 8
    bool write32;        // store Q over Y
};

// Enqueue Q = Y T for every request (all share KP, a multiple of 16 up to
// SC_KMAX) on `st`.
int run(const char *tag, const std::vector<Req> &reqs, int KP, hipStream_t st);

struct GemmReq {
    const float *A;      // [rows, K], row stride lda
    int64_t lda;
    int rows, K;
    const float *B;      // [K, N], row stride ldb; columns >= N read as zero
    int64_t ldb;
    int N;
    float *C32;          // [rows, nwrite] fp32, row stride ldc, or nullptr
    uint16_t *C16;       // the same in bf16, or nullptr
    int64_t ldc;
    int nwrite;
};

// Whether gemm() takes these operands: 16-byte aligned A and B whose row
// strides, K and N are multiples of 4, K and N at most SC_KMAX.
bool gemm_supported(const GemmReq &q);

// Enqueue C = A B for every request on `st`.
int gemm(const char *tag, const std::vector<GemmReq> &reqs, hipStream_t st);

// C = A^T B over the rows of two tall blocks, A [rows, NA], B [rows, NB]
// (NA, NB <= SC_KMAX), C [NA, NB] fp32 with row stride ldc: X = U^T T of the
// correction.  Workgroups sum row ranges into fp32 partials, which a second
// kernel adds in a fixed order; `part` holds part_blocks x NA x NB floats.
struct InnerReq {
    const float *A;
    int64_t lda;
    const float *B;
    int64_t ldb;
    int rows, NA, NB;
    float *C;
    int64_t ldc;
    float *part;
    int part_blocks;
};

// Whether inner() takes these operands (alignment as for gemm(), and room in
// `part` for at least one block of round_up(max(NA, NB), 32)^2 floats).
bool inner_supported(const InnerReq &q);
int inner(const char *tag, const std::vector<InnerReq> &reqs, hipStream_t st);

}  // namespace orth
}  // namespace acsc
