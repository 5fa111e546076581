// Streaming passes of the spectral corrector (internal; not part of the ABI).
//
// One pass multiplies a large bf16 matrix, read once from HBM, by a thin
// factor of up to SC_KMAX columns:
//   C[i, c] = sum_k opA[i, k] * B[k, c],  opA = A ([M, K] row-major) or A^T
//   (A stored [K, M] row-major),
// with B given transposed in bf16 (Bt[c][k], row stride ldbt, a multiple of 8).
// These are the power passes Y = M Z and Z = M^T Y of the anchor SVD and the
// product T = G V of the correction (Sec. 3.2).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <vector>

namespace acsc {
namespace pass {

struct Req {
    const uint16_t *A;
    int64_t lda;
    bool avec;          // A rows start 16-byte aligned (vector loads)
    const uint16_t *Bt;
    int64_t ldbt;
    float *C;           // [M, NP] fp32, row stride ldc
    int64_t ldc;
    int M, K, NP;       // NP = columns of the thin factor, a multiple of 16
    float *part;        // split-K partials, >= max_splits(M, K) * M * NP floats
};

// Largest number of K splits a pass over an [M x K] operand may use; the
// caller sizes `part` for it.
int max_splits(int64_t M, int64_t K);

// Enqueue one pass per request (all requests share NP) on `st`.
int run(const char *tag, bool trans, const std::vector<Req> &reqs, hipStream_t st);

// The anchor EMA fused with the first pass of the subspace iteration
// (Sec. 3.2): M <- a M + b G (the EMA: a = beta, b = 1 - beta; error
// feedback: a = b = 1; G may be null: M is kept), the bf16 shadow
// M16 = bf16(M) written for the later passes, and C = M16 * B in the same
// sweep over M, so that the first pass does not read the shadow back.
struct EmaReq {
    float *M;             // [m, n] fp32, row stride n
    const uint16_t *G;    // [m, n] bf16, or nullptr
    uint16_t *M16;        // [m, n] bf16, row stride n
    const uint16_t *Bt;   // thin factor transposed [NP, ldbt] bf16
    int64_t ldbt;
    float *C;             // [m, NP] fp32, row stride ldc
    int64_t ldc;
    int m, n, NP;
    float *part;          // split-k partials, >= max_splits(m, n) * m * NP floats, or nullptr (no split)
};

// Whether the fused kernel takes this batch: 16-byte aligned operands, n a
// multiple of 8, one NP, and enough row blocks over the batch to fill the
// GPU without splitting K.
bool ema_fusable(const std::vector<EmaReq> &reqs);

int ema_run(const char *tag, const std::vector<EmaReq> &reqs, float a, float b, hipStream_t st);

}  // namespace pass
}  // namespace acsc
