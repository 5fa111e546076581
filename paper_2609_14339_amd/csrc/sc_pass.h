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

}  // namespace pass
}  // namespace acsc
