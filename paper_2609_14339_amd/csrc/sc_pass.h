// Streaming passes of the spectral corrector (internal; not part of the ABI).
//
// One pass multiplies a large bf16 matrix, read once from HBM, by a thin
// factor of up to SC_KMAX columns:
//   C[i, c] = sum_k opA[i, k] * B[k, c],  opA = A ([M, K] row-major) or A^T
//   (A stored [K, M] row-major),
// with B given transposed in bf16 (Bt[c][k], row stride ldbt, a multiple of 8).
// These are the power passes Y = M Z and Z = M^T Y of the anchor SVD and the
// product T = G V of the correction (Sec. 3.2).
//
// The bf16 shadow of the EMA is kept in 64 x 64 tiles: element (i, j) of an
// [R x C] shadow sits at ((i / 64) * ntc + j / 64) * 4096 + (i % 64) * 64 + j % 64,
// ntc = ceil(C / 64), in a buffer of tiled_elems(R, C) elements.  A pass step
// then reads whole 8 KiB tiles (one per 64 rows of opA = A, four side by side
// for opA = A^T) instead of 128-byte pieces of 256 rows.
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
    int ntc;            // 0: A row-major with stride lda; > 0: A is a tiled shadow with ntc tiles per
                        // tile row (lda unused; requires avec)
};

inline int64_t tiles_per_row(int64_t C) { return (C + 63) / 64; }
inline int64_t tiled_elems(int64_t R, int64_t C) { return tiles_per_row(R) * tiles_per_row(C) * 4096; }

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
    uint16_t *M16;        // [m, n] bf16 in 64 x 64 tiles (tiled_elems(m, n) elements)
    const uint16_t *Bt;   // thin factor transposed [NP, ldbt] bf16
    int64_t ldbt;
    float *C;             // [m, NP] fp32, row stride ldc
    int64_t ldc;
    int m, n, NP;
    float *part;          // split-k partials, >= max_splits(m, n) * m * NP floats, or nullptr (no split)
    int *stall;           // set to kEmaStallMark if a wait of the kernel ran out of polls, or nullptr
};

// What the fused kernel writes to EmaReq::stall when one of its bounded waits
// for the other waves of a workgroup gave up (that workgroup's products are
// then not to be trusted); nothing is written otherwise.
constexpr int kEmaStallMark = 0x57A11ED0;
// Polls of a wait before it gives up (each about a microsecond or less).  The
// environment variable ACSC_EMA_SPIN_LIMIT, read by each call, lowers it (0
// gives up at the first unmet check), so that the report can be exercised.
constexpr int kEmaSpinLimit = 1 << 24;

// Whether the fused kernel takes this batch: 16-byte aligned operands, n a
// multiple of 8, one NP, and enough row blocks over the batch to fill the
// GPU without splitting K.
bool ema_fusable(const std::vector<EmaReq> &reqs);

int ema_run(const char *tag, const std::vector<EmaReq> &reqs, float a, float b, hipStream_t st);

}  // namespace pass
}  // namespace acsc
