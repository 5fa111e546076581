// Application of the CholeskyQR factor (internal; not part of the ABI):
//   Q = Y T  in place,  T = (L^{-1})^T  upper triangular  (KP x KP fp32),
// for a tall block Y [rows, KP] fp32 of the subspace iteration (Sec. 3.2
// basis construction), optionally with the bf16 transposed copy Qt16[c][i]
// that the next streaming pass reads.
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

}  // namespace orth
}  // namespace acsc
