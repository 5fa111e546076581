// Fused blend of the spectral correction (internal; not part of the ABI):
//   out = alpha * G + (1 - alpha) * P V^T
// with P = U X_f [m, RP] and V [n, RP] in bf16 (Sec. 3.2: G_proj = alpha G +
// (1 - alpha) U X_f V^T, the filtered gradient never materialised).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <vector>

namespace acsc {
namespace blend {

struct Req {
    const uint16_t *G;   // [m, n] bf16, row stride n
    uint16_t *out;       // [m, n] bf16 (may equal G)
    int m, n;
    const uint16_t *P;   // [m, RP] bf16
    const uint16_t *V;   // [n, RP] bf16
};

// Whether the streamed-tile kernel handles this padded rank.
bool supported(int RP);

// Enqueue the blend of every request (all share RP) on `st`.
int run(const char *tag, const std::vector<Req> &reqs, int RP, float alpha, hipStream_t st);

}  // namespace blend
}  // namespace acsc
