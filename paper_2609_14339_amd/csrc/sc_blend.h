// Fused blend of the spectral correction (internal; not part of the ABI):
//   out = alpha * G + (1 - alpha) * P V^T
// with P = U X_f [m, RP] and V [n, RP] in bf16 (Sec. 3.2: G_proj = alpha G +
// (1 - alpha) U X_f V^T, the filtered gradient never materialised).  The same
// streamed tiles serve the decompression of the data-parallel compressor
// (out = P_hat Q^T with error feedback; see run_feedback).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <vector>

namespace acsc {
namespace blend {

struct Req {
    const uint16_t *G;   // [m, n] bf16, row stride n
    uint16_t *out;       // [m, n] bf16 (may equal G); unused with an AdamW epilogue
    int m, n;
    const uint16_t *P;   // [m, RP] bf16
    const uint16_t *V;   // [n, RP] bf16
    float *W, *m1, *m2;  // AdamW epilogue: fp32 [m, n] weights and moments, in place
    float *E;            // feedback epilogue: fp32 [m, n] memory, holds M, takes M - out
};

// What a tile's product feeds: the stored blend, the AdamW step, or the
// decompression with error feedback.
enum Epilogue { kPlain = 0, kAdam = 1, kFeedback = 2 };

// Constants of the AdamW epilogue (Alg. 1 update; the optimiser of App. I):
// with g = coef * G_proj,
//   m1 <- beta1 m1 + (1 - beta1) g;  m2 <- beta2 m2 + (1 - beta2) g^2;
//   W  <- W (1 - lr wd) - (lr / bc1) m1 / (sqrt(m2) / sqrt(bc2) + eps),
// bc = 1 - beta^t; coef (device) is the clipping scale of the whole call.
struct AdamArgs {
    float beta1, beta2, omb1, omb2;
    float wdf;     // 1 - lr wd
    float step;    // lr / bc1
    float isbc2;   // 1 / sqrt(bc2)
    float eps;
    const float *coef;
};

// One element of the update; every corrected-AdamW kernel uses this.
__device__ __forceinline__ void adamw_elem(float g, float &w, float &m1, float &m2, const AdamArgs &a)
{
    m1 = a.beta1 * m1 + a.omb1 * g;
    m2 = a.beta2 * m2 + a.omb2 * (g * g);
    w = w * a.wdf - a.step * m1 / (__builtin_sqrtf(m2) * a.isbc2 + a.eps);
}

// Whether the streamed-tile kernel handles this padded rank.
bool supported(int RP);

// Enqueue the blend of every request (all share RP) on `st`; with `adam`,
// G_proj is not stored and the requests' W, m1, m2 take the AdamW step.
int run(const char *tag, const std::vector<Req> &reqs, int RP, float alpha, hipStream_t st,
        const AdamArgs *adam = nullptr);

// Decompression with error feedback (the data-parallel compressor):
//   out = bf16(P V^T),  E <- E - out  (E holds M on entry, fp32),
// for every request (G unused; all share RP) on `st`.
int run_feedback(const char *tag, const std::vector<Req> &reqs, int RP, hipStream_t st);

}  // namespace blend
}  // namespace acsc
