// Internal helpers shared by the library's translation units: error state,
// argument checks and bf16 bit conversions.  Not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>

#include "../../include/acsc.h"

namespace acsc {

// Per-thread text of the last error; set_error returns its code so that
// entry points can `return set_error(...)`.
int set_error(int code, const char *fmt, ...);
void clear_error();

#define ACSC_CHECK_ARG(cond, code, ...)            \
    do {                                           \
        if (!(cond))                               \
            return ::acsc::set_error(code, __VA_ARGS__); \
    } while (0)

// Optional per-kernel timing (acsc_stats_enable): ACSC_LAUNCH brackets a
// launch with HIP events on its stream when timing is on.
bool stats_on();
void *stats_begin(hipStream_t st, const char *tag);
void stats_end(hipStream_t st, void *token);

#define ACSC_LAUNCH(tag, kernel, grid, block, lds, st, ...)                         \
    do {                                                                          \
        void *acsc_tok_ = ::acsc::stats_on() ? ::acsc::stats_begin(st, tag) : nullptr; \
        hipLaunchKernelGGL(kernel, grid, block, lds, st, __VA_ARGS__);            \
        if (acsc_tok_)                                                            \
            ::acsc::stats_end(st, acsc_tok_);                                     \
    } while (0)

// Enqueue-time HIP error check; hipGetLastError also clears sticky launch
// errors left by this library's own launch.
inline int check_launch(const char *what)
{
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return set_error(ACSC_EHIP, "%s: %s", what, hipGetErrorString(e));
    return ACSC_OK;
}

inline bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Raise a kernel's dynamic-LDS limit (needed above the default 64 KiB).
template <typename F>
inline int allow_lds(F kernel, size_t bytes)
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



inline size_t dtype_size(acsc_dtype dt) { return dt == ACSC_BF16 ? 2 : 4; }

// One step of the anchor EMA, M <- beta M + (1 - beta) G (Sec. 3.2), with the
// contraction written out: every kernel that forms it rounds the same way
// (the product (1 - beta) G, then one fused multiply-add), so the fused and
// the separate EMA kernels agree bit for bit whatever the compiler would
// otherwise contract.
__device__ __forceinline__ float ema_step(float m, float g, float beta, float omb)
{
    return __builtin_fmaf(beta, m, omb * g);
}

// One element of the blend G_proj = alpha G + (1 - alpha) P V^T (Sec. 3.2),
// p = (P V^T)[i, j] in fp32, oma = 1 - alpha: one product and one fused
// multiply-add in a fixed order, so that every blend kernel rounds alike.
__device__ __forceinline__ float blend_step(float g, float p, float alpha, float oma)
{
    return __builtin_fmaf(alpha, g, oma * p);
}

// bf16 <-> fp32 on bit patterns.
__device__ __forceinline__ float bf16_to_f32(uint16_t h)
{
    return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// Round to nearest even on gfx950's v_cvt_pk_bf16_f32 (fp32 denormals are
// kept in the kernels' float mode, so they round like every other value); a
// NaN gives a quiet NaN.
typedef __bf16 acsc_bf16x2 __attribute__((ext_vector_type(2)));
typedef float acsc_f32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint16_t f32_to_bf16(float f)
{
    const __bf16 b = static_cast<__bf16>(f);
    uint16_t u;
    __builtin_memcpy(&u, &b, 2);
    return u;
}
// Two values in one instruction: lo in bits 0..15, hi in bits 16..31.
__device__ __forceinline__ uint32_t f32x2_to_bf16x2(float lo, float hi)
{
    const acsc_bf16x2 b = __builtin_convertvector(acsc_f32x2{lo, hi}, acsc_bf16x2);
    uint32_t u;
    __builtin_memcpy(&u, &b, 4);
    return u;
}

}  // namespace acsc
