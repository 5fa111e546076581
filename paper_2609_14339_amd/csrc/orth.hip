// Q = Y T on v_mfma_f32_32x32x2f32 for gfx950 (see sc_orth.h).
//
// One workgroup of 4 waves per 128 rows of Y; wave w owns rows 32 w .. 32 w + 31
// and every 32-column tile of Q.  Y and T stream through LDS in 32-deep
// chunks (the next chunk is loaded into registers while the current one is
// multiplied); since T is upper triangular, chunk kc only feeds column tiles
// kc and above.  The bf16 copy of Q^T is staged in LDS so that each column of
// it leaves as 16-byte stores along the rows.
#include "common.h"
#include "sc_orth.h"

#include <algorithm>

namespace acsc {
namespace orth {
namespace {

typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;

constexpr int kRows = 128;            // rows of Y per workgroup
constexpr int kKC = 32;               // depth of one chunk
constexpr int kYP = kKC + 1;          // Y chunk pitch in floats (column reads conflict-free)
constexpr int kSP = kRows + 8;        // staged Q^T pitch in bf16 (16-byte rows)
constexpr int kMaxJobs = 16;

struct Job {
    float *Y;
    int rows;
    const float *T;
    uint16_t *Qt16;
    int64_t ldq;
    int write32;
};
struct Batch {
    int count;
    Job j[kMaxJobs];
};

template <int NT>
struct Lds {
    static constexpr int TP = NT * 32;                            // T chunk pitch (floats)
    static constexpr int MAIN = kRows * kYP + kKC * TP;           // floats
    static constexpr int STAGE = (TP * kSP + 1) / 2;              // floats
    static constexpr int FLOATS = MAIN > STAGE ? MAIN : STAGE;
};

template <int NT>
__global__ __launch_bounds__(256) void orth_apply_kernel(const Batch jb, int KP)
{
    using L = Lds<NT>;
    constexpr int TP = L::TP;
    constexpr int YV = kRows * (kKC / 4) / 256;    // float4 of a Y chunk per thread
    constexpr int TV = kKC * (TP / 4) / 256;       // float4 of a T chunk per thread
    static_assert(YV * 256 == kRows * kKC / 4 && TV * 256 == kKC * TP / 4, "chunk split");
    __shared__ __attribute__((aligned(16))) float smem[L::FLOATS];
    float *Ys = smem, *Ts = smem + kRows * kYP;

    const Job &J = jb.j[blockIdx.z];
    const int rows = J.rows;
    const int row0 = blockIdx.x * kRows;
    if (row0 >= rows)
        return;
    const float *Y = J.Y;
    const float *T = J.T;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

    float4 yr[YV], tr[TV];
    auto load = [&](int kc) {
        const int k0 = kc * kKC;
#pragma unroll
        for (int u = 0; u < YV; ++u) {
            const int idx = tid + 256 * u;
            const int r = idx >> 3, c = k0 + (idx & 7) * 4;
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (row0 + r < rows && c < KP)
                v = *reinterpret_cast<const float4 *>(Y + static_cast<int64_t>(row0 + r) * KP + c);
            yr[u] = v;
        }
#pragma unroll
        for (int u = 0; u < TV; ++u) {
            const int idx = tid + 256 * u;
            const int kk = idx / (TP / 4), c = (idx % (TP / 4)) * 4;
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (k0 + kk < KP && c < KP)
                v = *reinterpret_cast<const float4 *>(T + static_cast<int64_t>(k0 + kk) * KP + c);
            tr[u] = v;
        }
    };
    auto stash = [&]() {
#pragma unroll
        for (int u = 0; u < YV; ++u) {
            const int idx = tid + 256 * u;
            float *d = Ys + (idx >> 3) * kYP + (idx & 7) * 4;
            d[0] = yr[u].x;
            d[1] = yr[u].y;
            d[2] = yr[u].z;
            d[3] = yr[u].w;
        }
#pragma unroll
        for (int u = 0; u < TV; ++u) {
            const int idx = tid + 256 * u;
            *reinterpret_cast<float4 *>(Ts + (idx / (TP / 4)) * TP + (idx % (TP / 4)) * 4) = tr[u];
        }
    };

    f32x16 acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int e = 0; e < 16; ++e)
            acc[t][e] = 0.f;

    load(0);
#pragma unroll
    for (int kc = 0; kc < NT; ++kc) {
        if (kc)
            __syncthreads();   // the previous chunk is consumed
        stash();
        __syncthreads();
        if (kc + 1 < NT)
            load(kc + 1);
        // A[i][k] = Y[32 wave + i][2 s + k] in lane i + 32 k; B[k][j] = T[2 s + k][32 t + j]
        const float *ya = Ys + (32 * wave + (lane & 31)) * kYP + (lane >> 5);
        const float *tb = Ts + (lane >> 5) * TP + (lane & 31);
#pragma unroll
        for (int s = 0; s < kKC / 2; ++s) {
            const float a = ya[2 * s];
#pragma unroll
            for (int t = kc; t < NT; ++t)
                acc[t] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, tb[2 * s * TP + 32 * t], acc[t], 0, 0, 0);
        }
    }

    // D[i][j] in lane j + 32 ((i / 4) % 2), element 4 (i / 8) + i % 4
    const int j = lane & 31, hi = lane >> 5;
    if (J.write32) {
        float *Yw = J.Y;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int col = 32 * t + j;
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int row = row0 + 32 * wave + 8 * (e >> 2) + 4 * hi + (e & 3);
                if (row < rows && col < KP)
                    Yw[static_cast<int64_t>(row) * KP + col] = acc[t][e];
            }
        }
    }
    if (J.Qt16) {
        __syncthreads();   // every wave is done with the chunk buffers
        uint16_t *St = reinterpret_cast<uint16_t *>(smem);
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                uint32_t w0 = static_cast<uint32_t>(f32_to_bf16(acc[t][4 * q])) |
                              (static_cast<uint32_t>(f32_to_bf16(acc[t][4 * q + 1])) << 16);
                uint32_t w1 = static_cast<uint32_t>(f32_to_bf16(acc[t][4 * q + 2])) |
                              (static_cast<uint32_t>(f32_to_bf16(acc[t][4 * q + 3])) << 16);
                *reinterpret_cast<uint2 *>(St + (32 * t + j) * kSP + 32 * wave + 8 * q + 4 * hi) = make_uint2(w0, w1);
            }
        __syncthreads();
        uint16_t *Q = J.Qt16;
        const int64_t ldq = J.ldq;
        for (int idx = tid; idx < TP * (kRows / 8); idx += 256) {
            const int col = idx / (kRows / 8), r8 = (idx % (kRows / 8)) * 8;
            if (col < KP && row0 + r8 < rows)
                *reinterpret_cast<uint4 *>(Q + col * ldq + row0 + r8) =
                    *reinterpret_cast<const uint4 *>(St + col * kSP + r8);
        }
    }
}

template <int NT>
void launch(const char *tag, const std::vector<Job> &jobs, int KP, hipStream_t st)
{
    for (size_t c0 = 0; c0 < jobs.size(); c0 += kMaxJobs) {
        Batch b{};
        b.count = static_cast<int>(std::min<size_t>(kMaxJobs, jobs.size() - c0));
        int gx = 1;
        for (int i = 0; i < b.count; ++i) {
            b.j[i] = jobs[c0 + i];
            gx = std::max(gx, (b.j[i].rows + kRows - 1) / kRows);
        }
        ACSC_LAUNCH(tag, orth_apply_kernel<NT>, dim3(gx, 1, b.count), dim3(256), 0, st, b, KP);
    }
}

}  // namespace

int run(const char *tag, const std::vector<Req> &reqs, int KP, hipStream_t st)
{
    if (KP < 16 || KP % 16 != 0 || KP > SC_KMAX)
        return set_error(ACSC_EINVAL, "orth: padded order %d not handled", KP);
    std::vector<Job> jobs;
    for (const Req &q : reqs) {
        if (q.rows < 1)
            continue;
        if (q.Qt16 && (q.ldq % 8 != 0 || q.ldq < q.rows || !aligned(q.Qt16, 16)))
            return set_error(ACSC_EINVAL, "orth: bf16 copy needs 16-byte rows of at least %d entries", q.rows);
        if (!aligned(q.Y, 16) || !aligned(q.T, 16))
            return set_error(ACSC_EINVAL, "orth: Y and T must be 16-byte aligned");
        jobs.push_back(Job{q.Y, q.rows, q.T, q.Qt16, q.ldq, q.write32 ? 1 : 0});
    }
    if (jobs.empty())
        return ACSC_OK;
    switch ((KP + 31) / 32) {
    case 1: launch<1>(tag, jobs, KP, st); break;
    case 2: launch<2>(tag, jobs, KP, st); break;
    case 3: launch<3>(tag, jobs, KP, st); break;
    case 4: launch<4>(tag, jobs, KP, st); break;
    case 5: launch<5>(tag, jobs, KP, st); break;
    default: launch<6>(tag, jobs, KP, st); break;
    }
    return ACSC_OK;
}

}  // namespace orth
}  // namespace acsc
