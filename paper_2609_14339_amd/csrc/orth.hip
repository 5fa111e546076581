// Tall-times-small products on v_mfma_f32_32x32x2f32 for gfx950 (see
// sc_orth.h).
//
// One workgroup of 4 waves per 128 rows of A; wave w owns rows 32 w .. 32 w + 31
// and every 32-column tile of C.  A and B stream through LDS in 32-deep
// chunks (the next chunk is loaded into registers while the current one is
// multiplied).  With an upper-triangular B (the CholeskyQR factor) chunk kc
// only feeds column tiles kc and above.  A bf16 copy of C^T is staged in LDS
// so that each of its rows leaves as 16-byte stores.
#include "common.h"
#include "sc_orth.h"

#include <algorithm>

namespace acsc {
namespace orth {
namespace {

typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;

constexpr int kRows = 128;            // rows of A per workgroup
constexpr int kKC = 32;               // depth of one chunk
constexpr int kYP = kKC + 1;          // A chunk pitch in floats (column reads conflict-free)
constexpr int kSP = kRows + 8;        // staged C^T pitch in bf16 (16-byte rows)
constexpr int kMaxJobs = 16;

struct Job {
    const float *A;
    int64_t lda;
    int rows, K;
    const float *B;
    int64_t ldb;
    int N, tri;
    float *C32;
    uint16_t *C16;
    int64_t ldc;
    int nwrite;
    uint16_t *Ct16;
    int64_t ldq;
};
struct Batch {
    int count;
    Job j[kMaxJobs];
};

template <int NT>
struct Lds {
    static constexpr int TP = NT * 32;                            // B chunk pitch (floats)
    static constexpr int MAIN = kRows * kYP + kKC * TP;           // floats
    static constexpr int STAGE = (TP * kSP + 1) / 2;              // floats
    static constexpr int FLOATS = MAIN > STAGE ? MAIN : STAGE;
};

template <int NT, bool TRI>
__global__ __launch_bounds__(256) void tall_small_kernel(const Batch jb)
{
    using L = Lds<NT>;
    constexpr int TP = L::TP;
    constexpr int YV = kRows * (kKC / 4) / 256;    // float4 of an A chunk per thread
    constexpr int TV = kKC * (TP / 4) / 256;       // float4 of a B chunk per thread
    static_assert(YV * 256 == kRows * kKC / 4 && TV * 256 == kKC * TP / 4, "chunk split");
    __shared__ __attribute__((aligned(16))) float smem[L::FLOATS];
    float *Ys = smem, *Ts = smem + kRows * kYP;

    const Job &J = jb.j[blockIdx.z];
    const int rows = J.rows;
    const int row0 = blockIdx.x * kRows;
    if (row0 >= rows)
        return;
    const float *A = J.A;
    const float *B = J.B;
    const int64_t lda = J.lda, ldb = J.ldb;
    const int K = J.K, N = J.N;
    const int nk = (K + kKC - 1) / kKC;
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
            if (row0 + r < rows && c < K)
                v = *reinterpret_cast<const float4 *>(A + static_cast<int64_t>(row0 + r) * lda + c);
            yr[u] = v;
        }
#pragma unroll
        for (int u = 0; u < TV; ++u) {
            const int idx = tid + 256 * u;
            const int kk = idx / (TP / 4), c = (idx % (TP / 4)) * 4;
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (k0 + kk < K && c < N)
                v = *reinterpret_cast<const float4 *>(B + static_cast<int64_t>(k0 + kk) * ldb + c);
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
    for (int kc = 0; kc < nk; ++kc) {
        if (kc)
            __syncthreads();   // the previous chunk is consumed
        stash();
        __syncthreads();
        if (kc + 1 < nk)
            load(kc + 1);
        // A[i][k] = A[32 wave + i][2 s + k] in lane i + 32 k; B[k][j] = B[2 s + k][32 t + j].
        // The chunk's 16 steps go in four groups of four; each group's
        // operands are read before the previous group's products are issued
        // (scheduling barriers: left alone, the compiler reads each operand
        // just before its product and waits for it there).
        constexpr int SG = 4;
        const float *ya = Ys + (32 * wave + (lane & 31)) * kYP + (lane >> 5);
        const float *tb = Ts + (lane >> 5) * TP + (lane & 31);
        float ah[2][SG], bh[2][SG][NT];
        auto rd = [&](int g) {
#pragma unroll
            for (int q = 0; q < SG; ++q) {
                const int s = SG * g + q;
                ah[g & 1][q] = ya[2 * s];
#pragma unroll
                for (int t = 0; t < NT; ++t)
                    bh[g & 1][q][t] = tb[2 * s * TP + 32 * t];
            }
        };
        auto mm = [&](int g) {
#pragma unroll
            for (int t = 0; t < NT; ++t)
                if (!TRI || t >= kc) {
#pragma unroll
                    for (int q = 0; q < SG; ++q)
                        acc[t] = __builtin_amdgcn_mfma_f32_32x32x2f32(ah[g & 1][q], bh[g & 1][q][t], acc[t], 0, 0,
                                                                      0);
                }
        };
        rd(0);
#pragma unroll
        for (int g = 0; g < kKC / 2 / SG; ++g) {
            __builtin_amdgcn_sched_barrier(0);
            if (g + 1 < kKC / 2 / SG)
                rd(g + 1);
            __builtin_amdgcn_sched_barrier(0);
            mm(g);
        }
    }

    // D[i][j] in lane j + 32 ((i / 4) % 2), element 4 (i / 8) + i % 4
    const int j = lane & 31, hi = lane >> 5;
    const int nwrite = J.nwrite;
    const int64_t ldc = J.ldc;
    if (J.C32 || J.C16) {
        float *C32 = J.C32;
        uint16_t *C16 = J.C16;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int col = 32 * t + j;
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int row = row0 + 32 * wave + 8 * (e >> 2) + 4 * hi + (e & 3);
                if (row < rows && col < nwrite) {
                    if (C32)
                        C32[static_cast<int64_t>(row) * ldc + col] = acc[t][e];
                    else
                        C16[static_cast<int64_t>(row) * ldc + col] = f32_to_bf16(acc[t][e]);
                }
            }
        }
    }
    if (J.Ct16) {
        __syncthreads();   // every wave is done with the chunk buffers
        uint16_t *St = reinterpret_cast<uint16_t *>(smem);
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                uint32_t w0 = f32x2_to_bf16x2(acc[t][4 * q], acc[t][4 * q + 1]);
                uint32_t w1 = f32x2_to_bf16x2(acc[t][4 * q + 2], acc[t][4 * q + 3]);
                *reinterpret_cast<uint2 *>(St + (32 * t + j) * kSP + 32 * wave + 8 * q + 4 * hi) = make_uint2(w0, w1);
            }
        __syncthreads();
        uint16_t *Q = J.Ct16;
        const int64_t ldq = J.ldq;
        for (int idx = tid; idx < TP * (kRows / 8); idx += 256) {
            const int col = idx / (kRows / 8), r8 = (idx % (kRows / 8)) * 8;
            if (col < nwrite && row0 + r8 < rows)
                *reinterpret_cast<uint4 *>(Q + col * ldq + row0 + r8) =
                    *reinterpret_cast<const uint4 *>(St + col * kSP + r8);
        }
    }
}

template <int NT>
void launch(const char *tag, const std::vector<Job> &jobs, hipStream_t st)
{
    for (size_t c0 = 0; c0 < jobs.size(); c0 += kMaxJobs) {
        Batch b{};
        b.count = static_cast<int>(std::min<size_t>(kMaxJobs, jobs.size() - c0));
        int gx = 1;
        for (int i = 0; i < b.count; ++i) {
            b.j[i] = jobs[c0 + i];
            gx = std::max(gx, (b.j[i].rows + kRows - 1) / kRows);
        }
        // run() and gemm() each make jobs of one kind (triangular B or not)
        if (b.j[0].tri)
            ACSC_LAUNCH(tag, (tall_small_kernel<NT, true>), dim3(gx, 1, b.count), dim3(256), 0, st, b);
        else
            ACSC_LAUNCH(tag, (tall_small_kernel<NT, false>), dim3(gx, 1, b.count), dim3(256), 0, st, b);
    }
}

int launch_all(const char *tag, const std::vector<Job> &jobs, hipStream_t st)
{
    if (jobs.empty())
        return ACSC_OK;
    int np = 16;
    for (const Job &j : jobs)
        np = std::max(np, std::max(j.N, j.nwrite));
    switch ((np + 31) / 32) {
    case 1: launch<1>(tag, jobs, st); break;
    case 2: launch<2>(tag, jobs, st); break;
    case 3: launch<3>(tag, jobs, st); break;
    case 4: launch<4>(tag, jobs, st); break;
    case 5: launch<5>(tag, jobs, st); break;
    default: launch<6>(tag, jobs, st); break;
    }
    return ACSC_OK;
}


// C = A^T B over row ranges: workgroup b of a job sums rows
// [b rpb, (b + 1) rpb) into its partial.  Rows arrive in 32-row chunks staged
// in LDS (A chunk, then B chunk, rows of NT x 32 floats); output tile
// (ti, tj) of 32 x 32 belongs to wave (ti NT + tj) % 4.
struct InnerJob {
    const float *A;
    int64_t lda;
    const float *B;
    int64_t ldb;
    int rows, NA, NB, rpb, blocks;
    float *part;
};
struct InnerBatch {
    int count;
    InnerJob j[kMaxJobs];
};

template <int NT>
__global__ __launch_bounds__(256) void tall_inner_kernel(const InnerBatch jb)
{
    constexpr int W = NT * 32;                 // staged row width (floats)
    constexpr int P = W + 4;                   // LDS row pitch (16-byte aligned)
    constexpr int TILES = NT * NT;
    constexpr int TPW = (TILES + 3) / 4;
    constexpr int CV = 32 * (W / 4);           // float4 of one operand chunk
    constexpr int PF = (CV + 255) / 256;       // float4 per thread and operand
    __shared__ __attribute__((aligned(16))) float As[32 * P], Bs[32 * P];
    const InnerJob &J = jb.j[blockIdx.z];
    if (static_cast<int>(blockIdx.x) >= J.blocks)
        return;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r0 = blockIdx.x * J.rpb;
    const int r1 = min(J.rows, r0 + J.rpb);
    const int NA = J.NA, NB = J.NB;

    f32x16 acc[TPW];
#pragma unroll
    for (int u = 0; u < TPW; ++u)
#pragma unroll
        for (int e = 0; e < 16; ++e)
            acc[u][e] = 0.f;

    float4 pa[PF], pb[PF];
    auto load = [&](int rb) {
#pragma unroll
        for (int u = 0; u < PF; ++u) {
            const int idx = tid + 256 * u;
            const int rr = idx / (W / 4), c = (idx % (W / 4)) * 4;
            const int gr = rb + rr;
            float4 a = make_float4(0.f, 0.f, 0.f, 0.f), b = a;
            if (idx < CV && gr < r1) {
                if (c < NA)
                    a = *reinterpret_cast<const float4 *>(J.A + static_cast<int64_t>(gr) * J.lda + c);
                if (c < NB)
                    b = *reinterpret_cast<const float4 *>(J.B + static_cast<int64_t>(gr) * J.ldb + c);
            }
            pa[u] = a;
            pb[u] = b;
        }
    };
    load(r0);
    for (int rb = r0; rb < r1; rb += 32) {
        __syncthreads();
#pragma unroll
        for (int u = 0; u < PF; ++u) {
            const int idx = tid + 256 * u;
            if (idx < CV) {
                const int o = (idx / (W / 4)) * P + (idx % (W / 4)) * 4;
                *reinterpret_cast<float4 *>(&As[o]) = pa[u];
                *reinterpret_cast<float4 *>(&Bs[o]) = pb[u];
            }
        }
        __syncthreads();
        if (rb + 32 < r1)
            load(rb + 32);
        // A'[i][k] = A[row 2 s + k][32 ti + i] in lane i + 32 k; B'[k][j] = B[row 2 s + k][32 tj + j]
#pragma unroll
        for (int s = 0; s < 16; ++s) {
            const int row = 2 * s + (lane >> 5);
#pragma unroll
            for (int u = 0; u < TPW; ++u) {
                const int t = wave + 4 * u;
                if (t < TILES) {
                    const int ti = t / NT, tj = t % NT;
                    acc[u] = __builtin_amdgcn_mfma_f32_32x32x2f32(As[row * P + 32 * ti + (lane & 31)],
                                                                  Bs[row * P + 32 * tj + (lane & 31)], acc[u], 0, 0, 0);
                }
            }
        }
    }
    // D[i][j] in lane j + 32 ((i / 4) % 2), element 4 (i / 8) + i % 4
    float *pp = J.part + static_cast<int64_t>(blockIdx.x) * W * W;
#pragma unroll
    for (int u = 0; u < TPW; ++u) {
        const int t = wave + 4 * u;
        if (t < TILES) {
            const int ti = t / NT, tj = t % NT;
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int i = 32 * ti + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
                pp[i * W + 32 * tj + (lane & 31)] = acc[u][e];
            }
        }
    }
}

struct InnerRedJob {
    const float *part;
    int blocks, NA, NB, W;
    float *C;
    int64_t ldc;
};
struct InnerRedBatch {
    int count;
    InnerRedJob j[kMaxJobs];
};

// C[i][j] = sum over blocks (fixed order) of part[b][i][j]
__global__ __launch_bounds__(256) void tall_inner_reduce_kernel(const InnerRedBatch jb)
{
    const InnerRedJob &J = jb.j[blockIdx.z];
    const int idx = blockIdx.x * 256 + threadIdx.x;
    if (idx >= J.NA * J.NB)
        return;
    const int i = idx / J.NB, j = idx - (idx / J.NB) * J.NB;
    const int64_t stride = static_cast<int64_t>(J.W) * J.W;
    const float *p = J.part + i * J.W + j;
    float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
    int b = 0;
    for (; b + 4 <= J.blocks; b += 4) {
        s0 += p[b * stride];
        s1 += p[(b + 1) * stride];
        s2 += p[(b + 2) * stride];
        s3 += p[(b + 3) * stride];
    }
    for (; b < J.blocks; ++b)
        s0 += p[b * stride];
    J.C[static_cast<int64_t>(i) * J.ldc + j] = (s0 + s1) + (s2 + s3);
}

template <int NT>
void launch_inner(const char *tag, const std::vector<InnerJob> &jobs, const std::vector<InnerRedJob> &red,
                  hipStream_t st)
{
    for (size_t c0 = 0; c0 < jobs.size(); c0 += kMaxJobs) {
        InnerBatch b{};
        InnerRedBatch rb{};
        b.count = rb.count = static_cast<int>(std::min<size_t>(kMaxJobs, jobs.size() - c0));
        int gx = 1, rx = 1;
        for (int i = 0; i < b.count; ++i) {
            b.j[i] = jobs[c0 + i];
            rb.j[i] = red[c0 + i];
            gx = std::max(gx, b.j[i].blocks);
            rx = std::max(rx, (rb.j[i].NA * rb.j[i].NB + 255) / 256);
        }
        ACSC_LAUNCH(tag, tall_inner_kernel<NT>, dim3(gx, 1, b.count), dim3(256), 0, st, b);
        ACSC_LAUNCH("sc_inner_reduce", tall_inner_reduce_kernel, dim3(rx, 1, rb.count), dim3(256), 0, st, rb);
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
        jobs.push_back(Job{q.Y, KP, q.rows, KP, q.T, KP, KP, 1, q.write32 ? q.Y : nullptr, nullptr, KP, KP,
                           q.Qt16, q.ldq});
    }
    return launch_all(tag, jobs, st);
}

bool gemm_supported(const GemmReq &q)
{
    return aligned(q.A, 16) && aligned(q.B, 16) && q.lda % 4 == 0 && q.ldb % 4 == 0 && q.K % 4 == 0 &&
           q.N % 4 == 0 && q.K >= 1 && q.K <= SC_KMAX && q.N >= 1 && q.N <= SC_KMAX && q.nwrite <= SC_KMAX &&
           q.lda >= q.K && q.ldb >= q.N && q.ldc >= q.nwrite;
}

int gemm(const char *tag, const std::vector<GemmReq> &reqs, hipStream_t st)
{
    std::vector<Job> jobs;
    for (const GemmReq &q : reqs) {
        if (!gemm_supported(q))
            return set_error(ACSC_EINVAL, "tall product: operands not aligned or sizes out of range");
        if (q.rows < 1)
            continue;
        jobs.push_back(Job{q.A, q.lda, q.rows, q.K, q.B, q.ldb, q.N, 0, q.C32, q.C16, q.ldc, q.nwrite, nullptr, 0});
    }
    return launch_all(tag, jobs, st);
}

bool inner_supported(const InnerReq &q)
{
    const int64_t W = (std::max(q.NA, q.NB) + 31) / 32 * 32;
    return aligned(q.A, 16) && aligned(q.B, 16) && q.lda % 4 == 0 && q.ldb % 4 == 0 && q.NA % 4 == 0 &&
           q.NB % 4 == 0 && q.NA >= 1 && q.NA <= SC_KMAX && q.NB >= 1 && q.NB <= SC_KMAX && q.lda >= q.NA &&
           q.ldb >= q.NB && q.ldc >= q.NB &&
           static_cast<int64_t>(q.part_blocks) * q.NA * q.NB >= W * W;   // room for one partial block
}

int inner(const char *tag, const std::vector<InnerReq> &reqs, hipStream_t st)
{
    int np = 32;
    int64_t total = 0;
    for (const InnerReq &q : reqs) {
        if (!inner_supported(q))
            return set_error(ACSC_EINVAL, "tall inner product: operands not aligned or sizes out of range");
        np = std::max(np, std::max(q.NA, q.NB));
        total += std::max(q.rows, 0);
    }
    const int NT = (np + 31) / 32, W = NT * 32;
    // one row count per block across the batch (about two workgroups per CU),
    // raised where a matrix's partial buffer holds fewer blocks
    const int64_t rpb_batch = std::max<int64_t>(32, (total + 511) / 512 + 31) / 32 * 32;
    std::vector<InnerJob> jobs;
    std::vector<InnerRedJob> red;
    for (const InnerReq &q : reqs) {
        if (q.rows < 1)
            continue;
        const int64_t cap = static_cast<int64_t>(q.part_blocks) * q.NA * q.NB / (static_cast<int64_t>(W) * W);
        if (cap < 1)
            return set_error(ACSC_EINVAL, "tall inner product: partial buffer too small");
        int64_t rpb = std::max<int64_t>(rpb_batch, (q.rows + cap - 1) / cap);
        rpb = (rpb + 31) / 32 * 32;
        const int blocks = static_cast<int>((q.rows + rpb - 1) / rpb);
        jobs.push_back(InnerJob{q.A, q.lda, q.B, q.ldb, q.rows, q.NA, q.NB, static_cast<int>(rpb), blocks, q.part});
        red.push_back(InnerRedJob{q.part, blocks, q.NA, q.NB, W, q.C, q.ldc});
    }
    if (jobs.empty())
        return ACSC_OK;
    switch (NT) {
    case 1: launch_inner<1>(tag, jobs, red, st); break;
    case 2: launch_inner<2>(tag, jobs, red, st); break;
    case 3: launch_inner<3>(tag, jobs, red, st); break;
    case 4: launch_inner<4>(tag, jobs, red, st); break;
    case 5: launch_inner<5>(tag, jobs, red, st); break;
    default: launch_inner<6>(tag, jobs, red, st); break;
    }
    return ACSC_OK;
}

}  // namespace orth
}  // namespace acsc
