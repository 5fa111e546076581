// Fused blend for gfx950 (see sc_blend.h), bf16 gradients.
//
// One workgroup per 128 x 128 tile of G.  The tile's 128 rows of P and 128
// rows of V (RP bf16 each) go straight from L2 into LDS (global_load_lds:
// lane L's 16 bytes land at the wave-uniform LDS address in M0 plus 16 L),
// XOR-swizzled in 128-byte groups; the G tile is loaded into registers right
// after and stays in flight while the four waves form P V^T on
// v_mfma_f32_32x32x16_bf16 (64 x 64 per wave).  The fp32 product is staged in
// LDS in G's row order, and each thread blends its own 16-byte chunks of G
// and writes them out.  Tiles are dealt so that XCD x owns the row blocks
// congruent to x mod 8 (each P slice stays in one L2) and walks them in bands
// of 64 columns (the band's V slices stay there too).
#include "common.h"
#include "sc_blend.h"

#include <algorithm>

namespace acsc {
namespace blend {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(short)))) short bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((address_space(3))) unsigned char lds_byte;
typedef unsigned int nu4 __attribute__((ext_vector_type(4)));
typedef float nf4 __attribute__((ext_vector_type(4)));

constexpr int kT = 128;          // tile edge
constexpr int kStPitch = 132;    // floats per staged product row (16-byte writes of 16 rows conflict-free)
constexpr int kMaxJobs = 16;
constexpr int kBand = 64;        // column blocks per band of the tile walk (2 MiB of V slices per XCD)

__host__ __device__ inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

struct Job {
    const uint16_t *G;
    uint16_t *out;
    int m, n;
    const uint16_t *P, *V;
    float *W, *m1, *m2;
    float *E;
    int vec;
};
struct Batch {
    int count;
    Job j[kMaxJobs];
};

// LDS slot of 16-byte chunk c of P / V row r (rows of RB bytes; an XOR, so
// the same map takes a slot back to its chunk).  Measured with the bank
// conflict counter on MI355X: 256-byte rows need all four chunk bits mixed
// with the row's low bits for the 16 rows a fragment read touches to spread
// over every bank; other row widths mix the low three bits with
// (r >> 1) ^ r.  Either way a fragment read runs without bank conflicts.
template <int RB>
__device__ __forceinline__ int slot_of(int c, int r)
{
    if constexpr (RB == 256)
        return c ^ (r & 15);
    else
        return (c & ~7) | ((c & 7) ^ (((r >> 1) ^ r) & 7));
}

// global_load_lds_dwordx4 takes its wave-uniform LDS address in M0.  The asm
// saves M0 in a scratch SGPR and restores it, so M0 holds, after the
// statement, whatever the compiler may have kept there; an LDS DMA needs one
// wait state after a scalar write of M0 (the GFX9-family hazard), hence the
// s_nop after each write (the compiler's hazard tracking does not see inside
// the statement).  (The compiler's own builtin for this instruction counts
// it in its LDS wait model and then waits for all fragment reads before the
// first MFMA of a step; kept opaque here, the explicit vmcnt waits of the
// kernel order the DMA.)
__device__ __forceinline__ void dma16(const void *gptr, uint32_t lds_addr)
{
    uint32_t saved;
    asm volatile("s_mov_b32 %0, m0\n\t"
                 "s_mov_b32 m0, %2\n\t"
                 "s_nop 0\n\t"
                 "global_load_lds_dwordx4 %1, off\n\t"
                 "s_mov_b32 m0, %0\n\t"
                 "s_nop 0"
                 : "=&s"(saved)
                 : "v"(gptr), "s"(lds_addr)
                 : "memory");
}

__device__ __forceinline__ void sync_lds()
{
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Wait until at most N vector-memory instructions of this wave are in
// flight (every older one has completed: they complete in issue order);
// N < 0 waits for all of them.
template <int N>
__device__ __forceinline__ void wait_vm()
{
    static_assert(N < 64, "vmcnt range");
    if constexpr (N < 0)
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    else
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// MODE kAdam: the blended values are not stored; they are the gradient of
// the AdamW step applied to the tile's weights and moments (fp32, in place).
// MODE kFeedback: no G; out = P V^T, and the fp32 memory E (holding M) takes
// M - out, with out as stored (bf16).
template <int RP, bool VEC, int MODE>
__global__ __launch_bounds__(256) void blend_kernel(const Batch jb, float alpha, const AdamArgs ad)
{
    constexpr bool ADAM = MODE == kAdam, EF = MODE == kFeedback;
    constexpr int RB = RP * 2;                  // bytes per P / V row
    constexpr int SLICE = kT * RB;              // bytes of one 128-row slice
    constexpr int NI = 2 * SLICE / 1024;        // DMA instructions for P and V
    static_assert(NI % 4 == 0 && RB % 128 == 0, "slice layout");
    constexpr int LDS = (2 * SLICE > kT * kStPitch * 4) ? 2 * SLICE : kT * kStPitch * 4;
    __shared__ __attribute__((aligned(1024))) unsigned char smem[LDS];

    const Job &J = jb.j[blockIdx.z];
    const int m = J.m, n = J.n;
    const int rb_n = static_cast<int>(cdiv(m, kT)), cb_n = static_cast<int>(cdiv(n, kT));
    // XCD x (= block % 8) owns the row blocks x, x + 8, ...; it walks them in
    // column bands of kBand column blocks, row blocks outer, so that a band's
    // V slices and the current P slice stay in its L2
    const int b = blockIdx.x;
    const int xcd = b & 7, t = b >> 3;
    const int nr = (rb_n - xcd + 7) / 8;
    if (t >= nr * cb_n)
        return;
    const int band = t / (nr * kBand);
    const int rem = t - band * nr * kBand;
    const int bw = min(kBand, cb_n - band * kBand);
    const int rb = xcd + 8 * (rem / bw);
    const int cb = band * kBand + rem % bw;
    const int row0 = rb * kT, col0 = cb * kT;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_byte *)smem));

    // P rows row0.. and V rows col0.. (clamped: rows past the end only feed
    // outputs that are never stored), 16 bytes per lane, swizzled per row
#pragma unroll
    for (int u = 0; u < NI / 4; ++u) {
        const int ins = u * 4 + wave;
        const int off = (ins * 1024 + lane * 16) % SLICE;   // byte offset within the slice
        const bool isV = ins * 1024 >= SLICE;
        const int r = off / RB;
        const int cl = (off % RB) / 16;
        const int c = slot_of<RB>(cl, r);
        const uint16_t *src = isV ? J.V + static_cast<int64_t>(min(col0 + r, n - 1)) * RP
                                  : J.P + static_cast<int64_t>(min(row0 + r, m - 1)) * RP;
        dma16(src + c * 8, lds0 + ins * 1024);
    }
    // the G tile into registers: thread q holds row q / 16, columns 8 (q % 16) ..
    // VEC: kRowLoads unconditional 16-byte loads per thread of kLoadsPerRow
    // instructions each (row and column clamped into G; what lies outside is
    // never stored), so that "at most kTail loads outstanding" below means
    // every slice DMA has landed.  Otherwise element loads, and the wait is
    // for everything.  kFeedback: the fp32 memory, two 16-byte loads a row.
    constexpr int kRowLoads = 8;
    constexpr int kLoadsPerRow = EF ? 2 : 1;
    constexpr int kTail = VEC ? kRowLoads * kLoadsPerRow : -1;
    static_assert(kT * kT / (256 * 8) == kRowLoads, "one 16-byte chunk of 8 elements per thread and load");
    uint4 g[kRowLoads];
    nf4 ev[kRowLoads * 2];
    if constexpr (EF) {
        if (VEC) {
#pragma unroll
            for (int u = 0; u < kRowLoads; ++u) {
                const int q = tid + 256 * u;
                const int gi = row0 + (q >> 4), gj = col0 + (q & 15) * 8;
                const nf4 *src = reinterpret_cast<const nf4 *>(J.E + static_cast<int64_t>(min(gi, m - 1)) * n +
                                                               min(gj, n - 8));
                ev[2 * u] = __builtin_nontemporal_load(src);
                ev[2 * u + 1] = __builtin_nontemporal_load(src + 1);
            }
        }
    }
#pragma unroll
    for (int u = 0; u < kRowLoads && !EF; ++u) {
        const int q = tid + 256 * u;
        const int gi = row0 + (q >> 4), gj = col0 + (q & 15) * 8;
        if (VEC) {
            // G streams through once: non-temporal, so that it does not push P and V out of L2
            const nu4 v = __builtin_nontemporal_load(
                reinterpret_cast<const nu4 *>(J.G + static_cast<int64_t>(min(gi, m - 1)) * n + min(gj, n - 8)));
            g[u] = make_uint4(v.x, v.y, v.z, v.w);
        } else {
            uint4 v = make_uint4(0u, 0u, 0u, 0u);
            if (gi < m) {
                const uint16_t *src = J.G + static_cast<int64_t>(gi) * n + gj;
                uint16_t e8[8];
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    e8[e] = gj + e < n ? src[e] : uint16_t(0);
                __builtin_memcpy(&v, e8, sizeof(v));
            }
            g[u] = v;
        }
    }
    wait_vm<kTail>();
    sync_lds();

    // P V^T: wave w computes rows 64 (w / 2) .., columns 64 (w % 2) .. as 2 x 2
    // tiles of 32 x 32; A[i][k] / B[k][j] in lane i (j) + 32 (k / 8), element k % 8
    const unsigned char *Ps = smem, *Vs = smem + SLICE;
    const int wr = (wave >> 1) * 64, wc = (wave & 1) * 64;
    f32x16 acc[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
            for (int e = 0; e < 16; ++e)
                acc[a][c][e] = 0.f;
#pragma unroll
    for (int kq = 0; kq < RP / 16; ++kq) {
        const int cs = kq * 2 + (lane >> 5);   // logical 16-byte chunk of the row
        bf16x8 af[2], bfr[2];
#pragma unroll
        for (int a = 0; a < 2; ++a) {
            const int r = wr + a * 32 + (lane & 31);
            af[a] = *reinterpret_cast<const bf16x8 *>(Ps + r * RB + 16 * slot_of<RB>(cs, r));
        }
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            const int r = wc + c * 32 + (lane & 31);
            bfr[c] = *reinterpret_cast<const bf16x8 *>(Vs + r * RB + 16 * slot_of<RB>(cs, r));
        }
        // (P V^T)^T = V P^T: V's rows as the A operand put four consecutive
        // columns of a G row in each lane's consecutive accumulators, so the
        // product is staged with 16-byte writes
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int c = 0; c < 2; ++c)
                acc[a][c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[c], af[a], acc[a][c], 0, 0, 0);
    }
    sync_lds();
    // stage the product: D^T[j][i] sits in lane i + 32 ((j / 4) % 2), element
    // 4 (j / 8) + j % 4, so elements 4 q .. 4 q + 3 are columns
    // j0 + 8 q + 4 (lane / 32) .. + 3 of row i = lane % 32 (row pitch 132
    // floats: the 16 rows a write touches fall on distinct banks)
    float *St = reinterpret_cast<float *>(smem);
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int i = wr + a * 32 + (lane & 31);
                const int j = wc + c * 32 + 8 * q + 4 * (lane >> 5);
                *reinterpret_cast<float4 *>(&St[i * kStPitch + j]) =
                    make_float4(acc[a][c][4 * q], acc[a][c][4 * q + 1], acc[a][c][4 * q + 2], acc[a][c][4 * q + 3]);
            }
    sync_lds();
    const float oma = 1.0f - alpha;
    if constexpr (EF) {
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int q = tid + 256 * u;
            const int rr = q >> 4, c8 = (q & 15) * 8;
            const int gi = row0 + rr, gj = col0 + c8;
            if (gi >= m)
                continue;
            const float4 p0 = *reinterpret_cast<const float4 *>(&St[rr * kStPitch + c8]);
            const float4 p1 = *reinterpret_cast<const float4 *>(&St[rr * kStPitch + c8 + 4]);
            const float pf[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
            uint16_t ob[8];
            float of[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                ob[e] = f32_to_bf16(pf[e]);
                of[e] = __uint_as_float(static_cast<uint32_t>(ob[e]) << 16);
            }
            const int64_t o = static_cast<int64_t>(gi) * n + gj;
            if (VEC && gj + 8 <= n) {
                nf4 e0 = ev[2 * u], e1 = ev[2 * u + 1];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    e0[e] = e0[e] - of[e];
                    e1[e] = e1[e] - of[4 + e];
                }
                const nu4 ov{static_cast<uint32_t>(ob[0]) | (static_cast<uint32_t>(ob[1]) << 16),
                             static_cast<uint32_t>(ob[2]) | (static_cast<uint32_t>(ob[3]) << 16),
                             static_cast<uint32_t>(ob[4]) | (static_cast<uint32_t>(ob[5]) << 16),
                             static_cast<uint32_t>(ob[6]) | (static_cast<uint32_t>(ob[7]) << 16)};
                __builtin_nontemporal_store(ov, reinterpret_cast<nu4 *>(J.out + o));
                __builtin_nontemporal_store(e0, reinterpret_cast<nf4 *>(J.E + o));
                __builtin_nontemporal_store(e1, reinterpret_cast<nf4 *>(J.E + o) + 1);
            } else {
                for (int e = 0; e < 8 && gj + e < n; ++e) {
                    J.out[o + e] = ob[e];
                    J.E[o + e] = J.E[o + e] - of[e];
                }
            }
        }
        return;
    }
    if constexpr (ADAM) {
        const float cf = *ad.coef;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int q = tid + 256 * u;
            const int rr = q >> 4, c8 = (q & 15) * 8;
            const int gi = row0 + rr, gj = col0 + c8;
            if (gi >= m)
                continue;
            const float4 p0 = *reinterpret_cast<const float4 *>(&St[rr * kStPitch + c8]);
            const float4 p1 = *reinterpret_cast<const float4 *>(&St[rr * kStPitch + c8 + 4]);
            const float pf[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
            const uint32_t w[4] = {g[u].x, g[u].y, g[u].z, g[u].w};
            float gp[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                gp[2 * e] = cf * blend_step(__uint_as_float(w[e] << 16), pf[2 * e], alpha, oma);
                gp[2 * e + 1] = cf * blend_step(__uint_as_float(w[e] & 0xFFFF0000u), pf[2 * e + 1], alpha, oma);
            }
            const int64_t o = static_cast<int64_t>(gi) * n + gj;
            if (VEC && gj + 8 <= n) {
                // the state streams through once: non-temporal both ways
                nf4 wv[2], mv[2], vv[2];
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    wv[h] = __builtin_nontemporal_load(reinterpret_cast<const nf4 *>(J.W + o) + h);
                    mv[h] = __builtin_nontemporal_load(reinterpret_cast<const nf4 *>(J.m1 + o) + h);
                    vv[h] = __builtin_nontemporal_load(reinterpret_cast<const nf4 *>(J.m2 + o) + h);
                }
#pragma unroll
                for (int h = 0; h < 2; ++h)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        float we = wv[h][e], me = mv[h][e], ve = vv[h][e];
                        adamw_elem(gp[4 * h + e], we, me, ve, ad);
                        wv[h][e] = we;
                        mv[h][e] = me;
                        vv[h][e] = ve;
                    }
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    __builtin_nontemporal_store(wv[h], reinterpret_cast<nf4 *>(J.W + o) + h);
                    __builtin_nontemporal_store(mv[h], reinterpret_cast<nf4 *>(J.m1 + o) + h);
                    __builtin_nontemporal_store(vv[h], reinterpret_cast<nf4 *>(J.m2 + o) + h);
                }
            } else {
                for (int e = 0; e < 8 && gj + e < n; ++e) {
                    float wv = J.W[o + e], mv = J.m1[o + e], vv = J.m2[o + e];
                    adamw_elem(gp[e], wv, mv, vv, ad);
                    J.W[o + e] = wv;
                    J.m1[o + e] = mv;
                    J.m2[o + e] = vv;
                }
            }
        }
        return;
    }
    // chunk u of this thread: row q / 16, columns 8 (q % 16) .. of the tile
    auto blended = [&](int u, int rr, int c8) {
        const float4 p0 = *reinterpret_cast<const float4 *>(&St[rr * kStPitch + c8]);
        const float4 p1 = *reinterpret_cast<const float4 *>(&St[rr * kStPitch + c8 + 4]);
        const float pf[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
        const uint32_t w[4] = {g[u].x, g[u].y, g[u].z, g[u].w};
        nu4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float lo = blend_step(__uint_as_float(w[e] << 16), pf[2 * e], alpha, oma);
            const float hi = blend_step(__uint_as_float(w[e] & 0xFFFF0000u), pf[2 * e + 1], alpha, oma);
            o[e] = f32x2_to_bf16x2(lo, hi);
        }
        return o;
    };
    if (VEC && row0 + kT <= m && col0 + kT <= n) {
        // a whole tile: every chunk is stored, with no bounds tests
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int q = tid + 256 * u;
            const int rr = q >> 4, c8 = (q & 15) * 8;
            const nu4 o = blended(u, rr, c8);
            __builtin_nontemporal_store(o, reinterpret_cast<nu4 *>(J.out + static_cast<int64_t>(row0 + rr) * n +
                                                                   col0 + c8));
        }
        return;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        const int q = tid + 256 * u;
        const int rr = q >> 4, c8 = (q & 15) * 8;
        const int gi = row0 + rr, gj = col0 + c8;
        if (gi >= m)
            continue;
        const nu4 o = blended(u, rr, c8);
        uint16_t *dst = J.out + static_cast<int64_t>(gi) * n + gj;
        if (VEC && gj + 8 <= n) {
            __builtin_nontemporal_store(o, reinterpret_cast<nu4 *>(dst));
        } else {
            const uint32_t ow[4] = {o.x, o.y, o.z, o.w};
            const uint16_t *e8 = reinterpret_cast<const uint16_t *>(ow);
            for (int e = 0; e < 8 && gj + e < n; ++e)
                dst[e] = e8[e];
        }
    }
}

template <int RP, int MODE>
void launch_rp(const char *tag, const std::vector<Job> &jobs, int tiles, float alpha, const AdamArgs &ad,
               hipStream_t st)
{
    std::vector<Job> part[2];
    for (const Job &j : jobs)
        part[j.vec ? 1 : 0].push_back(j);
    for (int v = 0; v < 2; ++v)
        for (size_t c0 = 0; c0 < part[v].size(); c0 += kMaxJobs) {
            Batch b{};
            b.count = static_cast<int>(std::min<size_t>(kMaxJobs, part[v].size() - c0));
            for (int i = 0; i < b.count; ++i)
                b.j[i] = part[v][c0 + i];
            if (v) {
                auto kern = blend_kernel<RP, true, MODE>;
                ACSC_LAUNCH(tag, kern, dim3(tiles, 1, b.count), dim3(256), 0, st, b, alpha, ad);
            } else {
                auto kern = blend_kernel<RP, false, MODE>;
                ACSC_LAUNCH(tag, kern, dim3(tiles, 1, b.count), dim3(256), 0, st, b, alpha, ad);
            }
        }
}

template <int MODE>
void launch_mode(const char *tag, int RP, const std::vector<Job> &jobs, int tiles, float alpha, const AdamArgs &ad,
                 hipStream_t st)
{
    switch (RP) {
    case 64: launch_rp<64, MODE>(tag, jobs, tiles, alpha, ad, st); break;
    case 128: launch_rp<128, MODE>(tag, jobs, tiles, alpha, ad, st); break;
    default: launch_rp<192, MODE>(tag, jobs, tiles, alpha, ad, st); break;
    }
}

int launch_all(const char *tag, const std::vector<Req> &reqs, int RP, float alpha, hipStream_t st,
               const AdamArgs *adam, bool feedback)
{
    if (!supported(RP))
        return set_error(ACSC_EINVAL, "blend: padded rank %d not handled by the streamed-tile kernel", RP);
    std::vector<Job> jobs;
    int tiles = 1;
    auto a16 = [](const void *p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; };
    for (const Req &q : reqs) {
        bool vec = q.n % 8 == 0 && q.n >= 8 && (feedback ? a16(q.E) : a16(q.G));
        vec = vec && (adam ? a16(q.W) && a16(q.m1) && a16(q.m2) : a16(q.out));
        jobs.push_back(Job{q.G, q.out, q.m, q.n, q.P, q.V, q.W, q.m1, q.m2, q.E, vec ? 1 : 0});
        const int64_t rbn = cdiv(q.m, kT), cbn = cdiv(q.n, kT);
        tiles = std::max<int>(tiles, static_cast<int>(cdiv(rbn, 8) * 8 * cbn));
    }
    const AdamArgs none{};
    const AdamArgs &ad = adam ? *adam : none;
    if (feedback)
        launch_mode<kFeedback>(tag, RP, jobs, tiles, alpha, ad, st);
    else if (adam)
        launch_mode<kAdam>(tag, RP, jobs, tiles, alpha, ad, st);
    else
        launch_mode<kPlain>(tag, RP, jobs, tiles, alpha, ad, st);
    return ACSC_OK;
}

}  // namespace

bool supported(int RP) { return RP == 64 || RP == 128 || RP == 192; }

int run(const char *tag, const std::vector<Req> &reqs, int RP, float alpha, hipStream_t st, const AdamArgs *adam)
{
    return launch_all(tag, reqs, RP, alpha, st, adam, false);
}

int run_feedback(const char *tag, const std::vector<Req> &reqs, int RP, hipStream_t st)
{
    return launch_all(tag, reqs, RP, 0.0f, st, nullptr, true);
}

}  // namespace blend
}  // namespace acsc
