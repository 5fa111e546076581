// Streaming passes for gfx950: a large bf16 matrix times a thin bf16 factor,
// fp32 accumulation on v_mfma_f32_16x16x32_bf16 (see sc_pass.h).
//
// The large operand is the HBM stream; the thin factor is small and is read
// from L2.  A workgroup owns 256 output rows (four waves of 64) and walks its
// K range in 64-deep steps.  Each step's slice of the thin factor is staged
// once in LDS and shared by the four waves; each wave stages its own 64 lines
// of A (128 contiguous bytes each) in LDS in the order they were loaded and
// reads its MFMA fragments back from there: 16-byte reads for opA = A,
// 16-bit gathers for opA = A^T.  Loads run two steps ahead in registers and
// the LDS tiles are double-buffered: one barrier per step.  Output rows are independent, so the K range is only
// split (into power-of-two slices, partials summed by a second kernel) when
// the batch has too few row blocks to give every CU one; block b works on
// split b % splits, which keeps each split on the same XCDs.
#include "common.h"
#include "sc_pass.h"

#include <algorithm>
#include <cstdlib>
#include <functional>
#include <map>
#include <mutex>

namespace acsc {
namespace pass {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(short)))) short bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
typedef __attribute__((address_space(3))) unsigned char lds_byte;

constexpr int kBM = 256;            // output rows per workgroup
constexpr int kBK = 64;             // depth of one step
constexpr int kBPitch = kBK + 8;    // bf16 per LDS row of the thin factor (144 B, 16-B aligned)
constexpr int kTPitch = 66;         // bf16 per k-row of a wave's A^T tile (33 dwords: conflict-free reads)
constexpr int kMaxNT = SC_KMAX / 16;
constexpr int kMaxJobs = 16;

__host__ __device__ inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
__host__ __device__ inline int64_t round_up(int64_t a, int64_t b) { return cdiv(a, b) * b; }

struct Job {
    const uint16_t *A;
    int64_t lda;
    const uint16_t *Bt;
    int64_t ldbt;
    float *C;
    int64_t ldc, split_stride;
    int M, K, kchunk, splits, nblocks, avec;
};

struct Batch {
    int count;
    Job j[kMaxJobs];
};

// Keep the first `avail` bf16 elements of an 8-element chunk, zero the rest.
__device__ __forceinline__ uint4 keep_first(uint4 v, int avail)
{
    auto m = [&](int e) -> uint32_t { return (e < avail ? 0xFFFFu : 0u) | (e + 1 < avail ? 0xFFFF0000u : 0u); };
    v.x &= m(0);
    v.y &= m(2);
    v.z &= m(4);
    v.w &= m(6);
    return v;
}

// 8 bf16 from a possibly unaligned address, elements >= avail read as zero.
__device__ __forceinline__ uint4 load8_scalar(const uint16_t *src, int avail)
{
    uint16_t e8[8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
        e8[e] = e < avail ? src[e] : uint16_t(0);
    uint4 v;
    __builtin_memcpy(&v, e8, sizeof(v));
    return v;
}

// Workgroup barrier that orders LDS accesses only.  __syncthreads() also
// fences global memory, which makes every wave wait for its outstanding
// global loads at the barrier and would drain the prefetch pipeline.
__device__ __forceinline__ void lds_barrier()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ __forceinline__ bf16x8 as_frag(const uint4 &v)
{
    bf16x8 f;
    __builtin_memcpy(&f, &v, sizeof(f));
    return f;
}

// VEC: A rows start 16-byte aligned and the row stride is a multiple of 8,
// so every 16-byte chunk that starts inside a row lies inside its padded
// extent.  Loads then need no guards: rows past the end are clamped to the
// last row (they only feed outputs that are never stored, or meet zero rows
// of the thin factor) and k is masked when a tail step is staged in LDS.
// !VEC: element loads with full guards (unaligned operands).
// NTK column tiles are computed; tiles at or past np / 16 read zeros and are
// not stored.
template <bool TRANS, int NTK, bool VEC>
__global__ __launch_bounds__(256) void pass_kernel(const Batch jb, int np)
{
    const Job &J = jb.j[blockIdx.z];
    if (static_cast<int>(blockIdx.x) >= J.nblocks)
        return;
    constexpr int NT = NTK;
    constexpr int NP = NT * 16;
    constexpr int BCH = NP * (kBK / 8);        // 16-byte chunks of one thin-factor step
    constexpr int BPT = (BCH + 255) / 256;
    // A step per wave: opA = A: [64 rows][kBPitch] (k contiguous);
    //                  opA = A^T: [64 k][kTPitch] (rows contiguous)
    constexpr int AW = TRANS ? kBK * kTPitch : 64 * kBPitch;
    __shared__ __attribute__((aligned(16))) uint16_t Bs[2][NP * kBPitch];
    __shared__ __attribute__((aligned(16))) uint16_t As[2][4 * AW];

    const uint16_t *__restrict__ A = J.A;
    const uint16_t *__restrict__ Bt = J.Bt;
    const int64_t lda = J.lda, ldbt = J.ldbt;
    const int M = J.M, splits = J.splits;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int split = static_cast<int>(blockIdx.x % splits);
    const int row0 = static_cast<int>(blockIdx.x / splits) * kBM;
    const int wrow0 = row0 + wave * 64;
    const int kbeg = split * J.kchunk;
    const int kend = min(J.K, kbeg + J.kchunk);
    const int nsteps = kend > kbeg ? static_cast<int>(cdiv(kend - kbeg, kBK)) : 0;
    const int bch_live = np * (kBK / 8);

    f32x4 acc[4][NT];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int t = 0; t < NT; ++t)
            acc[a][t] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Loads never post-process what they fetch (that would wait for the data
    // right after issue): addresses are clamped into the operand, and the
    // masking of a tail step happens when the registers are stored to LDS.
    uint4 rb[BPT];
    auto load_b = [&](int s) {
        const int k0 = kbeg + s * kBK;
#pragma unroll
        for (int j = 0; j < BPT; ++j) {
            const int q = min(tid + 256 * j, BCH - 1);
            const int c = min(q >> 3, np - 1);
            const int gk = k0 + (q & 7) * 8;
            rb[j] = *reinterpret_cast<const uint4 *>(Bt + static_cast<int64_t>(c) * ldbt + (gk < kend ? gk : kbeg));
        }
    };
    auto store_b = [&](int buf, int s) {
        const int k0 = kbeg + s * kBK;
        const bool full = k0 + kBK <= kend;
#pragma unroll
        for (int j = 0; j < BPT; ++j) {
            const int q = tid + 256 * j;
            if (q < BCH) {
                uint4 v = rb[j];
                if (!full)
                    v = keep_first(v, kend - (k0 + (q & 7) * 8));
                if (q >= bch_live)
                    v = make_uint4(0u, 0u, 0u, 0u);
                *reinterpret_cast<uint4 *>(&Bs[buf][(q >> 3) * kBPitch + (q & 7) * 8]) = v;
            }
        }
    };
    // One step of this wave's A: eight 16-byte chunks per lane, chunk j at
    // line j * 8 + lane / 8 (a row of A, or a k-row of A^T), 16-byte column
    // (lane % 8): each 128-byte line is read by eight consecutive lanes.
    auto load_a = [&](uint4 (&ra)[8], int s) {
        const int k0 = kbeg + s * kBK;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int line = j * 8 + (lane >> 3);
            const int c8 = (lane & 7) * 8;
            if (!TRANS) {
                const int gi = wrow0 + line;
                const int gk = k0 + c8;
                if (VEC) {
                    // rows past M only feed outputs that are never stored
                    ra[j] = *reinterpret_cast<const uint4 *>(A + static_cast<int64_t>(min(gi, M - 1)) * lda +
                                                             (gk < kend ? gk : kbeg));
                } else {
                    uint4 v = make_uint4(0u, 0u, 0u, 0u);
                    if (gi < M)
                        v = load8_scalar(A + static_cast<int64_t>(gi) * lda + gk, kend - gk);
                    ra[j] = v;
                }
            } else {
                const int gk = k0 + line;
                const int gi = wrow0 + c8;
                if (VEC) {
                    // k-rows past kend meet zero rows of the thin factor;
                    // columns past M only feed outputs that are never stored
                    ra[j] = *reinterpret_cast<const uint4 *>(A + static_cast<int64_t>(min(gk, kend - 1)) * lda +
                                                             min(gi, (M - 1) & ~7));
                } else {
                    uint4 v = make_uint4(0u, 0u, 0u, 0u);
                    if (gk < kend)
                        v = load8_scalar(A + static_cast<int64_t>(gk) * lda + gi, M - gi);
                    ra[j] = v;
                }
            }
        }
    };
    auto store_a = [&](const uint4 (&ra)[8], int buf, int s) {
        const int k0 = kbeg + s * kBK;
        const bool full = k0 + kBK <= kend;
        uint16_t *w = &As[buf][wave * AW];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int line = j * 8 + (lane >> 3);
            const int c8 = (lane & 7) * 8;
            if (!TRANS) {
                uint4 v = ra[j];
                if (VEC && !full)   // the padding past K may hold anything
                    v = keep_first(v, kend - (k0 + c8));
                *reinterpret_cast<uint4 *>(&w[line * kBPitch + c8]) = v;
            } else {
                // 33-dword rows: 4-byte stores
                uint32_t *dst = reinterpret_cast<uint32_t *>(&w[line * kTPitch + c8]);
                dst[0] = ra[j].x;
                dst[1] = ra[j].y;
                dst[2] = ra[j].z;
                dst[3] = ra[j].w;
            }
        }
    };
    auto compute = [&](int buf) {
        const uint16_t *w = &As[buf][wave * AW];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            bf16x8 af[4];
#pragma unroll
            for (int a = 0; a < 4; ++a) {
                if (!TRANS) {
                    af[a] = *reinterpret_cast<const bf16x8 *>(
                        &w[(a * 16 + (lane & 15)) * kBPitch + ks * 32 + (lane >> 4) * 8]);
                } else {
                    const uint16_t *col = &w[(ks * 32 + (lane >> 4) * 8) * kTPitch + a * 16 + (lane & 15)];
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        af[a][e] = static_cast<short>(col[e * kTPitch]);
                }
            }
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const bf16x8 b = *reinterpret_cast<const bf16x8 *>(
                    &Bs[buf][(t * 16 + (lane & 15)) * kBPitch + ks * 32 + (lane >> 4) * 8]);
#pragma unroll
                for (int a = 0; a < 4; ++a)
                    acc[a][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[a], b, acc[a][t], 0, 0, 0);
            }
        }
    };

    // Pipeline, step s: stage A(s + 1) and B(s + 1) from registers into the
    // other LDS buffers; issue B(s + 2), then A(s + 3) (two steps of A stay in
    // flight); multiply step s; barrier.  Every step issues the same loads
    // (step indices past the end are clamped to the last step, which is
    // still in L2), so the wait counts stay the same around the loop.
    if (nsteps > 0) {
        const int last = nsteps - 1;
        uint4 r0[8], r1[8];
        load_b(0);
        load_a(r0, 0);
        load_a(r1, min(1, last));
        store_b(0, 0);
        store_a(r0, 0, 0);
        load_b(min(1, last));
        load_a(r0, min(2, last));
        lds_barrier();
        auto step = [&](int s, uint4 (&nxt)[8]) {
            store_a(nxt, (s + 1) & 1, s + 1);
            store_b((s + 1) & 1, s + 1);
            load_b(min(s + 2, last));
            load_a(nxt, min(s + 3, last));
            compute(s & 1);
            lds_barrier();
        };
        int s = 0;
        for (; s + 2 <= nsteps; s += 2) {
            step(s, r1);
            step(s + 1, r0);
        }
        if (s < nsteps)
            step(s, r1);
    }

    float *Cs = J.C + static_cast<int64_t>(split) * J.split_stride;
    const int64_t ldc = J.ldc;
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int col = t * 16 + (lane & 15);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int row = wrow0 + a * 16 + (lane >> 4) * 4 + e;
                if (row < M && col < np)
                    Cs[static_cast<int64_t>(row) * ldc + col] = acc[a][t][e];
            }
        }
}

// ---------------------------------------------------------------------------
// Streaming pass with the loads going straight from HBM into LDS
// (global_load_lds_dwordx4: lane L's 16 bytes land at the wave-uniform LDS
// address in M0 plus 16 L).  An LDS ring of S stages holds, per step, the
// workgroup's 256 lines of A (a row of A, or a k-row of A^T: 128 bytes each)
// and the NP lines of the thin factor (128 bytes of k each).  Each line's
// eight 16-byte chunks are stored XOR-swizzled (slot = chunk ^ swz(line)) so
// that fragment reads from consecutive lines hit distinct banks: with
// swz = ((line >> 1) ^ line) & 7 neither the 16-byte reads of 16 lines nor
// the transposed 8-byte reads of four lines conflict (measured with the
// bank-conflict counter on MI355X; (line & 7) ^ ((line & 8) >> 1) cost four
// conflict cycles per 16-byte read).  No
// register staging: registers hold only the accumulators, and S - 1 steps of
// the stream are in flight while one is multiplied.  Used for 16-byte
// aligned operands (VEC); waits on the DMA counters are explicit.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int swz(int line) { return ((line >> 1) ^ line) & 7; }

// global_load_lds_dwordx4 takes its wave-uniform LDS address in M0.  The asm
// saves M0 in a scratch SGPR and restores it, so M0 holds, after the
// statement, whatever the compiler may have kept there; an LDS DMA needs one
// wait state after a scalar write of M0 (the GFX9-family hazard), hence the
// s_nop after each write (the compiler's hazard tracking does not see inside
// the statement).  (The compiler's own builtin for this instruction counts
// it in its LDS wait model and then waits for all fragment reads before the
// first MFMA of a step; kept opaque here, the explicit vmcnt waits of the
// kernel order the DMA.)  The LDS address is wave-uniform at every call;
// readfirstlane hands it to the statement in an SGPR.
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
                 : "v"(gptr), "s"(__builtin_amdgcn_readfirstlane(lds_addr))
                 : "memory");
}
// The same DMA with the non-temporal hint, for the streamed operand A: each
// line of it is read once per pass, so it is not kept in L2 at the expense of
// the thin factor, which every workgroup of an XCD re-reads.
__device__ __forceinline__ void dma16_nt(const void *gptr, uint32_t lds_addr)
{
    uint32_t saved;
    asm volatile("s_mov_b32 %0, m0\n\t"
                 "s_mov_b32 m0, %2\n\t"
                 "s_nop 0\n\t"
                 "global_load_lds_dwordx4 %1, off nt\n\t"
                 "s_mov_b32 m0, %0\n\t"
                 "s_nop 0"
                 : "=&s"(saved)
                 : "v"(gptr), "s"(__builtin_amdgcn_readfirstlane(lds_addr))
                 : "memory");
}

template <int N>
__device__ __forceinline__ void wait_dma()
{
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

__device__ __forceinline__ void sync_lds()
{
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// A run of workgroups over one job: row blocks rb0 .. rb0 + nrb - 1, each cut
// into `pieces` k ranges of kchunk (piece p of row block b is workgroup
// wg0 + (b - rb0) * pieces + p).  A single piece writes C; several write
// partials, which pass_reduce_kernel adds in piece order.
struct Seg {
    int job, wg0, rb0, nrb, pieces, kchunk;
};
struct DJob {
    const uint16_t *A;
    int64_t lda;
    const uint16_t *Bt;
    int64_t ldbt;
    float *C;
    int64_t ldc;
    float *part;      // partial of piece p at part + p * ss, row stride np
    int64_t ss;
    int M, K;
    int ntc;          // > 0: A is a tiled shadow (ntc tiles per tile row)
};
struct SegBatch {
    int njobs, nseg;
    DJob j[kMaxJobs];
    Seg s[2 * kMaxJobs];
};

// Eight waves, two per SIMD, one workgroup per CU (the LDS ring takes most of
// the 160 KiB).  The stage's 256 lines of A form four 64-line groups; wave w
// stages half (w / 4) of group (w % 4), 32 lines, and multiplies the 32
// output rows of that half against all NP columns.  For opA = A those are
// the lines it staged itself; for opA = A^T it also reads the other half's
// k-lines, so the per-step barrier (needed anyway for the shared thin
// factor) orders both.  With two waves per SIMD one wave's MFMAs overlap the
// other's waits, which one wave per SIMD could not do.  The 2 NT DMA
// instructions of the thin factor go round the eight waves.
//
// The product runs on v_mfma_f32_16x16x32_bf16 over exactly NP = 16 NT
// columns.  These passes run at a third of the MFMA peak, and with real data
// the MFMA's power draw, not HBM, sets their pace: covering 144 columns with
// 16-wide tiles (rather than padding to 160 for 32x32 tiles) takes 8% less
// time, and needs fewer fragment reads than 32x32 tiles plus a 16-wide one.
template <bool TRANS, int NT, int S>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2))) void pass_dma_kernel(const SegBatch sb,
                                                                                                  int np)
{
    const int wg = static_cast<int>(blockIdx.x);
    int si = 0;
    while (si + 1 < sb.nseg && wg >= sb.s[si + 1].wg0)
        ++si;
    const Seg &G = sb.s[si];
    const int rel = wg - G.wg0;
    if (rel >= G.nrb * G.pieces)
        return;   // padding between segments
    const DJob &J = sb.j[G.job];
    constexpr int NP = NT * 16;
    constexpr int A_BYTES = 256 * 128;
    constexpr int STAGE = A_BYTES + NP * 128;
    constexpr int BN = 2 * NT;                    // thin-factor DMA instructions per step
    constexpr int BI_LO = BN / 8, BI_HI = (BN + 7) / 8;
    constexpr int PER_A = 4;                      // A DMA instructions per wave and step
    static_assert(S >= 2 && (PER_A + BI_HI) * (S - 2) < 64, "vmcnt range");
    __shared__ __attribute__((aligned(1024))) unsigned char smem[S * STAGE];

    const uint16_t *__restrict__ A = J.A;
    const uint16_t *__restrict__ Bt = J.Bt;
    const int64_t lda = J.lda, ldbt = J.ldbt;
    const int M = J.M;
    const int piece = rel % G.pieces;
    const int row0 = (G.rb0 + rel / G.pieces) * kBM;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int grp = wave & 3, half = wave >> 2;
    const bool b_hi = wave < BN % 8;             // this wave issues BI_HI thin-factor instructions, else BI_LO
    const int grow0 = row0 + grp * 64;     // first line of this wave's group (a row of A, or a column of A^T)
    const int kbeg = piece * G.kchunk;
    const int kend = min(J.K, kbeg + G.kchunk);
    const int nsteps = kend > kbeg ? static_cast<int>(cdiv(kend - kbeg, kBK)) : 0;
    const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_byte *)smem));

    f32x4 acc[2][NT];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int t = 0; t < NT; ++t)
            acc[a][t] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Issue one step's DMA into stage `st`: this wave's 32 lines of A (4
    // instructions), and instructions w, w + 8, ... of the 2 NT of the thin
    // factor.  Addresses are clamped into the operands: rows past M feed
    // outputs that are never stored, thin-factor rows past np feed columns
    // that are never stored, k past kend is zeroed in LDS before the tail
    // step is used.
    auto issue = [&](int s, int st) {
        const int k0 = kbeg + s * kBK;
        const uint32_t sbase = lds0 + st * STAGE;
        const int sub = lane >> 3;            // line within the instruction
#pragma unroll
        for (int jj = 0; jj < PER_A; ++jj) {
            const int j = half * PER_A + jj;
            const int line = j * 8 + sub;     // line within the group's 64
            const int c = (lane & 7) ^ swz(line);
            const uint16_t *src;
            if (J.ntc > 0) {
                // tiled shadow: this wave's 64 lines are one tile (opA = A: rows
                // grow0.., k0..k0+63) or one tile's k-rows (opA = A^T: k-rows
                // k0.., columns grow0..grow0+63).  Row blocks past M re-read the
                // last tile row (outputs never stored); k-rows past kend are
                // clamped to kend - 1, so the zero rows of the thin factor never
                // meet the tile's unwritten padding.
                const int tg = min(grow0 >> 6, (M - 1) >> 6);
                if (!TRANS)
                    src = A + (static_cast<int64_t>(tg) * J.ntc + (k0 >> 6)) * 4096 + line * 64 + c * 8;
                else
                    src = A + (static_cast<int64_t>(k0 >> 6) * J.ntc + tg) * 4096 + min(line, kend - 1 - k0) * 64 +
                          c * 8;
            } else if (!TRANS) {
                const int gk = k0 + c * 8;
                src = A + static_cast<int64_t>(min(grow0 + line, M - 1)) * lda + (gk < kend ? gk : kbeg);
            } else {
                src = A + static_cast<int64_t>(min(k0 + line, kend - 1)) * lda + min(grow0 + c * 8, (M - 1) & ~7);
            }
            dma16_nt(src, sbase + grp * 8192 + j * 1024);
        }
#pragma unroll
        for (int b = 0; b < BI_HI; ++b) {
            if (b < BI_LO || b_hi) {
                const int m = b * 8 + wave;   // instruction index within the thin-factor tile
                const int line = m * 8 + sub;
                const int c = (lane & 7) ^ swz(line);
                const int gk = k0 + c * 8;
                const uint16_t *src = Bt + static_cast<int64_t>(min(line, np - 1)) * ldbt + (gk < kend ? gk : kbeg);
                dma16(src, sbase + A_BYTES + m * 1024);
            }
        }
    };
    // Tail step: zero k >= kend in the thin factor (and in A when k runs
    // along A's rows, whose padding may hold anything).
    auto fix_tail = [&](int st, int k0) {
        unsigned char *base = smem + st * STAGE;
        const int kk = kend - k0;
        const int nlines = (TRANS ? 0 : 256) + NP;
        for (int q = tid; q < nlines * 8; q += 512) {
            const int l = q >> 3, c = q & 7;
            if (c * 8 + 8 <= kk)
                continue;
            unsigned char *line = !TRANS && l < 256 ? base + l * 128 : base + A_BYTES + (l - (TRANS ? 0 : 256)) * 128;
            const int lidx = !TRANS && l < 256 ? (l & 63) : (l - (TRANS ? 0 : 256));
            uint4 *slot = reinterpret_cast<uint4 *>(line + 16 * (c ^ swz(lidx)));
            *slot = keep_first(*slot, kk - c * 8);
        }
    };
    // v_mfma_f32_16x16x32_bf16: A[i][k] / B[k][j] in lane i (j) + 16 (k / 8),
    // element k % 8.  The wave's 32 rows are two 16-row tiles, the NP columns
    // NT 16-wide tiles; a 64-deep step is two 32-deep halves.
    auto frags = [&](const unsigned char *aw, const unsigned char *bw, int kh, bf16x8 (&af)[2], bf16x8 (&bf)[NT]) {
        const int c = kh * 4 + (lane >> 4);   // 16-byte chunk: k = 8 c .. 8 c + 7 of the step
#pragma unroll
        for (int a = 0; a < 2; ++a) {
            if (!TRANS) {
                const int line = half * 32 + a * 16 + (lane & 15);
                af[a] = *reinterpret_cast<const bf16x8 *>(aw + line * 128 + 16 * (c ^ swz(line)));
            } else {
                // ds_read_b64_tr_b16: in each group of 16 lanes, result lane
                // L, element e = element L % 4 of what lane 4 e + L / 4 read.
                // Source lane 4 e + q of group g reads columns 4 q .. 4 q + 3
                // (of the tile's 16) from k-line 8 g + e, so lane L receives
                // column L of four consecutive k-lines; two reads give the
                // eight k of a fragment.
                const int l16 = lane & 15;
                const int col = half * 32 + a * 16 + (l16 & 3) * 4;
                const int line0 = kh * 32 + (lane >> 4) * 8 + (l16 >> 2);
                v4i16 h0, h1;
                {
                    const int line = line0;
                    h0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(reinterpret_cast<lds_v4i16 *>(
                        (lds_byte *)(aw + line * 128 + 16 * ((col >> 3) ^ swz(line)) + (col & 7) * 2)));
                }
                {
                    const int line = line0 + 4;
                    h1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(reinterpret_cast<lds_v4i16 *>(
                        (lds_byte *)(aw + line * 128 + 16 * ((col >> 3) ^ swz(line)) + (col & 7) * 2)));
                }
                af[a] = bf16x8{h0[0], h0[1], h0[2], h0[3], h1[0], h1[1], h1[2], h1[3]};
            }
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int line = t * 16 + (lane & 15);
            bf[t] = *reinterpret_cast<const bf16x8 *>(bw + line * 128 + 16 * (c ^ swz(line)));
        }
    };
    auto compute = [&](int st) {
        const unsigned char *base = smem + st * STAGE;
        const unsigned char *aw = base + grp * 8192;
        const unsigned char *bw = base + A_BYTES;
        bf16x8 af[2][2], bf[2][NT];
        frags(aw, bw, 0, af[0], bf[0]);
        frags(aw, bw, 1, af[1], bf[1]);
#pragma unroll
        for (int kh = 0; kh < 2; ++kh)
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
                for (int a = 0; a < 2; ++a)
                    acc[a][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[kh][a], bf[kh][t], acc[a][t], 0, 0, 0);
        // the second half's fragment reads go out under the first half's MFMAs
        constexpr int DS = (TRANS ? 4 : 2) + NT;
        __builtin_amdgcn_sched_group_barrier(0x100, DS, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, DS, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 2 * NT, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 2 * NT, 0);
    };

    if (nsteps > 0) {
        const int last = nsteps - 1;
#pragma unroll
        for (int p = 0; p < S - 1; ++p)
            issue(min(p, last), p);
        int st = 0;   // stage of step s
        for (int s = 0; s < nsteps; ++s) {
            // this wave's DMA for step s has landed
            if (b_hi)
                wait_dma<(PER_A + BI_HI) * (S - 2)>();
            else
                wait_dma<(PER_A + BI_LO) * (S - 2)>();
            sync_lds();                        // everyone's has; stage (s - 1) % S is free
            const int k0 = kbeg + s * kBK;
            if (k0 + kBK > kend) {
                fix_tail(st, k0);
                sync_lds();
            }
            int nst = st + S - 1;
            if (nst >= S)
                nst -= S;
            __builtin_amdgcn_s_setprio(1);   // the DMA leaves ahead of other waves' products
            issue(min(s + S - 1, last), nst);
            __builtin_amdgcn_s_setprio(0);
            compute(st);
            if (++st == S)
                st = 0;
        }
        wait_dma<0>();
    }

    // D[i][j] of a 16 x 16 tile: lane j + 16 (i / 4), element i % 4
    float *Cs = G.pieces > 1 ? J.part + static_cast<int64_t>(piece) * J.ss : J.C;
    const int64_t ldo = G.pieces > 1 ? static_cast<int64_t>(np) : J.ldc;
    const int wrow0 = grow0 + half * 32;
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int col = t * 16 + (lane & 15);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int row = wrow0 + a * 16 + 4 * (lane >> 4) + e;
                if (row < M && col < np)
                    Cs[static_cast<int64_t>(row) * ldo + col] = acc[a][t][e];
            }
        }
}

// C[i, c] = sum over splits of part[s][i, c] (NP columns, float4 when aligned).
struct RedJob {
    const float *part;
    int64_t split_stride;
    float *C;
    int64_t ldc;
    int M, NP, splits;
};
struct RedBatch {
    int count;
    RedJob j[kMaxJobs];
};

__global__ __launch_bounds__(256) void pass_reduce_kernel(const RedBatch jb)
{
    const RedJob &J = jb.j[blockIdx.z];
    const int64_t n4 = static_cast<int64_t>(J.M) * (J.NP / 4);
    const int q4 = J.NP / 4;
    for (int64_t idx = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; idx < n4;
         idx += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t i = idx / q4;
        const int c = static_cast<int>(idx % q4) * 4;
        float4 s = *reinterpret_cast<const float4 *>(J.part + i * J.NP + c);
        for (int p = 1; p < J.splits; ++p) {
            const float4 v = *reinterpret_cast<const float4 *>(J.part + p * J.split_stride + i * J.NP + c);
            s.x += v.x;
            s.y += v.y;
            s.z += v.z;
            s.w += v.w;
        }
        *reinterpret_cast<float4 *>(J.C + i * J.ldc + c) = s;
    }
}

// Element-load passes (operands that are not 16-byte aligned): one z slice
// of the grid per job.
template <bool TRANS>
void launch_scalar(const char *tag, const std::vector<Job> &jobs, int gx, int np, hipStream_t st)
{
    for (size_t c0 = 0; c0 < jobs.size(); c0 += kMaxJobs) {
        Batch b{};
        b.count = static_cast<int>(std::min<size_t>(kMaxJobs, jobs.size() - c0));
        for (int i = 0; i < b.count; ++i)
            b.j[i] = jobs[c0 + i];
        auto kern = pass_kernel<TRANS, kMaxNT, false>;
        ACSC_LAUNCH(tag, kern, dim3(gx, 1, b.count), dim3(256), 0, st, b, np);
    }
}

template <bool TRANS, int NTK>
void launch_segs(const char *tag, const SegBatch &b, int grid, int np, hipStream_t st)
{
    // three LDS stages while they fit in 160 KiB, else two
    constexpr int S = (3 * (256 * 128 + NTK * 16 * 128) <= 160 * 1024) ? 3 : 2;
    auto kern = pass_dma_kernel<TRANS, NTK, S>;
    ACSC_LAUNCH(tag, kern, dim3(grid), dim3(512), 0, st, b, np);
}

template <bool TRANS>
void launch_dma(const char *tag, const SegBatch &b, int grid, int np, hipStream_t st)
{
    switch (np / 16) {
    case 1: launch_segs<TRANS, 1>(tag, b, grid, np, st); break;
    case 2: launch_segs<TRANS, 2>(tag, b, grid, np, st); break;
    case 3: launch_segs<TRANS, 3>(tag, b, grid, np, st); break;
    case 4: launch_segs<TRANS, 4>(tag, b, grid, np, st); break;
    case 5: launch_segs<TRANS, 5>(tag, b, grid, np, st); break;
    case 6: launch_segs<TRANS, 6>(tag, b, grid, np, st); break;
    case 7: launch_segs<TRANS, 7>(tag, b, grid, np, st); break;
    case 8: launch_segs<TRANS, 8>(tag, b, grid, np, st); break;
    case 9: launch_segs<TRANS, 9>(tag, b, grid, np, st); break;
    case 10: launch_segs<TRANS, 10>(tag, b, grid, np, st); break;
    case 11: launch_segs<TRANS, 11>(tag, b, grid, np, st); break;
    default: launch_segs<TRANS, 12>(tag, b, grid, np, st); break;
    }
}

// ---------------------------------------------------------------------------
// Workgroup order of the DMA passes.  Workgroups go to the XCDs in turn
// (workgroup i to XCD i % X) and, within an XCD, to whichever CU frees up
// first; one pass workgroup fills a CU.  A batch that mixes long and short
// rows (the 70B-class build: 128 row blocks of 448 steps, 576 of 128) then
// ends with a round in which only some CUs work.  The plan below simulates
// that dispatch and, where it shortens the simulated makespan, moves the
// last-dispatched row blocks to the end of the grid as two k halves each
// (partials added by pass_reduce_kernel): for the 70B-class batch, 64 short
// row blocks halved make the long blocks' CUs finish with the others.
// ---------------------------------------------------------------------------
struct JobShape {
    int nrb, splits, kchunk, K;
    bool halvable;
};

struct SegPlan {
    std::vector<Seg> segs;
    std::vector<int> halved;   // per job: trailing row blocks cut in two k halves
    int grid = 0;
    int64_t makespan = 0;
};

int64_t simulate_dispatch(const std::vector<int> &cost, int xcds, int cus_per_xcd)
{
    std::vector<std::vector<int64_t>> free_at(static_cast<size_t>(xcds),
                                              std::vector<int64_t>(static_cast<size_t>(cus_per_xcd), 0));
    int64_t end = 0;
    for (size_t i = 0; i < cost.size(); ++i) {
        if (cost[i] == 0)
            continue;
        std::vector<int64_t> &h = free_at[i % static_cast<size_t>(xcds)];
        std::pop_heap(h.begin(), h.end(), std::greater<int64_t>());
        h.back() += cost[i];
        end = std::max(end, h.back());
        std::push_heap(h.begin(), h.end(), std::greater<int64_t>());
    }
    return end;
}

SegPlan layout(const std::vector<JobShape> &js, const std::vector<int> &halved, int xcds, int cus_per_xcd)
{
    SegPlan p;
    p.halved = halved;
    std::vector<int> cost;
    auto add = [&](int job, int rb0, int nrb, int pieces, int kc) {
        if (nrb <= 0)
            return;
        const int wg0 = static_cast<int>(round_up(static_cast<int64_t>(cost.size()), 8));
        cost.resize(static_cast<size_t>(wg0), 0);
        p.segs.push_back(Seg{job, wg0, rb0, nrb, pieces, kc});
        for (int b = 0; b < nrb; ++b)
            for (int pc = 0; pc < pieces; ++pc) {
                const int64_t kb = static_cast<int64_t>(pc) * kc;
                const int64_t ke = std::min<int64_t>(js[job].K, kb + kc);
                cost.push_back(ke > kb ? static_cast<int>(cdiv(ke - kb, kBK)) : 0);
            }
    };
    for (size_t j = 0; j < js.size(); ++j)
        add(static_cast<int>(j), 0, js[j].nrb - halved[j], js[j].splits, js[j].kchunk);
    for (size_t j = 0; j < js.size(); ++j)
        if (halved[j] > 0)
            add(static_cast<int>(j), js[j].nrb - halved[j], halved[j], 2,
                static_cast<int>(round_up(cdiv(js[j].K, 2), kBK)));
    p.grid = static_cast<int>(cost.size());
    p.makespan = simulate_dispatch(cost, xcds, cus_per_xcd);
    return p;
}

void device_cus(int &xcds, int &cus_per_xcd)
{
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
        cus = 256;
    xcds = std::max(1, cus / 32);   // 32 CUs per XCD on gfx950 (one XCD per partition in CPX mode)
    cus_per_xcd = std::max(1, cus / xcds);
}

// The plan depends only on the batch's shapes and the device, so it is made
// once per distinct batch and kept.
SegPlan plan(const std::vector<JobShape> &js)
{
    int xcds = 8, cpx = 32;
    device_cus(xcds, cpx);
    std::vector<int64_t> key{xcds, cpx};
    for (const JobShape &j : js)
        key.insert(key.end(), {j.nrb, j.splits, j.kchunk, j.K, j.halvable ? 1 : 0});
    static std::mutex mu;
    static std::map<std::vector<int64_t>, SegPlan> cache;
    {
        std::lock_guard<std::mutex> g(mu);
        auto it = cache.find(key);
        if (it != cache.end())
            return it->second;
    }
    std::vector<int> halved(js.size(), 0);
    SegPlan best = layout(js, halved, xcds, cpx);
    bool whole = true;
    int64_t wgs = 0;
    for (const JobShape &j : js) {
        whole = whole && j.splits == 1;
        wgs += static_cast<int64_t>(j.nrb) * j.splits;
    }
    if (whole && wgs >= static_cast<int64_t>(xcds) * cpx) {
        // trailing row blocks (in dispatch order) that may be halved
        int hmax = 0;
        for (size_t j = js.size(); j-- > 0 && js[j].halvable;)
            hmax += js[j].nrb;
        hmax = std::min(hmax, 2 * xcds * cpx);
        for (int h = 8; h <= hmax; h += 8) {
            std::vector<int> hv(js.size(), 0);
            int rest = h;
            for (size_t j = js.size(); j-- > 0 && rest > 0;) {
                hv[j] = std::min(rest, js[j].nrb);
                rest -= hv[j];
            }
            SegPlan p = layout(js, hv, xcds, cpx);
            if (p.makespan < best.makespan)
                best = p;
        }
    }
    std::lock_guard<std::mutex> g(mu);
    cache.emplace(key, best);
    return best;
}

// ---------------------------------------------------------------------------
// Anchor EMA fused with the first pass (see sc_pass.h).  A workgroup of 512
// threads owns 256 rows; per 64-deep step each thread takes eight 4-element pieces of M
// (16-byte loads, 16 lanes per row) and of G, forms the EMA, stores M
// (non-temporal) and the bf16 shadow, and drops the bf16 piece into the
// swizzled LDS layout of the streaming pass, where the step is multiplied on
// 16x16x32 MFMA.  All loads go through registers (the next step's are
// issued before this step's product), so the compiler's own wait counts are
// exact.
// ---------------------------------------------------------------------------
struct EmaJob {
    float *M;
    const uint16_t *G;
    uint16_t *M16;
    const uint16_t *Bt;
    int64_t ldbt;
    float *C;
    int64_t ldc;
    int m, n;
    float *part;      // pieces of a halved row block: partial p at part + p * ss, row stride np
    int64_t ss;
    int ntc;          // tiles per tile row of the shadow
    int *stall;       // EmaReq::stall
};
// Workgroups in the order of the streaming passes' dispatch plan (Seg runs
// over the jobs; see plan()), so that a batch that mixes long and short rows
// ends with every CU busy: whole rows, only the last-dispatched row blocks
// cut into two k halves.
struct EmaBatch {
    int njobs, nseg;
    EmaJob j[kMaxJobs];
    Seg s[2 * kMaxJobs];
};

// Workgroup-scope counters in LDS: a wave adds one when its part of a stage
// is written (or its reads of it are done); waiting waves poll.  Release and
// acquire order the stage's LDS accesses around the counters.
__device__ __forceinline__ void stage_signal(unsigned int *c, int lane)
{
    if (lane == 0)
        __hip_atomic_fetch_add(c, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
}
// Every wave of the workgroup reaches each of its signals, so a wait ends
// within a few steps' time; the poll count is bounded (about a second)
// so that a fault elsewhere cannot turn into a hung GPU.
// True once the counter has reached target; false if it had not after
// `spin` polls (the caller reports it: the stage's data may be stale).
__device__ __forceinline__ bool stage_wait(unsigned int *c, unsigned int target, int spin)
{
    if (__hip_atomic_load(c, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) >= target)
        return true;
    for (int i = 0; i < spin; ++i) {
        __builtin_amdgcn_s_sleep(1);
        if (__hip_atomic_load(c, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) >= target)
            return true;
    }
    return false;
}

// Eight waves per workgroup, two per SIMD (four waves left the stream with
// too few loads in flight).  Wave w loads, updates and multiplies rows
// 32 w .. 32 w + 31 of the block, staging their bf16 copy in an LDS region of
// its own, so the rows need no synchronisation between waves.  The thin
// factor's step is shared: each wave stages an eighth of it into a ring of
// kEmaStages buffers, and counters per buffer (parts written, readers done)
// replace the workgroup barrier, so that a wave waits for the others only
// when it is kEmaStages - 1 steps ahead (a barrier per step held the waves
// in lockstep on the slowest one's HBM loads).  Every wave runs every step,
// so every counter reaches its target.
constexpr int kEmaStages = 3;

template <int NT>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2))) void ema_pass_kernel(const EmaBatch jb, int np,
                                                                                                 float beta, float omb,
                                                                                                 int spin)
{
    const int wg = static_cast<int>(blockIdx.x);
    int si = 0;
    while (si + 1 < jb.nseg && wg >= jb.s[si + 1].wg0)
        ++si;
    const Seg &SG = jb.s[si];
    const int rel = wg - SG.wg0;
    if (rel >= SG.nrb * SG.pieces)
        return;   // padding between segments
    const EmaJob &J = jb.j[SG.job];
    constexpr int NP = NT * 16;
    constexpr int W = 8;                        // waves
    constexpr int A_WAVE = 32 * 128;            // a wave's 32 rows of one step (bf16)
    constexpr int A_BYTES = W * 2 * A_WAVE;     // two buffers per wave
    constexpr int B_STAGE = NP * 128;
    constexpr int NB = kEmaStages;
    constexpr int BCH = NP * 8;                 // 16-byte chunks of one thin-factor step
    constexpr int CPW = (BCH + W - 1) / W;      // chunks staged per wave
    constexpr int BPL = (CPW + 63) / 64;        // chunks per lane
    constexpr int PU = 8;                       // 4-element pieces of M per lane and step
    __shared__ __attribute__((aligned(1024))) unsigned char smem[A_BYTES + NB * B_STAGE];
    __shared__ unsigned int ready[NB], done[NB];

    float *__restrict__ M = J.M;
    const uint16_t *__restrict__ G = J.G;
    uint16_t *__restrict__ M16 = J.M16;
    const uint16_t *__restrict__ Bt = J.Bt;
    const int64_t ldbt = J.ldbt;
    const int m = J.m, n = J.n;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // workgroup -> (row block, piece): the k range [kbeg, kend) of the rows
    const int piece = rel % SG.pieces;
    const int row0 = (SG.rb0 + rel / SG.pieces) * kBM;
    const int kbeg = piece * SG.kchunk;
    const int kend = min(n, kbeg + SG.kchunk);
    const int nsteps = static_cast<int>(cdiv(kend - kbeg, kBK));
    const int wrow0 = row0 + wave * 32;
    if (tid < NB) {
        ready[tid] = 0u;
        done[tid] = 0u;
    }
    __syncthreads();

    f32x4 acc[2][NT];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int t = 0; t < NT; ++t)
            acc[a][t] = f32x4{0.f, 0.f, 0.f, 0.f};

    // piece u of this lane: row 4 u + lane / 16 of the wave's 32, 4 elements at
    // column 4 (lane % 16) of the step, so that 16 lanes cover a row's 256
    // bytes of M (128 of G) with one instruction
    float4 rm[PU];
    uint2 rg[PU];
    uint4 rb[BPL];
    // the thin factor's part first, so that its wait leaves M and G in flight
    // Loads are unconditional, from addresses clamped into the operands
    // (k past the end reads the piece's first step, rows past m the last
    // row; without a new gradient G is read from M's bytes), and what lies
    // outside is zeroed or skipped when the registers are used: the wait
    // for the thin factor's loads then counts exactly the M and G loads
    // issued after them and leaves those in flight.
    const uint16_t *__restrict__ Gs = G ? G : reinterpret_cast<const uint16_t *>(M);
    auto load_b = [&](int s) {
        const int k0 = kbeg + s * kBK;
#pragma unroll
        for (int j = 0; j < BPL; ++j) {
            const int q = min(wave * CPW + lane + 64 * j, BCH - 1);
            const int c = min(q >> 3, np - 1);
            const int gk = k0 + (q & 7) * 8;
            rb[j] = *reinterpret_cast<const uint4 *>(Bt + static_cast<int64_t>(c) * ldbt + (gk < kend ? gk : kbeg));
        }
    };
    auto load_mg = [&](int s) {
        const int k0 = kbeg + s * kBK;
#pragma unroll
        for (int u = 0; u < PU; ++u) {
            const int gi = min(wrow0 + 4 * u + (lane >> 4), m - 1), gk = k0 + (lane & 15) * 4;
            const int64_t o = static_cast<int64_t>(gi) * n + (gk < kend ? gk : kbeg);
            const f32x4 a = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(M + o));
            rm[u] = make_float4(a[0], a[1], a[2], a[3]);
            const unsigned long long gg = __builtin_nontemporal_load(reinterpret_cast<const unsigned long long *>(Gs + o));
            rg[u] = make_uint2(static_cast<uint32_t>(gg), static_cast<uint32_t>(gg >> 32));
        }
    };
    auto store_b = [&](int s) {
        const int k0 = kbeg + s * kBK;
        unsigned char *bw = smem + A_BYTES + (s % NB) * B_STAGE;
#pragma unroll
        for (int j = 0; j < BPL; ++j) {
            const int qi = lane + 64 * j;
            const int q = wave * CPW + qi;
            if (qi < CPW && q < BCH) {
                const int line = q >> 3, c = q & 7;
                uint4 v = rb[j];
                if (line >= np || k0 + c * 8 >= kend)
                    v = make_uint4(0u, 0u, 0u, 0u);
                *reinterpret_cast<uint4 *>(bw + line * 128 + 16 * (c ^ swz(line))) = v;
            }
        }
    };
    auto store_mg = [&](int s) {
        const int k0 = kbeg + s * kBK;
        unsigned char *aw = smem + (wave * 2 + (s & 1)) * A_WAVE;
#pragma unroll
        for (int u = 0; u < PU; ++u) {
            const int row = 4 * u + (lane >> 4), f = lane & 15;
            const int gi = wrow0 + row, gk = k0 + f * 4;
            float v[4] = {rm[u].x, rm[u].y, rm[u].z, rm[u].w};
            uint2 h = make_uint2(0u, 0u);
            if (gi < m && gk < kend) {
                const int64_t o = static_cast<int64_t>(gi) * n + gk;
                if (G) {
                    v[0] = ema_step(v[0], __uint_as_float(rg[u].x << 16), beta, omb);
                    v[1] = ema_step(v[1], __uint_as_float(rg[u].x & 0xFFFF0000u), beta, omb);
                    v[2] = ema_step(v[2], __uint_as_float(rg[u].y << 16), beta, omb);
                    v[3] = ema_step(v[3], __uint_as_float(rg[u].y & 0xFFFF0000u), beta, omb);
                    __builtin_nontemporal_store(f32x4{v[0], v[1], v[2], v[3]}, reinterpret_cast<f32x4 *>(M + o));
                }
                h.x = f32x2_to_bf16x2(v[0], v[1]);
                h.y = f32x2_to_bf16x2(v[2], v[3]);
                __builtin_nontemporal_store(static_cast<unsigned long long>(h.x) | (static_cast<unsigned long long>(h.y) << 32),
                                            reinterpret_cast<unsigned long long *>(M16 + (static_cast<int64_t>(gi >> 6) * J.ntc + (gk >> 6)) * 4096 +
                                                                                   (gi & 63) * 64 + (gk & 63)));
            }
            *reinterpret_cast<uint2 *>(aw + row * 128 + 16 * ((f >> 1) ^ swz(row)) + 8 * (f & 1)) = h;
        }
    };
    // v_mfma_f32_16x16x32_bf16 on the step in LDS, in the layout and order of
    // pass_dma_kernel<false> (the same products in the same order, so the
    // result equals the separate EMA and pass bit for bit); this wave's 32
    // rows are two 16-row tiles
    auto compute = [&](int s) {
        const unsigned char *aw = smem + (wave * 2 + (s & 1)) * A_WAVE;
        const unsigned char *bw = smem + A_BYTES + (s % NB) * B_STAGE;
        bf16x8 af[2][2], bf[2][NT];
#pragma unroll
        for (int kh = 0; kh < 2; ++kh) {
            const int c = kh * 4 + (lane >> 4);
#pragma unroll
            for (int a = 0; a < 2; ++a) {
                const int line = a * 16 + (lane & 15);
                af[kh][a] = *reinterpret_cast<const bf16x8 *>(aw + line * 128 + 16 * (c ^ swz(line)));
            }
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const int line = t * 16 + (lane & 15);
                bf[kh][t] = *reinterpret_cast<const bf16x8 *>(bw + line * 128 + 16 * (c ^ swz(line)));
            }
        }
#pragma unroll
        for (int kh = 0; kh < 2; ++kh)
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
                for (int a = 0; a < 2; ++a)
                    acc[a][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[kh][a], bf[kh][t], acc[a][t], 0, 0, 0);
    };
    // step s: its thin factor sits in buffer s % NB once ready[s % NB] has
    // reached W (s / NB + 1); the buffer may take step s + NB once done[s % NB]
    // has reached W (s / NB + 1)
    bool waited = true;   // every wait of this wave met its count
    auto put_b = [&](int s) {
        if (s >= NB)
            waited &= stage_wait(&done[s % NB], W * (s / NB), spin);
        store_b(s);
        stage_signal(&ready[s % NB], lane);
    };

    load_b(0);
    load_mg(0);
    put_b(0);
    store_mg(0);
    for (int s = 0; s < nsteps; ++s) {
        const bool more = s + 1 < nsteps;
        if (more) {
            // the next step's HBM loads leave at a raised wave priority, ahead
            // of the other wave of the SIMD's products
            __builtin_amdgcn_s_setprio(1);
            load_b(s + 1);
            load_mg(s + 1);
            __builtin_amdgcn_s_setprio(0);
            put_b(s + 1);
        }
        waited &= stage_wait(&ready[s % NB], W * (s / NB + 1), spin);
        compute(s);
        stage_signal(&done[s % NB], lane);
        if (more)
            store_mg(s + 1);
    }

    // D[i][j] of a 16 x 16 tile: lane j + 16 (i / 4), element i % 4;
    // a piece of a halved row block writes its partial (row stride np),
    // added up by pass_reduce_kernel
    if (!waited && lane == 0 && J.stall)
        __hip_atomic_store(J.stall, kEmaStallMark, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    float *Cout = SG.pieces > 1 ? J.part + piece * J.ss : J.C;
    const int64_t ldo = SG.pieces > 1 ? static_cast<int64_t>(np) : J.ldc;
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int col = t * 16 + (lane & 15);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int row = wrow0 + a * 16 + 4 * (lane >> 4) + e;
                if (row < m && col < np)
                    Cout[static_cast<int64_t>(row) * ldo + col] = acc[a][t][e];
            }
        }
}

template <int NT>
void ema_launch(const char *tag, const EmaBatch &b, int grid, int np, float a, float b_coef, int spin,
                hipStream_t st)
{
    ACSC_LAUNCH(tag, ema_pass_kernel<NT>, dim3(grid), dim3(512), 0, st, b, np, a, b_coef, spin);
}

}  // namespace

int max_splits(int64_t M, int64_t K)
{
    const int64_t mb = cdiv(M, kBM);
    int s = 1;
    while (s < 16 && mb * s < 256 && K / (2 * s) >= 512)
        s *= 2;
    return s;
}

int run(const char *tag, bool trans, const std::vector<Req> &reqs, hipStream_t st)
{
    if (reqs.empty())
        return ACSC_OK;
    const int NP = reqs[0].NP;
    if (NP < 16 || NP % 16 != 0 || NP > SC_KMAX)
        return set_error(ACSC_EINVAL, "pass with %d thin-factor columns (a multiple of 16 up to %d)", NP, SC_KMAX);
    for (const auto &q : reqs) {
        if (q.NP != NP)
            return set_error(ACSC_EINVAL, "pass: thin factors of one launch must have the same width");
        if (q.ntc > 0 && (!q.avec || q.ntc != tiles_per_row(trans ? q.M : q.K)))
            return set_error(ACSC_EINVAL, "pass: a tiled operand must be aligned and have ceil(columns / 64) tiles "
                                          "per tile row");
    }
    // Split K only as far as needed for one workgroup per CU over the batch.
    int64_t blocks = 0;
    for (const auto &q : reqs)
        blocks += cdiv(q.M, kBM);
    int want = 1;
    while (want < 16 && blocks * want < 256)
        want *= 2;
    // Longest K first: workgroups are dispatched in job order, so the long
    // row blocks start early and the short ones fill in behind them.
    std::vector<size_t> order(reqs.size());
    for (size_t i = 0; i < order.size(); ++i)
        order[i] = i;
    std::stable_sort(order.begin(), order.end(), [&](size_t a, size_t b) { return reqs[a].K > reqs[b].K; });
    std::vector<Job> sj;                 // element-load jobs
    std::vector<const Req *> vq;         // DMA jobs
    std::vector<int> vsplits, vchunk;
    std::vector<RedJob> red;
    int gx = 1;
    int64_t rtot = 1;
    for (size_t oi : order) {
        const Req &q = reqs[oi];
        int splits = std::min(want, max_splits(q.M, q.K));
        const int64_t chunk = round_up(cdiv(q.K, splits), kBK);
        splits = static_cast<int>(std::max<int64_t>(1, cdiv(q.K, chunk)));
        const int64_t ss = static_cast<int64_t>(q.M) * NP;
        if (splits > 1) {
            red.push_back(RedJob{q.part, ss, q.C, q.ldc, q.M, NP, splits});
            rtot = std::max<int64_t>(rtot, static_cast<int64_t>(q.M) * (NP / 4));
        }
        if (q.avec) {
            vq.push_back(&q);
            vsplits.push_back(splits);
            vchunk.push_back(static_cast<int>(chunk));
            continue;
        }
        const int nb = static_cast<int>(cdiv(q.M, kBM) * splits);
        gx = std::max(gx, nb);
        if (splits == 1)
            sj.push_back(Job{q.A, q.lda, q.Bt, q.ldbt, q.C, q.ldc, 0, q.M, q.K, static_cast<int>(chunk), 1, nb, 0});
        else
            sj.push_back(Job{q.A, q.lda, q.Bt, q.ldbt, q.part, NP, ss, q.M, q.K, static_cast<int>(chunk), splits, nb,
                             0});
    }
    gx = static_cast<int>(round_up(gx, 8));   // block -> XCD placement is the same for every job
    if (!sj.empty()) {
        if (trans)
            launch_scalar<true>(tag, sj, gx, NP, st);
        else
            launch_scalar<false>(tag, sj, gx, NP, st);
    }
    for (size_t c0 = 0; c0 < vq.size(); c0 += kMaxJobs) {
        const size_t cnt = std::min<size_t>(kMaxJobs, vq.size() - c0);
        std::vector<JobShape> js;
        SegBatch b{};
        b.njobs = static_cast<int>(cnt);
        for (size_t i = 0; i < cnt; ++i) {
            const Req &q = *vq[c0 + i];
            b.j[i] = DJob{q.A, q.lda, q.Bt, q.ldbt, q.C, q.ldc, q.part, static_cast<int64_t>(q.M) * NP, q.M, q.K, q.ntc};
            js.push_back(JobShape{static_cast<int>(cdiv(q.M, kBM)), vsplits[c0 + i], vchunk[c0 + i], q.K,
                                  q.part != nullptr && max_splits(q.M, q.K) >= 2 && q.K >= 2 * kBK});
        }
        const SegPlan pl = plan(js);
        b.nseg = static_cast<int>(pl.segs.size());
        for (size_t i = 0; i < pl.segs.size(); ++i)
            b.s[i] = pl.segs[i];
        if (trans)
            launch_dma<true>(tag, b, pl.grid, NP, st);
        else
            launch_dma<false>(tag, b, pl.grid, NP, st);
        for (size_t i = 0; i < cnt; ++i) {
            const int h = pl.halved[i];
            if (h <= 0)
                continue;
            const Req &q = *vq[c0 + i];
            const int64_t r0 = static_cast<int64_t>(js[i].nrb - h) * kBM;
            red.push_back(RedJob{q.part + r0 * NP, static_cast<int64_t>(q.M) * NP, q.C + r0 * q.ldc, q.ldc,
                                 static_cast<int>(q.M - r0), NP, 2});
            rtot = std::max<int64_t>(rtot, (q.M - r0) * (NP / 4));
        }
    }
    for (size_t c0 = 0; c0 < red.size(); c0 += kMaxJobs) {
        RedBatch b{};
        b.count = static_cast<int>(std::min<size_t>(kMaxJobs, red.size() - c0));
        for (int i = 0; i < b.count; ++i)
            b.j[i] = red[c0 + i];
        const unsigned g = static_cast<unsigned>(std::min<int64_t>(cdiv(rtot, 256), 8192));
        ACSC_LAUNCH("sc_split_reduce", pass_reduce_kernel, dim3(g, 1, b.count), dim3(256), 0, st, b);
    }
    return ACSC_OK;
}

bool ema_fusable(const std::vector<EmaReq> &reqs)
{
    if (reqs.empty())
        return false;
    int64_t blocks = 0;
    for (const EmaReq &q : reqs) {
        if (q.NP != reqs[0].NP || q.NP < 16 || q.NP % 16 != 0 || q.NP > SC_KMAX || q.n % 8 != 0 || q.ldbt % 8 != 0 ||
            !aligned(q.M, 16) || (q.G && !aligned(q.G, 16)) || !aligned(q.M16, 16) || !aligned(q.Bt, 16))
            return false;
        blocks += cdiv(q.m, kBM);
    }
    return blocks >= 256;
}

int ema_run(const char *tag, const std::vector<EmaReq> &reqs, float a, float b, hipStream_t st)
{
    if (!ema_fusable(reqs))
        return set_error(ACSC_EINVAL, "fused EMA pass: operands not aligned or batch too small");
    const int NP = reqs[0].NP;
    int spin = kEmaSpinLimit;
    if (const char *e = std::getenv("ACSC_EMA_SPIN_LIMIT"))
        spin = std::max(0, std::min(kEmaSpinLimit, std::atoi(e)));
    // longest rows first, as for the streaming passes, and the same dispatch
    // plan: for a batch of the same shapes the fused kernel multiplies the
    // same pieces in the same order as pass_dma_kernel<false>
    std::vector<size_t> order(reqs.size());
    for (size_t i = 0; i < order.size(); ++i)
        order[i] = i;
    std::stable_sort(order.begin(), order.end(), [&](size_t a, size_t b) { return reqs[a].n > reqs[b].n; });
    std::vector<RedJob> red;
    int64_t rtot = 1;
    for (size_t c0 = 0; c0 < order.size(); c0 += kMaxJobs) {
        const size_t cnt = std::min<size_t>(kMaxJobs, order.size() - c0);
        std::vector<JobShape> js;
        EmaBatch eb{};
        eb.njobs = static_cast<int>(cnt);
        for (size_t i = 0; i < cnt; ++i) {
            const EmaReq &q = reqs[order[c0 + i]];
            eb.j[i] = EmaJob{q.M, q.G, q.M16, q.Bt, q.ldbt, q.C, q.ldc, q.m, q.n, q.part,
                             static_cast<int64_t>(q.m) * NP, static_cast<int>(tiles_per_row(q.n)), q.stall};
            js.push_back(JobShape{static_cast<int>(cdiv(q.m, kBM)), 1, static_cast<int>(round_up(q.n, kBK)), q.n,
                                  q.part != nullptr && max_splits(q.m, q.n) >= 2 && q.n >= 2 * kBK});
        }
        const SegPlan pl = plan(js);
        eb.nseg = static_cast<int>(pl.segs.size());
        for (size_t i = 0; i < pl.segs.size(); ++i)
            eb.s[i] = pl.segs[i];
        switch (NP / 16) {
        case 1: ema_launch<1>(tag, eb, pl.grid, NP, a, b, spin, st); break;
        case 2: ema_launch<2>(tag, eb, pl.grid, NP, a, b, spin, st); break;
        case 3: ema_launch<3>(tag, eb, pl.grid, NP, a, b, spin, st); break;
        case 4: ema_launch<4>(tag, eb, pl.grid, NP, a, b, spin, st); break;
        case 5: ema_launch<5>(tag, eb, pl.grid, NP, a, b, spin, st); break;
        case 6: ema_launch<6>(tag, eb, pl.grid, NP, a, b, spin, st); break;
        case 7: ema_launch<7>(tag, eb, pl.grid, NP, a, b, spin, st); break;
        case 8: ema_launch<8>(tag, eb, pl.grid, NP, a, b, spin, st); break;
        case 9: ema_launch<9>(tag, eb, pl.grid, NP, a, b, spin, st); break;
        case 10: ema_launch<10>(tag, eb, pl.grid, NP, a, b, spin, st); break;
        case 11: ema_launch<11>(tag, eb, pl.grid, NP, a, b, spin, st); break;
        default: ema_launch<12>(tag, eb, pl.grid, NP, a, b, spin, st); break;
        }
        for (size_t i = 0; i < cnt; ++i) {
            const int h = pl.halved[i];
            if (h <= 0)
                continue;
            const EmaReq &q = reqs[order[c0 + i]];
            const int64_t r0 = static_cast<int64_t>(js[i].nrb - h) * kBM;
            red.push_back(RedJob{q.part + r0 * NP, static_cast<int64_t>(q.m) * NP, q.C + r0 * q.ldc, q.ldc,
                                 static_cast<int>(q.m - r0), NP, 2});
            rtot = std::max<int64_t>(rtot, (q.m - r0) * (NP / 4));
        }
    }
    for (size_t c0 = 0; c0 < red.size(); c0 += kMaxJobs) {
        RedBatch rb{};
        rb.count = static_cast<int>(std::min<size_t>(kMaxJobs, red.size() - c0));
        for (int i = 0; i < rb.count; ++i)
            rb.j[i] = red[c0 + i];
        const unsigned g = static_cast<unsigned>(std::min<int64_t>(cdiv(rtot, 256), 8192));
        ACSC_LAUNCH("sc_split_reduce", pass_reduce_kernel, dim3(g, 1, rb.count), dim3(256), 0, st, rb);
    }
    return ACSC_OK;
}

}  // namespace pass
}  // namespace acsc
