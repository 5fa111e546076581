// Activation-masking compressor for gfx950 (paper Sec. 3.1; Alg. 1; App. F).
//
// One wavefront owns one token row; a workgroup holds up to four rows.
//   pack:   keyed permutation -> kept-set bitmap in LDS -> wave prefix scan
//           of word popcounts -> ascending index list in LDS -> gather of the
//           kept values -> coalesced stores of vals (and uint16 idx).
//   unpack: bitmap (from the key, or from transmitted indices) -> per-word
//           exclusive prefix in LDS -> every lane writes whole 16-byte chunks
//           of the dense row: zeros, or scale * vals[rank] at kept slots.
// Rows are independent, so neither kernel needs more than wave-level and
// workgroup-level synchronisation, and the dense side is touched exactly once.
#include "common.h"

namespace acsc {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;
constexpr int kMaxWavesPerBlock = 4;
constexpr size_t kLdsBudget = 160 * 1024;

// SplitMix64 output function (Steele, Lea & Flood 2014).
__host__ __device__ __forceinline__ uint64_t mix64(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// MurmurHash3 32-bit finaliser (Appleby), the Feistel round function.
__device__ __forceinline__ uint32_t fmix32(uint32_t h)
{
    h ^= h >> 16;
    h *= 0x85EBCA6Bu;
    h ^= h >> 13;
    h *= 0xC2B2AE35u;
    h ^= h >> 16;
    return h;
}

// fmix32(h) & mask for masks of at most 8 bits (the Feistel round output,
// hb <= 8): those bits of the result are bits 0..7 and 16..23 of the second
// product, which depend only on the low 24 bits of its factors, so that
// product is taken on the full-rate 24-bit multiplier.  Equal to
// fmix32(h) & mask for every h.
__device__ __forceinline__ uint32_t fmix32_low8(uint32_t h, uint32_t mask)
{
    h ^= h >> 16;
    h *= 0x85EBCA6Bu;
    h ^= h >> 13;
    h = __umul24(h, 0xC2B2AE35u & 0xFFFFFFu);
    h ^= h >> 16;
    return h & mask;
}

// Key chain over the fields of g(layer, step, B, S, H), plus seed and microbatch.
__host__ __device__ __forceinline__ uint64_t chain_fields(uint64_t seed, uint64_t layer, uint64_t step,
                                                          uint64_t microbatch, uint64_t B, uint64_t S, uint64_t H)
{
    uint64_t z = seed;
    z = mix64((z ^ layer) + kGamma);
    z = mix64((z ^ step) + kGamma);
    z = mix64((z ^ microbatch) + kGamma);
    z = mix64((z ^ B) + kGamma);
    z = mix64((z ^ S) + kGamma);
    return mix64((z ^ H) + kGamma);
}

uint64_t chain_key(const ac_mask_key &k)
{
    return chain_fields(k.seed, k.layer, k.step, k.microbatch, k.B, k.S, k.H);
}

// What a launch over several boundaries needs besides the row data: the key
// of the first boundary (boundary l of the launch, blockIdx.y, is keyed with
// layer + l, Alg. 1's per-boundary mask) and the element strides between
// consecutive boundaries' tensors.
struct MaskBatch {
    uint64_t seed, step;
    uint32_t layer, microbatch, B, S, H;
    int64_t dense_stride;   // x (pack) or y (unpack)
    int64_t vals_stride;
    int64_t idx_stride;     // idx_in and idx_out

    __device__ __forceinline__ uint64_t key(uint32_t l) const
    {
        return chain_fields(seed, static_cast<uint64_t>(layer) + l, step, microbatch, B, S, H);
    }
};

int domain_bits(int H)
{
    int w = 2;
    while ((1ll << w) < H)
        w += 2;
    return w;
}

// Keyed permutation of [0, H) for one row: a balanced Feistel network on
// 2*hb bits, cycle-walked back into range.
template <int ROUNDS>
struct RowPerm {
    uint32_t sk[ROUNDS];
    uint32_t mask;
    int hb;
    uint32_t H;

    __device__ __forceinline__ RowPerm(uint64_t key, uint64_t row, int w, uint32_t H_) : H(H_)
    {
        uint64_t c = mix64((key ^ row) + kGamma);
#pragma unroll
        for (int j = 0; j < ROUNDS / 2; ++j) {
            sk[2 * j] = static_cast<uint32_t>(c);
            sk[2 * j + 1] = static_cast<uint32_t>(c >> 32);
            c = mix64(c + kGamma);
        }
        hb = w >> 1;
        mask = (1u << hb) - 1u;
    }

    __device__ __forceinline__ uint32_t feistel(uint32_t x) const
    {
        uint32_t L = x >> hb, R = x & mask;
#pragma unroll
        for (int j = 0; j < ROUNDS; ++j) {
            const uint32_t t = L ^ fmix32_low8(R ^ sk[j], mask);
            L = R;
            R = t;
        }
        return (L << hb) | R;
    }

    __device__ __forceinline__ uint32_t operator()(uint32_t i) const
    {
        uint32_t y = feistel(i);
        while (y >= H)
            y = feistel(y);
        return y;
    }
};

// The round function's output is masked to hb <= 8 bits and its input R has
// hb bits, so a row's whole round function is a table of ROUNDS x 2^hb bytes.
// Filling it costs ROUNDS * 2^hb mixer evaluations per row instead of ROUNDS
// per Feistel evaluation (about K * 2^w / H of those), which is what bounds
// the kernels when K is large next to 2^hb.  Rounds sit at a 256-byte stride
// so that the round offset is an immediate of the LDS read.
constexpr int kTabStride = 256;

template <int ROUNDS>
__host__ __device__ __forceinline__ constexpr int table_bytes() { return ROUNDS * kTabStride; }

// Whether a row's round table is cheaper than evaluating the round function
// per Feistel step: 2^hb entries per round against about K * 2^w / H
// evaluations (cycle walking rejects 1 - H / 2^w of them).
inline bool use_table(int H, int K, int w)
{
    const int hb = w >> 1;
    return hb <= 8 && static_cast<int64_t>(K) << w >= static_cast<int64_t>(H) << hb;
}

template <int ROUNDS>
struct TabPerm {
    const uint8_t *tab;
    uint32_t mask;
    int hb;

    // Every lane of the wave calls this; the caller orders the table writes
    // before the first read (wave_sync).
    __device__ __forceinline__ TabPerm(const RowPerm<ROUNDS> &p, uint8_t *t, int lane) : tab(t), mask(p.mask), hb(p.hb)
    {
        const int n = 1 << hb;
#pragma unroll
        for (int j = 0; j < ROUNDS; ++j)
            for (int r = lane; r < n; r += 64)
                t[j * kTabStride + r] = static_cast<uint8_t>(fmix32_low8(static_cast<uint32_t>(r) ^ p.sk[j], p.mask));
    }

    __device__ __forceinline__ uint32_t feistel(uint32_t x) const
    {
        uint32_t L = x >> hb, R = x & mask;
#pragma unroll
        for (int j = 0; j < ROUNDS; ++j) {
            const uint32_t t = L ^ tab[j * kTabStride + R];
            L = R;
            R = t;
        }
        return (L << hb) | R;
    }
};

__device__ __forceinline__ int wave_exclusive_scan(int v, int lane)
{
    int incl = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int t = __shfl_up(incl, off, 64);
        if (lane >= off)
            incl += t;
    }
    return incl - v;
}

// Each wave owns one row and its own slice of LDS, so the kernels only need
// their LDS accesses ordered within the wave (an LDS queue serves a wave in
// order); no workgroup barrier.
__device__ __forceinline__ void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Set the bits of pi(0) .. pi(K - 1) in the row bitmap.  Cycle walking takes a
// varying number of Feistel evaluations per index, so instead of one index
// per lane at a time (the wave waiting for its longest walk), every lane
// performs one evaluation per step and a lane whose walk ended takes the next
// unassigned index; the wave runs about 2 K / 64 steps for H about half the
// Feistel domain.
template <typename Perm>
__device__ __forceinline__ void mark_kept(const Perm &perm, int K, uint32_t H, uint32_t *bm, int lane,
                                          uint16_t *order = nullptr)
{
    int i = lane;
    bool live = i < K;
    uint32_t y = live ? perm.feistel(static_cast<uint32_t>(i)) : 0u;
    int next = 64;
    while (__ballot(live)) {
        const bool done = live && y < H;
        if (done) {
            atomicOr(&bm[y >> 5], 1u << (y & 31));
            if (order)
                order[i] = static_cast<uint16_t>(y);   // pi(i), before sorting
        }
        const unsigned long long fin = __ballot(done);
        const int before = __popcll(fin & ((1ull << lane) - 1ull));
        uint32_t src = y;
        if (done) {
            i = next + before;
            live = i < K;
            src = static_cast<uint32_t>(i);
        }
        if (live)
            y = perm.feistel(src);
        next += __popcll(fin);
    }
}

// Per-wave LDS layout of the pack kernel: bitmap[nw], uint16 order[K] (the
// kept indices in the order they were drawn), uint16 prefix[nw] (kept
// indices before each bitmap word).
__host__ __device__ __forceinline__ int pack_wave_words(int nw, int K) { return nw + (K + 1) / 2 + (nw + 1) / 2; }

// Per-wave LDS of the pack kernel in bytes: the words above, then (TABLE) the
// row's round table.
template <int ROUNDS, bool TABLE>
__host__ __device__ __forceinline__ int pack_wave_bytes(int nw, int K)
{
    return 4 * pack_wave_words(nw, K) + (TABLE ? table_bytes<ROUNDS>() : 0);
}

// Pack by given index lists (FROM_IDX): the row's K indices are read from
// idx_in, entries >= H give +0, and nothing of the mask is evaluated.  This is
// the pack of the direction that did not compute the mask: the receiving
// stage's backward pack reuses the index lists its key-driven unpack wrote.
template <typename E>
__global__ __launch_bounds__(256) void ac_pack_idx_kernel(const E *__restrict__ x, int64_t rows, int H,
                                                          int64_t ld_x, int K, MaskBatch mb,
                                                          const uint16_t *__restrict__ idx_in,
                                                          E *__restrict__ vals)
{
    const int lane = threadIdx.x & 63;
    const int wpb = blockDim.x >> 6;
    const int64_t row = static_cast<int64_t>(blockIdx.x) * wpb + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (row >= rows)
        return;
    const uint32_t layer = blockIdx.y;
    const E *xr = x + layer * mb.dense_stride + row * ld_x;
    const uint16_t *ir = idx_in + layer * mb.idx_stride + row * K;
    E *vr = vals + layer * mb.vals_stride + row * K;
    for (int base = 0; base < K; base += 256) {
        uint16_t jj[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int i = base + lane + 64 * u;
            jj[u] = i < K ? ir[i] : uint16_t(0);
        }
        E v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int i = base + lane + 64 * u;
            v[u] = (i < K && jj[u] < H) ? xr[jj[u]] : E(0);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int i = base + lane + 64 * u;
            if (i < K)
                vr[i] = v[u];
        }
    }
}

template <typename E, int ROUNDS, bool TABLE>
__global__ __launch_bounds__(256) void ac_pack_kernel(const E *__restrict__ x, int64_t rows, int H,
                                                      int64_t ld_x, int K, MaskBatch mb, int w,
                                                      E *__restrict__ vals,
                                                      uint16_t *__restrict__ idx)
{
    extern __shared__ uint32_t smem[];
    const int lane = threadIdx.x & 63;
    const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wpb = blockDim.x >> 6;
    const int nw = (H + 31) >> 5;
    uint32_t *bm = reinterpret_cast<uint32_t *>(reinterpret_cast<unsigned char *>(smem) +
                                                wid * pack_wave_bytes<ROUNDS, TABLE>(nw, K));
    uint16_t *order = reinterpret_cast<uint16_t *>(bm + nw);
    uint16_t *wpre = order + 2 * ((K + 1) / 2);
    const int64_t row = static_cast<int64_t>(blockIdx.x) * wpb + wid;
    const bool active = row < rows;

    if (!active)
        return;
    const uint32_t layer = blockIdx.y;
    const uint64_t key = mb.key(layer);
    x += layer * mb.dense_stride;
    vals += layer * mb.vals_stride;
    if (idx)
        idx += layer * mb.idx_stride;
    for (int i = lane; i < nw; i += 64)
        bm[i] = 0u;
    {
        const RowPerm<ROUNDS> perm(key, static_cast<uint64_t>(row), w, static_cast<uint32_t>(H));
        if (TABLE) {
            const TabPerm<ROUNDS> tp(perm, reinterpret_cast<uint8_t *>(bm + pack_wave_words(nw, K)), lane);
            wave_sync();
            mark_kept(tp, K, static_cast<uint32_t>(H), bm, lane, order);
        } else {
            wave_sync();
            mark_kept(perm, K, static_cast<uint32_t>(H), bm, lane, order);
        }
    }
    wave_sync();
    // The kept values are gathered in the order they were drawn, right after
    // the mask, and stored at their rank (the number of kept indices below
    // them) once the bitmap's word prefixes are known: the gather's HBM
    // latency overlaps the prefix scan instead of following the sorted list.
    const E *xr = x + row * ld_x;
    E *vr = vals + row * K;
    uint16_t *ir = idx ? idx + row * K : nullptr;
    bool scanned = false;
    for (int base = 0; base < K; base += 256) {
        E v[4];
        uint16_t jj[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int i = base + lane + 64 * u;
            jj[u] = i < K ? order[i] : uint16_t(0);
            v[u] = i < K ? xr[jj[u]] : E(0);
        }
        if (!scanned) {
            const int per = (nw + 63) >> 6;
            const int w0 = min(lane * per, nw), w1 = min(w0 + per, nw);
            int cnt = 0;
            for (int i = w0; i < w1; ++i)
                cnt += __popc(bm[i]);
            int pos = wave_exclusive_scan(cnt, lane);
            for (int i = w0; i < w1; ++i) {
                wpre[i] = static_cast<uint16_t>(pos);
                pos += __popc(bm[i]);
            }
            wave_sync();
            scanned = true;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int i = base + lane + 64 * u;
            if (i < K) {
                const uint32_t y = jj[u];
                const int rank = wpre[y >> 5] + __popc(bm[y >> 5] & ((1u << (y & 31)) - 1u));
                vr[rank] = v[u];
                if (ir)
                    ir[rank] = jj[u];
            }
        }
    }
}

// scale * v rounded once to the output type.
__device__ __forceinline__ uint32_t scaled(uint32_t vbits, float scale)
{
    return __float_as_uint(__uint_as_float(vbits) * scale);
}

// bf16: p = fl32(v * s) and e = v * s - p (exact, by fma) decide the rounding
// of the exact product: only when p sits exactly on a bf16 tie does the sign
// of e matter; otherwise rounding p to nearest even equals rounding v * s.
__device__ __forceinline__ uint16_t scaled(uint16_t vbits, float scale)
{
    const float v = bf16_to_f32(vbits);
    const float p = v * scale;
    const float e = __builtin_fmaf(v, scale, -p);
    uint32_t u = __float_as_uint(p);
    if ((u & 0x7F800000u) == 0x7F800000u)
        return (u & 0x007FFFFFu) ? static_cast<uint16_t>((u >> 16) | 0x0040u)
                                 : static_cast<uint16_t>(u >> 16);
    if ((u & 0xFFFFu) == 0x8000u && e != 0.0f) {
        const bool away = (e > 0.0f) == (p > 0.0f);
        u = away ? u + 0x8000u : (u & 0xFFFF0000u);
        return static_cast<uint16_t>(u >> 16);
    }
    u += 0x7FFFu + ((u >> 16) & 1u);
    return static_cast<uint16_t>(u >> 16);
}

template <typename E>
struct Vec16;
template <>
struct Vec16<uint16_t> {
    static constexpr int N = 8;
};
template <>
struct Vec16<uint32_t> {
    static constexpr int N = 4;
};

// Per-wave LDS of the staged pack: bitmap[nw], prefix[nw], then the packed
// row (K values) and its K indices.
constexpr int kSegWords = 64;   // bitmap words per segment of the Bernoulli kernels

__host__ __device__ __forceinline__ size_t staged_wave_bytes(int nw, int K, int esize)
{
    const size_t b = static_cast<size_t>(2 * nw) * 4 + static_cast<size_t>(K) * esize + static_cast<size_t>(K) * 2;
    return (b + 15) & ~static_cast<size_t>(15);
}

// Builds the kept-set bitmap of `row` (from the key, or from the transmitted
// indices) and the exclusive prefix of its word popcounts.  Every lane of the
// row's wave calls it.
// With TABLE, `tab` is the wave's round-table space (table_bytes<ROUNDS>()).
template <int ROUNDS, bool TABLE>
__device__ __forceinline__ void row_bitmap(uint32_t *bm, uint32_t *pre, int nw, bool active, uint64_t key,
                                           int64_t row, int w, int H, int K, int lane,
                                           const uint16_t *idx_row, uint8_t *tab)
{
    for (int i = lane; i < nw; i += 64)
        bm[i] = 0u;
    if (active && !idx_row) {
        const RowPerm<ROUNDS> perm(key, static_cast<uint64_t>(row), w, static_cast<uint32_t>(H));
        if (TABLE) {
            const TabPerm<ROUNDS> tp(perm, tab, lane);
            wave_sync();
            mark_kept(tp, K, static_cast<uint32_t>(H), bm, lane);
        } else {
            wave_sync();
            mark_kept(perm, K, static_cast<uint32_t>(H), bm, lane);
        }
    } else {
        wave_sync();
        if (active) {
            for (int i = lane; i < K; i += 64) {
                const uint32_t j = idx_row[i];
                if (j < static_cast<uint32_t>(H))
                    atomicOr(&bm[j >> 5], 1u << (j & 31));
            }
        }
    }
    wave_sync();
    if (active) {
        const int per = (nw + 63) >> 6;
        const int w0 = min(lane * per, nw), w1 = min(w0 + per, nw);
        int cnt = 0;
        for (int i = w0; i < w1; ++i)
            cnt += __popc(bm[i]);
        int pos = wave_exclusive_scan(cnt, lane);
        for (int i = w0; i < w1; ++i) {
            pre[i] = static_cast<uint32_t>(pos);
            pos += __popc(bm[i]);
        }
    }
    wave_sync();
}

// Pack, streaming form: each lane reads whole 16-byte chunks of the row that
// hold at least one kept entry (chunks with none are never fetched), drops the
// kept entries into their rank slots of an LDS copy of the packed row, and
// the packed row (and its indices) leaves with coalesced stores.
template <typename E, int ROUNDS, bool TABLE>
__global__ __launch_bounds__(256) void ac_pack_stream_kernel(const E *__restrict__ x, int64_t rows, int H,
                                                             int64_t ld_x, int K, MaskBatch mb, int w,
                                                             E *__restrict__ vals,
                                                             uint16_t *__restrict__ idx)
{
    extern __shared__ __attribute__((aligned(16))) uint32_t smem[];
    constexpr int N = Vec16<E>::N;
    const int lane = threadIdx.x & 63;
    const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wpb = blockDim.x >> 6;
    const int nw = (H + 31) >> 5;
    // the index slots are always reserved (they are written even when idx is NULL)
    const size_t staged = staged_wave_bytes(nw, K, sizeof(E));
    const size_t per_wave = staged + (TABLE ? table_bytes<ROUNDS>() : 0);
    uint32_t *bm = reinterpret_cast<uint32_t *>(reinterpret_cast<unsigned char *>(smem) + wid * per_wave);
    uint32_t *pre = bm + nw;
    E *kv = reinterpret_cast<E *>(pre + nw);
    uint16_t *ki = reinterpret_cast<uint16_t *>(kv + K);
    const int64_t row = static_cast<int64_t>(blockIdx.x) * wpb + wid;
    const bool active = row < rows;
    const uint32_t layer = blockIdx.y;
    const uint64_t key = mb.key(layer);
    x += layer * mb.dense_stride;
    vals += layer * mb.vals_stride;
    if (idx)
        idx += layer * mb.idx_stride;
    row_bitmap<ROUNDS, TABLE>(bm, pre, nw, active, key, row, w, H, K, lane, nullptr,
                              reinterpret_cast<uint8_t *>(bm) + staged);
    if (active) {
        const E *xr = x + row * ld_x;
        const int nch = H / N;
#pragma unroll 4
        for (int c = lane; c < nch; c += 64) {
            const int j0 = c * N;
            const uint32_t word = bm[j0 >> 5];
            const int sh = j0 & 31;
            const uint32_t bits = (word >> sh) & ((1u << N) - 1u);
            if (bits) {
                const uint4 v = *reinterpret_cast<const uint4 *>(xr + j0);
                const E *ve = reinterpret_cast<const E *>(&v);
                int rank = static_cast<int>(pre[j0 >> 5]) + __popc(word & ((1u << sh) - 1u));
#pragma unroll
                for (int e = 0; e < N; ++e) {
                    if (bits & (1u << e)) {
                        kv[rank] = ve[e];
                        ki[rank] = static_cast<uint16_t>(j0 + e);
                        ++rank;
                    }
                }
            }
        }
        for (int j = nch * N + lane; j < H; j += 64) {
            const uint32_t word = bm[j >> 5];
            const int b = j & 31;
            if ((word >> b) & 1u) {
                const int rank = static_cast<int>(pre[j >> 5]) + __popc(word & ((1u << b) - 1u));
                kv[rank] = xr[j];
                ki[rank] = static_cast<uint16_t>(j);
            }
        }
    }
    wave_sync();
    if (active) {
        E *vr = vals + row * K;
        uint16_t *ir = idx ? idx + row * K : nullptr;
        for (int i = lane; i < K; i += 64) {
            vr[i] = kv[i];
            if (ir)
                ir[i] = ki[i];
        }
    }
}

// Unpack, staged form: the packed row is first copied into LDS (coalesced),
// then the dense row is built in LDS segment by segment and streamed out.
// Every lane's work is uniform (zeroing and copying) except the drop of the
// few kept entries, where writing each 16-byte chunk with its kept entries in
// place made every lane of the wave pay for the chunks that hold one.
// Per wave the LDS holds the row bitmap, the packed row, one segment of
// kUSegWords bitmap words of the dense row and (TABLE) the round table; the
// rank of each kept entry comes from a wave scan of the segment's word
// popcounts, so no per-word prefix is stored.  Small per-wave LDS keeps many
// waves resident, which is what hides the mask's latency.
constexpr int kUSegWords = 32;

__host__ __device__ __forceinline__ size_t unpack_kv_offset(int nw) { return (static_cast<size_t>(nw) * 4 + 15) & ~static_cast<size_t>(15); }

__host__ __device__ __forceinline__ size_t unpack_seg_offset(int nw, int K, int esize)
{
    return (unpack_kv_offset(nw) + static_cast<size_t>(K) * esize + 15) & ~static_cast<size_t>(15);
}

__host__ __device__ __forceinline__ size_t unpack_wave_bytes(int nw, int K, int esize)
{
    return unpack_seg_offset(nw, K, esize) + static_cast<size_t>(kUSegWords) * 32 * esize;
}

template <typename E, int ROUNDS, bool FROM_IDX, bool VEC, bool TABLE>
__global__ __launch_bounds__(256) void ac_unpack_stream_kernel(const E *__restrict__ vals,
                                                               const uint16_t *__restrict__ idx,
                                                               int64_t rows, int H, int K, MaskBatch mb,
                                                               int w, float scale, E *__restrict__ y,
                                                               int64_t ld_y, uint16_t *__restrict__ idx_out)
{
    extern __shared__ __attribute__((aligned(16))) uint32_t smem[];
    const int lane = threadIdx.x & 63;
    const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wpb = blockDim.x >> 6;
    const int nw = (H + 31) >> 5;
    const size_t staged = unpack_wave_bytes(nw, K, sizeof(E));
    const size_t per_wave = staged + (TABLE ? table_bytes<ROUNDS>() : 0);
    unsigned char *wbase = reinterpret_cast<unsigned char *>(smem) + wid * per_wave;
    uint32_t *bm = reinterpret_cast<uint32_t *>(wbase);
    E *kv = reinterpret_cast<E *>(wbase + unpack_kv_offset(nw));
    E *seg = reinterpret_cast<E *>(wbase + unpack_seg_offset(nw, K, sizeof(E)));
    const int64_t row = static_cast<int64_t>(blockIdx.x) * wpb + wid;
    if (row >= rows)
        return;
    const uint32_t layer = blockIdx.y;
    vals += layer * mb.vals_stride + row * K;
    y += layer * mb.dense_stride + row * ld_y;
    // the row's first values are loaded into registers before the mask is
    // built and reach LDS after it, so their latency overlaps the mask
    constexpr int kPre = 4;
    E pv[kPre];
#pragma unroll
    for (int u = 0; u < kPre; ++u) {
        const int i = lane + 64 * u;
        pv[u] = i < K ? vals[i] : E(0);
    }
    for (int i = lane; i < nw; i += 64)
        bm[i] = 0u;
    if (FROM_IDX) {
        wave_sync();
        const uint16_t *ir = idx + layer * mb.idx_stride + row * K;
        for (int i = lane; i < K; i += 64) {
            const uint32_t j = ir[i];
            if (j < static_cast<uint32_t>(H))
                atomicOr(&bm[j >> 5], 1u << (j & 31));
        }
    } else {
        const RowPerm<ROUNDS> perm(mb.key(layer), static_cast<uint64_t>(row), w, static_cast<uint32_t>(H));
        if (TABLE) {
            const TabPerm<ROUNDS> tp(perm, wbase + staged, lane);
            wave_sync();
            mark_kept(tp, K, static_cast<uint32_t>(H), bm, lane);
        } else {
            wave_sync();
            mark_kept(perm, K, static_cast<uint32_t>(H), bm, lane);
        }
    }
#pragma unroll
    for (int u = 0; u < kPre; ++u) {
        const int i = lane + 64 * u;
        if (i < K)
            kv[i] = pv[u];
    }
    for (int i = lane + 64 * kPre; i < K; i += 64)
        kv[i] = vals[i];
    wave_sync();
    uint16_t *orow = (!FROM_IDX && idx_out) ? idx_out + layer * mb.idx_stride + row * K : nullptr;
    // The dense row is assembled in LDS one segment at a time: zero the
    // segment, drop the kept entries into it (lane l owns word l of the
    // segment), then write it out with whole 16-byte stores.  Global memory
    // only sees full lines.
    constexpr int N = Vec16<E>::N;
    int base = 0;   // kept entries before the segment
    for (int s0 = 0; s0 < nw; s0 += kUSegWords) {
        const int e0 = s0 * 32;                            // first element of the segment
        const int len = min(kUSegWords * 32, H - e0);      // elements in it
#pragma unroll
        for (int c = lane; c < kUSegWords * 32 / N; c += 64)
            reinterpret_cast<uint4 *>(seg)[c] = make_uint4(0u, 0u, 0u, 0u);
        const int wd = s0 + lane;
        uint32_t bits = (lane < kUSegWords && wd < nw) ? bm[wd] : 0u;
        const int cnt = __popc(bits);
        const int pre = wave_exclusive_scan(cnt, lane);
        const int total = __shfl(pre + cnt, 63, 64);
        wave_sync();
        int rank = base + pre;
        while (bits) {
            const int t = __ffs(bits) - 1;
            bits &= bits - 1u;
            seg[lane * 32 + t] = scaled(kv[rank], scale);
            if (orow)
                orow[rank] = static_cast<uint16_t>((wd << 5) + t);
            ++rank;
        }
        base += total;
        wave_sync();
        if (VEC) {
            const int nch = len / N;
            // non-temporal: the dense rows are not read again by this stage,
            // and stores that stay dirty in the memory-side cache are only
            // paid for by whichever kernel runs next
            for (int c = lane; c < nch; c += 64)
                __builtin_nontemporal_store(reinterpret_cast<const u32x4 *>(seg)[c],
                                            reinterpret_cast<u32x4 *>(y + e0 + c * N));
            for (int j = nch * N + lane; j < len; j += 64)
                y[e0 + j] = seg[j];
        } else {
            for (int j = lane; j < len; j += 64)
                y[e0 + j] = seg[j];
        }
        wave_sync();
    }
}

// The kept positions of a row, ascending, from its bitmap and word prefix:
// every lane walks its words and stores each set bit's position at its rank.
__device__ __forceinline__ void store_index_list(const uint32_t *bm, const uint32_t *pre, int nw, int lane,
                                                 uint16_t *__restrict__ out)
{
    for (int wd = lane; wd < nw; wd += 64) {
        uint32_t bits = bm[wd];
        int rank = static_cast<int>(pre[wd]);
        while (bits) {
            const int t = __ffs(bits) - 1;
            bits &= bits - 1u;
            out[rank++] = static_cast<uint16_t>((wd << 5) + t);
        }
    }
}

// Unpack without LDS staging of the dense row (for rows whose staged form does
// not fit the LDS budget).
template <typename E, int ROUNDS, bool FROM_IDX, bool VEC>
__global__ __launch_bounds__(256) void ac_unpack_kernel(const E *__restrict__ vals,
                                                        const uint16_t *__restrict__ idx,
                                                        int64_t rows, int H, int K, MaskBatch mb,
                                                        int w, float scale, E *__restrict__ y,
                                                        int64_t ld_y, uint16_t *__restrict__ idx_out)
{
    extern __shared__ uint32_t smem[];
    const int lane = threadIdx.x & 63;
    const int wid = threadIdx.x >> 6;
    const int wpb = blockDim.x >> 6;
    const int nw = (H + 31) >> 5;
    uint32_t *bm = smem + wid * 2 * nw;
    uint32_t *pre = bm + nw;
    const int64_t row = static_cast<int64_t>(blockIdx.x) * wpb + wid;
    const bool active = row < rows;
    const uint32_t layer = blockIdx.y;
    const uint64_t key = FROM_IDX ? 0 : mb.key(layer);
    vals += layer * mb.vals_stride;
    y += layer * mb.dense_stride;
    if (FROM_IDX)
        idx += layer * mb.idx_stride;

    for (int i = lane; i < nw; i += 64)
        bm[i] = 0u;
    wave_sync();
    if (active) {
        if (FROM_IDX) {
            const uint16_t *ir = idx + row * K;
            for (int i = lane; i < K; i += 64) {
                const uint32_t j = ir[i];
                if (j < static_cast<uint32_t>(H))
                    atomicOr(&bm[j >> 5], 1u << (j & 31));
            }
        } else {
            const RowPerm<ROUNDS> perm(key, static_cast<uint64_t>(row), w,
                                       static_cast<uint32_t>(H));
            for (int i = lane; i < K; i += 64) {
                const uint32_t j = perm(static_cast<uint32_t>(i));
                atomicOr(&bm[j >> 5], 1u << (j & 31));
            }
        }
    }
    wave_sync();
    if (active) {
        const int per = (nw + 63) >> 6;
        const int w0 = min(lane * per, nw), w1 = min(w0 + per, nw);
        int cnt = 0;
        for (int i = w0; i < w1; ++i)
            cnt += __popc(bm[i]);
        int pos = wave_exclusive_scan(cnt, lane);
        for (int i = w0; i < w1; ++i) {
            pre[i] = static_cast<uint32_t>(pos);
            pos += __popc(bm[i]);
        }
    }
    wave_sync();
    if (!active)
        return;
    if (!FROM_IDX && idx_out)
        store_index_list(bm, pre, nw, lane, idx_out + layer * mb.idx_stride + row * K);
    const E *vr = vals + row * K;
    E *yr = y + row * ld_y;
    int jtail = 0;
    if (VEC) {
        constexpr int N = Vec16<E>::N;
        const int nch = H / N;
        for (int c = lane; c < nch; c += 64) {
            const int j0 = c * N;
            const uint32_t word = bm[j0 >> 5];
            const int sh = j0 & 31;
            uint32_t bits = (word >> sh) & ((1u << N) - 1u);
            E out[N];
#pragma unroll
            for (int e = 0; e < N; ++e)
                out[e] = 0;
            if (bits) {
                int rank = static_cast<int>(pre[j0 >> 5]) + __popc(word & ((1u << sh) - 1u));
#pragma unroll
                for (int e = 0; e < N; ++e) {
                    if (bits & (1u << e))
                        out[e] = scaled(vr[rank++], scale);
                }
            }
            *reinterpret_cast<uint4 *>(yr + j0) = *reinterpret_cast<const uint4 *>(out);
        }
        jtail = nch * N;
    }
    for (int j = jtail + lane; j < H; j += 64) {
        const uint32_t word = bm[j >> 5];
        const int b = j & 31;
        E out = 0;
        if ((word >> b) & 1u) {
            const int rank = static_cast<int>(pre[j >> 5]) + __popc(word & ((1u << b) - 1u));
            out = scaled(vr[rank], scale);
        }
        yr[j] = out;
    }
}

// ---------------------------------------------------------------------------
// Bernoulli variant (App. F: every entry kept independently with probability
// 1 - p).  Rows keep a variable number of entries; the payload is laid out
// by row_ptr (row r owns vals[row_ptr[r] .. row_ptr[r + 1]), ascending).
// The draw (our specification, as the oracle): with k_r the row key, a and b
// its low and high 32 bits, entries 2q and 2q + 1 take the low and the high
// 16 bits of fmix32(fmix32(a ^ q) ^ b) and are kept when these are below T.
// The hashing runs once per key, in bern_mask_kernel, which stores the row
// bitmaps; pack and unpack read the bitmaps.
// ---------------------------------------------------------------------------
constexpr int kBernWaves = 4;

// One wave per row: the row's bitmap (bit j % 32 of word j / 32 is entry j)
// and its count, left at row_ptr[row + 1] for bern_scan_kernel.
__global__ __launch_bounds__(64 * kBernWaves) void bern_mask_kernel(int64_t rows, int H, uint32_t T, uint64_t key,
                                                                   int64_t *__restrict__ row_ptr,
                                                                   uint32_t *__restrict__ bits)
{
    const int lane = threadIdx.x & 63;
    const int64_t row = static_cast<int64_t>(blockIdx.x) * kBernWaves + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (row >= rows)
        return;
    const uint64_t kr = mix64((key ^ static_cast<uint64_t>(row)) + kGamma);
    const uint32_t a = static_cast<uint32_t>(kr), b = static_cast<uint32_t>(kr >> 32);
    const int nw = (H + 31) >> 5;
    uint32_t *br = bits + row * nw;
    int cnt = 0;
    for (int w = lane; w < nw; w += 64) {
        uint32_t word = 0;
#pragma unroll 4
        for (int p = 0; p < 16; ++p) {
            const uint32_t h = fmix32(fmix32(a ^ static_cast<uint32_t>(w * 16 + p)) ^ b);
            word |= ((h & 0xFFFFu) < T ? 1u : 0u) << (2 * p);
            word |= ((h >> 16) < T ? 1u : 0u) << (2 * p + 1);
        }
        const int left = H - w * 32;     // entries past H are never kept
        if (left < 32)
            word &= (1u << left) - 1u;
        br[w] = word;
        cnt += __popc(word);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
        cnt += __shfl_xor(cnt, off, 64);
    if (lane == 0)
        row_ptr[row + 1] = cnt;
}

// One workgroup: row_ptr[1 ..] holds the row counts; it becomes their
// inclusive prefix sum, row_ptr[0] = 0.  Tiles of 4096 rows: thread t loads
// rows t, t + 1024, .. of the tile (coalesced), the tile is scanned in LDS in
// a fixed order, and the running total carries to the next tile.
__global__ __launch_bounds__(1024) void bern_scan_kernel(int64_t rows, int64_t *__restrict__ row_ptr)
{
    constexpr int kTile = 4096;
    __shared__ int64_t v[kTile];
    __shared__ int64_t part[1024];
    const int t = threadIdx.x;
    int64_t carry = 0;
    for (int64_t r0 = 0; r0 < rows; r0 += kTile) {
        const int n = static_cast<int>(min<int64_t>(kTile, rows - r0));
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int i = t + 1024 * k;
            v[i] = i < n ? row_ptr[r0 + i + 1] : 0;
        }
        __syncthreads();
        // thread t scans its run of four, then the 1024 run sums
        int64_t s = 0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            s += v[4 * t + k];
            v[4 * t + k] = s;
        }
        part[t] = s;
        __syncthreads();
        for (int off = 1; off < 1024; off <<= 1) {
            const int64_t x = t >= off ? part[t - off] : 0;
            __syncthreads();
            part[t] += x;
            __syncthreads();
        }
        const int64_t before = carry + (t ? part[t - 1] : 0);
#pragma unroll
        for (int k = 0; k < 4; ++k)
            v[4 * t + k] += before;
        carry += part[1023];
        __syncthreads();
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int i = t + 1024 * k;
            if (i < n)
                row_ptr[r0 + i + 1] = v[i];
        }
        __syncthreads();
    }
    if (t == 0)
        row_ptr[0] = 0;
}

// One wave per row, 64 bitmap words (2048 entries) at a time: the segment's
// kept positions go to an LDS list in ascending order (word popcount prefix),
// then the wave gathers them and stores the payload contiguously.  Payload
// slots at or past cap are never written.
template <typename E>
__global__ __launch_bounds__(64 * kBernWaves) void bern_pack_kernel(const E *__restrict__ x, int64_t rows, int H,
                                                                   int64_t ld_x, const int64_t *__restrict__ row_ptr,
                                                                   const uint32_t *__restrict__ bits,
                                                                   E *__restrict__ vals, uint16_t *__restrict__ idx,
                                                                   int64_t cap)
{
    __shared__ uint16_t lists[kBernWaves][kSegWords * 32];
    const int lane = threadIdx.x & 63;
    const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t row = static_cast<int64_t>(blockIdx.x) * kBernWaves + wid;
    if (row >= rows)
        return;
    const int nw = (H + 31) >> 5;
    const uint32_t *br = bits + row * nw;
    const E *xr = x + row * ld_x;
    uint16_t *L = lists[wid];
    int64_t base = row_ptr[row];
    for (int s0 = 0; s0 < nw; s0 += kSegWords) {
        const int w = s0 + lane;
        uint32_t word = w < nw ? br[w] : 0u;
        const int left = H - w * 32;     // a bitmap never marks entries past H; do not trust it to
        if (left < 32)
            word &= left > 0 ? (1u << left) - 1u : 0u;
        const int c = __popc(word);
        const int pre = wave_exclusive_scan(c, lane);
        const int total = __shfl(pre + c, 63, 64);
        uint32_t bm = word;
        int pos = pre;
        while (bm) {
            const int t = __ffs(bm) - 1;
            bm &= bm - 1u;
            L[pos++] = static_cast<uint16_t>(w * 32 + t);
        }
        wave_sync();
        for (int i0 = 0; i0 < total; i0 += 256) {
            // four gathers in flight before any store
            E v[4];
            uint16_t jj[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int i = i0 + lane + 64 * u;
                jj[u] = i < total ? L[i] : uint16_t(0);
                v[u] = i < total ? xr[jj[u]] : E(0);
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int i = i0 + lane + 64 * u;
                const int64_t o = base + i;
                if (i < total && o < cap) {
                    vals[o] = v[u];
                    if (idx)
                        idx[o] = jj[u];
                }
            }
        }
        wave_sync();
        base += total;
    }
}

// One wave per row, a segment of the dense row at a time in LDS: zero it,
// drop scale * (kept value) at the kept entries, write it out with 16-byte
// non-temporal stores (element stores when the row is not 16-byte aligned).
// Payload slots at or past cap read as zero.
template <typename E, bool VEC>
__global__ __launch_bounds__(64 * kBernWaves) void bern_unpack_kernel(const E *__restrict__ vals, int64_t rows, int H,
                                                                     const int64_t *__restrict__ row_ptr,
                                                                     const uint32_t *__restrict__ bits, float scale,
                                                                     E *__restrict__ y, int64_t ld_y, int64_t cap)
{
    constexpr int N = Vec16<E>::N;
    __shared__ __attribute__((aligned(16))) E segs[kBernWaves][kSegWords * 32];
    const int lane = threadIdx.x & 63;
    const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t row = static_cast<int64_t>(blockIdx.x) * kBernWaves + wid;
    if (row >= rows)
        return;
    const int nw = (H + 31) >> 5;
    const uint32_t *br = bits + row * nw;
    E *seg = segs[wid];
    E *yr = y + row * ld_y;
    int64_t base = row_ptr[row];
    for (int s0 = 0; s0 < nw; s0 += kSegWords) {
        const int e0 = s0 * 32;
        const int len = min(kSegWords * 32, H - e0);
#pragma unroll
        for (int c = lane; c < kSegWords * 32 / N; c += 64)
            reinterpret_cast<uint4 *>(seg)[c] = make_uint4(0u, 0u, 0u, 0u);
        wave_sync();
        const int w = s0 + lane;
        const uint32_t word = w < nw ? br[w] : 0u;
        const int c = __popc(word);
        const int pre = wave_exclusive_scan(c, lane);
        const int total = __shfl(pre + c, 63, 64);
        uint32_t bm = word;
        int rank = pre;
        while (bm) {
            const int t = __ffs(bm) - 1;
            bm &= bm - 1u;
            const int64_t o = base + rank++;
            seg[lane * 32 + t] = o < cap ? scaled(vals[o], scale) : E(0);
        }
        wave_sync();
        if (VEC) {
            const int nch = len / N;
            for (int q = lane; q < nch; q += 64)
                __builtin_nontemporal_store(reinterpret_cast<const u32x4 *>(seg)[q],
                                            reinterpret_cast<u32x4 *>(yr + e0 + q * N));
            for (int j = nch * N + lane; j < len; j += 64)
                yr[e0 + j] = seg[j];
        } else {
            for (int j = lane; j < len; j += 64)
                yr[e0 + j] = seg[j];
        }
        wave_sync();
        base += total;
    }
}

int common_checks(acsc_dtype dt, int64_t rows, int H, int K, const ac_mask_key *key)
{
    ACSC_CHECK_ARG(dt == ACSC_F32 || dt == ACSC_BF16, ACSC_EDTYPE, "unknown dtype %d", (int)dt);
    ACSC_CHECK_ARG(key != nullptr, ACSC_EINVAL, "key is NULL");
    ACSC_CHECK_ARG(H >= 1 && H <= 65536, ACSC_EINVAL, "H=%d outside [1, 65536]", H);
    ACSC_CHECK_ARG(K >= 1 && K <= H, ACSC_EINVAL, "K=%d outside [1, H=%d]", K, H);
    ACSC_CHECK_ARG(rows >= 0, ACSC_EINVAL, "rows=%lld < 0", (long long)rows);
    ACSC_CHECK_ARG(key->H == static_cast<uint32_t>(H), ACSC_EINVAL, "key.H=%u != H=%d", key->H, H);
    ACSC_CHECK_ARG(static_cast<int64_t>(key->B) * key->S == rows, ACSC_EINVAL,
                   "rows=%lld != key.B*key.S=%llu", (long long)rows,
                   (unsigned long long)key->B * key->S);
    return ACSC_OK;
}

// Waves per workgroup such that the per-wave LDS fits the budget.
int waves_for(size_t per_wave_bytes)
{
    int wpb = kMaxWavesPerBlock;
    while (wpb > 1 && per_wave_bytes * wpb > kLdsBudget)
        --wpb;
    return wpb;
}

MaskBatch make_batch(const ac_mask_key &k, int64_t dense_stride, int64_t vals_stride, int64_t idx_stride)
{
    MaskBatch mb;
    mb.seed = k.seed;
    mb.step = k.step;
    mb.layer = k.layer;
    mb.microbatch = k.microbatch;
    mb.B = k.B;
    mb.S = k.S;
    mb.H = k.H;
    mb.dense_stride = dense_stride;
    mb.vals_stride = vals_stride;
    mb.idx_stride = idx_stride;
    return mb;
}

template <typename E, int ROUNDS, bool TABLE>
void launch_pack_t(const void *x, int nl, int64_t rows, int H, int64_t ld_x, bool vec, int K, const MaskBatch &mb,
                   int w, void *vals, uint16_t *idx, hipStream_t st)
{
    // The streaming form (whole 16-byte chunks) measured slower on MI355X than
    // the gather below at every keep fraction of the workloads; it stays
    // available for rows whose kept entries are dense (keep >= 1/4).
    const int nw = (H + 31) / 32;
    const size_t tab = TABLE ? table_bytes<ROUNDS>() : 0;
    const size_t sper = staged_wave_bytes(nw, K, sizeof(E)) + tab;
    const bool dense = 4 * static_cast<int64_t>(K) >= H;
    if (dense && vec && sper <= kLdsBudget &&
        allow_lds(ac_pack_stream_kernel<E, ROUNDS, TABLE>, sper * waves_for(sper)) == ACSC_OK) {
        const int wpb = waves_for(sper);
        const int64_t blocks = (rows + wpb - 1) / wpb;
        ACSC_LAUNCH("ac_pack", (ac_pack_stream_kernel<E, ROUNDS, TABLE>), dim3(static_cast<unsigned>(blocks), nl),
                    dim3(64 * wpb), sper * wpb, st, static_cast<const E *>(x), rows, H, ld_x, K, mb, w,
                    static_cast<E *>(vals), idx);
        return;
    }
    const size_t per = static_cast<size_t>(pack_wave_bytes<ROUNDS, TABLE>(nw, K));
    const int wpb = waves_for(per);
    allow_lds(ac_pack_kernel<E, ROUNDS, TABLE>, per * wpb);
    const int64_t blocks = (rows + wpb - 1) / wpb;
    ACSC_LAUNCH("ac_pack", (ac_pack_kernel<E, ROUNDS, TABLE>), dim3(static_cast<unsigned>(blocks), nl),
                dim3(64 * wpb), per * wpb, st, static_cast<const E *>(x), rows, H, ld_x, K,
                mb, w, static_cast<E *>(vals), idx);
}

template <typename E, int ROUNDS>
void launch_pack(const void *x, int nl, int64_t rows, int H, int64_t ld_x, bool vec, int K, const MaskBatch &mb,
                 int w, void *vals, uint16_t *idx, hipStream_t st)
{
    if (use_table(H, K, w))
        launch_pack_t<E, ROUNDS, true>(x, nl, rows, H, ld_x, vec, K, mb, w, vals, idx, st);
    else
        launch_pack_t<E, ROUNDS, false>(x, nl, rows, H, ld_x, vec, K, mb, w, vals, idx, st);
}

template <typename E>
void launch_pack_idx(const void *x, int nl, int64_t rows, int H, int64_t ld_x, int K, const MaskBatch &mb,
                     const uint16_t *idx_in, void *vals, hipStream_t st)
{
    const int64_t blocks = (rows + kMaxWavesPerBlock - 1) / kMaxWavesPerBlock;
    ACSC_LAUNCH("ac_pack_idx", ac_pack_idx_kernel<E>, dim3(static_cast<unsigned>(blocks), nl),
                dim3(64 * kMaxWavesPerBlock), 0, st, static_cast<const E *>(x), rows, H, ld_x, K, mb, idx_in,
                static_cast<E *>(vals));
}

template <typename E, int ROUNDS, bool FROM_IDX, bool VEC, bool TABLE>
bool launch_unpack_stream(const void *vals, const uint16_t *idx, int nl, int64_t rows, int H, int K,
                          const MaskBatch &mb, int w, float scale, void *y, int64_t ld_y, uint16_t *idx_out,
                          hipStream_t st)
{
    const int nw = (H + 31) / 32;
    const size_t sper = unpack_wave_bytes(nw, K, sizeof(E)) + (TABLE ? table_bytes<ROUNDS>() : 0);
    if (sper > kLdsBudget ||
        allow_lds(ac_unpack_stream_kernel<E, ROUNDS, FROM_IDX, VEC, TABLE>, sper * waves_for(sper)) != ACSC_OK)
        return false;
    const int wpb = waves_for(sper);
    const int64_t blocks = (rows + wpb - 1) / wpb;
    ACSC_LAUNCH(FROM_IDX ? "ac_unpack_idx" : "ac_unpack", (ac_unpack_stream_kernel<E, ROUNDS, FROM_IDX, VEC, TABLE>),
                dim3(static_cast<unsigned>(blocks), nl), dim3(64 * wpb), sper * wpb, st,
                static_cast<const E *>(vals), idx, rows, H, K, mb, w, scale, static_cast<E *>(y), ld_y, idx_out);
    return true;
}

template <typename E, int ROUNDS, bool FROM_IDX>
void launch_unpack(const void *vals, const uint16_t *idx, int nl, int64_t rows, int H, int K, const MaskBatch &mb,
                   int w, float scale, void *y, int64_t ld_y, bool vec, uint16_t *idx_out, hipStream_t st)
{
    // transmitted indices need no permutation, so no round table either
    const bool table = !FROM_IDX && use_table(H, K, w);
    bool done;
    if (vec)
        done = table ? launch_unpack_stream<E, ROUNDS, FROM_IDX, true, true>(vals, idx, nl, rows, H, K, mb, w, scale, y, ld_y, idx_out, st)
                     : launch_unpack_stream<E, ROUNDS, FROM_IDX, true, false>(vals, idx, nl, rows, H, K, mb, w, scale, y, ld_y, idx_out, st);
    else
        done = table ? launch_unpack_stream<E, ROUNDS, FROM_IDX, false, true>(vals, idx, nl, rows, H, K, mb, w, scale, y, ld_y, idx_out, st)
                     : launch_unpack_stream<E, ROUNDS, FROM_IDX, false, false>(vals, idx, nl, rows, H, K, mb, w, scale, y, ld_y, idx_out, st);
    if (done)
        return;
    const int nw = (H + 31) / 32;
    const size_t per = static_cast<size_t>(2 * nw) * 4;
    const int wpb = waves_for(per);
    allow_lds(ac_unpack_kernel<E, ROUNDS, FROM_IDX, true>, per * wpb);
    allow_lds(ac_unpack_kernel<E, ROUNDS, FROM_IDX, false>, per * wpb);
    const int64_t blocks = (rows + wpb - 1) / wpb;
    if (vec)
        ACSC_LAUNCH(FROM_IDX ? "ac_unpack_idx" : "ac_unpack", (ac_unpack_kernel<E, ROUNDS, FROM_IDX, true>),
                    dim3(static_cast<unsigned>(blocks), nl), dim3(64 * wpb), per * wpb, st,
                    static_cast<const E *>(vals), idx, rows, H, K, mb, w, scale,
                    static_cast<E *>(y), ld_y, idx_out);
    else
        ACSC_LAUNCH(FROM_IDX ? "ac_unpack_idx" : "ac_unpack", (ac_unpack_kernel<E, ROUNDS, FROM_IDX, false>),
                    dim3(static_cast<unsigned>(blocks), nl), dim3(64 * wpb), per * wpb, st,
                    static_cast<const E *>(vals), idx, rows, H, K, mb, w, scale,
                    static_cast<E *>(y), ld_y, idx_out);
}

// Checks shared by the batched mask calls: the boundary count, the layer ids
// it implies, and strides that keep every boundary's outputs apart.
int batch_checks(int nlayers, const ac_mask_key *key, int64_t rows, int64_t out_extent, int64_t out_stride,
                 const char *out_name)
{
    ACSC_CHECK_ARG(nlayers >= 0 && nlayers <= 65535, ACSC_EINVAL, "nlayers=%d outside [0, 65535]", nlayers);
    if (nlayers > 1) {
        ACSC_CHECK_ARG(static_cast<uint64_t>(key->layer) + static_cast<uint64_t>(nlayers - 1) <= 0xFFFFFFFFull,
                       ACSC_EINVAL, "key.layer + nlayers - 1 exceeds the 32-bit layer field");
        ACSC_CHECK_ARG(rows == 0 || out_stride >= out_extent, ACSC_EINVAL,
                       "%s layer stride %lld < %lld elements: boundaries would overlap", out_name,
                       (long long)out_stride, (long long)out_extent);
    }
    return ACSC_OK;
}

int mask_pack_impl(const void *x, acsc_dtype dt, int nlayers, int64_t rows, int H, int64_t ld_x, int64_t x_stride,
                   int K, const ac_mask_key *key, void *vals, int64_t vals_stride, const uint16_t *idx_in,
                   uint16_t *idx_out, int64_t idx_stride, hipStream_t stream)
{
    int rc = common_checks(dt, rows, H, K, key);
    if (rc)
        return rc;
    ACSC_CHECK_ARG(ld_x >= H, ACSC_EINVAL, "ld_x=%lld < H=%d", (long long)ld_x, H);
    if ((rc = batch_checks(nlayers, key, rows, rows * K, vals_stride, "vals")))
        return rc;
    if (idx_out && (rc = batch_checks(nlayers, key, rows, rows * K, idx_stride, "idx_out")))
        return rc;
    ACSC_CHECK_ARG(!(idx_in && idx_out), ACSC_EINVAL, "idx_in and idx_out are exclusive");
    ACSC_CHECK_ARG(nlayers <= 1 || (x_stride >= 0 && (!idx_in || idx_stride >= 0)), ACSC_EINVAL,
                   "negative layer stride");
    if (rows == 0 || nlayers == 0)
        return ACSC_OK;
    ACSC_CHECK_ARG(x && vals, ACSC_EINVAL, "x or vals is NULL");
    const size_t es = dtype_size(dt);
    ACSC_CHECK_ARG(aligned(x, es) && aligned(vals, es), ACSC_EALIGN,
                   "x and vals must be %zu-byte aligned", es);
    ACSC_CHECK_ARG((!idx_in || aligned(idx_in, 2)) && (!idx_out || aligned(idx_out, 2)), ACSC_EALIGN,
                   "idx must be 2-byte aligned");
    const bool vec = aligned(x, 16) && (static_cast<size_t>(ld_x) * es) % 16 == 0 &&
                     (nlayers <= 1 || (static_cast<size_t>(x_stride) * es) % 16 == 0);
    const MaskBatch mb = make_batch(*key, nlayers > 1 ? x_stride : 0, nlayers > 1 ? vals_stride : 0,
                                    nlayers > 1 ? idx_stride : 0);
    const int w = domain_bits(H);
    if (idx_in) {
        if (dt == ACSC_BF16)
            launch_pack_idx<uint16_t>(x, nlayers, rows, H, ld_x, K, mb, idx_in, vals, stream);
        else
            launch_pack_idx<uint32_t>(x, nlayers, rows, H, ld_x, K, mb, idx_in, vals, stream);
    } else if (dt == ACSC_BF16) {
        if (w <= 4)
            launch_pack<uint16_t, 12>(x, nlayers, rows, H, ld_x, vec, K, mb, w, vals, idx_out, stream);
        else
            launch_pack<uint16_t, 8>(x, nlayers, rows, H, ld_x, vec, K, mb, w, vals, idx_out, stream);
    } else {
        if (w <= 4)
            launch_pack<uint32_t, 12>(x, nlayers, rows, H, ld_x, vec, K, mb, w, vals, idx_out, stream);
        else
            launch_pack<uint32_t, 8>(x, nlayers, rows, H, ld_x, vec, K, mb, w, vals, idx_out, stream);
    }
    return check_launch("ac_mask_pack");
}

int unpack_impl(const void *vals, int64_t vals_stride, acsc_dtype dt, int nlayers, int64_t rows, int H, int K,
                const ac_mask_key *key, const uint16_t *idx_in, uint16_t *idx_out, int64_t idx_stride, float scale,
                void *y, int64_t ld_y, int64_t y_stride, hipStream_t stream)
{
    int rc = common_checks(dt, rows, H, K, key);
    if (rc)
        return rc;
    ACSC_CHECK_ARG(ld_y >= H, ACSC_EINVAL, "ld_y=%lld < H=%d", (long long)ld_y, H);
    ACSC_CHECK_ARG(std::isfinite(scale), ACSC_EINVAL, "scale must be finite");
    if ((rc = batch_checks(nlayers, key, rows, rows > 0 ? (rows - 1) * ld_y + H : 0, y_stride, "y")))
        return rc;
    if (idx_out && (rc = batch_checks(nlayers, key, rows, rows * K, idx_stride, "idx_out")))
        return rc;
    ACSC_CHECK_ARG(!(idx_in && idx_out), ACSC_EINVAL, "idx_in and idx_out are exclusive");
    ACSC_CHECK_ARG(nlayers <= 1 || (vals_stride >= 0 && (!idx_in || idx_stride >= 0)), ACSC_EINVAL,
                   "negative layer stride");
    if (rows == 0 || nlayers == 0)
        return ACSC_OK;
    ACSC_CHECK_ARG(vals && y, ACSC_EINVAL, "vals or y is NULL");
    const size_t es = dtype_size(dt);
    ACSC_CHECK_ARG(aligned(vals, es) && aligned(y, es), ACSC_EALIGN,
                   "vals and y must be %zu-byte aligned", es);
    ACSC_CHECK_ARG((!idx_in || aligned(idx_in, 2)) && (!idx_out || aligned(idx_out, 2)), ACSC_EALIGN,
                   "idx must be 2-byte aligned");
    const bool vec = aligned(y, 16) && (static_cast<size_t>(ld_y) * es) % 16 == 0 &&
                     (nlayers <= 1 || (static_cast<size_t>(y_stride) * es) % 16 == 0);
    const MaskBatch mb = make_batch(*key, nlayers > 1 ? y_stride : 0, nlayers > 1 ? vals_stride : 0,
                                    nlayers > 1 ? idx_stride : 0);
    const int w = domain_bits(H);
#define ACSC_UNPACK(E, R)                                                                                         \
    do {                                                                                                          \
        if (idx_in)                                                                                               \
            launch_unpack<E, R, true>(vals, idx_in, nlayers, rows, H, K, mb, w, scale, y, ld_y, vec, nullptr, stream); \
        else                                                                                                      \
            launch_unpack<E, R, false>(vals, nullptr, nlayers, rows, H, K, mb, w, scale, y, ld_y, vec, idx_out, stream); \
    } while (0)
    if (dt == ACSC_BF16) {
        if (w <= 4)
            ACSC_UNPACK(uint16_t, 12);
        else
            ACSC_UNPACK(uint16_t, 8);
    } else {
        if (w <= 4)
            ACSC_UNPACK(uint32_t, 12);
        else
            ACSC_UNPACK(uint32_t, 8);
    }
#undef ACSC_UNPACK
    return check_launch("ac_unpack_scatter");
}

}  // namespace
}  // namespace acsc

using namespace acsc;

extern "C" int ac_keep_count(int H, double keep, int *K)
{
    clear_error();
    ACSC_CHECK_ARG(K != nullptr, ACSC_EINVAL, "K is NULL");
    ACSC_CHECK_ARG(H >= 1 && H <= 65536, ACSC_EINVAL, "H=%d outside [1, 65536]", H);
    ACSC_CHECK_ARG(keep > 0.0 && keep <= 1.0, ACSC_EINVAL, "keep=%g outside (0, 1]", keep);
    const double k = std::floor(keep * static_cast<double>(H) + 0.5);
    ACSC_CHECK_ARG(k >= 1.0 && k <= static_cast<double>(H), ACSC_EINVAL,
                   "round(keep*H)=%g outside [1, H]", k);
    *K = static_cast<int>(k);
    return ACSC_OK;
}

extern "C" int ac_mask_pack(const void *x, acsc_dtype dt, int64_t rows, int H, int64_t ld_x, int K,
                            const ac_mask_key *key, void *vals, uint16_t *idx, hipStream_t stream)
{
    clear_error();
    return mask_pack_impl(x, dt, 1, rows, H, ld_x, 0, K, key, vals, 0, nullptr, idx, 0, stream);
}

extern "C" int ac_unpack_scatter(const void *vals, const uint16_t *idx, acsc_dtype dt, int64_t rows,
                                 int H, int K, const ac_mask_key *key, float scale, void *y,
                                 int64_t ld_y, hipStream_t stream)
{
    clear_error();
    return unpack_impl(vals, 0, dt, 1, rows, H, K, key, idx, nullptr, 0, scale, y, ld_y, 0, stream);
}

extern "C" int ac_mask_pack_batched(const void *x, acsc_dtype dt, int nlayers, int64_t rows, int H, int64_t ld_x,
                                    int64_t x_stride, int K, const ac_mask_key *key, void *vals,
                                    int64_t vals_stride, const uint16_t *idx_in, uint16_t *idx_out,
                                    int64_t idx_stride, hipStream_t stream)
{
    clear_error();
    return mask_pack_impl(x, dt, nlayers, rows, H, ld_x, x_stride, K, key, vals, vals_stride, idx_in, idx_out,
                          idx_stride, stream);
}

extern "C" int ac_unpack_scatter_batched(const void *vals, int64_t vals_stride, acsc_dtype dt, int nlayers,
                                         int64_t rows, int H, int K, const ac_mask_key *key,
                                         const uint16_t *idx_in, uint16_t *idx_out, int64_t idx_stride,
                                         float scale, void *y, int64_t ld_y, int64_t y_stride,
                                         hipStream_t stream)
{
    clear_error();
    return unpack_impl(vals, vals_stride, dt, nlayers, rows, H, K, key, idx_in, idx_out, idx_stride, scale, y,
                       ld_y, y_stride, stream);
}

// ---------------------------------------------------------------------------
// Bernoulli variant entry points.
// ---------------------------------------------------------------------------
namespace acsc {
namespace {

int bern_threshold(double keep, uint32_t *T)
{
    ACSC_CHECK_ARG(keep > 0.0 && keep <= 1.0, ACSC_EINVAL, "keep=%g outside (0, 1]", keep);
    const double t = std::floor(keep * 65536.0 + 0.5);
    ACSC_CHECK_ARG(t >= 1.0, ACSC_EINVAL, "keep=%g rounds to a zero threshold (keep >= 2^-17)", keep);
    *T = static_cast<uint32_t>(t > 65536.0 ? 65536.0 : t);
    return ACSC_OK;
}

int bern_shape(int64_t rows, int H)
{
    ACSC_CHECK_ARG(rows >= 0, ACSC_EINVAL, "rows=%lld < 0", (long long)rows);
    ACSC_CHECK_ARG(H >= 1 && H <= 65536, ACSC_EINVAL, "H=%d outside [1, 65536]", H);
    return ACSC_OK;
}

unsigned bern_blocks(int64_t rows)
{
    return static_cast<unsigned>((rows + kBernWaves - 1) / kBernWaves);
}

}  // namespace
}  // namespace acsc

extern "C" int ac_bern_mask(int64_t rows, int H, double keep, const ac_mask_key *key, int64_t *row_ptr,
                            uint32_t *bits, hipStream_t stream)
{
    clear_error();
    int rc = bern_shape(rows, H);
    if (rc)
        return rc;
    uint32_t T = 0;
    if ((rc = bern_threshold(keep, &T)))
        return rc;
    ACSC_CHECK_ARG(key != nullptr, ACSC_EINVAL, "key is NULL");
    ACSC_CHECK_ARG(key->H == static_cast<uint32_t>(H), ACSC_EINVAL, "key.H=%u != H=%d", key->H, H);
    ACSC_CHECK_ARG(static_cast<int64_t>(key->B) * key->S == rows, ACSC_EINVAL,
                   "rows=%lld != key.B*key.S=%llu", (long long)rows, (unsigned long long)key->B * key->S);
    ACSC_CHECK_ARG(row_ptr != nullptr && (rows == 0 || bits != nullptr), ACSC_EINVAL, "row_ptr or bits is NULL");
    ACSC_CHECK_ARG(aligned(row_ptr, 8) && aligned(bits, 4), ACSC_EALIGN, "row_ptr (8) or bits (4) misaligned");
    const uint64_t k = chain_key(*key);
    if (rows > 0)
        ACSC_LAUNCH("ac_bern_mask", bern_mask_kernel, dim3(bern_blocks(rows)), dim3(64 * kBernWaves), 0, stream,
                    rows, H, T, k, row_ptr, bits);
    ACSC_LAUNCH("ac_bern_scan", bern_scan_kernel, dim3(1), dim3(1024), 0, stream, rows, row_ptr);
    return check_launch("ac_bern_mask");
}

extern "C" int ac_bern_pack(const void *x, acsc_dtype dt, int64_t rows, int H, int64_t ld_x,
                            const int64_t *row_ptr, const uint32_t *bits, void *vals, uint16_t *idx,
                            int64_t cap, hipStream_t stream)
{
    clear_error();
    int rc = bern_shape(rows, H);
    if (rc)
        return rc;
    ACSC_CHECK_ARG(dt == ACSC_F32 || dt == ACSC_BF16, ACSC_EDTYPE, "unknown dtype %d", (int)dt);
    ACSC_CHECK_ARG(ld_x >= H, ACSC_EINVAL, "ld_x=%lld < H=%d", (long long)ld_x, H);
    ACSC_CHECK_ARG(cap >= 0, ACSC_EINVAL, "cap=%lld < 0", (long long)cap);
    if (rows == 0)
        return ACSC_OK;
    ACSC_CHECK_ARG(x && row_ptr && bits && (vals || cap == 0), ACSC_EINVAL, "null pointer argument");
    const size_t es = dtype_size(dt);
    ACSC_CHECK_ARG(aligned(x, es) && aligned(vals, es) && aligned(row_ptr, 8) && aligned(bits, 4) &&
                       (!idx || aligned(idx, 2)),
                   ACSC_EALIGN, "misaligned pointer argument");
    if (dt == ACSC_BF16)
        ACSC_LAUNCH("ac_bern_pack", bern_pack_kernel<uint16_t>, dim3(bern_blocks(rows)), dim3(64 * kBernWaves), 0,
                    stream, static_cast<const uint16_t *>(x), rows, H, ld_x, row_ptr, bits,
                    static_cast<uint16_t *>(vals), idx, cap);
    else
        ACSC_LAUNCH("ac_bern_pack", bern_pack_kernel<uint32_t>, dim3(bern_blocks(rows)), dim3(64 * kBernWaves), 0,
                    stream, static_cast<const uint32_t *>(x), rows, H, ld_x, row_ptr, bits,
                    static_cast<uint32_t *>(vals), idx, cap);
    return check_launch("ac_bern_pack");
}

extern "C" int ac_bern_unpack(const void *vals, acsc_dtype dt, int64_t rows, int H, const int64_t *row_ptr,
                              const uint32_t *bits, int64_t cap, float scale, void *y, int64_t ld_y,
                              hipStream_t stream)
{
    clear_error();
    int rc = bern_shape(rows, H);
    if (rc)
        return rc;
    ACSC_CHECK_ARG(dt == ACSC_F32 || dt == ACSC_BF16, ACSC_EDTYPE, "unknown dtype %d", (int)dt);
    ACSC_CHECK_ARG(ld_y >= H, ACSC_EINVAL, "ld_y=%lld < H=%d", (long long)ld_y, H);
    ACSC_CHECK_ARG(cap >= 0, ACSC_EINVAL, "cap=%lld < 0", (long long)cap);
    ACSC_CHECK_ARG(std::isfinite(scale), ACSC_EINVAL, "scale must be finite");
    if (rows == 0)
        return ACSC_OK;
    ACSC_CHECK_ARG(y && row_ptr && bits && (vals || cap == 0), ACSC_EINVAL, "null pointer argument");
    const size_t es = dtype_size(dt);
    ACSC_CHECK_ARG(aligned(y, es) && aligned(vals, es) && aligned(row_ptr, 8) && aligned(bits, 4), ACSC_EALIGN,
                   "misaligned pointer argument");
    const bool vec = aligned(y, 16) && (static_cast<size_t>(ld_y) * es) % 16 == 0;
#define ACSC_BERN_UNPACK(E, V)                                                                                   \
    ACSC_LAUNCH("ac_bern_unpack", (bern_unpack_kernel<E, V>), dim3(bern_blocks(rows)), dim3(64 * kBernWaves), 0, \
                stream, static_cast<const E *>(vals), rows, H, row_ptr, bits, scale, static_cast<E *>(y), ld_y, cap)
    if (dt == ACSC_BF16) {
        if (vec)
            ACSC_BERN_UNPACK(uint16_t, true);
        else
            ACSC_BERN_UNPACK(uint16_t, false);
    } else {
        if (vec)
            ACSC_BERN_UNPACK(uint32_t, true);
        else
            ACSC_BERN_UNPACK(uint32_t, false);
    }
#undef ACSC_BERN_UNPACK
    return check_launch("ac_bern_unpack");
}
