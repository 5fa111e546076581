/*
 * CPU oracle for the activation-masking compressor at a pipeline-parallel
 * boundary (paper Sec. 3.1; App. F).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, obviously correct
 * definition that the HIP path is checked against.  Only the test suite, the
 * smoke check and the benchmark's CPU-baseline leg may load it; the product
 * path never does.  It shares no code with the HIP library.
 *
 * What the paper fixes (Sec. 3.1): a hidden-state tensor h of T x H is masked
 * elementwise, keeping K = round((1-p) H) entries per token; the mask comes
 * from a shared deterministic pseudorandom function g(layer, step, B, S, H)
 * so that sender and receiver rebuild it and only the K kept values cross the
 * link; the backward pass uses the same mask.  App. F rescales by 1/(1-p) at
 * the receiver so the masked activation is unbiased.
 *
 * What the paper leaves open, and the reading taken here:
 *   - The PRF itself.  Key chain: SplitMix64's output mixer (Steele, Lea and
 *     Flood, OOPSLA 2014) folded over (layer, step, microbatch, B, S, H)
 *     starting from a seed.  Per-row subset: the first K outputs of a keyed
 *     balanced Feistel permutation on [0, 2^w) (Luby-Rackoff), with
 *     MurmurHash3's fmix32 finaliser (Appleby) as round function, restricted
 *     to [0, H) by cycle walking (Black-Rogaway 2002), then sorted ascending.
 *     8 rounds, or 12 when the halves have at most 2 bits (H <= 16): with
 *     4 rounds the induced K-subsets are measurably non-uniform at small w.
 *   - Fixed K per token (uniform K-subset) rather than iid Bernoulli entries.
 *   - round(): floor(keep * H + 0.5) evaluated in double.
 *   - The receiver scale is an explicit argument; the scaled value is the
 *     exact product rounded once to the output type (round to nearest even).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_GAMMA 0x9E3779B97F4A7C15ULL

/* SplitMix64 output function (mix64 / "variant 13"). */
uint64_t orc_mix64(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

/* MurmurHash3 32-bit finaliser. */
uint32_t orc_fmix32(uint32_t h)
{
    h ^= h >> 16;
    h *= 0x85EBCA6BU;
    h ^= h >> 13;
    h *= 0xC2B2AE35U;
    h ^= h >> 16;
    return h;
}

/* Mask key for g(layer, step, B, S, H) plus a seed and a microbatch id. */
uint64_t orc_mask_key(uint64_t seed, uint32_t layer, uint64_t step, uint32_t microbatch,
                      uint32_t B, uint32_t S, uint32_t H)
{
    uint64_t f[6];
    f[0] = layer; f[1] = step; f[2] = microbatch; f[3] = B; f[4] = S; f[5] = H;
    uint64_t k = seed;
    for (int i = 0; i < 6; ++i)
        k = orc_mix64((k ^ f[i]) + ORC_GAMMA);
    return k;
}

uint64_t orc_row_key(uint64_t key, uint64_t row)
{
    return orc_mix64((key ^ row) + ORC_GAMMA);
}

/* Smallest even w >= 2 with 2^w >= H. */
int orc_domain_bits(uint32_t H)
{
    int w = 2;
    while ((1ULL << w) < (uint64_t)H)
        w += 2;
    return w;
}

/* Number of Feistel rounds for a 2h-bit domain. */
int orc_feistel_rounds(int w)
{
    return w <= 4 ? 12 : 8;
}

/* Round subkeys: c_0 = row key, c_{j+1} = mix64(c_j + gamma);
 * sk[2j] = low 32 bits of c_j, sk[2j+1] = high 32 bits of c_j. */
static void subkeys(uint64_t row_key, int rounds, uint32_t sk[12])
{
    uint64_t c = row_key;
    for (int j = 0; 2 * j < rounds; ++j) {
        sk[2 * j] = (uint32_t)(c & 0xFFFFFFFFULL);
        sk[2 * j + 1] = (uint32_t)(c >> 32);
        c = orc_mix64(c + ORC_GAMMA);
    }
}

/* One pass of the balanced Feistel network on w-bit values:
 * (L, R) -> (R, L xor (fmix32(R xor sk_j) mod 2^h)) for each round j. */
uint32_t orc_feistel(uint32_t x, int w, uint64_t row_key)
{
    uint32_t sk[12];
    int rounds = orc_feistel_rounds(w);
    subkeys(row_key, rounds, sk);
    int h = w / 2;
    uint32_t mask = (1U << h) - 1U;
    uint32_t L = x >> h;
    uint32_t R = x & mask;
    for (int j = 0; j < rounds; ++j) {
        uint32_t t = L ^ (orc_fmix32(R ^ sk[j]) & mask);
        L = R;
        R = t;
    }
    return (L << h) | R;
}

/* The keyed permutation of [0, H): Feistel, cycle-walked back into range. */
uint32_t orc_perm(uint32_t i, uint32_t H, uint64_t row_key)
{
    int w = orc_domain_bits(H);
    uint32_t y = orc_feistel(i, w, row_key);
    while (y >= H)
        y = orc_feistel(y, w, row_key);
    return y;
}

int orc_keep_count(int H, double keep, int *K)
{
    if (H < 1 || H > 65536 || !(keep > 0.0) || !(keep <= 1.0))
        return -1;
    double k = floor(keep * (double)H + 0.5);
    if (k < 1.0 || k > (double)H)
        return -1;
    *K = (int)k;
    return 0;
}

static int cmp_u32(const void *a, const void *b)
{
    uint32_t x = *(const uint32_t *)a, y = *(const uint32_t *)b;
    return (x > y) - (x < y);
}

/* Kept indices of one row: sort{ pi_row(i) : 0 <= i < K }. */
int orc_row_indices(uint64_t key, uint64_t row, uint32_t H, uint32_t K, uint32_t *out)
{
    if (K < 1 || K > H)
        return -1;
    uint64_t rk = orc_row_key(key, row);
    for (uint32_t i = 0; i < K; ++i)
        out[i] = orc_perm(i, H, rk);
    qsort(out, K, sizeof(uint32_t), cmp_u32);
    return 0;
}

/* pack: vals[r, i] = x[r, I_r[i]] (bit copy), idx[r, i] = I_r[i].
 * esize is the element size in bytes (2 for bf16, 4 for fp32). */
int orc_pack(const void *x, int esize, int64_t rows, int H, int64_t ld_x, int K, uint64_t key,
             int64_t row0, void *vals, uint16_t *idx)
{
    uint32_t *I = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)K);
    if (!I)
        return -1;
    const unsigned char *xb = (const unsigned char *)x;
    unsigned char *vb = (unsigned char *)vals;
    for (int64_t r = 0; r < rows; ++r) {
        if (orc_row_indices(key, (uint64_t)(row0 + r), (uint32_t)H, (uint32_t)K, I) != 0) {
            free(I);
            return -1;
        }
        for (int i = 0; i < K; ++i) {
            memcpy(vb + ((size_t)r * K + i) * esize, xb + ((size_t)r * ld_x + I[i]) * esize,
                   (size_t)esize);
            if (idx)
                idx[(size_t)r * K + i] = (uint16_t)I[i];
        }
    }
    free(I);
    return 0;
}

/* Round a double to bfloat16 (8 significant bits), nearest with ties to even,
 * returning the 16-bit pattern.  Works on the value: the spacing of bf16
 * numbers at |v| is 2^(e-8) for v = f * 2^e, f in [0.5, 1), and 2^-133 below
 * the normal range. */
uint16_t orc_bf16_from_double(double v)
{
    if (isnan(v))
        return 0x7FC0;
    if (v == 0.0)
        return signbit(v) ? 0x8000 : 0x0000;
    if (isinf(v))
        return v > 0 ? 0x7F80 : 0xFF80;
    int e;
    frexp(v, &e);
    int q = e - 8;
    if (q < -133)
        q = -133;
    double t = nearbyint(ldexp(v, -q));   /* default rounding: ties to even */
    double rv = ldexp(t, q);
    if (fabs(rv) >= ldexp(1.0, 128))
        return v > 0 ? 0x7F80 : 0xFF80;
    float f = (float)rv;                   /* exact: rv has <= 8 significant bits */
    uint32_t b;
    memcpy(&b, &f, 4);
    if (rv == 0.0)
        return signbit(v) ? 0x8000 : 0x0000;
    return (uint16_t)(b >> 16);
}

double orc_bf16_to_double(uint16_t h)
{
    uint32_t b = (uint32_t)h << 16;
    float f;
    memcpy(&f, &b, 4);
    return (double)f;
}

/* unpack/scatter: y[r, :] = +0, then y[r, I_r[i]] = round(vals[r, i] * scale).
 * dtype 0 = fp32, 1 = bf16.  When idx is given, its row supplies the
 * positions instead of the key. */
int orc_unpack(const void *vals, const uint16_t *idx, int dtype, int64_t rows, int H, int K,
               uint64_t key, int64_t row0, float scale, void *y, int64_t ld_y)
{
    uint32_t *I = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)K);
    if (!I)
        return -1;
    for (int64_t r = 0; r < rows; ++r) {
        if (idx) {
            for (int i = 0; i < K; ++i)
                I[i] = idx[(size_t)r * K + i];
        } else if (orc_row_indices(key, (uint64_t)(row0 + r), (uint32_t)H, (uint32_t)K, I) != 0) {
            free(I);
            return -1;
        }
        if (dtype == 0) {
            float *yr = (float *)y + (size_t)r * ld_y;
            const float *vr = (const float *)vals + (size_t)r * K;
            for (int j = 0; j < H; ++j)
                yr[j] = 0.0f;
            for (int i = 0; i < K; ++i) {
                if (I[i] >= (uint32_t)H)
                    continue;
                double p = (double)vr[i] * (double)scale;   /* exact in double */
                yr[I[i]] = (float)p;                        /* one rounding */
            }
        } else {
            uint16_t *yr = (uint16_t *)y + (size_t)r * ld_y;
            const uint16_t *vr = (const uint16_t *)vals + (size_t)r * K;
            for (int j = 0; j < H; ++j)
                yr[j] = 0;
            for (int i = 0; i < K; ++i) {
                if (I[i] >= (uint32_t)H)
                    continue;
                double p = orc_bf16_to_double(vr[i]) * (double)scale;
                yr[I[i]] = orc_bf16_from_double(p);
            }
        }
    }
    free(I);
    return 0;
}

/* Dense mask of rows [row0, row0 + rows): m[r, j] = 1 if j is kept. */
int orc_mask_dense(int64_t rows, int H, int K, uint64_t key, int64_t row0, uint8_t *m)
{
    uint32_t *I = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)K);
    if (!I)
        return -1;
    for (int64_t r = 0; r < rows; ++r) {
        memset(m + (size_t)r * H, 0, (size_t)H);
        if (orc_row_indices(key, (uint64_t)(row0 + r), (uint32_t)H, (uint32_t)K, I) != 0) {
            free(I);
            return -1;
        }
        for (int i = 0; i < K; ++i)
            m[(size_t)r * H + I[i]] = 1;
    }
    free(I);
    return 0;
}

/* ------------------------------------------------------------------------
 * Bernoulli variant (App. F: each entry kept independently with probability
 * 1 - p; the receiver rescales by 1 / (1 - p)).  Rows keep a variable number
 * of entries, so the payload is laid out by rows: row_ptr[r] .. row_ptr[r+1]
 * index the kept values (and indices) of row r, ascending.
 *
 * The per-entry draw is our specification (the paper gives no PRF): with k_r
 * the row key above, a its low and b its high 32 bits, entries 2q and 2q + 1
 * of the row take the low and the high 16 bits of
 *     h_q = fmix32(fmix32(a ^ q) ^ b),
 * and entry j is kept iff its 16 bits are below T = floor(keep * 65536 + 0.5),
 * 1 <= T <= 65536: inclusion probability T / 65536.
 * ---------------------------------------------------------------------- */
int orc_bern_threshold(double keep, int *T)
{
    if (!(keep > 0.0 && keep <= 1.0))
        return -1;
    double t = floor(keep * 65536.0 + 0.5);
    if (t < 1.0)
        return -1;
    if (t > 65536.0)
        t = 65536.0;
    *T = (int)t;
    return 0;
}

int orc_bern_kept(uint64_t row_key, uint32_t j, int T)
{
    uint32_t a = (uint32_t)row_key, b = (uint32_t)(row_key >> 32);
    uint32_t h = orc_fmix32(orc_fmix32(a ^ (j >> 1)) ^ b);
    uint32_t u = (j & 1u) ? (h >> 16) : (h & 0xFFFFu);
    return u < (uint32_t)T;
}

/* row_ptr[0] = 0, row_ptr[r + 1] = row_ptr[r] + (entries kept in row row0 + r). */
int orc_bern_row_ptr(uint64_t key, int64_t rows, int H, int T, int64_t row0, int64_t *row_ptr)
{
    row_ptr[0] = 0;
    for (int64_t r = 0; r < rows; ++r) {
        uint64_t rk = orc_row_key(key, (uint64_t)(row0 + r));
        int64_t c = 0;
        for (int j = 0; j < H; ++j)
            c += orc_bern_kept(rk, (uint32_t)j, T);
        row_ptr[r + 1] = row_ptr[r] + c;
    }
    return 0;
}

/* pack: the kept entries of row r, ascending, at vals[row_ptr[r] ..] (bit
 * copies) and their positions at idx[row_ptr[r] ..] (if idx is given). */
int orc_bern_pack(const void *x, int esize, int64_t rows, int H, int64_t ld_x, int T, uint64_t key,
                  int64_t row0, const int64_t *row_ptr, void *vals, uint16_t *idx)
{
    const unsigned char *xb = (const unsigned char *)x;
    unsigned char *vb = (unsigned char *)vals;
    for (int64_t r = 0; r < rows; ++r) {
        uint64_t rk = orc_row_key(key, (uint64_t)(row0 + r));
        int64_t pos = row_ptr[r];
        for (int j = 0; j < H; ++j) {
            if (!orc_bern_kept(rk, (uint32_t)j, T))
                continue;
            memcpy(vb + (size_t)pos * esize, xb + ((size_t)r * ld_x + j) * esize, (size_t)esize);
            if (idx)
                idx[pos] = (uint16_t)j;
            ++pos;
        }
        if (pos != row_ptr[r + 1])
            return -1;
    }
    return 0;
}

/* unpack: y[r, :] = +0, then y[r, j] = round(scale * vals[...]) for the kept
 * j of the row in ascending order (positions from idx when given). */
int orc_bern_unpack(const void *vals, const uint16_t *idx, int dtype, int64_t rows, int H, int T,
                    uint64_t key, int64_t row0, const int64_t *row_ptr, float scale, void *y, int64_t ld_y)
{
    for (int64_t r = 0; r < rows; ++r) {
        uint64_t rk = orc_row_key(key, (uint64_t)(row0 + r));
        int64_t pos = row_ptr[r], end = row_ptr[r + 1];
        if (dtype == 0) {
            float *yr = (float *)y + (size_t)r * ld_y;
            for (int j = 0; j < H; ++j)
                yr[j] = 0.0f;
        } else {
            uint16_t *yr = (uint16_t *)y + (size_t)r * ld_y;
            for (int j = 0; j < H; ++j)
                yr[j] = 0;
        }
        for (int j = 0; j < H && pos < end; ++j) {
            int kept = idx ? (idx[pos] == (uint16_t)j) : orc_bern_kept(rk, (uint32_t)j, T);
            if (!kept)
                continue;
            if (dtype == 0) {
                double p = (double)((const float *)vals)[pos] * (double)scale;
                ((float *)y)[(size_t)r * ld_y + j] = (float)p;
            } else {
                double p = orc_bf16_to_double(((const uint16_t *)vals)[pos]) * (double)scale;
                ((uint16_t *)y)[(size_t)r * ld_y + j] = orc_bf16_from_double(p);
            }
            ++pos;
        }
    }
    return 0;
}
