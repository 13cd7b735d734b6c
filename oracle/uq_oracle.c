/*
 * uq_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously-correct CPU reference for the unbiased max-norm
 * quantisers of "Unbiased Single-scale and Multi-scale Quantizers for
 * Distributed Optimization" (arXiv 2109.12497).  Only the test suite, the
 * smoke check and the benchmark's CPU-baseline leg may load this file; the
 * product (the HIP library) never does and shares no code with it.
 *
 * Build: gcc -O2 -std=c99 -ffp-contract=off -fno-fast-math -shared -fPIC
 * (x86-64: SSE2 arithmetic, IEEE binary32/binary64, round-to-nearest-even,
 * no fused multiply-add, denormals preserved).
 *
 * Every function takes the paper's steps in the paper's order:
 *   Sec. 3.1 (QSGDMaxNorm): max-norm scale, Eq. (7)-(8) quantiser, integer
 *     code zeta = sign * s * xi, reconstruction Eq. (9) applied to the
 *     all-reduced (summed) codes with the 1/M of Algorithm 1;
 *   Sec. 3.2 (QSGDMaxNormMultiScale): per-coordinate scale rule Eq. (11),
 *     scale sharing by the minimum over workers, Eq. (10)/(12) quantiser,
 *     element-wise reconstruction Eq. (13) (Algorithm 2).
 *
 * Readings of points the paper leaves open (each pinned by a test):
 *   - the norm is the L2 norm of the whole flat vector, squares of the fp32
 *     values summed in fp64 in index order; W = fp32(sqrt(max_m S_m));
 *   - ratios are formed as x = |v| * fl32(s/W) (one rounding for the
 *     reciprocal table, one for the product), then clamped to x <= s_min so
 *     that |v| = W (a = 1, outside the paper's half-open level interval)
 *     gives the top level deterministically;
 *   - the Bernoulli choice of Eq. (8) uses a 32-bit uniform word r and the
 *     32-bit threshold t = floor(p * 2^32): round up iff r < t;
 *   - r comes from Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel
 *     random numbers: as easy as 1, 2, 3", SC'11) keyed by the 64-bit seed:
 *     coordinate i of worker m takes 16 bits from block (i/8, m, purpose 0)
 *     as the high half of r and 16 bits from block (i/8, m, purpose 1) as
 *     the low half;
 *   - zero, NaN and infinite coordinates give code 0; a scale W that is not
 *     a positive finite number, or for which s_min/W overflows, gives the
 *     all-zero output (scale index K-1 everywhere);
 *   - the all-reduce of the codes is an exact int32 sum; 1/M is folded into
 *     the reconstruction factor fl32(W / (M * s_k)).
 *
 * Sub-byte codes (the bit-packing the paper discusses in Sec. 5 and
 * Appendix A): with `bits` = 4 (s_min <= 7) or 2 (s_min <= 1) the code of
 * coordinate i is stored two's complement in bits (i % (8/bits)) * bits ..
 * +bits-1 of byte i / (8/bits), low bits first.
 *
 * GlobalRandK (Sec. 3.3-3.4): the K coordinates are a uniformly random
 * K-subset shared by all workers: coordinate i gets the 64-bit key
 * (hi, lo) = (word i%4 of Philox block (i/4, 0, purpose 2),
 *             word i%4 of Philox block (i/4, 0, purpose 3))
 * and the K coordinates with the smallest (key, i) are taken, listed in
 * increasing order.  The chosen coordinates of every worker are then
 * quantised as a K-dimensional problem (its own max norm, the same seed);
 * the reconstruction is written back to those coordinates and every other
 * coordinate of the averaged gradient is 0 (no d/K rescaling: the paper
 * applies the quantiser to the sampled coordinates and says nothing more).
 */
#include <float.h>
#include <math.h>
#include <stdint.h>
#include <stddef.h>
#include <stdlib.h>

/* ------------------------------------------------------------------------ */
/* Philox4x32-10, from the published round function: two 32x32->64 products  */
/* of counter words 0 and 2 with fixed multipliers, the high halves xored    */
/* with the other two counter words and the round key, the words permuted;  */
/* the two key words advance by Weyl constants between rounds.               */
/* ------------------------------------------------------------------------ */
void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    uint32_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        uint64_t prod_a = (uint64_t)0xD2511F53u * (uint64_t)x0;
        uint64_t prod_b = (uint64_t)0xCD9E8D57u * (uint64_t)x2;
        uint32_t y0 = (uint32_t)(prod_b >> 32) ^ x1 ^ k0;
        uint32_t y1 = (uint32_t)prod_b;
        uint32_t y2 = (uint32_t)(prod_a >> 32) ^ x3 ^ k1;
        uint32_t y3 = (uint32_t)prod_a;
        x0 = y0; x1 = y1; x2 = y2; x3 = y3;
    }
    out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/* The 32-bit uniform word r for coordinate i of worker m (see header). */
uint32_t orc_uniform_word(uint64_t seed, uint32_t worker, uint64_t i)
{
    uint64_t block = i / 8;
    unsigned j = (unsigned)(i % 8);
    unsigned word = j % 4;          /* coordinates 8q+0..3 -> words 0..3, low halves  */
    unsigned shift = (j / 4) * 16;  /* coordinates 8q+4..7 -> words 0..3, high halves */
    uint32_t key[2] = { (uint32_t)seed, (uint32_t)(seed >> 32) };
    uint32_t ctr[4] = { (uint32_t)block, (uint32_t)(block >> 32), worker, 0u };
    uint32_t first[4], second[4];
    orc_philox4x32_10(ctr, key, first);
    ctr[3] = 1u;
    orc_philox4x32_10(ctr, key, second);
    uint32_t hi = (first[word] >> shift) & 0xFFFFu;
    uint32_t lo = (second[word] >> shift) & 0xFFFFu;
    return (hi << 16) | lo;
}

/* ------------------------------------------------------------------------ */
/* Shared scale (Sec. 3.1/3.2: ||w||_2 = max_m ||g^m||_2, the MaxAllReduce   */
/* of Algorithm 1 and Algorithm 2).                                           */
/* ------------------------------------------------------------------------ */

/* S = sum_i v_i^2, each square exact in binary64, summed in index order. */
double orc_sum_of_squares(const float* v, int64_t n)
{
    double s = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        double x = (double)v[i];
        s = s + x * x;
    }
    return s;
}

/* W = fp32(sqrt(max_m S_m)); NaN if any S_m is NaN. */
float orc_max_norm(const double* sumsq, int32_t M)
{
    double best = 0.0;
    for (int32_t m = 0; m < M; ++m) {
        if (isnan(sumsq[m]))
            return NAN;
        if (sumsq[m] > best)
            best = sumsq[m];
    }
    return (float)sqrt(best);
}

/* All M rows (row stride ldg floats): per-row sums of squares, then W. */
float orc_shared_scale(const float* g, int64_t d, int32_t M, int64_t ldg, double* sumsq_out)
{
    for (int32_t m = 0; m < M; ++m)
        sumsq_out[m] = orc_sum_of_squares(g + (int64_t)m * ldg, d);
    return orc_max_norm(sumsq_out, M);
}

/* ------------------------------------------------------------------------ */
/* Tables derived from W: inv_k = fl32(s_k / W), deq_k = fl32(W / (M s_k)).  */
/* Returns 1 on the zero path (W not positive-finite, or s_min/W overflows), */
/* in which case both tables are zero.                                        */
/* ------------------------------------------------------------------------ */
int orc_tables(float W, const float* scales, int32_t K, int32_t M, float* inv, float* deq)
{
    int zero = !(W > 0.0f) || !(W <= FLT_MAX);
    if (!zero) {
        float first = scales[0] / W;
        zero = !(first <= FLT_MAX);
    }
    for (int32_t k = 0; k < K; ++k) {
        if (zero) {
            inv[k] = 0.0f;
            deq[k] = 0.0f;
        } else {
            inv[k] = scales[k] / W;
            deq[k] = W / ((float)M * scales[k]);
        }
    }
    return zero;
}

static int usable_magnitude(float a)
{
    return a > 0.0f && a <= FLT_MAX; /* false for 0, NaN and inf */
}

/* ------------------------------------------------------------------------ */
/* Per-coordinate scale rule, Eq. (11): the largest s_k in S with            */
/*   s_k <= (W / |v_i|) * min_j s_j,  i.e.  (|v_i| * s_k / W) <= s_0,         */
/* evaluated as fl32(|v_i| * inv_k) <= s_0.  No qualifying scale -> index 0;  */
/* a zero / non-finite coordinate -> the largest index K-1.                   */
/* ------------------------------------------------------------------------ */
void orc_scale_index_worker(const float* v, int64_t n, float W, const float* scales, int32_t K,
                            uint8_t* kstar)
{
    float inv[16], deq[16];
    int zero = orc_tables(W, scales, K, 1, inv, deq);
    float s0 = scales[0];
    for (int64_t i = 0; i < n; ++i) {
        float a = fabsf(v[i]);
        int chosen = K - 1;
        if (!zero && usable_magnitude(a)) {
            chosen = 0;
            for (int32_t k = K - 1; k >= 0; --k) {
                float x = a * inv[k];
                if (x <= s0) {
                    chosen = k;
                    break;
                }
            }
        }
        kstar[i] = (uint8_t)chosen;
    }
}

/* Scale sharing (Sec. 3.2, Algorithm 2): s*_i = min over workers of s*^m_i,
 * i.e. the smallest per-worker index. kstar_scratch holds n bytes. */
void orc_scale_index_shared(const float* g, int64_t d, int32_t M, int64_t ldg, float W,
                            const float* scales, int32_t K, uint8_t* idx, uint8_t* kstar_scratch)
{
    for (int64_t i = 0; i < d; ++i)
        idx[i] = (uint8_t)(K - 1);
    for (int32_t m = 0; m < M; ++m) {
        orc_scale_index_worker(g + (int64_t)m * ldg, d, W, scales, K, kstar_scratch);
        for (int64_t i = 0; i < d; ++i)
            if (kstar_scratch[i] < idx[i])
                idx[i] = kstar_scratch[i];
    }
}

/* ------------------------------------------------------------------------ */
/* Stochastic quantiser, Eq. (7)-(8) (single scale) and Eq. (10), (12)       */
/* (multi-scale with the shared per-coordinate scale).  Writes the integer   */
/* code zeta_i = sign(v_i) * s* * xi_i in {sign*l, sign*(l+1)}.               */
/*   v      : the n coordinates i0 .. i0+n-1 of worker `worker`              */
/*   idx    : shared scale index per coordinate (NULL: always scale 0);      */
/*            indices >= K are read as K-1                                     */
/* ------------------------------------------------------------------------ */
void orc_quantize(const float* v, int64_t n, int64_t i0, uint32_t worker, float W,
                  const float* scales, int32_t K, const uint8_t* idx, uint64_t seed, int8_t* codes)
{
    float inv[16], deq[16];
    int zero = orc_tables(W, scales, K, 1, inv, deq);
    float s0 = scales[0];
    for (int64_t j = 0; j < n; ++j) {
        float vi = v[j];
        float a = fabsf(vi);
        if (zero || !usable_magnitude(a)) {
            codes[j] = 0;
            continue;
        }
        int k = 0;
        if (idx != NULL) {
            k = idx[j];
            if (k > K - 1)
                k = K - 1;
        }
        /* x = a * s / W : the position of |v_i| on the grid of s* levels */
        float x = a * inv[k];
        if (x > s0)
            x = s0;
        float lf = floorf(x);          /* level l with x in [l, l+1) */
        int32_t l = (int32_t)lf;
        float p = x - lf;              /* p(a, s) = a s - l, exact */
        uint32_t t = (uint32_t)(p * 4294967296.0f); /* floor(p * 2^32) */
        uint32_t r = orc_uniform_word(seed, worker, (uint64_t)(i0 + j));
        int32_t mag = l + (r < t ? 1 : 0); /* l+1 with probability p */
        codes[j] = (int8_t)(vi < 0.0f ? -mag : mag);
    }
}

/* ------------------------------------------------------------------------ */
/* The all-reduce of Algorithm 1/2 on integer codes: an exact int32 sum.     */
/* ------------------------------------------------------------------------ */
void orc_sum_codes(const int8_t* codes, int64_t n, int32_t rows, int64_t ldc, int32_t* sum)
{
    for (int64_t i = 0; i < n; ++i) {
        int32_t acc = 0;
        for (int32_t m = 0; m < rows; ++m)
            acc += (int32_t)codes[(int64_t)m * ldc + i];
        sum[i] = acc;
    }
}

/* ------------------------------------------------------------------------ */
/* Reconstruction, Eq. (9) / Eq. (13) with the 1/M of Algorithm 1/2:          */
/*   ghat_i = W * (sum_m zeta^m_i) / (M * s*_i) = fl32(sum_i * deq_k).        */
/* ------------------------------------------------------------------------ */
void orc_dequantize(const int32_t* sum, int64_t n, int32_t M, float W, const float* scales,
                    int32_t K, const uint8_t* idx, float* out)
{
    float inv[16], deq[16];
    orc_tables(W, scales, K, M, inv, deq);
    for (int64_t i = 0; i < n; ++i) {
        int k = 0;
        if (idx != NULL) {
            k = idx[i];
            if (k > K - 1)
                k = K - 1;
        }
        out[i] = (float)sum[i] * deq[k];
    }
}

/* ------------------------------------------------------------------------ */
/* GlobalRandK selection (Sec. 3.3-3.4): keys, then the K smallest.          */
/* ------------------------------------------------------------------------ */

/* The 64-bit selection keys of coordinates i0 .. i0+n-1 as (hi, lo) words. */
void orc_randk_keys(uint64_t seed, int64_t i0, int64_t n, uint32_t* hi, uint32_t* lo)
{
    uint32_t key[2] = { (uint32_t)seed, (uint32_t)(seed >> 32) };
    for (int64_t j = 0; j < n; ++j) {
        uint64_t i = (uint64_t)(i0 + j);
        uint64_t block = i / 4;
        unsigned word = (unsigned)(i % 4);
        uint32_t ctr[4] = { (uint32_t)block, (uint32_t)(block >> 32), 0u, 2u };
        uint32_t out[4];
        orc_philox4x32_10(ctr, key, out);
        hi[j] = out[word];
        ctr[3] = 3u;
        orc_philox4x32_10(ctr, key, out);
        lo[j] = out[word];
    }
}

typedef struct { uint32_t hi, lo; uint32_t idx; } orc_key_t;

static int orc_key_cmp(const void* pa, const void* pb)
{
    const orc_key_t* a = (const orc_key_t*)pa;
    const orc_key_t* b = (const orc_key_t*)pb;
    if (a->hi != b->hi) return a->hi < b->hi ? -1 : 1;
    if (a->lo != b->lo) return a->lo < b->lo ? -1 : 1;
    if (a->idx != b->idx) return a->idx < b->idx ? -1 : 1;
    return 0;
}

static int orc_u32_cmp(const void* pa, const void* pb)
{
    uint32_t a = *(const uint32_t*)pa, b = *(const uint32_t*)pb;
    return a < b ? -1 : (a > b ? 1 : 0);
}

/* The K coordinates of [0, d) with the smallest (key, index), ascending.
 * scratch holds d entries of 12 bytes (orc_key_t). */
void orc_randk_select(int64_t d, int64_t K, uint64_t seed, uint32_t* out, void* scratch)
{
    orc_key_t* keys = (orc_key_t*)scratch;
    uint32_t hi, lo;
    for (int64_t i = 0; i < d; ++i) {
        orc_randk_keys(seed, i, 1, &hi, &lo);
        keys[i].hi = hi;
        keys[i].lo = lo;
        keys[i].idx = (uint32_t)i;
    }
    qsort(keys, (size_t)d, sizeof(orc_key_t), orc_key_cmp);
    for (int64_t j = 0; j < K; ++j)
        out[j] = keys[j].idx;
    qsort(out, (size_t)K, sizeof(uint32_t), orc_u32_cmp);
}

/* ------------------------------------------------------------------------ */
/* Sub-byte codes: packing, unpacking and the integer sum of packed rows.    */
/* ------------------------------------------------------------------------ */

void orc_pack_codes(const int8_t* codes, int64_t n, int32_t bits, uint8_t* out)
{
    int per = 8 / bits;
    uint32_t field = (1u << bits) - 1u;
    for (int64_t b = 0; b < (n + per - 1) / per; ++b)
        out[b] = 0;
    for (int64_t i = 0; i < n; ++i) {
        uint32_t v = (uint32_t)(int32_t)codes[i] & field;
        out[i / per] = (uint8_t)(out[i / per] | (v << ((i % per) * bits)));
    }
}

void orc_unpack_codes(const uint8_t* packed, int64_t n, int32_t bits, int8_t* out)
{
    int per = 8 / bits;
    uint32_t field = (1u << bits) - 1u;
    for (int64_t i = 0; i < n; ++i) {
        uint32_t v = ((uint32_t)packed[i / per] >> ((i % per) * bits)) & field;
        int32_t x = (int32_t)v;
        if (x >= (1 << (bits - 1)))
            x -= 1 << bits; /* sign extension */
        out[i] = (int8_t)x;
    }
}

/* sum_i = sum over rows of the unpacked code of coordinate i (row stride ldp bytes). */
void orc_sum_packed(const uint8_t* packed, int64_t n, int32_t rows, int64_t ldp, int32_t bits, int32_t* sum)
{
    for (int64_t i = 0; i < n; ++i)
        sum[i] = 0;
    int8_t one;
    for (int32_t m = 0; m < rows; ++m) {
        const uint8_t* row = packed + (int64_t)m * ldp;
        for (int64_t i = 0; i < n; ++i) {
            int per = 8 / bits;
            uint8_t byte = row[i / per];
            uint8_t sub[1] = { (uint8_t)(byte >> ((i % per) * bits)) };
            orc_unpack_codes(sub, 1, bits, &one);
            sum[i] += one;
        }
    }
}
