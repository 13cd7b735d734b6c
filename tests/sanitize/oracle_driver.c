/*
 * The CPU oracle under AddressSanitizer and UndefinedBehaviorSanitizer (a
 * test driver, built and run by tests/test_oracle_sanitized.py; never part of
 * the product).  Every buffer is allocated at its exact size, so that a read
 * or write past any of them is reported.  It runs the worked examples of the
 * quantisers (Sec. 3.1-3.2), every stage of Algorithms 1-2 on small random
 * rows with zeros, negative zeros, NaN, infinities and denormals, sub-byte
 * packing (Sec. 5) and the GlobalRandK selection (Sec. 3.3), and checks the
 * results that those definitions fix.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

float orc_shared_scale(const float* g, int64_t d, int32_t M, int64_t ldg, double* sumsq_out);
int orc_tables(float W, const float* scales, int32_t K, int32_t M, float* inv, float* deq);
void orc_scale_index_shared(const float* g, int64_t d, int32_t M, int64_t ldg, float W, const float* scales,
                            int32_t K, uint8_t* idx, uint8_t* kstar_scratch);
void orc_quantize(const float* v, int64_t n, int64_t i0, uint32_t worker, float W, const float* scales, int32_t K,
                  const uint8_t* idx, uint64_t seed, int8_t* codes);
void orc_sum_codes(const int8_t* codes, int64_t n, int32_t rows, int64_t ldc, int32_t* sum);
void orc_dequantize(const int32_t* sum, int64_t n, int32_t M, float W, const float* scales, int32_t K,
                    const uint8_t* idx, float* out);
void orc_randk_keys(uint64_t seed, int64_t i0, int64_t n, uint32_t* hi, uint32_t* lo);
void orc_randk_select(int64_t d, int64_t K, uint64_t seed, uint32_t* out, void* scratch);
void orc_pack_codes(const int8_t* codes, int64_t n, int32_t bits, uint8_t* out);
void orc_unpack_codes(const uint8_t* packed, int64_t n, int32_t bits, int8_t* out);
void orc_sum_packed(const uint8_t* packed, int64_t n, int32_t rows, int64_t ldp, int32_t bits, int32_t* sum);

static int failures = 0;
#define CHECK(cond)                                                       \
    do {                                                                  \
        if (!(cond)) {                                                    \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
            ++failures;                                                   \
        }                                                                 \
    } while (0)

static void* xmalloc(size_t n)
{
    void* p = malloc(n ? n : 1);
    if (!p) {
        fprintf(stderr, "out of memory\n");
        exit(2);
    }
    return p;
}

static uint64_t rng = 0x2109124970ull;
static uint32_t next_u32(void)
{
    rng = rng * 6364136223846793005ull + 1442695040888963407ull;
    return (uint32_t)(rng >> 33);
}

/* Example A: M = 1, s = 5, g = (3, -4, 0, 0) * 2^-10: W = 5 * 2^-10, the codes
 * are (3, -4, 0, 0) for every seed and the reconstruction equals g. */
static void example_a(void)
{
    const float s = 5.0f;
    float* g = xmalloc(4 * sizeof(float));
    g[0] = ldexpf(3.0f, -10);
    g[1] = ldexpf(-4.0f, -10);
    g[2] = 0.0f;
    g[3] = 0.0f;
    double* S = xmalloc(sizeof(double));
    const float W = orc_shared_scale(g, 4, 1, 4, S);
    CHECK(W == ldexpf(5.0f, -10));
    int8_t* codes = xmalloc(4);
    int32_t* sum = xmalloc(4 * sizeof(int32_t));
    float* out = xmalloc(4 * sizeof(float));
    for (uint64_t seed = 0; seed < 64; ++seed) {
        orc_quantize(g, 4, 0, 0, W, &s, 1, NULL, seed, codes);
        CHECK(codes[0] == 3 && codes[1] == -4 && codes[2] == 0 && codes[3] == 0);
    }
    orc_sum_codes(codes, 4, 1, 4, sum);
    orc_dequantize(sum, 4, 1, W, &s, 1, NULL, out);
    for (int i = 0; i < 4; ++i)
        CHECK(out[i] == g[i]);
    free(g), free(S), free(codes), free(sum), free(out);
}

/* Example B: s = 127, g = (2^-3, 0, 0, 0): |g_0| = W gives code 127. */
static void example_b(void)
{
    const float s = 127.0f;
    float* g = xmalloc(4 * sizeof(float));
    memset(g, 0, 4 * sizeof(float));
    g[0] = 0.125f;
    double* S = xmalloc(sizeof(double));
    const float W = orc_shared_scale(g, 4, 1, 4, S);
    int8_t* codes = xmalloc(4);
    orc_quantize(g, 4, 0, 0, W, &s, 1, NULL, 7, codes);
    CHECK(W == 0.125f && codes[0] == 127 && codes[1] == 0);
    free(g), free(S), free(codes);
}

/* Example C: s = 3, g = 0.5 * (1, -1, 1, -1): every code is +-1 or +-2 with
 * the sign of g, both levels occurring over many seeds. */
static void example_c(void)
{
    const float s = 3.0f;
    float* g = xmalloc(4 * sizeof(float));
    for (int i = 0; i < 4; ++i)
        g[i] = (i & 1) ? -0.5f : 0.5f;
    double* S = xmalloc(sizeof(double));
    const float W = orc_shared_scale(g, 4, 1, 4, S);
    CHECK(W == 1.0f);
    int8_t* codes = xmalloc(4);
    int ones = 0, twos = 0;
    for (uint64_t seed = 0; seed < 256; ++seed) {
        orc_quantize(g, 4, 0, 0, W, &s, 1, NULL, seed, codes);
        for (int i = 0; i < 4; ++i) {
            const int mag = abs(codes[i]);
            CHECK(mag == 1 || mag == 2);
            CHECK((codes[i] < 0) == (g[i] < 0.0f));
            ones += mag == 1;
            twos += mag == 2;
        }
    }
    CHECK(ones > 300 && twos > 300);
    free(g), free(S), free(codes);
}

/* Example D: several scales, W = 1, S = (7, 112): |v| = 1/64 takes scale
 * index 1, |v| = 1/4 index 0, |v| = 1/16 index 1 with the deterministic top
 * code 7; shared by two workers the index is the minimum. */
static void example_d(void)
{
    const float S2[2] = {7.0f, 112.0f};
    float* g = xmalloc(6 * sizeof(float));
    const float a[3] = {1.0f / 64, 0.25f, 1.0f / 16};
    for (int i = 0; i < 3; ++i) {
        g[i] = a[i];
        g[3 + i] = a[(i + 1) % 3];
    }
    uint8_t* idx = xmalloc(3);
    uint8_t* scratch = xmalloc(3);
    orc_scale_index_shared(g, 3, 1, 3, 1.0f, S2, 2, idx, scratch);
    CHECK(idx[0] == 1 && idx[1] == 0 && idx[2] == 1);
    int8_t* codes = xmalloc(3);
    orc_quantize(g, 3, 0, 0, 1.0f, S2, 2, idx, 11, codes);
    CHECK(codes[2] == 7 && (codes[0] == 1 || codes[0] == 2) && (codes[1] == 1 || codes[1] == 2));
    orc_scale_index_shared(g, 3, 2, 3, 1.0f, S2, 2, idx, scratch);
    CHECK(idx[0] == 0 && idx[1] == 0 && idx[2] == 1);
    free(g), free(idx), free(scratch), free(codes);
}

static float random_value(void)
{
    const uint32_t u = next_u32() % 100;
    if (u < 5)
        return 0.0f;
    if (u < 7)
        return -0.0f;
    if (u < 8)
        return NAN;
    if (u < 9)
        return (next_u32() & 1) ? INFINITY : -INFINITY;
    if (u < 12)
        return ldexpf((float)(next_u32() % 1000 + 1), -149 + 0) * 1.0f; /* denormals */
    const float x = ldexpf((float)((int32_t)(next_u32() % 2000001) - 1000000), -20 - (int)(next_u32() % 20));
    return x;
}

/* Every stage of Algorithms 1-2 on small random rows (finite rows, and rows
 * holding NaN or infinity, which select the zero path). */
static void random_rows(void)
{
    const int64_t dims[] = {1, 2, 7, 8, 9, 100, 1001};
    const float scales[4] = {7.0f, 112.0f, 1792.0f, 28672.0f};
    for (size_t di = 0; di < sizeof dims / sizeof dims[0]; ++di) {
        const int64_t d = dims[di];
        for (int finite = 0; finite < 2; ++finite)
            for (int32_t K = 1; K <= 4; K += 3) {
                const int32_t M = 3;
                float* g = xmalloc((size_t)(M * d) * sizeof(float));
                for (int64_t i = 0; i < M * d; ++i) {
                    float x = random_value();
                    if (finite && !isfinite(x))
                        x = 0.5f;
                    g[i] = x;
                }
                double* S = xmalloc((size_t)M * sizeof(double));
                const float W = orc_shared_scale(g, d, M, d, S);
                float* inv = xmalloc((size_t)K * sizeof(float));
                float* deq = xmalloc((size_t)K * sizeof(float));
                const int zero = orc_tables(W, scales, K, M, inv, deq);
                CHECK(zero == !(isfinite(W) && W > 0.0f));
                uint8_t* idx = NULL;
                if (K > 1) {
                    idx = xmalloc((size_t)d);
                    uint8_t* scratch = xmalloc((size_t)d);
                    orc_scale_index_shared(g, d, M, d, W, scales, K, idx, scratch);
                    for (int64_t i = 0; i < d; ++i)
                        CHECK(idx[i] < K);
                    free(scratch);
                }
                int8_t* codes = xmalloc((size_t)(M * d));
                for (int32_t m = 0; m < M; ++m)
                    orc_quantize(g + m * d, d, 0, (uint32_t)m, W, scales, K, idx, 99, codes + m * d);
                int32_t* sum = xmalloc((size_t)d * sizeof(int32_t));
                orc_sum_codes(codes, d, M, d, sum);
                float* out = xmalloc((size_t)d * sizeof(float));
                orc_dequantize(sum, d, M, W, scales, K, idx, out);
                for (int64_t i = 0; i < d; ++i) {
                    int32_t t = 0;
                    for (int32_t m = 0; m < M; ++m) {
                        const int8_t c = codes[m * d + i];
                        CHECK(abs(c) <= (int)scales[0]);
                        if (zero || !isfinite(g[m * d + i]) || g[m * d + i] == 0.0f)
                            CHECK(c == 0);
                        t += c;
                    }
                    CHECK(sum[i] == t);
                    CHECK(isfinite(out[i]));
                }
                free(g), free(S), free(inv), free(deq), free(idx), free(codes), free(sum), free(out);
            }
    }
}

/* Packing: every code of a field width round-trips at ragged lengths, and the
 * packed rows sum to the int8 rows' sum. */
static void packing(void)
{
    const int32_t widths[2] = {4, 2};
    for (int w = 0; w < 2; ++w) {
        const int32_t bits = widths[w];
        const int per = 8 / bits;
        const int lo = -(1 << (bits - 1)), hi = (1 << (bits - 1)) - 1;
        for (int64_t n = 1; n <= 37; ++n) {
            const int32_t rows = 3;
            const int64_t ldp = (n + per - 1) / per;
            int8_t* codes = xmalloc((size_t)(rows * n));
            for (int64_t i = 0; i < rows * n; ++i)
                codes[i] = (int8_t)(lo + (int)(next_u32() % (uint32_t)(hi - lo + 1)));
            uint8_t* packed = xmalloc((size_t)(rows * ldp));
            for (int32_t r = 0; r < rows; ++r)
                orc_pack_codes(codes + r * n, n, bits, packed + r * ldp);
            int8_t* back = xmalloc((size_t)n);
            for (int32_t r = 0; r < rows; ++r) {
                orc_unpack_codes(packed + r * ldp, n, bits, back);
                CHECK(memcmp(back, codes + r * n, (size_t)n) == 0);
            }
            int32_t* s1 = xmalloc((size_t)n * sizeof(int32_t));
            int32_t* s2 = xmalloc((size_t)n * sizeof(int32_t));
            orc_sum_codes(codes, n, rows, n, s1);
            orc_sum_packed(packed, n, rows, ldp, bits, s2);
            CHECK(memcmp(s1, s2, (size_t)n * sizeof(int32_t)) == 0);
            free(codes), free(packed), free(back), free(s1), free(s2);
        }
    }
}

/* GlobalRandK: the K smallest keys, ascending coordinates, all distinct;
 * K = d takes every coordinate. */
static void randk(void)
{
    const int64_t d = 1000;
    const int64_t Ks[3] = {1, 17, 1000};
    for (int k = 0; k < 3; ++k) {
        const int64_t K = Ks[k];
        uint32_t* sel = xmalloc((size_t)K * sizeof(uint32_t));
        void* scratch = xmalloc((size_t)d * 12);
        orc_randk_select(d, K, 42, sel, scratch);
        for (int64_t j = 0; j < K; ++j) {
            CHECK(sel[j] < d);
            if (j > 0)
                CHECK(sel[j] > sel[j - 1]);
        }
        if (K == d)
            for (int64_t j = 0; j < K; ++j)
                CHECK(sel[j] == (uint32_t)j);
        free(sel), free(scratch);
    }
    uint32_t* hi = xmalloc(5 * sizeof(uint32_t));
    uint32_t* lo = xmalloc(5 * sizeof(uint32_t));
    orc_randk_keys(42, 3, 5, hi, lo);
    free(hi), free(lo);
}

int main(void)
{
    example_a();
    example_b();
    example_c();
    example_d();
    random_rows();
    packing();
    randk();
    if (failures) {
        fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    printf("oracle sanitized run: ok\n");
    return 0;
}
