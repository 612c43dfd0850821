/*
 * Plain C restatement of the oracle's blockwise / groupwise E4M3 quantisation.
 * TEST INFRASTRUCTURE ONLY: it exists so that exhaustive and full-size checks
 * (about 1e9 elements) finish in seconds on the host.  It is pinned to the
 * numpy oracle (oracle/quant.py) and to torch's float8_e4m3fn cast by the CPU
 * test suite.  The HIP library never links or calls it.
 *
 * What it computes (paper section 2.1.1, Eq. (1); 128x128 weight blocks,
 * 1x128 per-token activation groups, fp32 scales):
 *   amax  = largest |x| of the block / group (bf16 widened exactly to fp32)
 *   scale = amax / 448 in IEEE fp32 (1.0 when amax == 0)
 *   code  = E4M3(fl32(x / scale)), round to nearest even on the E4M3 grid,
 *           saturating at 448, sign of x kept.
 *
 * The power-of-two (UE8M0) variant (section 2.4.3) replaces the scale by 2^k,
 * k the smallest integer with amax <= 448 * 2^k (clamped at -127; 1.0 for
 * amax == 0), and the quotient by the exact product x * 2^-k.
 *
 * Build: gcc -O2 -fopenmp -ffp-contract=off -fno-fast-math -shared -fPIC
 * (no flag that changes IEEE behaviour; x86-64 SSE keeps subnormals).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

static float bf16_to_f32(uint16_t h) {
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

/* E4M3 grid rounding of one fp32 value (RNE, saturate to 448, keep sign). */
static uint8_t e4m3_encode(float v) {
    uint32_t u;
    memcpy(&u, &v, 4);
    uint8_t sign = (uint8_t)((u >> 31) << 7);
    double a = fabs((double)v);          /* exact widening */
    if (isnan(a)) return 0x7F;
    if (a >= 448.0) return (uint8_t)(sign | 0x7E);
    int code;
    if (a < 0x1p-6) {
        /* subnormal grid, step 2^-9; nearbyint rounds half to even */
        code = (int)nearbyint(a * 0x1p9);
    } else {
        int e;
        double m = frexp(a, &e);         /* a = m * 2^e, m in [0.5, 1) */
        e -= 1;                          /* a = (2m) * 2^e, 2m in [1, 2) */
        int n = (int)nearbyint(ldexp(a, 3 - e));   /* in [8, 16] */
        code = ((e + 7) << 3) + (n - 8);
        (void)m;
    }
    if (code > 0x7E) code = 0x7E;
    return (uint8_t)(sign | code);
}

static float scale_of(float amax) {
    return amax == 0.0f ? 1.0f : amax / 448.0f;
}

/* W [n][ldw] bf16 bits -> q [n][ldq], scale [n/128][k/128].  n, k multiples of 128. */
void oracle_quant_weight_block128(const uint16_t* w, int64_t n, int64_t k, int64_t ldw,
                                  uint8_t* q, int64_t ldq, float* scale) {
    int64_t nbn = n / 128, nbk = k / 128;
    #pragma omp parallel for schedule(dynamic, 16)
    for (int64_t b = 0; b < nbn * nbk; ++b) {
        int64_t bi = b / nbk, bj = b % nbk;
        float amax = 0.0f;
        for (int64_t r = 0; r < 128; ++r)
            for (int64_t c = 0; c < 128; ++c) {
                float x = fabsf(bf16_to_f32(w[(bi * 128 + r) * ldw + bj * 128 + c]));
                if (x > amax) amax = x;
            }
        float s = scale_of(amax);
        scale[bi * nbk + bj] = s;
        for (int64_t r = 0; r < 128; ++r)
            for (int64_t c = 0; c < 128; ++c) {
                float x = bf16_to_f32(w[(bi * 128 + r) * ldw + bj * 128 + c]);
                volatile float quot = x / s;
                q[(bi * 128 + r) * ldq + bj * 128 + c] = e4m3_encode(quot);
            }
    }
}

/* A [m][lda] bf16 bits -> q [m][ldq], scale [k/128][ld_scale]. */
void oracle_quant_act_token_group128(const uint16_t* a, int64_t m, int64_t k, int64_t lda,
                                     uint8_t* q, int64_t ldq, float* scale, int64_t ld_scale) {
    int64_t ng = k / 128;
    #pragma omp parallel for schedule(dynamic, 64)
    for (int64_t t = 0; t < m * ng; ++t) {
        int64_t row = t / ng, g = t % ng;
        const uint16_t* src = a + row * lda + g * 128;
        float amax = 0.0f;
        for (int c = 0; c < 128; ++c) {
            float x = fabsf(bf16_to_f32(src[c]));
            if (x > amax) amax = x;
        }
        float s = scale_of(amax);
        scale[g * ld_scale + row] = s;
        for (int c = 0; c < 128; ++c) {
            volatile float quot = bf16_to_f32(src[c]) / s;
            q[row * ldq + g * 128 + c] = e4m3_encode(quot);
        }
    }
}

/* Element map alone: codes for x[i] quantised against the group maximum amax[i]. */
void oracle_e4m3_of_quotient(const uint16_t* x, const uint16_t* amax, int64_t count, uint8_t* out) {
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i) {
        float s = scale_of(fabsf(bf16_to_f32(amax[i])));
        volatile float quot = bf16_to_f32(x[i]) / s;
        out[i] = e4m3_encode(quot);
    }
}

/* Power-of-two scale: 2^k with k the smallest integer such that amax <= 448 * 2^k
 * (every comparison exact in double), clamped at 2^-127; 1.0 for amax == 0. */
static int pow2_k(float amax) {
    if (amax == 0.0f) return 0;
    int k = (int)ceil(log2((double)amax / 448.0));
    while ((double)amax > 448.0 * ldexp(1.0, k)) ++k;
    while ((double)amax <= 448.0 * ldexp(1.0, k - 1)) --k;
    return k < -127 ? -127 : k;
}

static uint8_t e4m3_pow2(float x, int k) {
    return e4m3_encode((float)ldexp((double)x, -k));   /* exact above 2^-126; below, E4M3 gives +-0 */
}

void oracle_quant_weight_block128_ue8m0(const uint16_t* w, int64_t n, int64_t k, int64_t ldw,
                                        uint8_t* q, int64_t ldq, float* scale) {
    int64_t nbn = n / 128, nbk = k / 128;
    #pragma omp parallel for schedule(dynamic, 16)
    for (int64_t b = 0; b < nbn * nbk; ++b) {
        int64_t bi = b / nbk, bj = b % nbk;
        float amax = 0.0f;
        for (int64_t r = 0; r < 128; ++r)
            for (int64_t c = 0; c < 128; ++c) {
                float x = fabsf(bf16_to_f32(w[(bi * 128 + r) * ldw + bj * 128 + c]));
                if (x > amax) amax = x;
            }
        int e = pow2_k(amax);
        scale[bi * nbk + bj] = ldexpf(1.0f, e);
        for (int64_t r = 0; r < 128; ++r)
            for (int64_t c = 0; c < 128; ++c)
                q[(bi * 128 + r) * ldq + bj * 128 + c] = e4m3_pow2(bf16_to_f32(w[(bi * 128 + r) * ldw + bj * 128 + c]), e);
    }
}

void oracle_quant_act_token_group128_ue8m0(const uint16_t* a, int64_t m, int64_t k, int64_t lda,
                                           uint8_t* q, int64_t ldq, float* scale, int64_t ld_scale) {
    int64_t ng = k / 128;
    #pragma omp parallel for schedule(dynamic, 64)
    for (int64_t t = 0; t < m * ng; ++t) {
        int64_t row = t / ng, g = t % ng;
        const uint16_t* src = a + row * lda + g * 128;
        float amax = 0.0f;
        for (int c = 0; c < 128; ++c) {
            float x = fabsf(bf16_to_f32(src[c]));
            if (x > amax) amax = x;
        }
        int e = pow2_k(amax);
        scale[g * ld_scale + row] = ldexpf(1.0f, e);
        for (int c = 0; c < 128; ++c) q[row * ldq + g * 128 + c] = e4m3_pow2(bf16_to_f32(src[c]), e);
    }
}
