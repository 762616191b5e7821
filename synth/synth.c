/*
 * Seeded synthetic inputs shared by the oracle and the GPU path: model
 * weights drawn from N(0, std) and uniform random prompt token ids.
 *
 * This file holds none of the decoding method's arithmetic.  It only turns
 * (seed, tensor id, element index) into numbers, so that both sides of a
 * parity test receive bit-identical inputs.
 *
 * Random source: Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random
 * numbers: as easy as 1, 2, 3", SC'11), written from its published
 * description.  Normals: inversion of the normal CDF on 16-bit uniforms.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

static void philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
    uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
    uint32_t k0 = key_in[0], k1 = key_in[1];
    for (int round = 0; round < 10; ++round) {
        uint64_t p0 = (uint64_t)0xD2511F53u * c0;
        uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t n0 = hi1 ^ c1 ^ k0;
        uint32_t n2 = hi0 ^ c3 ^ k1;
        c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Exposed for the generator's own known-answer test. */
void synth_philox(const uint32_t *ctr, const uint32_t *key, uint32_t *out) {
    philox4x32_10(ctr, key, out);
}

static inline uint16_t f32_to_bf16_rne(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return 0x7FC0; /* NaN */
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

/*
 * Normal draws by table inversion: a 16-bit uniform u selects the midpoint
 * quantile Phi^-1((u + 0.5) / 65536) of the standard normal.  The table is
 * computed once by bisection on Phi(x) = erfc(-x / sqrt 2) / 2 in double.
 * Each Philox call yields eight 16-bit uniforms, so eight normals: element i
 * comes from call i / 8, word (i % 8) / 2, half i % 2 (low half first).
 * Draws are truncated at about 4.3 sigma, which is immaterial for a random
 * initialisation.
 */
static double g_quantile[65536];
static int g_quantile_ready = 0;

static void build_quantile_table(void) {
    if (g_quantile_ready) return;
    for (int i = 0; i < 65536; ++i) {
        double p = ((double)i + 0.5) / 65536.0;
        double lo = -10.0, hi = 10.0;
        for (int it = 0; it < 80; ++it) {
            double mid = 0.5 * (lo + hi);
            double phi = 0.5 * erfc(-mid * 0.70710678118654752440);
            if (phi < p) lo = mid; else hi = mid;
        }
        g_quantile[i] = 0.5 * (lo + hi);
    }
    g_quantile_ready = 1;
}

static inline void normals8(uint64_t call, uint32_t tensor_id, uint32_t seed, double out[8]) {
    uint32_t ctr[4] = {(uint32_t)call, (uint32_t)(call >> 32), tensor_id, 0xB0C5u};
    uint32_t key[2] = {seed, 0x5EED5EEDu};
    uint32_t w[4];
    philox4x32_10(ctr, key, w);
    for (int j = 0; j < 4; ++j) {
        out[2 * j] = g_quantile[w[j] & 0xFFFFu];
        out[2 * j + 1] = g_quantile[w[j] >> 16];
    }
}

/* out[i] = bf16_rne(float(std * normal(seed, tensor_id, i))), i in [0, n). */
void synth_normal_bf16(uint16_t *out, int64_t n, uint32_t seed, uint32_t tensor_id, double std) {
    build_quantile_table();
    int64_t calls = (n + 7) / 8;
#pragma omp parallel for schedule(static)
    for (int64_t c = 0; c < calls; ++c) {
        double v[8];
        normals8((uint64_t)c, tensor_id, seed, v);
        for (int j = 0; j < 8; ++j) {
            int64_t i = c * 8 + j;
            if (i < n) out[i] = f32_to_bf16_rne((float)(std * v[j]));
        }
    }
}

/* out[i] = float(std * normal(seed, tensor_id, i)). */
void synth_normal_f32(float *out, int64_t n, uint32_t seed, uint32_t tensor_id, double std) {
    build_quantile_table();
    int64_t calls = (n + 7) / 8;
#pragma omp parallel for schedule(static)
    for (int64_t c = 0; c < calls; ++c) {
        double v[8];
        normals8((uint64_t)c, tensor_id, seed, v);
        for (int j = 0; j < 8; ++j) {
            int64_t i = c * 8 + j;
            if (i < n) out[i] = (float)(std * v[j]);
        }
    }
}

/* Uniform token ids: out[i] = floor(word0 * vocab / 2^32). */
void synth_tokens(int32_t *out, int64_t n, int32_t vocab, uint32_t seed) {
    for (int64_t i = 0; i < n; ++i) {
        uint32_t ctr[4] = {(uint32_t)i, (uint32_t)((uint64_t)i >> 32), 1u, 0u};
        uint32_t key[2] = {seed, 0u};
        uint32_t w[4];
        philox4x32_10(ctr, key, w);
        out[i] = (int32_t)(((uint64_t)w[0] * (uint64_t)vocab) >> 32);
    }
}
