/*
 * Seeded synthetic-input generator shared by the CPU oracle and the GPU path.
 *
 * It holds none of the decoding method's arithmetic: it only turns
 * (seed, stream, index) into numbers.  Every synthetic tensor (weights,
 * prefix K/V, token ids, ragged lengths) is drawn here, once, on the host,
 * so both sides consume identical bits.
 *
 * Counter-based generator: Philox-4x32 with 10 rounds, as published by
 * Salmon, Moraes, Dror and Shaw, "Parallel Random Numbers: As Easy as
 * 1, 2, 3" (SC'11).  Key = (seed, stream); counter = (block index low,
 * block index high, 0, 0); one block yields four 32-bit words.
 *
 *  - normals: words (w0,w1) and (w2,w3) of block i/4 feed Box-Muller in
 *    double precision, u = (w + 0.5) / 2^32; element i takes
 *    r*cos(2*pi*u2) / r*sin(2*pi*u2) of its pair.  The value times `std`
 *    is rounded to float (round-to-nearest-even), then to bfloat16 (RNE).
 *  - integers in [lo, hi]: word i%4 of block i/4, mapped by
 *    lo + floor(w * (hi - lo + 1) / 2^32).
 */
#include <stdint.h>
#include <string.h>
#include <math.h>

#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

void synth_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4])
{
    uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
    uint32_t k0 = key_in[0], k1 = key_in[1];
    for (int round = 0; round < 10; ++round) {
        uint64_t p0 = (uint64_t)PHILOX_M0 * c0;
        uint64_t p1 = (uint64_t)PHILOX_M1 * c2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t n0 = hi1 ^ c1 ^ k0;
        uint32_t n1 = lo1;
        uint32_t n2 = hi0 ^ c3 ^ k1;
        uint32_t n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
        k0 += PHILOX_W0;
        k1 += PHILOX_W1;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

static inline void block_words(uint32_t seed, uint32_t stream, uint64_t block, uint32_t w[4])
{
    uint32_t ctr[4] = { (uint32_t)block, (uint32_t)(block >> 32), 0u, 0u };
    uint32_t key[2] = { seed, stream };
    synth_philox4x32_10(ctr, key, w);
}

/* float -> bfloat16 bits, round to nearest even (inputs here are finite). */
uint16_t synth_f32_to_bf16(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

static inline void normals4(uint32_t seed, uint32_t stream, uint64_t block, double z[4])
{
    uint32_t w[4];
    block_words(seed, stream, block, w);
    const double two32 = 4294967296.0, two_pi = 6.283185307179586476925286766559;
    for (int p = 0; p < 2; ++p) {
        double u1 = ((double)w[2 * p] + 0.5) / two32;
        double u2 = ((double)w[2 * p + 1] + 0.5) / two32;
        double r = sqrt(-2.0 * log(u1));
        z[2 * p] = r * cos(two_pi * u2);
        z[2 * p + 1] = r * sin(two_pi * u2);
    }
}

void synth_normal_f64(uint32_t seed, uint32_t stream, uint64_t offset, uint64_t n, double* out)
{
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < (int64_t)n; ++i) {
        uint64_t e = offset + (uint64_t)i;
        double z[4];
        normals4(seed, stream, e >> 2, z);
        out[i] = z[e & 3];
    }
}

void synth_normal_bf16(uint32_t seed, uint32_t stream, uint64_t offset, uint64_t n, double std, uint16_t* out)
{
    /* Whole 4-element blocks are generated once each; the ragged head and
       tail fall back to per-element generation. */
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < (int64_t)n; ++i) {
        uint64_t e = offset + (uint64_t)i;
        if ((e & 3) != 0 && i != 0) continue;          /* handled with its block */
        double z[4];
        normals4(seed, stream, e >> 2, z);
        for (uint64_t j = e & 3; j < 4; ++j) {
            int64_t dst = i + (int64_t)(j - (e & 3));
            if (dst >= (int64_t)n) break;
            out[dst] = synth_f32_to_bf16((float)(z[j] * std));
        }
    }
}

void synth_uniform_int(uint32_t seed, uint32_t stream, uint64_t offset, uint64_t n, int32_t lo, int32_t hi, int32_t* out)
{
    uint64_t range = (uint64_t)((int64_t)hi - (int64_t)lo + 1);
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < (int64_t)n; ++i) {
        uint64_t e = offset + (uint64_t)i;
        uint32_t w[4];
        block_words(seed, stream, e >> 2, w);
        out[i] = (int32_t)((int64_t)lo + (int64_t)(((uint64_t)w[e & 3] * range) >> 32));
    }
}
