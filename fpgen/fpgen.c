/*
 * Seeded synthetic-input generator (host C, built with gcc).
 *
 * Produces the synthetic weights, norm gains and prompt hidden states that
 * stand in for a real checkpoint and real prompts.  It holds none of the
 * fingerprint layer's arithmetic: it only draws numbers.
 *
 * Generator: SplitMix64 (Steele, Lea & Flood, "Fast splittable pseudorandom
 * number generators", OOPSLA 2014) used as a counter-based hash.
 *   mix64(z): z ^= z>>30; z *= 0xBF58476D1CE4E5B9; z ^= z>>27;
 *             z *= 0x94D049BB133111EB; z ^= z>>31
 *   key      = mix64(mix64(seed) + G * (((layer+1) << 8) | tensor))
 *   word c   = mix64(key + G * (c+1))          (G = 0x9E3779B97F4A7C15)
 * Element i sums the 12 unsigned 16-bit lanes of words 3i, 3i+1, 3i+2
 * (Irwin-Hall of 12 uniforms), S in [0, 786420]; z = float(S - 393210) * 2^-16
 * is exactly representable, has mean 0 and variance 1 - 2^-32.
 * The stored value is bf16_rne(float(mean + float(sigma * z))).
 */
#include <stdint.h>
#include <stddef.h>

#define FPGEN_GAMMA 0x9E3779B97F4A7C15ULL

static inline uint64_t mix64(uint64_t z) {
    z ^= z >> 30; z *= 0xBF58476D1CE4E5B9ULL;
    z ^= z >> 27; z *= 0x94D049BB133111EBULL;
    z ^= z >> 31;
    return z;
}

static inline uint16_t bf16_rne_bits(float f) {
    union { float f; uint32_t u; } v; v.f = f;
    uint32_t u = v.u;
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

uint64_t fpgen_mix64(uint64_t z) { return mix64(z); }

uint64_t fpgen_key(uint64_t seed, int32_t layer, int32_t tensor) {
    uint64_t id = ((uint64_t)(int64_t)(layer + 1) << 8) | (uint64_t)(uint32_t)tensor;
    return mix64(mix64(seed) + FPGEN_GAMMA * id);
}

/* z-scores (exact float32) for elements [start, start+n) of one stream */
void fpgen_z(uint64_t seed, int32_t layer, int32_t tensor, int64_t start, int64_t n, float* out) {
    uint64_t key = fpgen_key(seed, layer, tensor);
    #pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < n; ++j) {
        uint64_t i = (uint64_t)(start + j);
        uint32_t s = 0;
        for (int c = 0; c < 3; ++c) {
            uint64_t w = mix64(key + FPGEN_GAMMA * (3 * i + (uint64_t)c + 1));
            s += (uint32_t)(w & 0xFFFF) + (uint32_t)((w >> 16) & 0xFFFF)
               + (uint32_t)((w >> 32) & 0xFFFF) + (uint32_t)(w >> 48);
        }
        out[j] = (float)((int32_t)s - 393210) * (1.0f / 65536.0f);
    }
}

/* bf16 bit patterns bf16_rne(float(mean + float(sigma*z))) */
void fpgen_bf16(uint64_t seed, int32_t layer, int32_t tensor, int64_t start, int64_t n,
                float mean, float sigma, uint16_t* out) {
    uint64_t key = fpgen_key(seed, layer, tensor);
    #pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < n; ++j) {
        uint64_t i = (uint64_t)(start + j);
        uint32_t s = 0;
        for (int c = 0; c < 3; ++c) {
            uint64_t w = mix64(key + FPGEN_GAMMA * (3 * i + (uint64_t)c + 1));
            s += (uint32_t)(w & 0xFFFF) + (uint32_t)((w >> 16) & 0xFFFF)
               + (uint32_t)((w >> 32) & 0xFFFF) + (uint32_t)(w >> 48);
        }
        float z = (float)((int32_t)s - 393210) * (1.0f / 65536.0f);
        float t = sigma * z;      /* rounded product; built with -ffp-contract=off */
        out[j] = bf16_rne_bits(mean + t);
    }
}
