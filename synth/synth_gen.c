/*
 * The counter-based value generator of synth/__init__.py, in C for sizes the
 * numpy version takes minutes on (hundreds of millions of values per session
 * batch).  Same definition, step for step (SplitMix64 finaliser: Steele, Lea
 * and Flood, OOPSLA 2014):
 *
 *   c     = kind << 62 | sid << 42 | layer << 36 | head << 32 | token << 8 | dim
 *   h     = mix(mix(seed) ^ c),   mix(x) = finaliser of x + 0x9E3779B97F4A7C15
 *   s     = sum of the four 16-bit fields of h - 131070
 *   value = float32(s) * mult     (one float32 multiply, correctly rounded)
 *   bf16  = round to nearest even of the float32 bit pattern
 *
 * This file only draws numbers: it holds no attention arithmetic, no page
 * layout and no allocation policy.  Built with gcc by synth.build().
 */
#include <stdint.h>
#include <string.h>

static uint64_t mix(uint64_t x) {
    uint64_t z = x + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

static float value_of(uint64_t key, uint64_t c, float mult) {
    const uint64_t h = mix(key ^ c);
    const int64_t s = (int64_t)(h & 0xFFFF) + (int64_t)((h >> 16) & 0xFFFF) + (int64_t)((h >> 32) & 0xFFFF) +
                      (int64_t)(h >> 48) - 131070;
    const float f = (float)s;  /* exact: |s| < 2^24 */
    return f * mult;
}

static uint16_t bf16_bits(float x) {
    uint32_t b;
    memcpy(&b, &x, 4);
    return (uint16_t)(((uint64_t)b + 0x7FFF + ((b >> 16) & 1)) >> 16);
}

/*
 * K (kind 0) and V (kind 1) of one session and layer as logical arrays
 * [seq_len][num_kv_heads][head_dim]: uint16 bf16 bit patterns when bf16 != 0,
 * float32 otherwise.
 */
void synth_session_kv(uint64_t seed, int64_t sid, int64_t seq_len, int32_t layer, int32_t num_kv_heads,
                      int32_t head_dim, float mult, int32_t bf16, void* k_out, void* v_out) {
    const uint64_t key = mix(seed);
    const int64_t per_token = (int64_t)num_kv_heads * head_dim;
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < seq_len; ++t) {
        for (int32_t g = 0; g < num_kv_heads; ++g) {
            for (int32_t d = 0; d < head_dim; ++d) {
                const uint64_t base = ((uint64_t)sid << 42) | ((uint64_t)layer << 36) | ((uint64_t)g << 32) |
                                      ((uint64_t)t << 8) | (uint64_t)d;
                const float kf = value_of(key, base, mult);
                const float vf = value_of(key, (1ull << 62) | base, mult);
                const int64_t i = t * per_token + (int64_t)g * head_dim + d;
                if (bf16) {
                    ((uint16_t*)k_out)[i] = bf16_bits(kf);
                    ((uint16_t*)v_out)[i] = bf16_bits(vf);
                } else {
                    ((float*)k_out)[i] = kf;
                    ((float*)v_out)[i] = vf;
                }
            }
        }
    }
}
