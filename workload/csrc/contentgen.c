/* Content-addressed synthetic values, C version of workload/contentgen.py.
 *
 * Same definitions, bit for bit: SplitMix64 (Steele, Lea, Flood, OOPSLA 2014)
 * used as a counter-based generator, a prefix hash chain over token ids, and
 * an Irwin-Hall sum of twelve 16-bit uniforms rounded to bf16 with integer
 * operations.  Holds no attention or radix-tree arithmetic.  Built with gcc
 * and OpenMP; used to regenerate large inputs quickly on the host.
 */
#include <stdint.h>
#include <string.h>

#define CG_GAMMA 0x9E3779B97F4A7C15ULL
#define CG_STREAM_SALT 0xD1B54A32D192ED03ULL
#define CG_BASE_SALT 0x5851F42D4C957F2DULL
#define CG_IH_OFFSET 393210

static inline uint64_t cg_mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

uint64_t cg_base_hash(uint64_t seed) { return cg_mix64(seed ^ CG_BASE_SALT); }

void cg_prefix_hashes(const int32_t* tokens, int64_t n, uint64_t seed, uint64_t* out) {
  uint64_t h = cg_base_hash(seed);
  for (int64_t p = 0; p < n; ++p) {
    h = cg_mix64((h ^ (uint64_t)(int64_t)tokens[p]) + CG_GAMMA);
    out[p] = h;
  }
}

static inline uint16_t cg_f32_bits_to_bf16_rne(uint32_t b) {
  return (uint16_t)(((uint64_t)b + 0x7FFFu + ((b >> 16) & 1u)) >> 16);
}

static inline uint16_t cg_value(uint64_t key, uint64_t e) {
  int64_t acc = 0;
  for (uint64_t k = 0; k < 3; ++k) {
    uint64_t w = cg_mix64(key + (3 * e + k + 1) * CG_GAMMA);
    acc += (int64_t)(w & 0xFFFF) + (int64_t)((w >> 16) & 0xFFFF) +
           (int64_t)((w >> 32) & 0xFFFF) + (int64_t)(w >> 48);
  }
  float z = (float)(int32_t)(acc - CG_IH_OFFSET) * (1.0f / 65536.0f);
  uint32_t bits;
  memcpy(&bits, &z, 4);
  return cg_f32_bits_to_bf16_rne(bits);
}

void cg_values_bf16(const uint64_t* hashes, int64_t n, int32_t stream, int32_t n_elem,
                    uint16_t* out) {
#pragma omp parallel for schedule(static)
  for (int64_t p = 0; p < n; ++p) {
    uint64_t key = cg_mix64(hashes[p] ^ ((uint64_t)stream * CG_STREAM_SALT));
    uint16_t* o = out + p * (int64_t)n_elem;
    for (int32_t e = 0; e < n_elem; ++e) o[e] = cg_value(key, (uint64_t)e);
  }
}

/* Token ids for segments of synthetic text: token i of the run named by key
 * is mix(key + (i + 1) * GAMMA) mod vocab. */
void cg_run_tokens(uint64_t key, int64_t n, int32_t vocab, int32_t* out) {
  for (int64_t i = 0; i < n; ++i)
    out[i] = (int32_t)(cg_mix64(key + (uint64_t)(i + 1) * CG_GAMMA) % (uint64_t)vocab);
}
