/* Host implementation of the seeded input generator (bitwise the same values as the torch
 * implementation in wisp_inputs/__init__.py): a 32-bit integer mixer over element indices,
 * then a table lookup (normal quantiles) or an 8-bit field (synthetic KV).
 * Holds none of the verification method's arithmetic. */
#include <stdint.h>
#include <string.h>

static inline uint32_t mix32(uint32_t h) {
  h ^= h >> 16;
  h *= 0x45D9F3Bu;
  h ^= h >> 16;
  h *= 0x45D9F3Bu;
  h ^= h >> 16;
  return h;
}

static inline uint32_t hashed(uint32_t k0, uint32_t k1, uint64_t i) {
  return mix32(mix32((uint32_t)i ^ k0) ^ k1);
}

void gen_table16(const uint16_t *table, uint32_t k0, uint32_t k1, uint64_t start, uint64_t n, uint16_t *out) {
#pragma omp parallel for schedule(static)
  for (int64_t e = 0; e < (int64_t)n; e++) out[e] = table[hashed(k0, k1, start + (uint64_t)e) >> 16];
}

void gen_table32(const float *table, uint32_t k0, uint32_t k1, uint64_t start, uint64_t n, float *out) {
#pragma omp parallel for schedule(static)
  for (int64_t e = 0; e < (int64_t)n; e++) out[e] = table[hashed(k0, k1, start + (uint64_t)e) >> 16];
}

/* (2k - 255) / 128 with k the top 8 bits: exact in fp32 and bf16 */
void gen_kv32(uint32_t k0, uint32_t k1, uint64_t start, uint64_t n, float *out) {
#pragma omp parallel for schedule(static)
  for (int64_t e = 0; e < (int64_t)n; e++) {
    float k8 = (float)(hashed(k0, k1, start + (uint64_t)e) >> 24);
    out[e] = (k8 * 2.0f - 255.0f) * (1.0f / 128.0f);
  }
}

void gen_kv16(uint32_t k0, uint32_t k1, uint64_t start, uint64_t n, uint16_t *out) {
#pragma omp parallel for schedule(static)
  for (int64_t e = 0; e < (int64_t)n; e++) {
    float k8 = (float)(hashed(k0, k1, start + (uint64_t)e) >> 24);
    float v = (k8 * 2.0f - 255.0f) * (1.0f / 128.0f);
    uint32_t u;
    memcpy(&u, &v, 4);
    out[e] = (uint16_t)(u >> 16);   /* exact: at most 8 significant bits */
  }
}
