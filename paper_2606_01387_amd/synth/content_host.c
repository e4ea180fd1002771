/*
 * content_host.c -- seeded synthetic KV-pool content, host side.
 *
 * Part of the input generator shared by the tests, the oracle side and the
 * benchmark.  It holds none of the checker's arithmetic: content comes from
 * Philox4x32-10 (Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as
 * easy as 1, 2, 3", SC 2011), a different counter-based generator from the
 * one the checker keys its digests with.  fill.hip implements the same
 * definition on the GPU; a GPU test compares the two byte for byte.
 *
 * Content definition.  The pool is laid out [plane][block][chunk] and every
 * chunk is a whole number of 16-byte units.  Unit v of chunk (plane p,
 * block b) is:
 *   - bf16 pools: three Philox calls with counter (3v + r, b, p, TAG_BF16),
 *     r = 0, 1, 2, and key (seed low, seed high) give 24 16-bit halves
 *     (word w gives half 2w from its low 16 bits, 2w+1 from its high 16
 *     bits).  Element t = 0..7 takes s = half[3t] + half[3t+1] + half[3t+2]
 *     (Irwin-Hall of three uniforms), x = (2s - 196605) / 65536, which is
 *     exact in fp32 and has mean 0 and variance 1 - 2^-32, and stores x
 *     rounded to bf16 (round to nearest, ties to even) little-endian;
 *   - raw-byte pools (fp8 e4m3 payloads, never interpreted): one Philox call
 *     with counter (v, b, p, TAG_BYTES), its four words little-endian.
 */

#include <stdint.h>
#include <string.h>

#define TAG_BF16 0x6B760000u
#define TAG_BYTES 0x6B760001u

void synth_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
  uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
  uint32_t k0 = key_in[0], k1 = key_in[1];
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    uint64_t p0 = (uint64_t)0xD2511F53u * c0;
    uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
    uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
    uint32_t n1 = (uint32_t)p1;
    uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
    uint32_t n3 = (uint32_t)p0;
    c0 = n0;
    c1 = n1;
    c2 = n2;
    c3 = n3;
  }
  out[0] = c0;
  out[1] = c1;
  out[2] = c2;
  out[3] = c3;
}

static uint16_t bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

/* One 16-byte unit of content. */
static void unit(uint64_t seed, int raw_bytes, uint32_t p, uint32_t b, uint32_t v,
                 uint8_t out[16]) {
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  if (raw_bytes) {
    uint32_t ctr[4] = {v, b, p, TAG_BYTES};
    uint32_t w[4];
    synth_philox4x32_10(ctr, key, w);
    for (int i = 0; i < 4; ++i)
      for (int k = 0; k < 4; ++k) out[4 * i + k] = (uint8_t)(w[i] >> (8 * k));
    return;
  }
  uint32_t w[12];
  for (uint32_t r = 0; r < 3; ++r) {
    uint32_t ctr[4] = {3u * v + r, b, p, TAG_BF16};
    synth_philox4x32_10(ctr, key, w + 4 * r);
  }
  for (int t = 0; t < 8; ++t) {
    uint32_t s = 0;
    for (int k = 0; k < 3; ++k) {
      int idx = 3 * t + k;
      s += (w[idx / 2] >> (16 * (idx % 2))) & 0xFFFFu;
    }
    int32_t n = 2 * (int32_t)s - 196605;
    float x = (float)n * (1.0f / 65536.0f);
    uint16_t h = bf16_rne(x);
    out[2 * t] = (uint8_t)h;
    out[2 * t + 1] = (uint8_t)(h >> 8);
  }
}

/* Canonical bytes of block b (planes concatenated): planes * chunk_bytes. */
int synth_block_canonical(uint64_t seed, int raw_bytes, uint32_t planes, uint64_t chunk_bytes,
                          uint32_t b, uint8_t* out) {
  if (chunk_bytes % 16) return -1;
  for (uint32_t p = 0; p < planes; ++p)
    for (uint64_t v = 0; v < chunk_bytes / 16; ++v)
      unit(seed, raw_bytes, p, b, (uint32_t)v, out + p * chunk_bytes + 16 * v);
  return 0;
}

/* Whole pool in its [plane][block][chunk] layout (small pools only). */
int synth_pool_host(uint64_t seed, int raw_bytes, uint32_t planes, uint32_t num_blocks,
                    uint64_t chunk_bytes, uint8_t* out) {
  if (chunk_bytes % 16) return -1;
  for (uint32_t p = 0; p < planes; ++p)
    for (uint32_t b = 0; b < num_blocks; ++b)
      for (uint64_t v = 0; v < chunk_bytes / 16; ++v)
        unit(seed, raw_bytes, p, b, (uint32_t)v,
             out + ((uint64_t)p * num_blocks + b) * chunk_bytes + 16 * v);
  return 0;
}
