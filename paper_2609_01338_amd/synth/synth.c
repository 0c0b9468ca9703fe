/*
 * Seeded synthetic inputs for the restore-and-prefill path: normally distributed
 * weights encoded as Q4_0 blocks.  This file draws and encodes inputs only; it
 * holds no step of the method (no dequantization, no model arithmetic).
 *
 * Random numbers: Philox4x32-10, the counter-based generator of Salmon, Moraes,
 * Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3" (SC'11), turned
 * into normals with the Box-Muller transform.  Element e of a tensor (row-major
 * [out][in] index, padding excluded) takes word e%4 of the block
 * philox(counter = {e/4 low, e/4 high, 0, 0}, key = {seed, tensor_id}), so the
 * draws do not depend on the thread count.
 *
 * Q4_0 encoding (GGUF-compatible): 32 consecutive `in` elements per block; the
 * block holds an IEEE half scale d followed by 16 bytes whose low nibble is
 * element j and high nibble element j+16 (j < 16).  The encoder takes the signed
 * element of largest magnitude m, sets d = m / -8, and stores
 * q = min(15, trunc(x / d + 8.5)); a zero block stores d = 0, q = 8.  Rows whose
 * `in` length is not a multiple of 32 are padded with zeros.
 */
#define _GNU_SOURCE
#include <math.h>
#include <stdint.h>
#include <string.h>

#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

void mz_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
  uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
  uint32_t k0 = key_in[0], k1 = key_in[1];
  for (int r = 0; r < 10; ++r) {
    uint64_t p0 = (uint64_t)PHILOX_M0 * c0;
    uint64_t p1 = (uint64_t)PHILOX_M1 * c2;
    uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
    uint32_t n1 = (uint32_t)p1;
    uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
    uint32_t n3 = (uint32_t)p0;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    k0 += PHILOX_W0; k1 += PHILOX_W1;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Four standard normals for counter block b (Box-Muller in single precision). */
static void normals4(uint64_t b, uint32_t seed, uint32_t tensor_id, float z[4]) {
  uint32_t ctr[4] = {(uint32_t)b, (uint32_t)(b >> 32), 0u, 0u};
  uint32_t key[2] = {seed, tensor_id};
  uint32_t w[4];
  mz_philox4x32_10(ctr, key, w);
  for (int i = 0; i < 4; i += 2) {
    /* 24-bit uniforms in (0, 1): log is finite */
    float u1 = ((float)(w[i] >> 8) + 0.5f) * (1.0f / 16777216.0f);
    float u2 = ((float)(w[i + 1] >> 8) + 0.5f) * (1.0f / 16777216.0f);
    float r = sqrtf(-2.0f * logf(u1));
    float s, c;
    sincosf(6.2831853071795864f * u2, &s, &c);
    z[i] = r * c;
    z[i + 1] = r * s;
  }
}

void mz_synth_normal(uint32_t seed, uint32_t tensor_id, uint64_t start, uint64_t n, float stddev,
                     float *out) {
  #pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < (int64_t)n; ++i) {
    uint64_t e = start + (uint64_t)i;
    float z[4];
    normals4(e >> 2, seed, tensor_id, z);
    out[i] = stddev * z[e & 3];
  }
}

/* IEEE binary32 -> binary16, round to nearest even (finite inputs of the ranges used here,
   subnormals and overflow handled). */
static uint16_t f32_to_f16_bits(float f) {
  uint32_t x;
  memcpy(&x, &f, 4);
  uint32_t sign = (x >> 16) & 0x8000u;
  uint32_t absx = x & 0x7FFFFFFFu;
  if (absx >= 0x7F800000u) return (uint16_t)(sign | (absx > 0x7F800000u ? 0x7E00u : 0x7C00u));
  if (absx >= 0x477FF000u) return (uint16_t)(sign | 0x7C00u);          /* rounds to >= 65520 */
  if (absx < 0x38800000u) {                                            /* below 2^-14: subnormal */
    if (absx < 0x33000000u) return (uint16_t)sign;                     /* < 2^-25 rounds to 0 */
    uint32_t mant = (absx & 0x7FFFFFu) | 0x800000u;
    int exp = (int)(absx >> 23);                                       /* 102..112 */
    int shift = 126 - exp;                                             /* 14..24 */
    uint32_t q = mant >> shift;
    uint32_t rem = mant & ((1u << shift) - 1u);
    uint32_t half = 1u << (shift - 1);
    if (rem > half || (rem == half && (q & 1u))) q++;
    return (uint16_t)(sign | q);
  }
  uint32_t q = ((absx - 0x38000000u) >> 13);                           /* rebias 127 -> 15 */
  uint32_t rem = absx & 0x1FFFu;
  if (rem > 0x1000u || (rem == 0x1000u && (q & 1u))) q++;
  return (uint16_t)(sign | q);
}

void mz_f32_to_f16(const float *in, uint16_t *out, uint64_t n) {
  for (uint64_t i = 0; i < n; ++i) out[i] = f32_to_f16_bits(in[i]);
}

/* Encode one block of 32 floats. */
static void encode_block(const float *x, uint8_t *dst) {
  float amax = 0.f, m = 0.f;
  for (int j = 0; j < 32; ++j) {
    float a = fabsf(x[j]);
    if (a > amax) { amax = a; m = x[j]; }
  }
  float d = m / -8.f;
  float id = d != 0.f ? 1.f / d : 0.f;
  uint16_t dh = f32_to_f16_bits(d);
  dst[0] = (uint8_t)(dh & 0xFF);
  dst[1] = (uint8_t)(dh >> 8);
  for (int j = 0; j < 16; ++j) {
    int q0 = (int)(x[j] * id + 8.5f);
    int q1 = (int)(x[j + 16] * id + 8.5f);
    if (q0 > 15) q0 = 15;
    if (q1 > 15) q1 = 15;
    dst[2 + j] = (uint8_t)(q0 | (q1 << 4));
  }
}

/* Draw a [rows][cols] N(0, stddev^2) tensor and write it as Q4_0 rows of
   ceil(cols/32) blocks (18 bytes each). */
void mz_synth_q4_0(uint32_t seed, uint32_t tensor_id, int64_t rows, int64_t cols, float stddev,
                   uint8_t *dst) {
  int64_t nb = (cols + 31) / 32;
  #pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r) {
    float buf[32];
    float z[4];
    uint64_t zb = UINT64_MAX;
    for (int64_t b = 0; b < nb; ++b) {
      for (int j = 0; j < 32; ++j) {
        int64_t c = b * 32 + j;
        if (c < cols) {
          uint64_t e = (uint64_t)r * (uint64_t)cols + (uint64_t)c;
          if ((e >> 2) != zb) { zb = e >> 2; normals4(zb, seed, tensor_id, z); }
          buf[j] = stddev * z[e & 3];
        } else {
          buf[j] = 0.f;
        }
      }
      encode_block(buf, dst + (r * nb + b) * 18);
    }
  }
}

/* Encode caller-supplied floats [rows][cols] as Q4_0 (same rules as above). */
void mz_encode_q4_0(const float *x, int64_t rows, int64_t cols, uint8_t *dst) {
  int64_t nb = (cols + 31) / 32;
  #pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r) {
    float buf[32];
    for (int64_t b = 0; b < nb; ++b) {
      for (int j = 0; j < 32; ++j) {
        int64_t c = b * 32 + j;
        buf[j] = c < cols ? x[r * cols + c] : 0.f;
      }
      encode_block(buf, dst + (r * nb + b) * 18);
    }
  }
}
