/*
 * inputs_native.c - seeded synthetic input generation for paged decode attention.
 *
 * This file produces INPUT BYTES only (random normals, their bf16 rounding and an
 * fp8-e4m3fn quantisation of KV tiles).  It contains none of the attention
 * arithmetic; both the CPU oracle and the GPU library consume what it writes.
 *
 * Random numbers: Philox4x32-10, the counter-based generator of Salmon, Moraes,
 * Dror and Shaw ("Parallel random numbers: as easy as 1, 2, 3", SC'11), keyed by a
 * 64-bit seed, with a 128-bit counter (element block index, stream id).  Each
 * counter value yields four 32-bit words, turned into four N(0,1) draws by the
 * Box-Muller transform.  Element i of a stream is therefore a pure function of
 * (seed, stream, i), independent of threading and of how a buffer is chunked.
 *
 * Built with gcc -O2 -fopenmp as a plain shared library (no GPU code).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

static void philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
  uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
  uint32_t k0 = key_in[0], k1 = key_in[1];
  for (int r = 0; r < 10; ++r) {
    uint64_t p0 = (uint64_t)PHILOX_M0 * c0;
    uint64_t p1 = (uint64_t)PHILOX_M1 * c2;
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    uint32_t n0 = hi1 ^ c1 ^ k0;
    uint32_t n2 = hi0 ^ c3 ^ k1;
    c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
    k0 += PHILOX_W0; k1 += PHILOX_W1;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Four N(0,1) draws for block `blk` of (seed, stream). */
static void normal_block(uint64_t seed, uint64_t stream, uint64_t blk, double z[4]) {
  uint32_t ctr[4] = {(uint32_t)blk, (uint32_t)(blk >> 32), (uint32_t)stream, (uint32_t)(stream >> 32)};
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  uint32_t w[4];
  philox4x32_10(ctr, key, w);
  const double two_pi = 6.283185307179586476925286766559;
  const double inv32 = 1.0 / 4294967296.0;
  for (int p = 0; p < 2; ++p) {
    double u1 = ((double)w[2 * p] + 1.0) * inv32; /* (0, 1] keeps log finite */
    double u2 = (double)w[2 * p + 1] * inv32;     /* [0, 1) */
    double r = sqrt(-2.0 * log(u1));
    z[2 * p] = r * cos(two_pi * u2);
    z[2 * p + 1] = r * sin(two_pi * u2);
  }
}

static uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x0040u);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

/* Round |a| (finite, >= 0, <= 448) to the nearest OCP E4M3FN value, ties to even. */
static uint8_t e4m3fn_encode_mag(double a) {
  if (a >= 448.0) return 0x7E;
  if (a < 0.015625) {                      /* below 2^-6: subnormal grid of 2^-9 */
    double m = nearbyint(a * 512.0);       /* 0..8; 8 is the smallest normal 0x08 */
    return (uint8_t)m;
  }
  int e2;
  double fr = frexp(a, &e2);               /* a = fr * 2^e2, fr in [0.5, 1) */
  int e = e2 - 1;                          /* a = (2 fr) * 2^e, 2fr in [1, 2) */
  double m = nearbyint((2.0 * fr - 1.0) * 8.0);
  if (m >= 8.0) { m = 0.0; e += 1; }
  int code = ((e + 7) << 3) | (int)m;
  if (code > 0x7E) code = 0x7E;
  return (uint8_t)code;
}

static uint8_t e4m3fn_encode(double x) {
  uint8_t s = (x < 0.0 || (x == 0.0 && signbit(x))) ? 0x80 : 0x00;
  return (uint8_t)(s | e4m3fn_encode_mag(fabs(x)));
}

/* ---------------------------------------------------------------- exports */

/* Fill out[0..n) with elements [offset, offset+n) of stream (seed, stream). */
#define FILL_BODY(STORE)                                                          \
  uint64_t b0 = offset >> 2, b1 = (offset + (uint64_t)n + 3) >> 2;                \
  _Pragma("omp parallel for schedule(static)")                                    \
  for (int64_t blk = (int64_t)b0; blk < (int64_t)b1; ++blk) {                      \
    double z[4];                                                                  \
    normal_block(seed, stream, (uint64_t)blk, z);                                 \
    for (int e = 0; e < 4; ++e) {                                                 \
      int64_t i = (int64_t)((uint64_t)blk * 4 + (uint64_t)e) - (int64_t)offset;   \
      if (i >= 0 && i < n) { STORE; }                                             \
    }                                                                             \
  }

void inputs_fill_normal_f32(uint64_t seed, uint64_t stream, uint64_t offset, int64_t n, float* out) {
  FILL_BODY(out[i] = (float)z[e])
}

void inputs_fill_normal_bf16(uint64_t seed, uint64_t stream, uint64_t offset, int64_t n, uint16_t* out) {
  FILL_BODY(out[i] = f32_to_bf16_rne((float)z[e]))
}

void inputs_f32_to_bf16(const float* in, int64_t n, uint16_t* out) {
  #pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) out[i] = f32_to_bf16_rne(in[i]);
}

void inputs_f32_to_e4m3fn(const float* in, int64_t n, uint8_t* out) {
  #pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    double x = in[i];
    if (x > 448.0) x = 448.0;
    if (x < -448.0) x = -448.0;
    out[i] = e4m3fn_encode(x);
  }
}

/*
 * Generate `ntiles` KV tiles of `rows` x `cols` N(0,1) values (tile t holds stream
 * elements [t*rows*cols, (t+1)*rows*cols)), and quantise each to E4M3FN with one fp32
 * scale per tile: scale = amax/448 over the first nvalid[t] rows (1 when that amax is
 * 0), byte = RNE(x/scale) clamped to +-448.  Rows >= nvalid[t] are quantised with the
 * same scale (they are poisoned by the caller afterwards).
 */
void inputs_gen_fp8_tiles(uint64_t seed, uint64_t stream, int64_t ntiles, int rows, int cols,
                          const int8_t* nvalid, uint8_t* out, float* scales) {
  const int64_t te = (int64_t)rows * cols;
  #pragma omp parallel
  {
    double buf[16 * 256];
    #pragma omp for schedule(static)
    for (int64_t t = 0; t < ntiles; ++t) {
      double amax = 0.0;
      int nv = nvalid[t];
      for (int64_t e0 = 0; e0 < te; e0 += 4) {   /* te is a multiple of 4 */
        double z[4];
        normal_block(seed, stream, (uint64_t)(t * te + e0) >> 2, z);
        for (int e = 0; e < 4; ++e) {
          double v = (double)(float)z[e];
          buf[e0 + e] = v;
          if (e0 + e < (int64_t)nv * cols && fabs(v) > amax) amax = fabs(v);
        }
      }
      float sc = amax > 0.0 ? (float)(amax / 448.0) : 1.0f;
      scales[t] = sc;
      for (int64_t e = 0; e < te; ++e) {
        double x = buf[e] / (double)sc;
        if (x > 448.0) x = 448.0;
        if (x < -448.0) x = -448.0;
        out[t * te + e] = e4m3fn_encode(x);
      }
    }
  }
}

/* Raw Philox4x32-10 block, exported for the generator's known-answer test. */
void inputs_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  philox4x32_10(ctr, key, out);
}
