/*
 * oracle.c - fp64 CPU oracle for batched decode attention over a paged KV cache.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may call, link or load
 * this file; only the tests, the package smoke check and the bench's CPU-baseline
 * leg use it.  It shares no code, header or helper with the GPU library.
 *
 * What it computes.  The rollout stage the paper schedules is dominated by
 * autoregressive decode over a KV cache whose size per token is the paper's
 * b_kv = 2 L H_kv d_head b_dtype / tp (App. A.1.2, rollout model) and whose decode
 * cost grows with the history attended, the H_dec term of the decode predictor
 * (App. A.1.2).  The operation evaluated at each step, per layer, is exact softmax
 * attention of one new query token per sequence over that sequence's cached tokens:
 *
 *     o[b,h,:] = sum_t softmax_t( scale * q[b,h,:] . k_t ) * v_t,
 *     t = 0 .. seq_lens[b]-1,   k_t, v_t taken from KV head kv_head_of_q[h],
 *
 * with scale = 1/sqrt(d) unless given.  The paper does not write this formula; the
 * readings used here (seq_len counts the current token, empty sequence -> zeros,
 * token t in page block_table[b][t / P] slot t % P, fp8 value = decode(byte) *
 * per-(page, KV head) scale) are stated with the build's design notes.
 *
 * How.  The plain definition, in fp64, one (sequence, KV head) at a time:
 * explicit gather of every token through the block table, all scores, the row
 * maximum, exponentials, their sum, then the weighted sum of V - two passes over
 * the tokens in ascending order, no splitting, no online rescaling.
 *
 * Multi-token queries.  Rollout also runs prefill over prompt tokens before it
 * decodes (Sec. 3, rollout; App. A.1.2, the prefill cost whose attention term
 * grows with the square of the prompt length).  A prefill chunk of n_b tokens of
 * sequence b sits at the end of its seq_lens[b] cached tokens (their K/V already
 * written); its query token i (0 <= i < n_b) is at position
 * pos = seq_lens[b] - n_b + i and attends causally to positions 0 .. pos:
 *
 *     o[r,h,:] = sum_{t <= pos} softmax_t( scale * q[r,h,:] . k_t ) * v_t,
 *     r = q_start[b] + i,
 *
 * i.e. the decode definition above with history pos + 1.  Decode is the case
 * n_b = 1.  oracle_multi_query_attention evaluates exactly that, one query token
 * at a time, with the same two-pass routine.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { ORC_F32 = 0, ORC_BF16 = 1, ORC_FP8_E4M3FN = 2 };

enum {
  ORC_OK = 0,
  ORC_BAD_ARG = -1,
  ORC_BAD_LEN = -2,
  ORC_BAD_PAGE = -3,
  ORC_NO_MEM = -4,
  ORC_BAD_QLEN = -5
};

/* bf16: the upper 16 bits of an IEEE binary32. */
static double orc_bf16(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* OCP 8-bit floating point, E4M3 ("FN") encoding: 1 sign, 4 exponent (bias 7),
 * 3 mantissa bits; exponent 0 is subnormal (m/8 * 2^-6); S.1111.111 is NaN; no
 * infinities; largest finite 448. */
static double orc_e4m3fn(uint8_t byte) {
  int sign = byte >> 7;
  int e = (byte >> 3) & 0xF;
  int m = byte & 0x7;
  double mag;
  if (e == 0xF && m == 0x7) return NAN;
  if (e == 0)
    mag = ldexp((double)m / 8.0, -6);
  else
    mag = ldexp(1.0 + (double)m / 8.0, e - 7);
  return sign ? -mag : mag;
}

static double orc_load(const void* base, int dtype, int64_t idx) {
  switch (dtype) {
    case ORC_F32: return (double)((const float*)base)[idx];
    case ORC_BF16: return orc_bf16(((const uint16_t*)base)[idx]);
    default: return orc_e4m3fn(((const uint8_t*)base)[idx]);
  }
}

/* Scalar decode hook for the decoder tests. */
double oracle_decode_scalar(int dtype, uint32_t bits) {
  switch (dtype) {
    case ORC_F32: { float f; memcpy(&f, &bits, 4); return (double)f; }
    case ORC_BF16: return orc_bf16((uint16_t)bits);
    case ORC_FP8_E4M3FN: return orc_e4m3fn((uint8_t)bits);
  }
  return NAN;
}

typedef struct {
  int batch, num_q_heads, num_kv_heads, head_dim, page_size, max_pages_per_seq, num_pages;
  int q_dtype, kv_dtype;
  const void *q, *k_cache, *v_cache;
  const float *k_scale, *v_scale;
  int64_t stride_page, stride_head, stride_slot;
  const int32_t *block_table, *seq_lens, *kv_head_of_q;
  double scale;
  double* out;
} orc_args;

/* One (sequence b, KV head g): every query head h with kv_head_of_q[h] == g
 * attends to the first L tokens of sequence b; its query and output are row
 * `row` of q and out ([row][num_q_heads][head_dim]). */
static int orc_one(const orc_args* a, int b, int g, int L, int64_t row, double* kbuf, double* vbuf, double* s,
                   int* heads) {
  const int d = a->head_dim, P = a->page_size;
  int nh = 0;
  for (int h = 0; h < a->num_q_heads; ++h)
    if (a->kv_head_of_q[h] == g) heads[nh++] = h;

  if (L == 0) {
    for (int i = 0; i < nh; ++i)
      for (int j = 0; j < d; ++j) a->out[(row * a->num_q_heads + heads[i]) * d + j] = 0.0;
    return ORC_OK;
  }

  /* Pass 1: gather k_t and scores s[i][t]. */
  for (int t = 0; t < L; ++t) {
    int pid = a->block_table[(int64_t)b * a->max_pages_per_seq + t / P];
    int slot = t % P;
    if (pid < 0 || pid >= a->num_pages) return ORC_BAD_PAGE;
    int64_t base = (int64_t)pid * a->stride_page + (int64_t)g * a->stride_head + (int64_t)slot * a->stride_slot;
    double ks = (a->kv_dtype == ORC_FP8_E4M3FN) ? (double)a->k_scale[(int64_t)pid * a->num_kv_heads + g] : 1.0;
    for (int j = 0; j < d; ++j) kbuf[j] = orc_load(a->k_cache, a->kv_dtype, base + j) * ks;
    for (int i = 0; i < nh; ++i) {
      int64_t qb = (row * a->num_q_heads + heads[i]) * d;
      double dot = 0.0;
      for (int j = 0; j < d; ++j) dot += orc_load(a->q, a->q_dtype, qb + j) * kbuf[j];
      s[(int64_t)i * L + t] = a->scale * dot;
    }
  }

  /* Softmax weights per head: w_t = exp(s_t - max s), Z = sum_t w_t. */
  for (int i = 0; i < nh; ++i) {
    double* si = s + (int64_t)i * L;
    double m = -INFINITY;
    for (int t = 0; t < L; ++t) m = si[t] > m ? si[t] : m;
    for (int t = 0; t < L; ++t) si[t] = exp(si[t] - m);
  }

  /* Pass 2: out = sum_t w_t v_t / Z. */
  for (int i = 0; i < nh; ++i) {
    double* o = a->out + (row * a->num_q_heads + heads[i]) * d;
    for (int j = 0; j < d; ++j) o[j] = 0.0;
  }
  for (int t = 0; t < L; ++t) {
    int pid = a->block_table[(int64_t)b * a->max_pages_per_seq + t / P];
    int slot = t % P;
    int64_t base = (int64_t)pid * a->stride_page + (int64_t)g * a->stride_head + (int64_t)slot * a->stride_slot;
    double vs = (a->kv_dtype == ORC_FP8_E4M3FN) ? (double)a->v_scale[(int64_t)pid * a->num_kv_heads + g] : 1.0;
    for (int j = 0; j < d; ++j) vbuf[j] = orc_load(a->v_cache, a->kv_dtype, base + j) * vs;
    for (int i = 0; i < nh; ++i) {
      double w = s[(int64_t)i * L + t];
      double* o = a->out + (row * a->num_q_heads + heads[i]) * d;
      for (int j = 0; j < d; ++j) o[j] += w * vbuf[j];
    }
  }
  for (int i = 0; i < nh; ++i) {
    double z = 0.0;
    const double* si = s + (int64_t)i * L;
    for (int t = 0; t < L; ++t) z += si[t];
    double* o = a->out + (row * a->num_q_heads + heads[i]) * d;
    for (int j = 0; j < d; ++j) o[j] /= z;
  }
  return ORC_OK;
}

typedef struct { int b, g, L; int64_t row; } orc_unit;

static int orc_longest_first(const void* x, const void* y) {
  const orc_unit* u = (const orc_unit*)x;
  const orc_unit* v = (const orc_unit*)y;
  if (u->L != v->L) return v->L - u->L;
  if (u->b != v->b) return u->b - v->b;
  return u->g - v->g;
}

/* Evaluate every unit (longest first, dynamic schedule); the first failure wins. */
static int orc_run_units(const orc_args* ap, orc_unit* units, int nunits, int maxL, int num_threads) {
  const orc_args a = *ap;
  const int head_dim = a.head_dim, num_q_heads = a.num_q_heads;
  qsort(units, (size_t)nunits, sizeof(orc_unit), orc_longest_first);

  int status = ORC_OK;
  if (num_threads <= 0) num_threads = omp_get_max_threads();
  #pragma omp parallel num_threads(num_threads)
  {
    double* kbuf = (double*)malloc(sizeof(double) * (size_t)head_dim);
    double* vbuf = (double*)malloc(sizeof(double) * (size_t)head_dim);
    double* s = (double*)malloc(sizeof(double) * (size_t)num_q_heads * (size_t)(maxL > 0 ? maxL : 1));
    int* heads = (int*)malloc(sizeof(int) * (size_t)num_q_heads);
    int local = (kbuf && vbuf && s && heads) ? ORC_OK : ORC_NO_MEM;
    #pragma omp for schedule(dynamic, 1)
    for (int u = 0; u < nunits; ++u) {
      if (local != ORC_OK) continue;
      int r = orc_one(&a, units[u].b, units[u].g, units[u].L, units[u].row, kbuf, vbuf, s, heads);
      if (r != ORC_OK) local = r;
    }
    #pragma omp critical
    { if (local != ORC_OK) status = local; }
    free(kbuf); free(vbuf); free(s); free(heads);
  }
  return status;
}

/*
 * Compute out[b][h][:] (fp64, [batch][num_q_heads][head_dim]) for every b with
 * batch_mask == NULL or batch_mask[b] != 0; rows of other sequences are untouched.
 * Returns ORC_OK, or a negative code for inconsistent arguments, a seq_len beyond
 * max_pages_per_seq * page_size, or a page id outside [0, num_pages).
 * num_threads <= 0 uses the OpenMP default.
 */
int oracle_decode_attention(int batch, int num_q_heads, int num_kv_heads, int head_dim, int page_size,
                            int max_pages_per_seq, int num_pages, int q_dtype, int kv_dtype, const void* q,
                            const void* k_cache, const void* v_cache, const float* k_scale,
                            const float* v_scale, int64_t stride_page, int64_t stride_head,
                            int64_t stride_slot, const int32_t* block_table, const int32_t* seq_lens,
                            const int32_t* kv_head_of_q, double scale, const uint8_t* batch_mask,
                            double* out, int num_threads) {
  if (batch < 0 || num_q_heads <= 0 || num_kv_heads <= 0 || head_dim <= 0 || page_size <= 0) return ORC_BAD_ARG;
  if (q_dtype != ORC_F32 && q_dtype != ORC_BF16) return ORC_BAD_ARG;
  if (kv_dtype < ORC_F32 || kv_dtype > ORC_FP8_E4M3FN) return ORC_BAD_ARG;
  if (kv_dtype == ORC_FP8_E4M3FN && (!k_scale || !v_scale)) return ORC_BAD_ARG;
  for (int h = 0; h < num_q_heads; ++h)
    if (kv_head_of_q[h] < 0 || kv_head_of_q[h] >= num_kv_heads) return ORC_BAD_ARG;
  int maxL = 0;
  for (int b = 0; b < batch; ++b) {
    if (batch_mask && !batch_mask[b]) continue;
    if (seq_lens[b] < 0 || (int64_t)seq_lens[b] > (int64_t)max_pages_per_seq * page_size) return ORC_BAD_LEN;
    if (seq_lens[b] > maxL) maxL = seq_lens[b];
  }

  orc_args a = {batch, num_q_heads, num_kv_heads, head_dim, page_size, max_pages_per_seq, num_pages,
                q_dtype, kv_dtype, q, k_cache, v_cache, k_scale, v_scale, stride_page, stride_head,
                stride_slot, block_table, seq_lens, kv_head_of_q,
                scale > 0.0 ? scale : 1.0 / sqrt((double)head_dim), out};

  int nunits = 0;
  orc_unit* units = (orc_unit*)malloc(sizeof(orc_unit) * (size_t)(batch > 0 ? batch : 1) * num_kv_heads);
  if (!units) return ORC_NO_MEM;
  for (int b = 0; b < batch; ++b) {
    if (batch_mask && !batch_mask[b]) continue;
    for (int g = 0; g < num_kv_heads; ++g) units[nunits++] = (orc_unit){b, g, seq_lens[b], b};
  }
  int status = orc_run_units(&a, units, nunits, maxL, num_threads);
  free(units);
  return status;
}

/*
 * Multi-token queries: compute out[r][h][:] (fp64, [total_q][num_q_heads][head_dim])
 * for every query row r = q_start[b] + i, 0 <= i < n_b = q_start[b+1] - q_start[b],
 * of every b with batch_mask == NULL or batch_mask[b] != 0; q is
 * [total_q][num_q_heads][head_dim] with total_q = q_start[batch].  Row r attends
 * causally to the first seq_lens[b] - n_b + i + 1 tokens of sequence b.  Rows of
 * other sequences are untouched.  Returns ORC_BAD_QLEN when q_start is not
 * non-decreasing from 0 or a selected sequence has more query tokens than cached
 * tokens, otherwise as oracle_decode_attention.
 */
int oracle_multi_query_attention(int batch, int num_q_heads, int num_kv_heads, int head_dim, int page_size,
                                 int max_pages_per_seq, int num_pages, int q_dtype, int kv_dtype, const void* q,
                                 const void* k_cache, const void* v_cache, const float* k_scale,
                                 const float* v_scale, int64_t stride_page, int64_t stride_head,
                                 int64_t stride_slot, const int32_t* block_table, const int32_t* seq_lens,
                                 const int32_t* q_start, const int32_t* kv_head_of_q, double scale,
                                 const uint8_t* batch_mask, double* out, int num_threads) {
  if (batch < 0 || num_q_heads <= 0 || num_kv_heads <= 0 || head_dim <= 0 || page_size <= 0) return ORC_BAD_ARG;
  if (q_dtype != ORC_F32 && q_dtype != ORC_BF16) return ORC_BAD_ARG;
  if (kv_dtype < ORC_F32 || kv_dtype > ORC_FP8_E4M3FN) return ORC_BAD_ARG;
  if (kv_dtype == ORC_FP8_E4M3FN && (!k_scale || !v_scale)) return ORC_BAD_ARG;
  for (int h = 0; h < num_q_heads; ++h)
    if (kv_head_of_q[h] < 0 || kv_head_of_q[h] >= num_kv_heads) return ORC_BAD_ARG;
  if (q_start[0] != 0) return ORC_BAD_QLEN;
  int64_t nunits_all = 0;
  int maxL = 0;
  for (int b = 0; b < batch; ++b) {
    const int n = q_start[b + 1] - q_start[b];
    if (n < 0) return ORC_BAD_QLEN;
    if (batch_mask && !batch_mask[b]) continue;
    if (seq_lens[b] < 0 || (int64_t)seq_lens[b] > (int64_t)max_pages_per_seq * page_size) return ORC_BAD_LEN;
    if (n > seq_lens[b]) return ORC_BAD_QLEN;
    if (seq_lens[b] > maxL) maxL = seq_lens[b];
    nunits_all += (int64_t)n * num_kv_heads;
  }

  orc_args a = {batch, num_q_heads, num_kv_heads, head_dim, page_size, max_pages_per_seq, num_pages,
                q_dtype, kv_dtype, q, k_cache, v_cache, k_scale, v_scale, stride_page, stride_head,
                stride_slot, block_table, seq_lens, kv_head_of_q,
                scale > 0.0 ? scale : 1.0 / sqrt((double)head_dim), out};

  /* One unit per (query token, KV head): the decode definition with history pos + 1. */
  if (nunits_all > 0x7fffffff) return ORC_BAD_ARG;
  orc_unit* units = (orc_unit*)malloc(sizeof(orc_unit) * (size_t)(nunits_all > 0 ? nunits_all : 1));
  if (!units) return ORC_NO_MEM;
  int nunits = 0;
  for (int b = 0; b < batch; ++b) {
    if (batch_mask && !batch_mask[b]) continue;
    const int n = q_start[b + 1] - q_start[b];
    for (int i = 0; i < n; ++i) {
      const int pos = seq_lens[b] - n + i;
      for (int g = 0; g < num_kv_heads; ++g) units[nunits++] = (orc_unit){b, g, pos + 1, (int64_t)q_start[b] + i};
    }
  }
  int status = orc_run_units(&a, units, nunits, maxL, num_threads);
  free(units);
  return status;
}

/* Threads a default-sized parallel region of this library uses. */
int oracle_max_threads(void) { return omp_get_max_threads(); }
