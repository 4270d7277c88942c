/*
 * echo_oracle.c -- plain fp64 CPU reference for one mixed serving iteration
 * over a paged KV cache.  TEST INFRASTRUCTURE ONLY (see echo_oracle.h): only
 * the tests, the smoke check and the benchmark's CPU-baseline leg use it.
 *
 * Everything here follows the definitions directly: a scatter for append, a
 * byte copy for block copy, and for attention a gather of each row's logical
 * key/value sequence followed by textbook softmax attention in fp64 with sums
 * taken in ascending key order.  There is no tiling, no online softmax and no
 * split of the key range.
 */
#include "echo_oracle.h"

#include <math.h>
#include <pthread.h>
#include <stdatomic.h>
#include <stdlib.h>
#include <string.h>

#define BS 16

/* ------------------------------------------------------------------ codecs */

double orc_bf16_value(uint16_t bits) {
    /* bf16 is the upper half of an IEEE binary32 */
    uint32_t w = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &w, sizeof f);
    return (double)f;
}

/* OCP 8-bit floating point, E4M3 ("e4m3fn"): 1 sign, 4 exponent (bias 7),
 * 3 mantissa bits; no infinities; S.1111.111 is NaN; largest finite 448;
 * exponent field 0 holds subnormals m * 2^-9. */
double orc_e4m3_value(uint8_t code) {
    int s = code >> 7, e = (code >> 3) & 15, m = code & 7;
    double v;
    if (e == 15 && m == 7) return NAN;
    if (e == 0)
        v = ldexp((double)m, -9);
    else
        v = ldexp((double)(8 + m), e - 10);
    return s ? -v : v;
}

static double round_half_even(double v) {
    double fl = floor(v), d = v - fl;
    if (d > 0.5) return fl + 1.0;
    if (d < 0.5) return fl;
    return fmod(fl, 2.0) == 0.0 ? fl : fl + 1.0;
}

/* Nearest e4m3 value to x, ties to even mantissa, saturating to +-448. */
uint8_t orc_e4m3_encode(float x) {
    if (isnan(x)) return 0x7F;
    uint8_t sign = signbit(x) ? 0x80 : 0x00;
    double a = fabs((double)x);
    if (a >= 448.0) return sign | 0x7E;
    if (a < ldexp(1.0, -6)) {
        int m = (int)round_half_even(a * 512.0); /* a / 2^-9, exact */
        return sign | (uint8_t)m;                 /* m == 8 is 2^-6, code 0x08 */
    }
    int ex;
    frexp(a, &ex);                 /* a = f * 2^ex, f in [0.5, 1) */
    int e = ex - 1;                /* a = 1.x * 2^e */
    double frac = ldexp(a, -e) - 1.0;
    int m = (int)round_half_even(frac * 8.0);
    if (m == 8) { m = 0; e += 1; }
    int field = e + 7;
    if (field > 15 || (field == 15 && m > 6)) return sign | 0x7E;
    return sign | (uint8_t)((field << 3) | m);
}

float orc_e4m3_fresh_scale(float amax) {
    if (amax == 0.0f) return 1.0f;
    return (float)((double)amax / 448.0);
}

/* ----------------------------------------------------------------- helpers */

static size_t k_index(const orc_pool *p, int32_t blk, int32_t h, int32_t slot, int32_t d) {
    return (((size_t)blk * p->num_kv_heads + h) * BS + slot) * p->head_dim + d;
}

static size_t v_index(const orc_pool *p, int32_t blk, int32_t h, int32_t slot, int32_t d) {
    return (((size_t)blk * p->num_kv_heads + h) * p->head_dim + d) * BS + slot;
}

static int batch_ok(const orc_pool *p, const orc_batch *b) {
    if (b->num_rows < 0 || b->q_start[0] != 0) return 0;
    for (int32_t r = 0; r < b->num_rows; ++r) {
        int32_t q = b->q_start[r + 1] - b->q_start[r];
        int32_t L = b->seq_lens[r];
        if (q < 1 || L < q) return 0;
        if ((L + BS - 1) / BS > b->max_blocks_per_row) return 0;
        for (int32_t j = 0; j < (L + BS - 1) / BS; ++j) {
            int32_t blk = b->block_tables[(size_t)r * b->max_blocks_per_row + j];
            if (blk < 0 || blk >= p->num_blocks) return 0;
        }
    }
    return 1;
}

/* ------------------------------------------------------------------ append */

int orc_kv_append(const orc_pool *p, const orc_batch *b, const uint16_t *k_new,
                  const uint16_t *v_new) {
    if (!batch_ok(p, b)) return -1;
    const int32_t H = p->num_kv_heads, D = p->head_dim;
    for (int32_t r = 0; r < b->num_rows; ++r) {
        const int32_t t0 = b->q_start[r];
        const int32_t L = b->seq_lens[r];
        const int32_t p0 = L - (b->q_start[r + 1] - t0); /* first new position */
        for (int32_t j = p0 / BS; j <= (L - 1) / BS; ++j) {
            const int32_t blk = b->block_tables[(size_t)r * b->max_blocks_per_row + j];
            const int32_t lo = p0 > BS * j ? p0 : BS * j;          /* positions written */
            const int32_t hi = L < BS * (j + 1) ? L : BS * (j + 1);
            const int fresh = (BS * j >= p0);                      /* slot 0 written now */
            for (int32_t h = 0; h < H; ++h) {
                if (!p->kv_fp8) {
                    uint16_t *K = (uint16_t *)p->k, *V = (uint16_t *)p->v;
                    for (int32_t pos = lo; pos < hi; ++pos) {
                        const size_t src = ((size_t)(t0 + pos - p0) * H + h) * D;
                        for (int32_t d = 0; d < D; ++d) {
                            K[k_index(p, blk, h, pos % BS, d)] = k_new[src + d];
                            V[v_index(p, blk, h, pos % BS, d)] = v_new[src + d];
                        }
                    }
                    continue;
                }
                uint8_t *K = (uint8_t *)p->k, *V = (uint8_t *)p->v;
                const size_t si = (size_t)blk * H + h;
                if (fresh) {
                    double ak = 0.0, av = 0.0;
                    for (int32_t pos = lo; pos < hi; ++pos) {
                        const size_t src = ((size_t)(t0 + pos - p0) * H + h) * D;
                        for (int32_t d = 0; d < D; ++d) {
                            double x = fabs(orc_bf16_value(k_new[src + d]));
                            double y = fabs(orc_bf16_value(v_new[src + d]));
                            if (x > ak) ak = x;
                            if (y > av) av = y;
                        }
                    }
                    p->k_scale[si] = orc_e4m3_fresh_scale((float)ak);
                    p->v_scale[si] = orc_e4m3_fresh_scale((float)av);
                }
                const double sk = (double)p->k_scale[si], sv = (double)p->v_scale[si];
                for (int32_t pos = lo; pos < hi; ++pos) {
                    const size_t src = ((size_t)(t0 + pos - p0) * H + h) * D;
                    for (int32_t d = 0; d < D; ++d) {
                        /* x / s correctly rounded to binary32, then encoded */
                        float qk = (float)(orc_bf16_value(k_new[src + d]) / sk);
                        float qv = (float)(orc_bf16_value(v_new[src + d]) / sv);
                        K[k_index(p, blk, h, pos % BS, d)] = orc_e4m3_encode(qk);
                        V[v_index(p, blk, h, pos % BS, d)] = orc_e4m3_encode(qv);
                    }
                }
            }
        }
    }
    return 0;
}

/* -------------------------------------------------------------- block copy */

int orc_block_copy(const orc_pool *p, const int32_t *pairs, int32_t n) {
    const size_t elems = (size_t)p->num_kv_heads * BS * p->head_dim;
    const size_t bytes = elems * (p->kv_fp8 ? 1 : 2);
    for (int32_t i = 0; i < n; ++i) {
        int32_t s = pairs[2 * i], d = pairs[2 * i + 1];
        if (s < 0 || s >= p->num_blocks || d < 0 || d >= p->num_blocks) return -1;
    }
    for (int32_t i = 0; i < n; ++i) {
        int32_t s = pairs[2 * i], d = pairs[2 * i + 1];
        memmove((char *)p->k + (size_t)d * bytes, (char *)p->k + (size_t)s * bytes, bytes);
        memmove((char *)p->v + (size_t)d * bytes, (char *)p->v + (size_t)s * bytes, bytes);
        if (p->kv_fp8) {
            for (int32_t h = 0; h < p->num_kv_heads; ++h) {
                p->k_scale[(size_t)d * p->num_kv_heads + h] =
                    p->k_scale[(size_t)s * p->num_kv_heads + h];
                p->v_scale[(size_t)d * p->num_kv_heads + h] =
                    p->v_scale[(size_t)s * p->num_kv_heads + h];
            }
        }
    }
    return 0;
}

/* --------------------------------------------------------------- attention */

static double k_value(const orc_pool *p, int32_t blk, int32_t h, int32_t slot, int32_t d) {
    if (!p->kv_fp8) return orc_bf16_value(((const uint16_t *)p->k)[k_index(p, blk, h, slot, d)]);
    return orc_e4m3_value(((const uint8_t *)p->k)[k_index(p, blk, h, slot, d)]) *
           (double)p->k_scale[(size_t)blk * p->num_kv_heads + h];
}

static double v_value(const orc_pool *p, int32_t blk, int32_t h, int32_t slot, int32_t d) {
    if (!p->kv_fp8) return orc_bf16_value(((const uint16_t *)p->v)[v_index(p, blk, h, slot, d)]);
    return orc_e4m3_value(((const uint8_t *)p->v)[v_index(p, blk, h, slot, d)]) *
           (double)p->v_scale[(size_t)blk * p->num_kv_heads + h];
}

typedef struct {
    const orc_pool *p;
    const orc_batch *b;
    const uint16_t *q;
    int32_t hq;
    double scale;
    const int32_t *sel;
    int32_t n;
    double *out;
    atomic_int next;
} attn_job;

static int32_t row_of_token(const orc_batch *b, int32_t t) {
    int32_t lo = 0, hi = b->num_rows - 1; /* last row with q_start[row] <= t */
    while (lo < hi) {
        int32_t mid = (lo + hi + 1) / 2;
        if (b->q_start[mid] <= t) lo = mid; else hi = mid - 1;
    }
    return lo;
}

/* out = sum_j softmax_j(scale * q . k_j) v_j over keys j = 0..pos of the row */
static void attend_one(const attn_job *J, int32_t qi, double *s, double *out) {
    const orc_pool *p = J->p;
    const orc_batch *b = J->b;
    const int32_t D = p->head_dim;
    const int32_t t = qi / J->hq, h = qi % J->hq;
    const int32_t g = h / (J->hq / p->num_kv_heads);
    const int32_t r = row_of_token(b, t);
    const int32_t qlen = b->q_start[r + 1] - b->q_start[r];
    const int32_t pos = b->seq_lens[r] - qlen + (t - b->q_start[r]);
    const int32_t *bt = b->block_tables + (size_t)r * b->max_blocks_per_row;
    const uint16_t *qv = J->q + ((size_t)t * J->hq + h) * D;

    double m = -INFINITY;
    for (int32_t j = 0; j <= pos; ++j) {
        double dot = 0.0;
        for (int32_t d = 0; d < D; ++d)
            dot += orc_bf16_value(qv[d]) * k_value(p, bt[j / BS], g, j % BS, d);
        s[j] = J->scale * dot;
        if (s[j] > m) m = s[j];
    }
    double z = 0.0;
    for (int32_t j = 0; j <= pos; ++j) {
        s[j] = exp(s[j] - m);
        z += s[j];
    }
    for (int32_t d = 0; d < D; ++d) out[d] = 0.0;
    for (int32_t j = 0; j <= pos; ++j) {
        const double w = s[j] / z;
        for (int32_t d = 0; d < D; ++d) out[d] += w * v_value(p, bt[j / BS], g, j % BS, d);
    }
}

static void *attn_worker(void *arg) {
    attn_job *J = (attn_job *)arg;
    int32_t maxlen = 1;
    for (int32_t r = 0; r < J->b->num_rows; ++r)
        if (J->b->seq_lens[r] > maxlen) maxlen = J->b->seq_lens[r];
    double *s = (double *)malloc(sizeof(double) * (size_t)maxlen);
    if (!s) return NULL;
    for (;;) {
        int32_t i = atomic_fetch_add(&J->next, 1);
        if (i >= J->n) break;
        int32_t qi = J->sel ? J->sel[i] : i;
        attend_one(J, qi, s, J->out + (size_t)i * J->p->head_dim);
    }
    free(s);
    return NULL;
}

int orc_attention(const orc_pool *p, const orc_batch *b, const uint16_t *q, int32_t hq,
                  float sm_scale, const int32_t *sel, int32_t n_sel, double *out,
                  int32_t n_threads) {
    if (!batch_ok(p, b) || hq <= 0 || hq % p->num_kv_heads != 0) return -1;
    const int32_t T = b->q_start[b->num_rows];
    const int32_t n = sel ? n_sel : T * hq;
    for (int32_t i = 0; sel && i < n; ++i)
        if (sel[i] < 0 || sel[i] >= T * hq) return -1;
    attn_job J = {p, b, q, hq, (double)sm_scale, sel, n, out, 0};
    atomic_init(&J.next, 0);
    if (n_threads < 1) n_threads = 1;
    if (n_threads > 256) n_threads = 256;
    pthread_t th[256];
    int32_t started = 0;
    for (; started < n_threads - 1; ++started)
        if (pthread_create(&th[started], NULL, attn_worker, &J) != 0) break;
    attn_worker(&J);
    for (int32_t i = 0; i < started; ++i) pthread_join(th[i], NULL);
    return 0;
}
