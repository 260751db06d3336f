/*
 * Reference oracle for batched paged decode attention and the KV append.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, obviously correct
 * CPU definition that the GPU library is checked against.  Only the test
 * suite, the smoke check and the benchmark's CPU-baseline leg may load it.
 * It shares no code, header, table or helper with the GPU library and is
 * compiled by gcc, never by hipcc.
 *
 * What is computed.  The paper (beLLMan, Sec. 3, "Our key proposal" and
 * "Setup and trace") serves an LLM through vLLM and watches the
 * time-between-tokens of the decode loop; the cost of each decode step is
 * attention of one new query token per request over that request's KV cache,
 * whose length is the prompt plus the tokens generated so far.  The paper
 * itself prints no attention formula; the definition below is textbook
 * scaled dot-product attention with grouped-query heads:
 *
 *   for request b and query head h (kv head g = h / G, G = H_q / H_kv):
 *     s_t   = scale * sum_d q[b,h,d] * k_t[d]          for t < L_b
 *     w_t   = exp(s_t - max_u s_u),   Z = sum_t w_t
 *     out   = sum_t (w_t / Z) * v_t
 *
 * everything in IEEE binary64, with no reordering, blocking or splitting.
 *
 * Paged layout read here (the library's contract, restated independently):
 *   K pool  [NP, H_kv, D/x, 16, x]   x = 16 bytes / element size
 *   V pool  [NP, H_kv, D, 16]
 *   token t of request b lives in page block_table[b][t/16], slot t%16.
 * Element codes: bf16 (the upper half of an IEEE binary32) or OCP fp8
 * e4m3fn (1 sign, 4 exponent bits with bias 7, 3 mantissa bits, subnormals at
 * exponent 0, S.1111.111 is NaN, no infinities).  For fp8 pools each
 * (request, kv head) carries one fp32 scale for K and one for V; the real value
 * of a code is decode(code) * scale, formed exactly in binary64.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_PAGE 16

enum { ORACLE_BF16 = 1, ORACLE_FP8_E4M3FN = 2 };

/* bf16 bit pattern -> binary64.  A bf16 value is exactly the binary32 whose
 * upper 16 bits are the pattern and whose lower 16 bits are zero. */
double oracle_bf16_to_f64(uint16_t bits)
{
    uint32_t w = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &w, sizeof f);
    return (double)f;
}

/* OCP e4m3fn code -> binary64, from the format definition. */
double oracle_e4m3fn_to_f64(uint8_t code)
{
    int sign = (code >> 7) & 1;
    int e = (code >> 3) & 0xF;
    int m = code & 0x7;
    double mag;
    if (e == 0xF && m == 0x7)
        return NAN;
    if (e == 0)
        mag = ldexp((double)m / 8.0, 1 - 7);          /* subnormal */
    else
        mag = ldexp(1.0 + (double)m / 8.0, e - 7);    /* normal */
    return sign ? -mag : mag;
}

/* Threads the parallel loops below will use (for reporting). */
int oracle_num_threads(void) { return omp_get_max_threads(); }

static double load_code(const void *base, int64_t idx, int dtype)
{
    if (dtype == ORACLE_BF16)
        return oracle_bf16_to_f64(((const uint16_t *)base)[idx]);
    return oracle_e4m3fn_to_f64(((const uint8_t *)base)[idx]);
}

static int elem_bytes(int dtype) { return dtype == ORACLE_BF16 ? 2 : 1; }

/* Offset (in elements) of K element (page, kv head g, slot, dim d). */
static int64_t k_offset(int64_t page, int g, int slot, int d, int H_kv, int D, int x)
{
    int64_t tile = page * H_kv + g;                 /* one (page, head) tile */
    int64_t chunk = tile * (D / x) + d / x;         /* x-element chunk of dims */
    return (chunk * ORACLE_PAGE + slot) * x + d % x;
}

/* Offset (in elements) of V element (page, kv head g, dim d, slot). */
static int64_t v_offset(int64_t page, int g, int slot, int d, int H_kv, int D)
{
    int64_t tile = page * H_kv + g;
    return (tile * D + d) * ORACLE_PAGE + slot;
}

/*
 * Decode attention, one full forward step, in binary64.
 *   q        [B, H_q, D] bf16 bit patterns
 *   k_scale, v_scale  [B, H_kv] fp32, used only for fp8 pools (may be NULL
 *            for bf16)
 *   seq_lens [B] attention lengths (the length after this step's append)
 *   out      [B, H_q, D] binary64
 * A request with length 0 gets an all-zero output row.
 * Returns 0, or -1 when a used block-table entry or a length is out of range.
 */
/* One query row against the first L tokens of request b's KV head g: the
 * definition above, into o[0..D).  Returns 0, or -2 if out of memory. */
static int attend(const uint16_t *qrow, int b, int g, int L, int H_kv, int D, int kv_dtype,
                  const void *k_pages, const void *v_pages, double ks, double vs,
                  const int32_t *block_table, int max_pages, float scale, double *o)
{
    const int x = 16 / elem_bytes(kv_dtype);
    double *s;
    double m, Z;

    for (int d = 0; d < D; ++d)
        o[d] = 0.0;
    if (L == 0)
        return 0;
    s = (double *)malloc(sizeof(double) * (size_t)L);
    if (!s)
        return -2;

    /* scores */
    for (int t = 0; t < L; ++t) {
        int64_t pg = block_table[(int64_t)b * max_pages + t / ORACLE_PAGE];
        int slot = t % ORACLE_PAGE;
        double dot = 0.0;
        for (int d = 0; d < D; ++d) {
            double kv = load_code(k_pages, k_offset(pg, g, slot, d, H_kv, D, x), kv_dtype) * ks;
            dot += oracle_bf16_to_f64(qrow[d]) * kv;
        }
        s[t] = (double)scale * dot;
    }

    /* softmax weights */
    m = s[0];
    for (int t = 1; t < L; ++t)
        if (s[t] > m)
            m = s[t];
    Z = 0.0;
    for (int t = 0; t < L; ++t) {
        s[t] = exp(s[t] - m);
        Z += s[t];
    }

    /* weighted sum of values */
    for (int t = 0; t < L; ++t) {
        int64_t pg = block_table[(int64_t)b * max_pages + t / ORACLE_PAGE];
        int slot = t % ORACLE_PAGE;
        double w = s[t] / Z;
        for (int d = 0; d < D; ++d) {
            double vv = load_code(v_pages, v_offset(pg, g, slot, d, H_kv, D), kv_dtype) * vs;
            o[d] += w * vv;
        }
    }
    free(s);
    return 0;
}

/* Every used block-table entry of every request lies in the pool, and the
 * lengths fit the table. */
static int check_table(int B, const int32_t *seq_lens, const int32_t *block_table, int max_pages,
                       int64_t num_pages)
{
    for (int b = 0; b < B; ++b) {
        int L = seq_lens[b];
        if (L < 0 || L > max_pages * ORACLE_PAGE)
            return -1;
        for (int p = 0; p < (L + ORACLE_PAGE - 1) / ORACLE_PAGE; ++p) {
            int32_t pg = block_table[(int64_t)b * max_pages + p];
            if (pg < 0 || pg >= num_pages)
                return -1;
        }
    }
    return 0;
}

int oracle_decode_attention(int B, int H_q, int H_kv, int D, int kv_dtype,
                            const uint16_t *q,
                            const void *k_pages, const void *v_pages, int64_t num_pages,
                            const float *k_scale, const float *v_scale,
                            const int32_t *block_table, int max_pages,
                            const int32_t *seq_lens, float scale, double *out)
{
    const int G = H_q / H_kv;
    int bad = 0;

    if (check_table(B, seq_lens, block_table, max_pages, num_pages))
        return -1;

#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int b = 0; b < B; ++b) {
        for (int h = 0; h < H_q; ++h) {
            const int g = h / G;
            double ks = 1.0, vs = 1.0;
            if (kv_dtype == ORACLE_FP8_E4M3FN) {
                ks = (double)k_scale[(int64_t)b * H_kv + g];
                vs = (double)v_scale[(int64_t)b * H_kv + g];
            }
            if (attend(q + ((int64_t)b * H_q + h) * D, b, g, seq_lens[b], H_kv, D, kv_dtype, k_pages, v_pages,
                       ks, vs, block_table, max_pages, scale, out + ((int64_t)b * H_q + h) * D))
                bad = 1;
        }
    }
    return bad ? -2 : 0;
}

/*
 * Prefill (prompt) attention over the paged cache: request b contributes the
 * query tokens q_start[b] .. q_start[b+1]-1, the last n_b of its L_b =
 * seq_lens[b] tokens (their keys and values are already in the cache), and
 * query token i, at position p = L_b - n_b + (i - q_start[b]), attends the
 * tokens 0..p (causal self-attention, the prefill that produces a request's
 * first output token).  That is the decode definition above applied to each
 * query token with length p + 1.  q and out are [T, H_q, D] with T =
 * q_start[B].  Returns 0, -1 for a malformed table, -2 if out of memory.
 */
int oracle_prefill_attention(int B, int H_q, int H_kv, int D, int kv_dtype,
                             const uint16_t *q,
                             const void *k_pages, const void *v_pages, int64_t num_pages,
                             const float *k_scale, const float *v_scale,
                             const int32_t *block_table, int max_pages,
                             const int32_t *seq_lens, const int32_t *q_start, float scale, double *out)
{
    const int G = H_q / H_kv;
    int bad = 0;
    int64_t T;

    if (check_table(B, seq_lens, block_table, max_pages, num_pages))
        return -1;
    if (q_start[0] != 0)
        return -1;
    for (int b = 0; b < B; ++b)
        if (q_start[b + 1] < q_start[b] || q_start[b + 1] - q_start[b] > seq_lens[b])
            return -1;
    T = q_start[B];

#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int64_t i = 0; i < T; ++i) {
        for (int h = 0; h < H_q; ++h) {
            int b = 0;
            while (q_start[b + 1] <= i)
                ++b;
            const int n = q_start[b + 1] - q_start[b];
            const int p = seq_lens[b] - n + (int)(i - q_start[b]);
            const int g = h / G;
            double ks = 1.0, vs = 1.0;
            if (kv_dtype == ORACLE_FP8_E4M3FN) {
                ks = (double)k_scale[(int64_t)b * H_kv + g];
                vs = (double)v_scale[(int64_t)b * H_kv + g];
            }
            if (attend(q + (i * H_q + h) * D, b, g, p + 1, H_kv, D, kv_dtype, k_pages, v_pages, ks, vs,
                       block_table, max_pages, scale, out + (i * H_q + h) * D))
                bad = 1;
        }
    }
    return bad ? -2 : 0;
}

uint8_t oracle_quantize_e4m3fn(float x, float scale)
{
    float v = x / scale;
    int sign = signbit(v) ? 0x80 : 0;
    double a = fabs((double)v);
    double step, scaled, r, fl;
    int e, code;
    if (isnan(v))
        return (uint8_t)(sign | 0x7F);
    if (a >= 448.0)
        return (uint8_t)(sign | 0x7E);
    if (a < ldexp(1.0, -6)) {
        step = ldexp(1.0, -9);                         /* subnormal spacing */
    } else {
        e = (int)floor(log2(a));
        if (ldexp(1.0, e) > a) e -= 1;                 /* guard log2 rounding */
        if (ldexp(1.0, e + 1) <= a) e += 1;
        step = ldexp(1.0, e - 3);                      /* 3 mantissa bits */
    }
    scaled = a / step;                                 /* exact: power-of-two step */
    fl = floor(scaled);
    r = scaled - fl;
    if (r > 0.5 || (r == 0.5 && fmod(fl, 2.0) != 0.0))
        fl += 1.0;
    a = fl * step;                                     /* rounded magnitude */
    if (a >= 448.0)
        return (uint8_t)(sign | 0x7E);
    if (a < ldexp(1.0, -6)) {
        code = (int)(a / ldexp(1.0, -9));              /* 0..7 */
    } else {
        e = (int)floor(log2(a));
        if (ldexp(1.0, e) > a) e -= 1;
        if (ldexp(1.0, e + 1) <= a) e += 1;
        code = ((e + 7) << 3) | (int)(a / ldexp(1.0, e - 3) - 8.0);
    }
    return (uint8_t)(sign | code);
}

/*
 * KV append, on host copies of the pools: for each request b the new token's
 * K and V rows ([B, H_kv, D]) are written into page block_table[b][L/16],
 * slot L%16, with L = seq_lens[b]; then seq_lens[b] becomes L + 1.  Nothing
 * else is written.  new_dtype == pool dtype: the rows are codes of that type,
 * copied byte for byte.  bf16 rows into fp8 pools: each value x of head g is
 * stored as oracle_quantize_e4m3fn(x, scale[b, g]) with that request's K or
 * V scale.  Returns 0, or -1 (and writes nothing) when a slot falls outside
 * the block table or the page pool.
 */
int oracle_kv_append(int B, int H_kv, int D, int kv_dtype, int new_dtype,
                     const void *k_new, const void *v_new,
                     void *k_pages, void *v_pages, int64_t num_pages,
                     const float *k_scale, const float *v_scale,
                     const int32_t *block_table, int max_pages, int32_t *seq_lens)
{
    const int eb = elem_bytes(kv_dtype);
    const int x = 16 / eb;
    const int quant = kv_dtype == ORACLE_FP8_E4M3FN && new_dtype == ORACLE_BF16;

    for (int b = 0; b < B; ++b) {
        int L = seq_lens[b];
        int32_t pg;
        if (L < 0 || L / ORACLE_PAGE >= max_pages)
            return -1;
        pg = block_table[(int64_t)b * max_pages + L / ORACLE_PAGE];
        if (pg < 0 || pg >= num_pages)
            return -1;
    }

    for (int b = 0; b < B; ++b) {
        int L = seq_lens[b];
        int64_t pg = block_table[(int64_t)b * max_pages + L / ORACLE_PAGE];
        int slot = L % ORACLE_PAGE;
        for (int g = 0; g < H_kv; ++g) {
            for (int d = 0; d < D; ++d) {
                int64_t src = ((int64_t)b * H_kv + g) * D + d;
                char *kdst = (char *)k_pages + k_offset(pg, g, slot, d, H_kv, D, x) * eb;
                char *vdst = (char *)v_pages + v_offset(pg, g, slot, d, H_kv, D) * eb;
                if (quant) {
                    float kx = (float)oracle_bf16_to_f64(((const uint16_t *)k_new)[src]);
                    float vx = (float)oracle_bf16_to_f64(((const uint16_t *)v_new)[src]);
                    *(uint8_t *)kdst = oracle_quantize_e4m3fn(kx, k_scale[(int64_t)b * H_kv + g]);
                    *(uint8_t *)vdst = oracle_quantize_e4m3fn(vx, v_scale[(int64_t)b * H_kv + g]);
                } else {
                    memcpy(kdst, (const char *)k_new + src * eb, (size_t)eb);
                    memcpy(vdst, (const char *)v_new + src * eb, (size_t)eb);
                }
            }
        }
        seq_lens[b] = L + 1;
    }
    return 0;
}

/*
 * Write a prompt's keys and values into the paged cache: request b's tokens
 * q_start[b] .. q_start[b+1]-1 of k_new / v_new ([T, H_kv, D], the pool's
 * element type) go to positions seq_lens[b], seq_lens[b] + 1, ... (page
 * block_table[b][pos / 16], slot pos % 16), byte for byte, and seq_lens[b]
 * grows by their count.  Nothing else is written.  Returns 0 or -1.
 */
int oracle_kv_write(int B, int H_kv, int D, int kv_dtype, const void *k_new, const void *v_new,
                    void *k_pages, void *v_pages, int64_t num_pages,
                    const int32_t *block_table, int max_pages, int32_t *seq_lens, const int32_t *q_start)
{
    const int eb = elem_bytes(kv_dtype);
    const int x = 16 / eb;

    if (q_start[0] != 0)
        return -1;
    for (int b = 0; b < B; ++b) {
        int L = seq_lens[b], n = q_start[b + 1] - q_start[b];
        if (n < 0 || L < 0 || (n > 0 && (L + n - 1) / ORACLE_PAGE >= max_pages))
            return -1;
        for (int pos = L; pos < L + n; ++pos) {
            int32_t pg = block_table[(int64_t)b * max_pages + pos / ORACLE_PAGE];
            if (pg < 0 || pg >= num_pages)
                return -1;
        }
    }
    for (int b = 0; b < B; ++b) {
        int L = seq_lens[b];
        for (int64_t i = q_start[b]; i < q_start[b + 1]; ++i) {
            int pos = L + (int)(i - q_start[b]);
            int64_t pg = block_table[(int64_t)b * max_pages + pos / ORACLE_PAGE];
            int slot = pos % ORACLE_PAGE;
            for (int g = 0; g < H_kv; ++g) {
                for (int d = 0; d < D; ++d) {
                    int64_t src = (i * H_kv + g) * D + d;
                    memcpy((char *)k_pages + k_offset(pg, g, slot, d, H_kv, D, x) * eb,
                           (const char *)k_new + src * eb, (size_t)eb);
                    memcpy((char *)v_pages + v_offset(pg, g, slot, d, H_kv, D) * eb,
                           (const char *)v_new + src * eb, (size_t)eb);
                }
            }
        }
        seq_lens[b] = L + (q_start[b + 1] - q_start[b]);
    }
    return 0;
}
