/*
 * attention_oracle.c -- CPU oracle for one decoder self-attention block at a
 * single decode position.  TEST INFRASTRUCTURE ONLY (see moe_oracle.c); it
 * shares no code with the HIP library.
 *
 * The paper runs its model with a 4096-token context and attention on the
 * accelerator (sec. 6, the primary configuration) but describes no attention
 * arithmetic; the block here is our reading of a Qwen3-class decoder layer:
 *   h = rmsnorm(x) (unit gain); [q; k; v] = W_qkv h, with n_heads query heads
 *   and n_kv key/value heads of head_dim each (grouped-query attention: query
 *   head j reads key/value head j / (n_heads / n_kv)); every query and key head
 *   is RMS-normalised (unit gain) and then rotated by the rotary position
 *   embedding of the rotate-half form (dims i and i + head_dim/2 turned by the
 *   angle p * theta^(-2i/head_dim)); the token's key and value are stored at
 *   position p of a bf16 cache (round to nearest even); each query head attends
 *   over positions 0..p with softmax(q . k / sqrt(head_dim)); the heads'
 *   outputs, concatenated, go through W_o and are added to x.
 * Arithmetic in fp64; sums in index order.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define AO_OK 0
#define AO_ERR_ARG (-1)

static double bf16_to_double(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* bf16 of a value, round to nearest even (through its fp32 value) */
static uint16_t double_to_bf16(double v)
{
    float f = (float)v;
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    uint32_t lsb = (u >> 16) & 1u;
    u += 0x7fffu + lsb;
    return (uint16_t)(u >> 16);
}

/* Rotary position embedding of one head vector v[d] (d even) at position p. */
void oracle_rope(double *v, int d, int p, double theta)
{
    const int half = d / 2;
    for (int i = 0; i < half; i++) {
        const double ang = (double)p * pow(theta, -2.0 * i / d);
        const double c = cos(ang), s = sin(ang);
        const double a = v[i], b = v[i + half];
        v[i] = a * c - b * s;
        v[i + half] = b * c + a * s;
    }
}

static void rms_normalise(double *v, int n, double eps)
{
    double ss = 0.0;
    for (int i = 0; i < n; i++)
        ss += v[i] * v[i];
    const double inv = 1.0 / sqrt(ss / n + eps);
    for (int i = 0; i < n; i++)
        v[i] *= inv;
}

/*
 * x        fp32 [H] input of the block
 * w_qkv    bf16 [(n_heads + 2 n_kv) * head_dim x H]: the query rows, then the key rows, then the value rows
 * w_o      bf16 [H x n_heads * head_dim]
 * k_cache, v_cache: bf16 [n_kv][max_pos][head_dim]; positions < p are inputs, position p is written
 * y        fp64 [H] = x + W_o concat_j(attention output of query head j)
 */
int oracle_attention_decode(const float *x, int H, int n_heads, int n_kv, int head_dim, const uint16_t *w_qkv,
                            const uint16_t *w_o, uint16_t *k_cache, uint16_t *v_cache, int max_pos, int p,
                            double theta, double eps, double *y)
{
    if (!x || !w_qkv || !w_o || !k_cache || !v_cache || !y || H < 1 || n_heads < 1 || n_kv < 1 ||
        n_heads % n_kv || head_dim < 2 || head_dim % 2 || p < 0 || p >= max_pos)
        return AO_ERR_ARG;
    const int d = head_dim, group = n_heads / n_kv, rows = (n_heads + 2 * n_kv) * d;
    double *h = malloc(sizeof(double) * (size_t)H);
    double *qkv = malloc(sizeof(double) * (size_t)rows);
    double *att = calloc((size_t)n_heads * d, sizeof(double));
    double *sc = malloc(sizeof(double) * (size_t)(p + 1));
    for (int i = 0; i < H; i++)
        h[i] = x[i];
    rms_normalise(h, H, eps);
    for (int r = 0; r < rows; r++) {
        double acc = 0.0;
        for (int i = 0; i < H; i++)
            acc += bf16_to_double(w_qkv[(size_t)r * H + i]) * h[i];
        qkv[r] = acc;
    }
    double *q = qkv, *k = qkv + (size_t)n_heads * d, *v = k + (size_t)n_kv * d;
    for (int j = 0; j < n_heads; j++) {
        rms_normalise(q + (size_t)j * d, d, eps);
        oracle_rope(q + (size_t)j * d, d, p, theta);
    }
    for (int g = 0; g < n_kv; g++) {
        rms_normalise(k + (size_t)g * d, d, eps);
        oracle_rope(k + (size_t)g * d, d, p, theta);
        for (int i = 0; i < d; i++) {
            k_cache[((size_t)g * max_pos + p) * d + i] = double_to_bf16(k[(size_t)g * d + i]);
            v_cache[((size_t)g * max_pos + p) * d + i] = double_to_bf16(v[(size_t)g * d + i]);
        }
    }
    const double scale = 1.0 / sqrt((double)d);
    for (int j = 0; j < n_heads; j++) {
        const int g = j / group;
        double mx = -INFINITY;
        for (int t = 0; t <= p; t++) {
            double s = 0.0;
            for (int i = 0; i < d; i++)
                s += q[(size_t)j * d + i] * bf16_to_double(k_cache[((size_t)g * max_pos + t) * d + i]);
            sc[t] = s * scale;
            if (sc[t] > mx)
                mx = sc[t];
        }
        double sum = 0.0;
        for (int t = 0; t <= p; t++) {
            sc[t] = exp(sc[t] - mx);
            sum += sc[t];
        }
        for (int t = 0; t <= p; t++)
            for (int i = 0; i < d; i++)
                att[(size_t)j * d + i] += sc[t] / sum * bf16_to_double(v_cache[((size_t)g * max_pos + t) * d + i]);
    }
    for (int r = 0; r < H; r++) {
        double acc = 0.0;
        for (int i = 0; i < n_heads * d; i++)
            acc += bf16_to_double(w_o[(size_t)r * n_heads * d + i]) * att[i];
        y[r] = (double)x[r] + acc;
    }
    free(h);
    free(qkv);
    free(att);
    free(sc);
    return AO_OK;
}
