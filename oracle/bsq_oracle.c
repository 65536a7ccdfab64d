/*
 * CPU oracle for the binary spherical (BSQ) weight codec and the products
 * that consume it.
 *
 * TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the
 * benchmark's CPU baseline may load this library. It shares no code, header,
 * table or constant generator with the HIP library under
 * paper_2607_08643_amd/csrc, and it must stay plain: every loop below follows
 * the order in which the paper (Section III) states the method, with the
 * readings listed next to each step where the paper is silent.
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fno-fast-math -fopenmp -shared
 * (no contraction, no fast-math; rows are independent, so the OpenMP row loop
 * gives the same bits for every thread count).
 *
 * Canonical fp32 arithmetic contract for the encoder (the GPU reproduces it
 * bit for bit, because stage-2 codes depend on the stage-1 reconstruction):
 *   - fmaf() is the fused multiply-add of IEEE 754 (one rounding);
 *   - '/' is IEEE division, round to nearest even;
 *   - fp32 -> fp16 is round to nearest even, with finite overflow saturated;
 *   - subnormals are kept.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_OK 0
#define ORC_ERR_ARG 1
#define ORC_ERR_NONFINITE 6

#define KIND_IDENTITY 0
#define KIND_LINEAR 1
#define KIND_MLP 2
#define KIND_MLP_RES1 3

#define FMT_INT8 0
#define FMT_E4M3 1
#define FMT_E5M2 2

#define MAX_CODE_BITS 16
#define MAX_HIDDEN 256
#define MAX_STAGES 4

/* ------------------------------------------------------------------------ */
/* binary16 conversions, written from the IEEE 754 binary16 definition.      */
/* ------------------------------------------------------------------------ */

/* fp32 -> fp16 bits, round to nearest, ties to even. Values whose rounded
 * magnitude exceeds 65504 become infinity (IEEE behaviour). */
uint16_t orc_f32_to_f16(float f)
{
    uint32_t x;
    memcpy(&x, &f, 4);
    uint16_t sign = (uint16_t)((x >> 16) & 0x8000u);
    if (isnan(f)) return (uint16_t)(sign | 0x7e00u);
    if (isinf(f)) return (uint16_t)(sign | 0x7c00u);
    double a = fabs((double)f);
    if (a == 0.0) return sign;
    int e2;
    frexp(a, &e2);            /* a in [2^(e2-1), 2^e2) */
    int E = e2 - 1;           /* unbiased binary exponent of a */
    if (E < -14) {
        /* subnormal range: spacing 2^-24; n = 1024 is the smallest normal */
        double n = nearbyint(a * 0x1p24);
        return (uint16_t)(sign | (uint16_t)n);
    }
    double n = nearbyint(ldexp(a, 10 - E));   /* in [1024, 2048] */
    uint32_t bits = ((uint32_t)(E + 15) << 10) + ((uint32_t)n - 1024u);
    if (bits >= 0x7c00u) return (uint16_t)(sign | 0x7c00u);
    return (uint16_t)(sign | bits);
}

float orc_f16_to_f32(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int ex = (h >> 10) & 0x1f;
    int man = h & 0x3ff;
    double v;
    if (ex == 0x1f) v = man ? NAN : INFINITY;
    else if (ex == 0) v = ldexp((double)man, -24);
    else v = ldexp((double)(1024 + man), ex - 25);
    return (float)(sign ? -v : v);
}

/* Gain storage rule: fp16, round to nearest even, finite overflow saturated
 * to +-65504 (the largest finite binary16). */
uint16_t orc_gain_to_f16(float alpha)
{
    uint16_t h = orc_f32_to_f16(alpha);
    if ((h & 0x7fffu) == 0x7c00u) h = (uint16_t)((h & 0x8000u) | 0x7bffu);
    return h;
}

/* ------------------------------------------------------------------------ */
/* Decoders (Section III-C; Table "BSQ codec components").                   */
/* ------------------------------------------------------------------------ */

/* Spherical code value: q_j = sign_j / sqrt(b). The stored bit is 1 for +.  */
float orc_code_scale(int b)
{
    return (float)(1.0 / sqrt((double)b));
}

/* D_theta(q) for one b-bit code.
 *  identity: y = q (requires d == b)
 *  linear:   y_m = beta_m + sum_j M[m][j] q_j          (fmaf chain over j)
 *  mlp:      a_k = relu(b1_k + sum_j W1[k][j] q_j)      (fmaf chain over j)
 *            y_m = b2_m + sum_k W2[m][k] a_k            (fmaf chain over k)
 *  mlp with one residual block (the symmetric decoder's res1 row of the
 *  codec ablation; reading: the block acts on the hidden layer):
 *            a_k as above;
 *            t_k = relu(cr_k + sum_l R[k][l] a_l)       (fmaf chain over l)
 *            a'_k = a_k + t_k                           (one fp32 add)
 *            y_m = b2_m + sum_k W2[m][k] a'_k           (fmaf chain over k)
 *  relu(a) = (a > 0) ? a : +0.0f. */
int orc_decoder_eval(int kind, int d, int b, int h,
                     const float *W1, const float *b1,
                     const float *W2, const float *b2,
                     const float *R, const float *cr,
                     uint32_t code, float *y)
{
    if (b < 1 || b > MAX_CODE_BITS || d < 1 || d > MAX_CODE_BITS) return ORC_ERR_ARG;
    float q[MAX_CODE_BITS];
    float c = orc_code_scale(b);
    for (int j = 0; j < b; ++j) q[j] = ((code >> j) & 1u) ? c : -c;
    if (kind == KIND_IDENTITY) {
        if (d != b) return ORC_ERR_ARG;
        for (int j = 0; j < d; ++j) y[j] = q[j];
    } else if (kind == KIND_LINEAR) {
        for (int m = 0; m < d; ++m) {
            float acc = b1[m];
            for (int j = 0; j < b; ++j) acc = fmaf(W1[m * b + j], q[j], acc);
            y[m] = acc;
        }
    } else if (kind == KIND_MLP || kind == KIND_MLP_RES1) {
        if (h < 1 || h > MAX_HIDDEN) return ORC_ERR_ARG;
        float a[MAX_HIDDEN];
        for (int k = 0; k < h; ++k) {
            float acc = b1[k];
            for (int j = 0; j < b; ++j) acc = fmaf(W1[k * b + j], q[j], acc);
            a[k] = (acc > 0.0f) ? acc : 0.0f;
        }
        if (kind == KIND_MLP_RES1) {
            if (!R || !cr) return ORC_ERR_ARG;
            float t[MAX_HIDDEN];
            for (int k = 0; k < h; ++k) {
                float acc = cr[k];
                for (int l = 0; l < h; ++l) acc = fmaf(R[k * h + l], a[l], acc);
                t[k] = (acc > 0.0f) ? acc : 0.0f;
            }
            for (int k = 0; k < h; ++k) a[k] = a[k] + t[k];
        }
        for (int m = 0; m < d; ++m) {
            float acc = b2[m];
            for (int k = 0; k < h; ++k) acc = fmaf(W2[m * h + k], a[k], acc);
            y[m] = acc;
        }
    } else {
        return ORC_ERR_ARG;
    }
    return ORC_OK;
}

/* Every code's decoded vector, table[code * d + m]. This is the function
 * above evaluated for each of the 2^b codes (memoised; same bits). */
int orc_decoder_table(int kind, int d, int b, int h,
                      const float *W1, const float *b1,
                      const float *W2, const float *b2,
                      const float *R, const float *c, float *table)
{
    uint32_t n = 1u << b;
    for (uint32_t code = 0; code < n; ++code) {
        int rc = orc_decoder_eval(kind, d, b, h, W1, b1, W2, b2, R, c, code, table + (size_t)code * d);
        if (rc) return rc;
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Protected input channels (Section III-E, eq. protected_channel_selection) */
/* ------------------------------------------------------------------------ */

/* Column energy key_j = g_j^2 * sum_i w_ij^2 in fp64, rows summed in order
 * i = 0 .. d_out-1; g defaults to 1. Ranking by key is ranking by
 * g_j * ||W[:, j]||_2 since both are monotone in it. */
void orc_column_keys(const float *w, int64_t d_out, int64_t d_in, const float *g, double *key)
{
    for (int64_t j = 0; j < d_in; ++j) {
        double s = 0.0;
        for (int64_t i = 0; i < d_out; ++i) {
            double v = (double)w[i * d_in + j];
            s = s + v * v;
        }
        if (g) {
            double gj = (double)g[j];
            s = (gj * gj) * s;
        }
        key[j] = s;
    }
}

static const double *g_sort_keys;
static int cmp_key_desc_index_asc(const void *pa, const void *pb)
{
    int64_t a = *(const int64_t *)pa, b = *(const int64_t *)pb;
    double ka = g_sort_keys[a], kb = g_sort_keys[b];
    if (ka > kb) return -1;
    if (ka < kb) return 1;
    return (a < b) ? -1 : (a > b);
}
static int cmp_i32_asc(const void *pa, const void *pb)
{
    int32_t a = *(const int32_t *)pa, b = *(const int32_t *)pb;
    return (a > b) - (a < b);
}

/* TopK over given keys: the k largest of key[0 .. n-1], equal keys -> lower
 * index first; returned in ascending index order. Not thread-safe (qsort
 * comparator state); the oracle calls it from one thread. */
int orc_topk(const double *key, int64_t n, int64_t k, int32_t *idx)
{
    if (k < 0 || k > n) return ORC_ERR_ARG;
    int64_t *order = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    if (!order) return ORC_ERR_ARG;
    for (int64_t j = 0; j < n; ++j) order[j] = j;
    g_sort_keys = key;
    qsort(order, (size_t)n, sizeof(int64_t), cmp_key_desc_index_asc);
    for (int64_t p = 0; p < k; ++p) idx[p] = (int32_t)order[p];
    qsort(idx, (size_t)k, sizeof(int32_t), cmp_i32_asc);
    free(order);
    return ORC_OK;
}

/* P = TopK_j(key, k) over the column keys. */
int orc_protect_select(const float *w, int64_t d_out, int64_t d_in, const float *g,
                       int64_t k, int32_t *idx, double *key_out)
{
    if (k < 0 || k > d_in) return ORC_ERR_ARG;
    double *key = key_out ? key_out : (double *)malloc(sizeof(double) * (size_t)(d_in > 0 ? d_in : 1));
    if (!key) return ORC_ERR_ARG;
    orc_column_keys(w, d_out, d_in, g, key);
    int rc = orc_topk(key, d_in, k, idx);
    if (!key_out) free(key);
    return rc;
}

/* Output-channel energy key_i = g_i^2 * sum_j w_ij^2 in fp64, columns summed
 * in order j = 0 .. d_in-1; g (one value per output row) defaults to 1. This
 * is the score of eq. protected_channel_selection applied to rows, the
 * output-channel axis of the protection-axis ablation (Section IV-D). */
void orc_row_keys(const float *w, int64_t d_out, int64_t d_in, const float *g, double *key)
{
    for (int64_t i = 0; i < d_out; ++i) {
        double s = 0.0;
        for (int64_t j = 0; j < d_in; ++j) {
            double v = (double)w[i * d_in + j];
            s = s + v * v;
        }
        if (g) {
            double gi = (double)g[i];
            s = (gi * gi) * s;
        }
        key[i] = s;
    }
}

/* Coupled MLP intermediate-channel score (eq. mlp_coupled_protection). For
 * gate and up ([d_ffn][d_model]) channel j is output row j; for down
 * ([d_model][d_ffn]) it is input column j:
 *   S_j = |g^gate_j| ||W_gate[j, :]|| + |g^up_j| ||W_up[j, :]|| + |g^down_j| ||W_down[:, j]||
 * Each squared norm is an fp64 sum in element order, the norm its correctly
 * rounded fp64 square root, and the three terms are added left to right. The
 * statistics g are magnitudes (absolute value taken); NULL means ones.
 * P = TopK_j(S, k) as orc_topk. score (may be NULL) receives S. */
int orc_coupled_select(const float *wg, const float *wu, const float *wd, int64_t d_model, int64_t d_ffn,
                       const float *gg, const float *gu, const float *gd, int64_t k, int32_t *idx,
                       double *score_out)
{
    if (k < 0 || k > d_ffn || d_model < 0) return ORC_ERR_ARG;
    size_t n = (size_t)(d_ffn > 0 ? d_ffn : 1);
    double *sg = (double *)malloc(sizeof(double) * n), *su = (double *)malloc(sizeof(double) * n);
    double *sd = (double *)malloc(sizeof(double) * n);
    double *score = score_out ? score_out : (double *)malloc(sizeof(double) * n);
    if (!sg || !su || !sd || !score) return ORC_ERR_ARG;
    orc_row_keys(wg, d_ffn, d_model, NULL, sg);
    orc_row_keys(wu, d_ffn, d_model, NULL, su);
    orc_column_keys(wd, d_model, d_ffn, NULL, sd);
    for (int64_t j = 0; j < d_ffn; ++j) {
        double a = gg ? fabs((double)gg[j]) : 1.0;
        double b = gu ? fabs((double)gu[j]) : 1.0;
        double c = gd ? fabs((double)gd[j]) : 1.0;
        score[j] = (a * sqrt(sg[j]) + b * sqrt(su[j])) + c * sqrt(sd[j]);
    }
    int rc = orc_topk(score, d_ffn, k, idx);
    free(sg);
    free(su);
    free(sd);
    if (!score_out) free(score);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* Protected payload formats (Table "BSQ codec components": the protected    */
/* path stored as INT8, FP8-E4M3 or FP8-E5M2). Each stored element is one    */
/* byte; its value times the slice's fp32 scale is the weight.               */
/*   INT8: two's complement, -127..127.                                     */
/*   E4M3: sign, 4 exponent bits (bias 7), 3 fraction bits; subnormals;      */
/*         no infinities, S.1111.111 is NaN; largest finite 448.            */
/*   E5M2: sign, 5 exponent bits (bias 15), 2 fraction bits; subnormals;     */
/*         S.11111.00 is infinity; largest finite 57344.                    */
/* (The OCP 8-bit floating point formats; reading: a protected slice is      */
/* scaled so that its largest magnitude lands on the format's largest        */
/* finite value, as the int8 path lands it on 127.)                          */
/* ------------------------------------------------------------------------ */

float orc_payload_max(int fmt)
{
    if (fmt == FMT_E4M3) return 448.0f;
    if (fmt == FMT_E5M2) return 57344.0f;
    return 127.0f;
}

/* The value of one stored byte, from the field definitions above. */
float orc_payload_value(uint8_t q, int fmt)
{
    if (fmt == FMT_INT8) return (float)(int8_t)q;
    int ebits = (fmt == FMT_E4M3) ? 4 : 5, mbits = 7 - ebits;
    int bias = (1 << (ebits - 1)) - 1;
    int sign = q >> 7;
    int ex = (q >> mbits) & ((1 << ebits) - 1);
    int man = q & ((1 << mbits) - 1);
    double v;
    if (fmt == FMT_E4M3 && ex == 15 && man == 7) v = NAN;
    else if (fmt == FMT_E5M2 && ex == 31) v = man ? NAN : INFINITY;
    else if (ex == 0) v = ldexp((double)man, 1 - bias - mbits);
    else v = ldexp((double)((1 << mbits) + man), ex - bias - mbits);
    return (float)(sign ? -v : v);
}

/* The stored byte for v (already divided by the scale).
 *   INT8: clamp(round_half_even(v), -127, 127).
 *   FP8:  the finite value nearest to v, ties to the even code (fraction
 *         LSB 0), the sign of v kept (so -0 and negative values that round
 *         to zero give the negative zero code); |v| above the largest finite
 *         value saturates to it. Found by trying every finite non-negative
 *         code, in double precision (every candidate and v are exact there). */
uint8_t orc_payload_quant(float v, int fmt)
{
    if (fmt == FMT_INT8) {
        float t = nearbyintf(v);
        if (t > 127.0f) t = 127.0f;
        if (t < -127.0f) t = -127.0f;
        return (uint8_t)(int8_t)t;
    }
    double a = fabs((double)v);
    uint8_t sign = signbit(v) ? 0x80u : 0u;
    uint8_t best = 0;
    double best_err = INFINITY;
    for (int code = 0; code < 128; ++code) {
        double cv = (double)orc_payload_value((uint8_t)code, fmt);
        if (!isfinite(cv)) continue;
        double err = fabs(cv - a);
        if (err < best_err || (err == best_err && (code & 1) == 0)) {
            best_err = err;
            best = (uint8_t)code;
        }
    }
    if (a >= (double)orc_payload_max(fmt)) best = (fmt == FMT_E4M3) ? 0x7eu : 0x7bu;
    return (uint8_t)(sign | best);
}

/* Q8 of the protected columns (eq. protected_8bit_scatter; reading: symmetric,
 * one fp32 scale per protected column):
 *   m_j = max_i |w_ij|;  s_j = m_j / max(fmt)   (127, 448 or 57344);
 *   q_ij = orc_payload_quant(w_ij / s_j, fmt), and the zero byte when s_j = 0.
 * Layout: q8[i * k + p] for protected column idx[p]. */
void orc_q8(const float *w, int64_t d_out, int64_t d_in, const int32_t *idx, int64_t k,
            int fmt, uint8_t *q8, float *scale)
{
    for (int64_t p = 0; p < k; ++p) {
        int64_t j = idx[p];
        float m = 0.0f;
        for (int64_t i = 0; i < d_out; ++i) {
            float a = fabsf(w[i * d_in + j]);
            if (a > m) m = a;
        }
        float s = m / orc_payload_max(fmt);
        scale[p] = s;
        for (int64_t i = 0; i < d_out; ++i)
            q8[i * k + p] = (s != 0.0f) ? orc_payload_quant(w[i * d_in + j] / s, fmt) : 0u;
    }
}

/* Q8 of protected output rows (eq. protected_8bit_scatter with row slices;
 * reading: symmetric, one fp32 scale per protected row):
 *   m_p = max_j |w[idx_p][j]|;  s_p = m_p / max(fmt);
 *   q8[p * d_in + j] = orc_payload_quant(w[idx_p][j] / s_p, fmt), and the
 *   zero byte when s_p = 0. */
void orc_q8_rows(const float *w, int64_t d_out, int64_t d_in, const int32_t *idx, int64_t k,
                 int fmt, uint8_t *q8, float *scale)
{
    (void)d_out;
    for (int64_t p = 0; p < k; ++p) {
        const float *row = w + (int64_t)idx[p] * d_in;
        float m = 0.0f;
        for (int64_t j = 0; j < d_in; ++j) {
            float a = fabsf(row[j]);
            if (a > m) m = a;
        }
        float s = m / orc_payload_max(fmt);
        scale[p] = s;
        for (int64_t j = 0; j < d_in; ++j)
            q8[p * d_in + j] = (s != 0.0f) ? orc_payload_quant(row[j] / s, fmt) : 0u;
    }
}

/* ------------------------------------------------------------------------ */
/* Encoder: sphere map + sign code + residual stage (Sections III-C, III-D). */
/* ------------------------------------------------------------------------ */

/* Encode one matrix w [d_out][d_in] (fp32, row-major) into S stages.
 *
 * Chunk (i, c) is w[i, c*d : (c+1)*d] (reading: d consecutive inputs of one
 * output row). The encoder gives z = E(r) in R^b (Section III-C): the
 * identity (b = d, z = r), or a learned linear map z = E r with E [b][d]
 * (enc[s] non-NULL; reading: the fmaf chain z_m = sum_j E[m][j] r_j from +0,
 * j in order). For ||z|| > 0 the sign of u = z / ||z|| equals the sign of z,
 * so the code of a chunk is
 *   bit_m = (z_m >= 0)                   (reading: +0 and -0 give 1)
 *   code  = sum_m bit_m << m             (element m -> bit m, LSB first)
 * Stage s (r^(0) = chunk with protected positions zeroed):
 *   y      = D_s(q)
 *   num    = fmaf chain over unprotected j of r_j * y_j, from +0
 *   den    = fmaf chain over unprotected j of y_j * y_j, from +0
 *   alpha  = den > 0 ? num / den : 0;   NaN -> 0
 *   gain   = fp16(alpha) (saturating);  a = (float)gain
 *   r_j    = fmaf(-a, y_j, r_j) for unprotected j
 * (reading: each stage stores a least-squares fp16 gain so that the stage
 * never increases the reconstruction error, whatever its decoder).
 *
 * Outputs, each row padded to `pitch` chunks (padding: code 0, gain +0):
 *   codes[s]  uint8 (b <= 8) or uint16 (b > 8), [d_out][pitch]
 *   gains[s]  fp16 bits,                         [d_out][pitch]
 *   idx[k] ascending protected columns, q8[d_out][k], scale[k].
 *
 * tables[s] is the decoder table of stage s (orc_decoder_table). */
/* The per-chunk stages of every row i with skip[i] == 0 (skip may be NULL);
 * positions j with prot[j] != 0 are masked out of BSQ. Rows with skip[i] set
 * and padding chunks get code 0 and gain +0. */
static void encode_rows(int d, int b, int stages, const float *const *tables, const float *const *enc,
                        const float *w, int64_t d_out,
                        int64_t d_in, int64_t pitch, const unsigned char *prot, const unsigned char *skip,
                        void *const *codes, uint16_t *const *gains, int nthreads)
{
    int64_t C = d_in / d;
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 16)
#else
    (void)nthreads;
#endif
    for (int64_t i = 0; i < d_out; ++i) {
        float r[MAX_CODE_BITS];
        for (int64_t c = 0; c < pitch; ++c) {
            if (c >= C || (skip && skip[i])) {
                for (int s = 0; s < stages; ++s) {
                    if (b <= 8) ((uint8_t *)codes[s])[i * pitch + c] = 0;
                    else ((uint16_t *)codes[s])[i * pitch + c] = 0;
                    gains[s][i * pitch + c] = 0;
                }
                continue;
            }
            for (int j = 0; j < d; ++j) {
                int64_t col = c * d + j;
                r[j] = prot[col] ? 0.0f : w[i * d_in + col];
            }
            for (int s = 0; s < stages; ++s) {
                uint32_t code = 0;
                if (enc && enc[s]) {
                    /* learned linear encoder: z_m = sum_j E[m][j] r_j, an
                     * fmaf chain from +0 in j order; bit m = (z_m >= 0) */
                    for (int m = 0; m < b; ++m) {
                        float z = 0.0f;
                        for (int j = 0; j < d; ++j) z = fmaf(enc[s][m * d + j], r[j], z);
                        if (z >= 0.0f) code |= 1u << m;
                    }
                } else {
                    for (int j = 0; j < d; ++j)
                        if (r[j] >= 0.0f) code |= 1u << j;
                }
                const float *y = tables[s] + (size_t)code * d;
                float num = 0.0f, den = 0.0f;
                for (int j = 0; j < d; ++j) {
                    if (prot[c * d + j]) continue;
                    num = fmaf(r[j], y[j], num);
                    den = fmaf(y[j], y[j], den);
                }
                float alpha = (den > 0.0f) ? num / den : 0.0f;
                if (alpha != alpha) alpha = 0.0f;
                uint16_t gh = orc_gain_to_f16(alpha);
                float a = orc_f16_to_f32(gh);
                for (int j = 0; j < d; ++j) {
                    if (prot[c * d + j]) continue;
                    r[j] = fmaf(-a, y[j], r[j]);
                }
                if (b <= 8) ((uint8_t *)codes[s])[i * pitch + c] = (uint8_t)code;
                else ((uint16_t *)codes[s])[i * pitch + c] = (uint16_t)code;
                gains[s][i * pitch + c] = gh;
            }
        }
    }
}

int orc_encode(int d, int b, int stages, const float *const *tables, const float *const *enc,
               const float *w, int64_t d_out, int64_t d_in, const float *g,
               int64_t k, int64_t pitch, int fmt,
               void *const *codes, uint16_t *const *gains,
               int32_t *idx, uint8_t *q8, float *scale, int nthreads)
{
    if (d < 1 || d > MAX_CODE_BITS || stages < 1 || stages > MAX_STAGES) return ORC_ERR_ARG;
    if (b < 1 || b > MAX_CODE_BITS || (b != d && !enc)) return ORC_ERR_ARG;
    if (d_in % d != 0 || k < 0 || k > d_in) return ORC_ERR_ARG;
    int64_t C = d_in / d;
    if (pitch < C) return ORC_ERR_ARG;
    for (int64_t t = 0; t < d_out * d_in; ++t)
        if (!isfinite(w[t])) return ORC_ERR_NONFINITE;

    /* protected set, Q8 payload and the complement mask */
    unsigned char *prot = (unsigned char *)calloc((size_t)(d_in > 0 ? d_in : 1), 1);
    if (!prot) return ORC_ERR_ARG;
    if (k > 0) {
        int rc = orc_protect_select(w, d_out, d_in, g, k, idx, NULL);
        if (rc) { free(prot); return rc; }
        orc_q8(w, d_out, d_in, idx, k, fmt, q8, scale);
        for (int64_t p = 0; p < k; ++p) prot[idx[p]] = 1;
    }
    encode_rows(d, b, stages, tables, enc, w, d_out, d_in, pitch, prot, NULL, codes, gains, nthreads);
    free(prot);
    return ORC_OK;
}

/* Encode with a given protected set idx[k] (strictly ascending, in range;
 * ORC_ERR_ARG otherwise):
 *   axis 0 (input columns): Q8 of those columns (orc_q8, q8 [d_out][k]) and
 *          BSQ on the rest of every row, exactly as orc_encode does after its
 *          own selection;
 *   axis 1 (output rows): Q8 of those rows (orc_q8_rows, q8 [k][d_in]); BSQ
 *          on every other row with no position masked (the complement of a
 *          row slice is whole rows); the protected rows are not BSQ-coded and
 *          keep code 0 and gain +0 in the planes.
 * This is how the coupled MLP set of eq. mlp_coupled_protection reaches the
 * three matrices: rows of gate and up, columns of down. */
int orc_encode_set(int d, int b, int stages, const float *const *tables, const float *const *enc,
                   const float *w, int64_t d_out, int64_t d_in, int axis,
                   const int32_t *idx, int64_t k, int64_t pitch, int fmt,
                   void *const *codes, uint16_t *const *gains,
                   uint8_t *q8, float *scale, int nthreads)
{
    if (d < 1 || d > MAX_CODE_BITS || stages < 1 || stages > MAX_STAGES) return ORC_ERR_ARG;
    if (b < 1 || b > MAX_CODE_BITS || (b != d && !enc)) return ORC_ERR_ARG;
    if (axis != 0 && axis != 1) return ORC_ERR_ARG;
    int64_t n = axis ? d_out : d_in;
    if (d_in % d != 0 || k < 0 || k > n) return ORC_ERR_ARG;
    if (pitch < d_in / d) return ORC_ERR_ARG;
    for (int64_t p = 0; p < k; ++p)
        if (idx[p] < 0 || idx[p] >= n || (p > 0 && idx[p] <= idx[p - 1])) return ORC_ERR_ARG;
    for (int64_t t = 0; t < d_out * d_in; ++t)
        if (!isfinite(w[t])) return ORC_ERR_NONFINITE;
    unsigned char *prot = (unsigned char *)calloc((size_t)(d_in > 0 ? d_in : 1), 1);
    unsigned char *skip = (unsigned char *)calloc((size_t)(d_out > 0 ? d_out : 1), 1);
    if (!prot || !skip) { free(prot); free(skip); return ORC_ERR_ARG; }
    if (axis == 0) {
        orc_q8(w, d_out, d_in, idx, k, fmt, q8, scale);
        for (int64_t p = 0; p < k; ++p) prot[idx[p]] = 1;
    } else {
        orc_q8_rows(w, d_out, d_in, idx, k, fmt, q8, scale);
        for (int64_t p = 0; p < k; ++p) skip[idx[p]] = 1;
    }
    encode_rows(d, b, stages, tables, enc, w, d_out, d_in, pitch, prot, skip, codes, gains, nthreads);
    free(prot);
    free(skip);
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Decoder assembly (eq. parallel_stage_decode, eq. protected_8bit_scatter). */
/* ------------------------------------------------------------------------ */

/* W_hat[i][j] = sum over stages of gain_s * D_s(code_s)[j], as an fmaf chain
 * over s from +0 (each stage decoded independently, then summed); protected
 * columns are then overwritten with value(q8) * scale (fp32 product). */
int orc_decode(int d, int b, int stages, const float *const *tables,
               int64_t d_out, int64_t d_in, int64_t pitch,
               const void *const *codes, const uint16_t *const *gains,
               const int32_t *idx, const uint8_t *q8, const float *scale, int64_t k, int fmt,
               float *w_hat, int nthreads)
{
    if (d < 1 || d > MAX_CODE_BITS || stages < 1 || stages > MAX_STAGES) return ORC_ERR_ARG;
    if (d_in % d != 0) return ORC_ERR_ARG;
    int64_t C = d_in / d;
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 16)
#endif
    for (int64_t i = 0; i < d_out; ++i) {
        for (int64_t c = 0; c < C; ++c) {
            for (int j = 0; j < d; ++j) {
                float v = 0.0f;
                for (int s = 0; s < stages; ++s) {
                    uint32_t code = (b <= 8) ? ((const uint8_t *)codes[s])[i * pitch + c]
                                             : ((const uint16_t *)codes[s])[i * pitch + c];
                    float a = orc_f16_to_f32(gains[s][i * pitch + c]);
                    v = fmaf(a, tables[s][(size_t)code * d + j], v);
                }
                w_hat[i * d_in + c * d + j] = v;
            }
        }
        for (int64_t p = 0; p < k; ++p)
            w_hat[i * d_in + idx[p]] = orc_payload_value(q8[i * k + p], fmt) * scale[p];
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Fused product route, fp64: y_i = sum_c sum_s gain * <D_s(code), x~_c>      */
/*   + sum_p scale_p value(q8_ip) x_{idx_p} + sum_r B_ir (A x)_r              */
/* x~ is x with the protected positions zeroed. This route never forms W_hat. */
/* ------------------------------------------------------------------------ */
int orc_gemv_fused(int d, int b, int stages, const float *const *tables,
                   int64_t d_out, int64_t d_in, int64_t pitch,
                   const void *const *codes, const uint16_t *const *gains,
                   const int32_t *idx, const uint8_t *q8, const float *scale, int64_t k, int fmt,
                   const double *x, int rank, const double *A, const double *B,
                   double *y, int nthreads)
{
    if (d < 1 || d > MAX_CODE_BITS || stages < 1 || stages > MAX_STAGES) return ORC_ERR_ARG;
    int64_t C = d_in / d;
    double *xt = (double *)malloc(sizeof(double) * (size_t)(d_in > 0 ? d_in : 1));
    double t[64];
    if (!xt || rank > 64) { free(xt); return ORC_ERR_ARG; }
    for (int64_t j = 0; j < d_in; ++j) xt[j] = x[j];
    for (int64_t p = 0; p < k; ++p) xt[idx[p]] = 0.0;
    for (int r = 0; r < rank; ++r) {
        double acc = 0.0;
        for (int64_t j = 0; j < d_in; ++j) acc += A[(int64_t)r * d_in + j] * x[j];
        t[r] = acc;
    }
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 16)
#endif
    for (int64_t i = 0; i < d_out; ++i) {
        double acc = 0.0;
        for (int64_t c = 0; c < C; ++c) {
            for (int s = 0; s < stages; ++s) {
                uint32_t code = (b <= 8) ? ((const uint8_t *)codes[s])[i * pitch + c]
                                         : ((const uint16_t *)codes[s])[i * pitch + c];
                double a = (double)orc_f16_to_f32(gains[s][i * pitch + c]);
                const float *yv = tables[s] + (size_t)code * d;
                double dot = 0.0;
                for (int j = 0; j < d; ++j) dot += (double)yv[j] * xt[c * d + j];
                acc += a * dot;
            }
        }
        for (int64_t p = 0; p < k; ++p)
            acc += (double)scale[p] * (double)orc_payload_value(q8[i * k + p], fmt) * x[idx[p]];
        for (int r = 0; r < rank; ++r) acc += B[i * rank + r] * t[r];
        y[i] = acc;
    }
    free(xt);
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Codec training (Section III-C, eq. codec_loss_terms): the decisions of one */
/* forward pass, taken in fp32 so that the training kernels and the oracle   */
/* agree on them exactly (the values of the pass are fp64 in oracle/train.py) */
/* ------------------------------------------------------------------------ */

/* For chunks x [n][d] (fp32): the code of z = E x (E [b][d], the fmaf chain
 * from +0 in j order, bit m = (z_m >= 0)), and the ReLU mask of the decoder's
 * hidden pre-activation at q = sign(z) / sqrt(b) (pre_k = fmaf chain from
 * b1_k over j of W1[k][j] q_j; mask bit k = (pre_k > 0)). codes [n], masks
 * [n][h] (0 or 1). */
void orc_train_decisions(int d, int b, int h, const float *E, const float *W1, const float *b1,
                         const float *x, int64_t n, uint32_t *codes, unsigned char *masks)
{
    float c = orc_code_scale(b);
    for (int64_t i = 0; i < n; ++i) {
        uint32_t code = 0;
        float q[MAX_CODE_BITS];
        for (int m = 0; m < b; ++m) {
            float z = 0.0f;
            for (int j = 0; j < d; ++j) z = fmaf(E[m * d + j], x[i * d + j], z);
            if (z >= 0.0f) code |= 1u << m;
            q[m] = (z >= 0.0f) ? c : -c;
        }
        codes[i] = code;
        for (int k = 0; k < h; ++k) {
            float acc = b1[k];
            for (int j = 0; j < b; ++j) acc = fmaf(W1[k * b + j], q[j], acc);
            masks[i * h + k] = (acc > 0.0f) ? 1 : 0;
        }
    }
}

int orc_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
