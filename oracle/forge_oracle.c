/*
 * forge_oracle.c -- plain, slow, obviously-correct CPU reference for one fused
 * weight-gradient + AdamW step of a linear layer (FORGE, Sec. 2.2, Algorithm 1).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or call
 * this file; only the test-suite, the smoke check and the CPU-baseline leg of the
 * benchmark do.  It shares no code, header, table or constant with the HIP
 * library: it is written from the paper's definitions alone.
 *
 * What it computes (all floating point in fp64 unless stated):
 *   1. G = dY^T X, G[p][q] = sum_{t=0}^{T-1} dY[t][p] * X[t][q], summed in token
 *      order t = 0..T-1 (Eq. wgrad; App. A "Setup").  bf16 x bf16 products are
 *      exact in fp64.
 *   2. Decode the stored moments (fp32 / bf16 as they are; int8 as scale * code,
 *      with the second moment stored through its square root).
 *   3. AdamW exactly as Algorithm 1 states it: the two moment recurrences, the
 *      bias corrections 1 - beta^t, and the decoupled weight update
 *      W' = (1 - lr*wd) W - lr * mhat / (sqrt(vhat) + eps).
 *   4. Round to the storage dtypes with round-to-nearest-even: W' to bf16 straight
 *      from fp64; m', v' to fp32 or bf16 straight from fp64.
 *   5. int8 moments (block-absmax scheme of App. B, with 256-row blocks along
 *      d_out and sqrt(v) storage): per block and column, a = max |x|, scale
 *      s = a/127, code = clamp(round_half_even(x/s)).  The paper keeps this
 *      arithmetic in fp32, so the code decision is taken in fp32 here: x is
 *      rounded to fp32, s is an fp32 division, x/s is an fp32 division.  The
 *      second-moment codes are floored at 1 inside non-zero blocks (App. B: v is
 *      kept away from zero).  The weight update reads the unquantized fp64 m', v'.
 *
 * Hyper-parameters arrive as the fp32 values the GPU receives; they are promoted
 * to fp64 here, so lr = 1e-3 means (double)(float)1e-3.
 *
 * The paper's own int8 layout (App. B), forge_oracle_adamw_i8row: one scale per 64
 * consecutive elements of a row (along d_in), a = max |x| over the block, s = a/127,
 * code = round_half_even(x/s) clamped to [-127, 127], for m and for v itself (no square
 * root), the v codes floored at 1 inside non-zero blocks; decision in fp32 as above.
 *
 * fp8 encodings (forge_oracle_adamw_fp8; App. E's per-tensor delayed-scaled fp8 states and
 * the fp8-weight recipe of Sec. 3): OCP E4M3 codes (1 sign, 4 exponent bits with bias 7,
 * 3 mantissa bits, largest finite 448, subnormals below 2^-6), encoded round-half-even from
 * the fp32 quotient x/s clamped to [-448, 448]; one scale per tensor, s = amax/448 from a
 * previous step's amax (1 while there is none), kept in a ring of 4 amax slots: step t
 * decodes with slot (t-2)%4, encodes with slot (t-1)%4, max-reduces the fp32 magnitudes of
 * its new values (|W'|, |m'|, sqrt(v')) into slot t%4 and clears slot (t+1)%4.  sqrt(v) is
 * what is stored for the second moment, and a positive one never encodes to zero.
 *
 * Other update rules (forge_oracle_rule_step): the coordinate-wise optimizer families of
 * the paper's family table (App. I) and Muon's momentum accumulate (regime 2 of App. A).
 * The paper states that each was checked against its reference implementation and does
 * not restate the rules, so each is written here from that implementation's published
 * algorithm (torch.optim's documentation for SGD, Adagrad, RMSprop, NAdam, RAdam, Adamax;
 * the Lion paper's algorithm for Lion), in fp64, coupled weight decay (gg = g + wd w)
 * where those algorithms use it, decoupled for Lion.
 *
 * The layer-level backward adds one more quantity, computed before the update:
 *   0. the input gradient dX = dY W from the pre-update weight (Algorithm 1, first
 *      line; the ordering remark of App. A), dX[t][q] = sum_p dY[t][p] * W[p][q],
 *      summed in order p = 0..d_out-1, in fp64.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_I8_BLOCK 256

enum { ORACLE_MOMENT_F32 = 0, ORACLE_MOMENT_BF16 = 1, ORACLE_MOMENT_I8 = 2, ORACLE_MOMENT_I8_ROW64 = 3 };
#define ORACLE_ROW_BLOCK 64

/* ---------------------------------------------------------------- bf16 helpers */

/* bf16 bit pattern -> exact fp64 value (bf16 is the top half of an fp32). */
double forge_oracle_bf16_to_f64(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/*
 * fp64 -> bf16 with round-to-nearest, ties to even, in one rounding step.
 * bf16 carries 8 significant bits; its subnormal spacing is 2^-133.  The value is
 * scaled by a power of two so that one unit in the last place becomes 1, rounded
 * to an integer with rint (ties-to-even under the default rounding mode) and
 * scaled back.  Overflow past the largest bf16 gives infinity.
 */
uint16_t forge_oracle_f64_to_bf16(double x)
{
    if (isnan(x)) return (uint16_t)0x7FC0;
    uint16_t sign = signbit(x) ? (uint16_t)0x8000 : (uint16_t)0;
    double ax = fabs(x);
    if (ax == 0.0) return sign;
    if (isinf(ax)) return (uint16_t)(sign | 0x7F80);
    int e;
    (void)frexp(ax, &e);            /* ax = f * 2^e, 0.5 <= f < 1 */
    int ulp_exp = e - 8;            /* 8 significant bits */
    if (ulp_exp < -133) ulp_exp = -133;
    double n = rint(ldexp(ax, -ulp_exp));
    double r = ldexp(n, ulp_exp);   /* exactly representable in bf16, or 2^128 */
    float rf = (float)r;            /* exact, or +inf on overflow */
    uint32_t u;
    memcpy(&u, &rf, sizeof u);
    return (uint16_t)(sign | (uint16_t)(u >> 16));
}

/* ------------------------------------------------------------- 1. weight gradient */

/*
 * G[p*d_in + q] = sum_t dY[t*d_out + p] * X[t*d_in + q]   (Eq. wgrad, App. A)
 * X: bf16 [T, d_in], dY: bf16 [T, d_out], both row-major.  G: fp64 [d_out, d_in].
 * For every element the sum runs over t = 0..T-1 in order.
 */
void forge_oracle_wgrad(const uint16_t *X, const uint16_t *dY, int64_t T,
                        int64_t d_in, int64_t d_out, double *G)
{
    double *Xd = (double *)malloc(sizeof(double) * (size_t)(T * d_in > 0 ? T * d_in : 1));
    for (int64_t i = 0; i < T * d_in; ++i) Xd[i] = forge_oracle_bf16_to_f64(X[i]);

#pragma omp parallel for schedule(dynamic, 4)
    for (int64_t p = 0; p < d_out; ++p) {
        double *row = G + p * d_in;
        for (int64_t q = 0; q < d_in; ++q) row[q] = 0.0;
        for (int64_t t = 0; t < T; ++t) {
            double a = forge_oracle_bf16_to_f64(dY[t * d_out + p]);
            const double *xr = Xd + t * d_in;
            for (int64_t q = 0; q < d_in; ++q) row[q] += a * xr[q];
        }
    }
    free(Xd);
}

/* Elementwise forge_oracle_f64_to_bf16 over n values. */
void forge_oracle_f64_to_bf16_array(const double *x, int64_t n, uint16_t *out)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = forge_oracle_f64_to_bf16(x[i]);
}

/* ------------------------------------------------------------- 0. input gradient */

/*
 * dX[t*d_in + q] = sum_p dY[t*d_out + p] * W[p*d_in + q]   (chain rule through
 * Y = X W^T, Eq. fwd; Algorithm 1, first line).  dY: bf16 [T, d_out], W: bf16
 * [d_out, d_in], both row-major.  dX: fp64 [T, d_in].  Every element's sum runs over
 * p = 0..d_out-1 in order; d_out == 0 gives zeros.
 */
void forge_oracle_input_grad(const uint16_t *dY, const uint16_t *W, int64_t T, int64_t d_in,
                             int64_t d_out, double *dX)
{
    double *Wd = (double *)malloc(sizeof(double) * (size_t)(d_out * d_in > 0 ? d_out * d_in : 1));
    for (int64_t i = 0; i < d_out * d_in; ++i) Wd[i] = forge_oracle_bf16_to_f64(W[i]);

#pragma omp parallel for schedule(dynamic, 4)
    for (int64_t t = 0; t < T; ++t) {
        double *row = dX + t * d_in;
        for (int64_t q = 0; q < d_in; ++q) row[q] = 0.0;
        for (int64_t p = 0; p < d_out; ++p) {
            double a = forge_oracle_bf16_to_f64(dY[t * d_out + p]);
            const double *wr = Wd + p * d_in;
            for (int64_t q = 0; q < d_in; ++q) row[q] += a * wr[q];
        }
    }
    free(Wd);
}

/* ------------------------------------------------------------- int8 quantizer */

/*
 * Quantize one block column: n values x[i*stride] (fp64) -> codes, returning the
 * fp32 scale.  floor_one: second-moment codes are clamped to [1, 127] when the
 * block is non-zero.  quot (optional): the fp32 quotient x/s before rounding,
 * which tests use to recognise rounding ties.
 */
static float quantize_column(const double *x, int64_t n, int64_t stride, int floor_one,
                             int8_t *codes, int64_t code_stride, double *quot)
{
    float a = 0.0f;
    for (int64_t i = 0; i < n; ++i) {
        float xi = fabsf((float)x[i * stride]);
        if (xi > a) a = xi;
    }
    float s = a / 127.0f;  /* fp32 division, correctly rounded */
    for (int64_t i = 0; i < n; ++i) {
        int code = 0;
        float qf = 0.0f;
        if (s > 0.0f) {
            qf = (float)x[i * stride] / s;   /* fp32 division */
            float r = rintf(qf);             /* ties to even */
            if (r > 127.0f) r = 127.0f;
            if (r < -127.0f) r = -127.0f;
            if (floor_one && r < 1.0f) r = 1.0f;
            code = (int)r;
        }
        codes[i * code_stride] = (int8_t)code;
        if (quot) quot[i * code_stride] = (double)qf;
    }
    return s;
}

/*
 * Quantize a full [d_out, d_in] fp64 matrix into int8 codes + fp32 scales
 * [ceil(d_out/256), d_in]; the last block may hold fewer than 256 rows.
 * is_second_moment: x holds v itself; the stored quantity is sqrt(v) with the
 * floor-at-one rule.
 */
void forge_oracle_quantize_i8(const double *x, int64_t d_in, int64_t d_out,
                              int is_second_moment, int8_t *codes, float *scales)
{
    int64_t nblk = (d_out + ORACLE_I8_BLOCK - 1) / ORACLE_I8_BLOCK;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < nblk; ++b) {
        int64_t r0 = b * ORACLE_I8_BLOCK;
        int64_t n = d_out - r0 < ORACLE_I8_BLOCK ? d_out - r0 : ORACLE_I8_BLOCK;
        double *col = (double *)malloc(sizeof(double) * (size_t)n);
        for (int64_t q = 0; q < d_in; ++q) {
            for (int64_t i = 0; i < n; ++i) {
                double xv = x[(r0 + i) * d_in + q];
                col[i] = is_second_moment ? sqrt(xv) : xv;
            }
            scales[b * d_in + q] = quantize_column(col, n, 1, is_second_moment,
                                                   codes + r0 * d_in + q, d_in, NULL);
        }
        free(col);
    }
}

/* ------------------------------------------------------------- 2-5. AdamW step */

/*
 * One AdamW step (Algorithm 1, state update then weight update) on a given fp64
 * gradient G [d_out, d_in].
 *
 * W        bf16 [d_out, d_in], updated in place (RNE from fp64).
 * m, v     moments in place: float* (F32), uint16_t* bf16 bits (BF16), or int8
 *          codes (I8) with m_scale / v_scale fp32 [ceil(d_out/256), d_in].
 * round_grad_to_bf16  round G to bf16 (RNE) before use: the gradient a two-kernel
 *          path would have stored in a bf16 buffer (App. B, truncation bias).
 * W64, m64, v64   optional fp64 outputs of the unrounded new values.
 * qm, qv   optional (I8 only): the fp32 quotients x/s the codes were rounded from.
 */
void forge_oracle_adamw(const double *G, uint16_t *W, void *m, void *v,
                        float *m_scale, float *v_scale, int64_t d_in, int64_t d_out,
                        int moment_dtype, float lr, float beta1, float beta2, float eps,
                        float weight_decay, int64_t step, int round_grad_to_bf16,
                        double *W64, double *m64, double *v64, double *qm, double *qv)
{
    const double b1 = (double)beta1, b2 = (double)beta2;
    const double eta = (double)lr, lam = (double)weight_decay, ep = (double)eps;
    const double bc1 = 1.0 - pow(b1, (double)step);
    const double bc2 = 1.0 - pow(b2, (double)step);
    const double wdf = 1.0 - eta * lam;
    const int64_t nblk = (d_out + ORACLE_I8_BLOCK - 1) / ORACLE_I8_BLOCK;

#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t b = 0; b < nblk; ++b) {
        int64_t r0 = b * ORACLE_I8_BLOCK;
        int64_t n = d_out - r0 < ORACLE_I8_BLOCK ? d_out - r0 : ORACLE_I8_BLOCK;
        double *mnew = NULL, *vroot = NULL;
        if (moment_dtype == ORACLE_MOMENT_I8) {
            mnew = (double *)malloc(sizeof(double) * (size_t)(n * d_in));
            vroot = (double *)malloc(sizeof(double) * (size_t)(n * d_in));
        }
        for (int64_t i = 0; i < n; ++i) {
            int64_t p = r0 + i;
            for (int64_t q = 0; q < d_in; ++q) {
                int64_t k = p * d_in + q;
                double g = G[k];
                if (round_grad_to_bf16) g = forge_oracle_bf16_to_f64(forge_oracle_f64_to_bf16(g));

                double m0, v0;
                switch (moment_dtype) {
                case ORACLE_MOMENT_F32:
                    m0 = (double)((const float *)m)[k];
                    v0 = (double)((const float *)v)[k];
                    break;
                case ORACLE_MOMENT_BF16:
                    m0 = forge_oracle_bf16_to_f64(((const uint16_t *)m)[k]);
                    v0 = forge_oracle_bf16_to_f64(((const uint16_t *)v)[k]);
                    break;
                default: {
                    double sm = (double)m_scale[b * d_in + q];
                    double sv = (double)v_scale[b * d_in + q];
                    double root = sv * (double)((const int8_t *)v)[k];
                    m0 = sm * (double)((const int8_t *)m)[k];
                    v0 = root * root;
                    break;
                }
                }

                /* Algorithm 1: state update A ... */
                double m1 = b1 * m0 + (1.0 - b1) * g;
                double v1 = b2 * v0 + (1.0 - b2) * g * g;
                /* ... then weight update U, reading the new state. */
                double mhat = m1 / bc1;
                double vhat = v1 / bc2;
                double w0 = forge_oracle_bf16_to_f64(W[k]);
                double w1 = wdf * w0 - eta * mhat / (sqrt(vhat) + ep);

                W[k] = forge_oracle_f64_to_bf16(w1);
                if (W64) W64[k] = w1;
                if (m64) m64[k] = m1;
                if (v64) v64[k] = v1;
                switch (moment_dtype) {
                case ORACLE_MOMENT_F32:
                    ((float *)m)[k] = (float)m1;
                    ((float *)v)[k] = (float)v1;
                    break;
                case ORACLE_MOMENT_BF16:
                    ((uint16_t *)m)[k] = forge_oracle_f64_to_bf16(m1);
                    ((uint16_t *)v)[k] = forge_oracle_f64_to_bf16(v1);
                    break;
                default:
                    mnew[i * d_in + q] = m1;
                    vroot[i * d_in + q] = sqrt(v1);
                    break;
                }
            }
        }
        if (moment_dtype == ORACLE_MOMENT_I8) {
            int8_t *mc = (int8_t *)m, *vc = (int8_t *)v;
            for (int64_t q = 0; q < d_in; ++q) {
                m_scale[b * d_in + q] = quantize_column(
                    mnew + q, n, d_in, 0, mc + r0 * d_in + q, d_in, qm ? qm + r0 * d_in + q : NULL);
                v_scale[b * d_in + q] = quantize_column(
                    vroot + q, n, d_in, 1, vc + r0 * d_in + q, d_in, qv ? qv + r0 * d_in + q : NULL);
            }
            free(mnew);
            free(vroot);
        }
    }
}

/* ------------------------------------------------------- the whole fused step */

/* G = dY^T X, then the AdamW step; G is returned in G_out when it is non-NULL. */
void forge_oracle_linear_step(const uint16_t *X, const uint16_t *dY, uint16_t *W, void *m,
                              void *v, float *m_scale, float *v_scale, int64_t T,
                              int64_t d_in, int64_t d_out, int moment_dtype, float lr,
                              float beta1, float beta2, float eps, float weight_decay,
                              int64_t step, int round_grad_to_bf16, double *G_out,
                              double *W64, double *m64, double *v64, double *qm, double *qv)
{
    double *G = G_out ? G_out : (double *)malloc(sizeof(double) * (size_t)(d_in * d_out > 0 ? d_in * d_out : 1));
    forge_oracle_wgrad(X, dY, T, d_in, d_out, G);
    forge_oracle_adamw(G, W, m, v, m_scale, v_scale, d_in, d_out, moment_dtype, lr, beta1,
                       beta2, eps, weight_decay, step, round_grad_to_bf16, W64, m64, v64, qm, qv);
    if (!G_out) free(G);
}

/* ------------------------------------------------------------- int8, 64-wide row blocks */

/* Quantize row blocks: x fp64 [d_out, d_in] -> codes [d_out, d_in], scales [d_out, nb]. */
void forge_oracle_quantize_i8_row64(const double *x, int64_t d_in, int64_t d_out, int second_moment,
                                    int8_t *codes, float *scales, double *quot)
{
    const int64_t nb = (d_in + ORACLE_ROW_BLOCK - 1) / ORACLE_ROW_BLOCK;
#pragma omp parallel for schedule(static)
    for (int64_t p = 0; p < d_out; ++p)
        for (int64_t b = 0; b < nb; ++b) {
            const int64_t q0 = b * ORACLE_ROW_BLOCK;
            const int64_t n = d_in - q0 < ORACLE_ROW_BLOCK ? d_in - q0 : ORACLE_ROW_BLOCK;
            const int64_t k = p * d_in + q0;
            scales[p * nb + b] = quantize_column(x + k, n, 1, second_moment, codes + k, 1, quot ? quot + k : NULL);
        }
}

/*
 * AdamW (Algorithm 1) with the moments in the 64-wide row-block int8 layout: decode
 * m = s_m q_m and v = s_v q_v, update in fp64, W' from the unquantised m', v' (App. B: the
 * update arithmetic stays in full precision), then re-quantise m' and v' per row block.
 */
void forge_oracle_adamw_i8row(const double *G, uint16_t *W, int8_t *m, int8_t *v, float *m_scale,
                              float *v_scale, int64_t d_in, int64_t d_out, float lr, float beta1,
                              float beta2, float eps, float weight_decay, int64_t step, double *W64,
                              double *m64, double *v64, double *qm, double *qv)
{
    const double b1 = (double)beta1, b2 = (double)beta2;
    const double eta = (double)lr, lam = (double)weight_decay, ep = (double)eps;
    const double bc1 = 1.0 - pow(b1, (double)step);
    const double bc2 = 1.0 - pow(b2, (double)step);
    const double wdf = 1.0 - eta * lam;
    const int64_t nb = (d_in + ORACLE_ROW_BLOCK - 1) / ORACLE_ROW_BLOCK;
    double *mn = (double *)malloc(sizeof(double) * (size_t)(d_in * d_out > 0 ? d_in * d_out : 1));
    double *vn = (double *)malloc(sizeof(double) * (size_t)(d_in * d_out > 0 ? d_in * d_out : 1));
#pragma omp parallel for schedule(static)
    for (int64_t k = 0; k < d_in * d_out; ++k) {
        const int64_t p = k / d_in, q = k % d_in;
        const double m0 = (double)m_scale[p * nb + q / ORACLE_ROW_BLOCK] * (double)m[k];
        const double v0 = (double)v_scale[p * nb + q / ORACLE_ROW_BLOCK] * (double)v[k];
        const double g = G[k];
        const double m1 = b1 * m0 + (1.0 - b1) * g;
        const double v1 = b2 * v0 + (1.0 - b2) * g * g;
        const double w0 = forge_oracle_bf16_to_f64(W[k]);
        const double w1 = wdf * w0 - eta * (m1 / bc1) / (sqrt(v1 / bc2) + ep);
        W[k] = forge_oracle_f64_to_bf16(w1);
        mn[k] = m1;
        vn[k] = v1;
        if (W64) W64[k] = w1;
        if (m64) m64[k] = m1;
        if (v64) v64[k] = v1;
    }
    forge_oracle_quantize_i8_row64(mn, d_in, d_out, 0, m, m_scale, qm);
    forge_oracle_quantize_i8_row64(vn, d_in, d_out, 1, v, v_scale, qv);
    free(mn);
    free(vn);
}

/* ------------------------------------------------------------- fp8 (E4M3) encodings */

/* E4M3 code -> value (the OCP definition; codes 0x7F and 0xFF are NaN). */
double forge_oracle_e4m3_decode(uint8_t c)
{
    const int sign = c >> 7, e = (c >> 3) & 0xF, m = c & 7;
    if (e == 15 && m == 7) return NAN;
    const double v = e == 0 ? ldexp((double)m / 8.0, -6) : ldexp(1.0 + (double)m / 8.0, e - 7);
    return sign ? -v : v;
}

/* fp32 value, already within [-448, 448] -> nearest E4M3 code, ties to even. */
uint8_t forge_oracle_e4m3_encode(float x)
{
    const uint8_t sign = signbit(x) ? 0x80 : 0;
    double a = fabs((double)x);
    if (a > 448.0) a = 448.0;
    if (a < ldexp(1.0, -6)) {                   /* subnormal range: steps of 2^-9 */
        const double q = rint(ldexp(a, 9));      /* 0..8; 8 is the smallest normal, code 8 */
        return (uint8_t)(sign | (uint8_t)q);
    }
    int e;
    (void)frexp(a, &e);                          /* a = f * 2^e, 0.5 <= f < 1: exponent e - 1 */
    e -= 1;
    double q = rint(ldexp(a, 3 - e));            /* 8..16: the significand with 3 fraction bits */
    if (q == 16.0) {
        q = 8.0;
        e += 1;
    }
    return (uint8_t)(sign | (uint8_t)(((e + 7) << 3) | ((int)q - 8)));
}

void forge_oracle_e4m3_encode_array(const float *x, int64_t n, uint8_t *out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = forge_oracle_e4m3_encode(x[i]);
}

static float fp8_scale_of(float amax) { return amax > 0.0f ? amax / 448.0f : 1.0f; }

static float clamp448(float x) { return x > 448.0f ? 448.0f : (x < -448.0f ? -448.0f : x); }

/*
 * One AdamW step (Algorithm 1, fp64) with fp8 tensors.  w_fp8: W holds E4M3 codes with ring
 * w_ring, else bf16 bits.  m_fp8: m, v hold E4M3 codes of m and sqrt(v) with rings m_ring,
 * v_ring, else bf16 bits.  W64, m64, v64 (optional): unrounded fp64 results; qw, qm, qv
 * (optional): the fp32 quotients x/s that were encoded (0 where a tensor is bf16).
 */
void forge_oracle_adamw_fp8(const double *G, void *W, int w_fp8, float *w_ring, void *m, void *v, int m_fp8,
                            float *m_ring, float *v_ring, int64_t d_in, int64_t d_out, float lr, float beta1,
                            float beta2, float eps, float weight_decay, int64_t step, double *W64, double *m64,
                            double *v64, double *qw, double *qm, double *qv)
{
    const double b1 = beta1, b2 = beta2, eta = lr, lam = weight_decay, ep = eps;
    const double bc1 = 1.0 - pow(b1, (double)step), bc2 = 1.0 - pow(b2, (double)step);
    const double wdf = 1.0 - eta * lam;
    const int slot = (int)(step % 4), enc = (slot + 3) % 4, dec = (slot + 2) % 4, clr = (slot + 1) % 4;
    const float w_dec = w_fp8 ? fp8_scale_of(w_ring[dec]) : 1.0f, w_enc = w_fp8 ? fp8_scale_of(w_ring[enc]) : 1.0f;
    const float m_dec = m_fp8 ? fp8_scale_of(m_ring[dec]) : 1.0f, m_enc = m_fp8 ? fp8_scale_of(m_ring[enc]) : 1.0f;
    const float v_dec = m_fp8 ? fp8_scale_of(v_ring[dec]) : 1.0f, v_enc = m_fp8 ? fp8_scale_of(v_ring[enc]) : 1.0f;
    float aw = 0.0f, am = 0.0f, av = 0.0f;
    for (int64_t k = 0; k < d_in * d_out; ++k) {
        double w0, m0, v0;
        if (w_fp8) w0 = (double)w_dec * forge_oracle_e4m3_decode(((uint8_t *)W)[k]);
        else w0 = forge_oracle_bf16_to_f64(((uint16_t *)W)[k]);
        if (m_fp8) {
            m0 = (double)m_dec * forge_oracle_e4m3_decode(((uint8_t *)m)[k]);
            const double r0 = (double)v_dec * forge_oracle_e4m3_decode(((uint8_t *)v)[k]);
            v0 = r0 * r0;
        } else {
            m0 = forge_oracle_bf16_to_f64(((uint16_t *)m)[k]);
            v0 = forge_oracle_bf16_to_f64(((uint16_t *)v)[k]);
        }
        const double g = G[k];
        const double m1 = b1 * m0 + (1.0 - b1) * g;
        const double v1 = b2 * v0 + (1.0 - b2) * g * g;
        const double w1 = wdf * w0 - eta * (m1 / bc1) / (sqrt(v1 / bc2) + ep);
        const double r1 = sqrt(v1);
        if (W64) W64[k] = w1;
        if (m64) m64[k] = m1;
        if (v64) v64[k] = v1;
        if (w_fp8) {
            const float qf = (float)w1 / w_enc;
            ((uint8_t *)W)[k] = forge_oracle_e4m3_encode(clamp448(qf));
            if (qw) qw[k] = qf;
            if (fabsf((float)w1) > aw) aw = fabsf((float)w1);
        } else {
            ((uint16_t *)W)[k] = forge_oracle_f64_to_bf16(w1);
            if (qw) qw[k] = 0.0;
        }
        if (m_fp8) {
            const float qmf = (float)m1 / m_enc, qvf = (float)r1 / v_enc;
            uint8_t cv = forge_oracle_e4m3_encode(clamp448(qvf));
            if (r1 > 0.0 && (cv & 0x7F) == 0) cv = 1;
            ((uint8_t *)m)[k] = forge_oracle_e4m3_encode(clamp448(qmf));
            ((uint8_t *)v)[k] = cv;
            if (qm) qm[k] = qmf;
            if (qv) qv[k] = qvf;
            if (fabsf((float)m1) > am) am = fabsf((float)m1);
            if ((float)r1 > av) av = (float)r1;
        } else {
            ((uint16_t *)m)[k] = forge_oracle_f64_to_bf16(m1);
            ((uint16_t *)v)[k] = forge_oracle_f64_to_bf16(v1);
            if (qm) qm[k] = 0.0;
            if (qv) qv[k] = 0.0;
        }
    }
    if (w_fp8) {
        if (aw > w_ring[slot]) w_ring[slot] = aw;
        w_ring[clr] = 0.0f;
    }
    if (m_fp8) {
        if (am > m_ring[slot]) m_ring[slot] = am;
        if (av > v_ring[slot]) v_ring[slot] = av;
        m_ring[clr] = 0.0f;
        v_ring[clr] = 0.0f;
    }
}

/* ------------------------------------------------------------- other update rules */

enum {
    ORACLE_OPT_ADAMW = 0, ORACLE_OPT_SGD = 1, ORACLE_OPT_SGD_MOMENTUM = 2, ORACLE_OPT_ADAGRAD = 3,
    ORACLE_OPT_RMSPROP = 4, ORACLE_OPT_LION = 5, ORACLE_OPT_NADAM = 6, ORACLE_OPT_RADAM = 7,
    ORACLE_OPT_ADAMAX = 8, ORACLE_OPT_MUON = 9
};

static double load_state(const void *s, int64_t k, int dtype)
{
    if (!s) return 0.0;
    if (dtype == ORACLE_MOMENT_F32) return (double)((const float *)s)[k];
    return forge_oracle_bf16_to_f64(((const uint16_t *)s)[k]);
}

static void store_state(void *s, int64_t k, int dtype, double x)
{
    if (!s) return;
    if (dtype == ORACLE_MOMENT_F32) ((float *)s)[k] = (float)x;   /* C cast: round to nearest even */
    else ((uint16_t *)s)[k] = forge_oracle_f64_to_bf16(x);
}

/*
 * One step of update rule `opt` on the fp64 gradient G [d_out, d_in] (AdamW has its own
 * routine above).  W: bf16 bits [d_out, d_in], in/out (untouched by the Muon accumulate).
 * s1, s2: state tensors in `state_dtype` (fp32 or bf16), in/out; NULL for a state the rule
 * does not have.  W64, S1, S2 (optional): the unrounded fp64 results.  AUX (optional): the
 * argument of Lion's sign, which a test needs to recognise elements where the sign is
 * decided within rounding error.  Hyper-parameters are promoted from fp32 to fp64.
 *
 *   SGD       gg = g + wd w;  w' = w - lr gg
 *   SGD-m     b' = beta1 b + gg;  w' = w - lr b'            (dampening 0, no Nesterov)
 *   Adagrad   s' = s + gg^2;  w' = w - clr gg / (sqrt(s') + eps),  clr = lr / (1 + (t-1) lr_decay)
 *   RMSprop   a' = beta2 a + (1 - beta2) gg^2;  w' = w - lr gg / (sqrt(a') + eps)
 *   Lion      c = beta1 m + (1 - beta1) g;  w' = w (1 - lr wd) - lr sign(c);
 *             m' = beta2 m + (1 - beta2) g
 *   NAdam     mu_i = beta1 (1 - 0.5 * 0.96^(i psi)), P_t = prod_{i<=t} mu_i;
 *             m', v' the Adam moments of gg;  d = sqrt(v' / (1 - beta2^t)) + eps;
 *             w' = w - lr (1 - mu_t) / (1 - P_t) gg / d - lr mu_{t+1} / (1 - P_t mu_{t+1}) m' / d
 *   RAdam     m', v' the Adam moments of gg;  mhat = m' / (1 - beta1^t);
 *             rho_inf = 2 / (1 - beta2) - 1;  rho_t = rho_inf - 2 t beta2^t / (1 - beta2^t);
 *             rho_t > 5: w' = w - lr mhat r sqrt(1 - beta2^t) / (sqrt(v') + eps),
 *                        r = sqrt((rho_t - 4)(rho_t - 2) rho_inf / ((rho_inf - 4)(rho_inf - 2) rho_t));
 *             else       w' = w - lr mhat
 *   Adamax    m' = beta1 m + (1 - beta1) gg;  u' = max(beta2 u, |gg| + eps);
 *             w' = w - lr / (1 - beta1^t) m' / u'
 *   Muon      B' = beta1 B + g  (W unchanged)
 */
void forge_oracle_rule_step(const double *G, uint16_t *W, void *s1, void *s2, int64_t d_in, int64_t d_out,
                            int opt, int state_dtype, float lr, float beta1, float beta2, float eps,
                            float weight_decay, float lr_decay, float momentum_decay, int64_t step,
                            double *W64, double *S1, double *S2, double *AUX)
{
    const double eta = lr, b1 = beta1, b2 = beta2, ep = eps, lam = weight_decay, t = (double)step;
    const double bc1 = 1.0 - pow(b1, t), bc2 = 1.0 - pow(b2, t);
    /* NAdam's momentum schedule */
    double mu_t = 0.0, mu_next = 0.0, prod = 1.0;
    if (opt == ORACLE_OPT_NADAM) {
        for (int64_t i = 1; i <= step; ++i)
            prod *= b1 * (1.0 - 0.5 * pow(0.96, (double)i * (double)momentum_decay));
        mu_t = b1 * (1.0 - 0.5 * pow(0.96, t * (double)momentum_decay));
        mu_next = b1 * (1.0 - 0.5 * pow(0.96, (t + 1.0) * (double)momentum_decay));
    }
    /* RAdam's rectification */
    double rho_inf = 0.0, rho_t = 0.0, rect = 0.0;
    if (opt == ORACLE_OPT_RADAM) {
        rho_inf = 2.0 / (1.0 - b2) - 1.0;
        rho_t = rho_inf - 2.0 * t * pow(b2, t) / bc2;
        if (rho_t > 5.0)
            rect = sqrt((rho_t - 4.0) * (rho_t - 2.0) * rho_inf / ((rho_inf - 4.0) * (rho_inf - 2.0) * rho_t));
    }
    const double clr = eta / (1.0 + (t - 1.0) * (double)lr_decay);

#pragma omp parallel for schedule(static)
    for (int64_t k = 0; k < d_in * d_out; ++k) {
        const double g = G[k];
        const double w = forge_oracle_bf16_to_f64(W[k]);
        const double a = load_state(s1, k, state_dtype);
        const double b = load_state(s2, k, state_dtype);
        const double gg = g + lam * w;
        double w1 = w, a1 = a, bb1 = b, aux = 0.0;
        switch (opt) {
        case ORACLE_OPT_SGD:
            w1 = w - eta * gg;
            break;
        case ORACLE_OPT_SGD_MOMENTUM:
            a1 = b1 * a + gg;
            w1 = w - eta * a1;
            break;
        case ORACLE_OPT_ADAGRAD:
            a1 = a + gg * gg;
            w1 = w - clr * gg / (sqrt(a1) + ep);
            break;
        case ORACLE_OPT_RMSPROP:
            a1 = b2 * a + (1.0 - b2) * gg * gg;
            w1 = w - eta * gg / (sqrt(a1) + ep);
            break;
        case ORACLE_OPT_LION: {
            const double c = b1 * a + (1.0 - b1) * g;
            const double sg = c > 0.0 ? 1.0 : (c < 0.0 ? -1.0 : 0.0);
            aux = c;
            w1 = w * (1.0 - eta * lam) - eta * sg;
            a1 = b2 * a + (1.0 - b2) * g;
            break;
        }
        case ORACLE_OPT_NADAM: {
            a1 = b1 * a + (1.0 - b1) * gg;
            bb1 = b2 * b + (1.0 - b2) * gg * gg;
            const double d = sqrt(bb1 / bc2) + ep;
            w1 = w - eta * (1.0 - mu_t) / (1.0 - prod) * gg / d - eta * mu_next / (1.0 - prod * mu_next) * a1 / d;
            break;
        }
        case ORACLE_OPT_RADAM: {
            a1 = b1 * a + (1.0 - b1) * gg;
            bb1 = b2 * b + (1.0 - b2) * gg * gg;
            const double mhat = a1 / bc1;
            if (rho_t > 5.0) w1 = w - eta * mhat * rect * sqrt(bc2) / (sqrt(bb1) + ep);
            else w1 = w - eta * mhat;
            break;
        }
        case ORACLE_OPT_ADAMAX: {
            a1 = b1 * a + (1.0 - b1) * gg;
            const double n = fabs(gg) + ep;
            bb1 = b2 * b > n ? b2 * b : n;
            w1 = w - eta / bc1 * a1 / bb1;
            break;
        }
        case ORACLE_OPT_MUON:
            a1 = b1 * a + g;
            w1 = w;
            break;
        default:
            break;
        }
        if (opt != ORACLE_OPT_MUON) W[k] = forge_oracle_f64_to_bf16(w1);
        store_state(s1, k, state_dtype, a1);
        store_state(s2, k, state_dtype, bb1);
        if (W64) W64[k] = w1;
        if (S1) S1[k] = a1;
        if (S2) S2[k] = bb1;
        if (AUX) AUX[k] = aux;
    }
}

int forge_oracle_num_threads(void)
{
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads the oracle's parallel loops use from now on (n >= 1); for timing runs. */
void forge_oracle_set_num_threads(int n)
{
#ifdef _OPENMP
    extern void omp_set_num_threads(int);
    if (n >= 1) omp_set_num_threads(n);
#else
    (void)n;
#endif
}
