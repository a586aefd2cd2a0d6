/*
 * mpfa_oracle.c -- plain, slow CPU oracle for QK4PV8 FlashAttention (MpFA).
 *
 * TEST INFRASTRUCTURE ONLY: loaded by the tests, the smoke check and the CPU
 * baseline leg of the benchmark; never by the product library.  It shares no
 * code with the HIP path.
 *
 * Each function follows a passage of the paper (cited in its comment).  All
 * arithmetic between the method's rounding points is FP64; the rounding
 * points themselves (R2..R8, see the header) are taken exactly as specified,
 * with FP32 where the method computes in FP32 (means, centering, the scale
 * division, the Delta_S dot product).
 *
 * Build: gcc -std=c11 -O2 -ffp-contract=off -fopenmp -fPIC -shared (no
 * fast-math: IEEE semantics are part of the specification).
 */
#include "mpfa_oracle.h"

#include <assert.h>
#include <float.h>
#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* -------------------------------------------------------------------------- */
/* Number formats                                                              */
/* -------------------------------------------------------------------------- */

/* E2M1 (Sec. 2.1, Eq. 1; rho = 6 is its largest magnitude): one sign bit, two
 * exponent bits, one mantissa bit.  Magnitudes by code 0..7. */
static const double E2M1_MAG[8] = {0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0};

double orc_e2m1_value(uint8_t code)
{
    double v = E2M1_MAG[code & 7];
    return (code & 8) ? -v : v;
}

/* Round to the nearest E2M1 value; a tie goes to the even code (the one whose
 * mantissa bit is 0); magnitudes above 6 saturate to 6.  The sign of the input
 * is kept, also for results of magnitude zero. */
uint8_t orc_e2m1_encode(double y)
{
    assert(!isnan(y));
    uint8_t sign = signbit(y) ? 8 : 0;
    double a = fabs(y);
    if (a >= 6.0) return (uint8_t)(sign | 7);   /* saturate (also avoids cancellation) */
    int best = 0;
    double bestd = a;
    for (int c = 1; c < 8; ++c) {
        double d = fabs(a - E2M1_MAG[c]);
        if (d < bestd || (d == bestd && (c % 2) == 0)) {
            best = c;
            bestd = d;
        }
    }
    return (uint8_t)(sign | best);
}

/* OCP FP8 E4M3 ("FN" variant): bias 7, no infinities, S.1111.111 is NaN, so
 * the largest finite magnitude is 448 (Sec. 4.1 uses 448 as the fixed P
 * scale for exactly that reason). */
double orc_e4m3_value(uint8_t code)
{
    int e = (code >> 3) & 15;
    int m = code & 7;
    double v;
    if (e == 15 && m == 7) return NAN;
    if (e == 0)
        v = ldexp((double)m / 8.0, -6);
    else
        v = ldexp(1.0 + (double)m / 8.0, e - 7);
    return (code & 0x80) ? -v : v;
}

/* Round to the nearest finite E4M3 value (codes 0x00..0x7E are increasing in
 * magnitude); ties to the even code; magnitudes above 448 saturate to 448. */
uint8_t orc_e4m3_encode(double x)
{
    assert(!isnan(x));
    uint8_t sign = signbit(x) ? 0x80 : 0;
    double a = fabs(x);
    if (a >= 448.0) return (uint8_t)(sign | 0x7E);
    /* largest code c with value(c) <= a, by bisection over 0..0x7E */
    int lo = 0, hi = 0x7E;
    while (lo < hi) {
        int mid = (lo + hi + 1) / 2;
        if (orc_e4m3_value((uint8_t)mid) <= a) lo = mid; else hi = mid - 1;
    }
    int c = lo;
    double d0 = a - orc_e4m3_value((uint8_t)c);
    double d1 = orc_e4m3_value((uint8_t)(c + 1)) - a;
    int pick;
    if (d0 < d1) pick = c;
    else if (d1 < d0) pick = c + 1;
    else pick = (c % 2 == 0) ? c : c + 1;
    return (uint8_t)(sign | pick);
}

float orc_bf16_value(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

/* Nearest BF16 value of a finite double (BF16 keeps the upper 16 bits of an
 * FP32 pattern): among the BF16 neighbours of x the closer one, the one with
 * an even last bit on a tie.  Finite inputs only. */
static uint16_t bf16_nearest(double x)
{
    float f = (float)x;
    uint32_t u;
    memcpy(&u, &f, 4);
    if (isnan(x)) return (uint16_t)((u >> 16) | 0x40);
    uint16_t base = (uint16_t)(u >> 16);
    uint16_t lo_lim = (base & 0x8000) ? 0x8000 : 0x0000;
    uint16_t hi_lim = (base & 0x8000) ? 0xFF80 : 0x7F80;
    uint16_t best = base;
    double bestd = fabs(x - (double)orc_bf16_value(base));
    uint16_t cand[2];
    int nc = 0;
    if (base > lo_lim) cand[nc++] = (uint16_t)(base - 1);
    if ((uint16_t)(base + 1) < hi_lim) cand[nc++] = (uint16_t)(base + 1);
    for (int i = 0; i < nc; ++i) {
        double d = fabs(x - (double)orc_bf16_value(cand[i]));
        if (d < bestd || (d == bestd && (cand[i] & 1) == 0)) {
            best = cand[i];
            bestd = d;
        }
    }
    return best;
}

uint16_t orc_bf16_encode(float x) { return bf16_nearest((double)x); }

uint16_t orc_bf16_encode_f64(double x) { return bf16_nearest(x); }

void orc_e4m3_encode_f32_array(const float* x, int64_t n, uint8_t* out)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = isnan(x[i]) ? 0x7F : orc_e4m3_encode((double)x[i]);
}

void orc_e2m1_encode_f32_array(const float* x, int64_t n, uint8_t* out)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = isnan(x[i]) ? 0xFF : orc_e2m1_encode((double)x[i]);
}

void orc_bf16_encode_f32_array(const float* x, int64_t n, uint16_t* out)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = orc_bf16_encode(x[i]);
}

/* -------------------------------------------------------------------------- */
/* Quantization pass (the steps of Algorithm 1 before its main loop)           */
/* -------------------------------------------------------------------------- */

/* Second-level scale of NVFP4: a power of two chosen so that the largest
 * group scale amax/(6t) lands in (224, 448], i.e. the smallest t = 2^k with
 * 6 * 448 * t >= amax.  A power of two keeps every fold of t exact.  k is
 * clamped to [-63, 63] so that the product of a query and a key tensor scale,
 * and its inverse, stay normal FP32 numbers (2^-126 .. 2^126). */
float orc_tensor_scale(float amax)
{
    if (!(amax > 0.0f)) return 1.0f;
    double a = (double)amax;
    int k = (int)ceil(log2(a / 2688.0));
    /* correct any log2 rounding with exact comparisons */
    while (k > -200 && ldexp(2688.0, k - 1) >= a) --k;
    while (ldexp(2688.0, k) < a) ++k;
    if (k < -63) k = -63;
    if (k > 63) k = 63;
    return (float)ldexp(1.0, k);
}

/* Eq. 7: the per-(sequence, head) mean over the valid tokens, summed in FP32
 * in a fixed order (sequentially inside 128-token blocks, then the block
 * partials sequentially), divided in FP32 and rounded to BF16. */
void orc_stats_one(const uint16_t* x, int64_t n_tok, int64_t stride, int smooth,
                   int tscale_unit, uint16_t* mean_out, float* tscale_out)
{
    float meanf[ORC_D];
    for (int c = 0; c < ORC_D; ++c) {
        uint16_t mb = 0;
        if (smooth && n_tok > 0) {
            float total = 0.0f;
            for (int64_t b0 = 0; b0 < n_tok; b0 += 128) {
                float part = 0.0f;
                int64_t b1 = b0 + 128 < n_tok ? b0 + 128 : n_tok;
                for (int64_t t = b0; t < b1; ++t) part += orc_bf16_value(x[t * stride + c]);
                total += part;
            }
            float mean = total / (float)n_tok;
            mb = orc_bf16_encode(mean);
        }
        mean_out[c] = mb;
        meanf[c] = orc_bf16_value(mb);
    }
    float amax = 0.0f;
    for (int64_t t = 0; t < n_tok; ++t)
        for (int c = 0; c < ORC_D; ++c) {
            float xc = orc_bf16_value(x[t * stride + c]) - meanf[c];
            float ax = fabsf(xc);
            if (ax > amax) amax = ax;
        }
    *tscale_out = tscale_unit ? 1.0f : orc_tensor_scale(amax);
}

/* amax of the centered values of one (sequence, head) against a given mean. */
static float centered_amax(const uint16_t* x, int64_t n_tok, int64_t stride, const uint16_t* mean)
{
    float amax = 0.0f;
    for (int64_t t = 0; t < n_tok; ++t)
        for (int c = 0; c < ORC_D; ++c) {
            float xc = orc_bf16_value(x[t * stride + c]) - orc_bf16_value(mean[c]);
            float ax = fabsf(xc);
            if (ax > amax) amax = ax;
        }
    return amax;
}

/* Eq. 1 with a 16-element group and an E4M3 group scale s_g = amax/rho,
 * rho = 6, on top of the power-of-two tensor scale t:
 *   s_code = E4M3(amax / (6 t)),   code = E2M1(x / (t * dec(s_code))).
 * The divisions are FP32 IEEE divisions.  A group whose scale rounds to zero
 * keeps only the signs of its elements. */
void orc_nvfp4_row(const float* xc, float t, uint8_t* codes64, uint8_t* scales8)
{
    uint8_t code[ORC_D];
    for (int g = 0; g < ORC_NG; ++g) {
        float a = 0.0f;
        for (int i = 0; i < ORC_G; ++i) {
            float ax = fabsf(xc[g * ORC_G + i]);
            if (ax > a) a = ax;
        }
        float six_t = 6.0f * t;
        float ratio = a / six_t;
        uint8_t s = orc_e4m3_encode((double)ratio);
        scales8[g] = s;
        double sd = orc_e4m3_value(s);
        for (int i = 0; i < ORC_G; ++i) {
            float x = xc[g * ORC_G + i];
            if (sd == 0.0) {
                code[g * ORC_G + i] = signbit(x) ? 8 : 0;
            } else {
                float scale = t * (float)sd;       /* exact: t is a power of two */
                float y = x / scale;
                code[g * ORC_G + i] = orc_e2m1_encode((double)y);
            }
        }
    }
    for (int j = 0; j < ORC_D / 2; ++j)
        codes64[j] = (uint8_t)(code[2 * j] | (code[2 * j + 1] << 4));
}

void orc_nvfp4_dequant_row(const uint8_t* codes64, const uint8_t* scales8, double t, double* out)
{
    for (int c = 0; c < ORC_D; ++c) {
        uint8_t byte = codes64[c / 2];
        uint8_t code = (c & 1) ? (byte >> 4) : (byte & 15);
        out[c] = t * orc_e4m3_value(scales8[c / ORC_G]) * orc_e2m1_value(code);
    }
}

void orc_mxfp4_row(const float* xc, uint8_t* codes64, uint8_t* scales8)
{
    uint8_t code[ORC_D];
    for (int g = 0; g < 4; ++g) {
        double a = 0.0;
        for (int i = 0; i < 32; ++i) {
            double ax = fabs((double)xc[g * 32 + i]);
            if (ax > a) a = ax;
        }
        int e = -127;
        if (a > 0.0) {
            int ex;
            frexp(a, &ex);                 /* a = m * 2^ex, m in [0.5, 1) */
            e = (ex - 1) - 2;              /* floor(log2 a) - 2 */
            if (e < -127) e = -127;
            if (e > 127) e = 127;
        }
        scales8[g] = (uint8_t)(e + 127);
        for (int i = 0; i < 32; ++i) {
            double y = ldexp((double)xc[g * 32 + i], -e);    /* exact */
            code[g * 32 + i] = orc_e2m1_encode(y);
        }
    }
    for (int g = 4; g < 8; ++g) scales8[g] = 0;
    for (int j = 0; j < ORC_D / 2; ++j)
        codes64[j] = (uint8_t)(code[2 * j] | (code[2 * j + 1] << 4));
}

void orc_mxfp4_dequant_row(const uint8_t* codes64, const uint8_t* scales8, double* out)
{
    for (int c = 0; c < ORC_D; ++c) {
        uint8_t byte = codes64[c / 2];
        uint8_t code = (c & 1) ? (byte >> 4) : (byte & 15);
        out[c] = ldexp(orc_e2m1_value(code), (int)scales8[c / 32] - 127);
    }
}

/* Algorithm 1 stage one, fused with the cache write (Sec. 5.1, Sec. 6):
 * statistics (first prefill only, then frozen), centering, NVFP4 Q and K,
 * FP8 V (no scale, not centered, Sec. 4.2), and Delta_S = Qbar . K_c per key
 * and query head (Eq. 9) as an FP32 fused multiply-add chain over the
 * channels, rounded to BF16 (the compensation is carried in BF16, Sec. 7.4).
 * Query head h uses KV head h / (h_q / h_kv). */
/* V as NVFP4 along keys (characterization of Sec. 3.1): for every page a
 * sequence of this call occupies and every (KV head, channel), the page's 64
 * values (absent slots as zero) form four 16-key groups, quantized with the
 * same group rule as Q/K rows (Eq. 1) and tensor scale 1.  The row quantizer
 * takes 8 groups; the page fills the first four. */
static void nvfp4_v_pages(const orc_quant_args* a, int64_t n_pages)
{
    const int Hkv = a->h_kv;
    uint8_t* aux = (uint8_t*)a->v_aux;
    uint8_t* aux_scales = aux + n_pages * Hkv * ORC_D * 32;
    for (int b = 0; b < a->batch; ++b) {
        int64_t t0 = a->cu_seqlens[b], n = a->cu_seqlens[b + 1] - t0;
        for (int64_t p0 = 0; p0 < n; p0 += ORC_PAGE) {
            int64_t page = a->slot_mapping[t0 + p0] / ORC_PAGE;
            int64_t cnt = n - p0 < ORC_PAGE ? n - p0 : ORC_PAGE;
            for (int h = 0; h < Hkv; ++h) {
                for (int c = 0; c < ORC_D; ++c) {
                    float vals[ORC_D];
                    uint8_t codes[64], scales[8];
                    for (int j = 0; j < ORC_D; ++j) vals[j] = 0.0f;
                    for (int64_t j = 0; j < cnt; ++j)
                        vals[j] = orc_bf16_value(a->v[((t0 + p0 + j) * Hkv + h) * ORC_D + c]);
                    orc_nvfp4_row(vals, 1.0f, codes, scales);
                    const int64_t r = (page * Hkv + h) * ORC_D + c;
                    memcpy(aux + r * 32, codes, 32);
                    memcpy(aux_scales + r * 4, scales, 4);
                }
            }
        }
    }
}

int orc_quantize_qk(const orc_quant_args* a)
{
    const int B = a->batch, Hq = a->h_q, Hkv = a->h_kv;
    if (B < 0 || Hq <= 0 || Hkv <= 0 || Hkv > 64 || Hq % Hkv) return -1;
    const int smooth = (a->flags & ORC_SMOOTH) != 0;
    const int stats = (a->flags & ORC_COMPUTE_STATS) != 0;
    const int mx = (a->flags & ORC_MXFP4) != 0;
    const int tunit = (a->flags & ORC_TSCALE_UNIT) != 0 || mx;   /* MXFP4: no tensor scale */
    const int grp = Hq / Hkv;

    for (int b = 0; b < B; ++b) {
        int64_t t0 = a->cu_seqlens[b], n = a->cu_seqlens[b + 1] - a->cu_seqlens[b];
        for (int h = 0; h < Hq; ++h) {
            const uint16_t* x = a->q + (t0 * Hq + h) * ORC_D;
            uint16_t* mean = a->q_mean + ((int64_t)b * Hq + h) * ORC_D;
            if (stats) {
                orc_stats_one(x, n, (int64_t)Hq * ORC_D, smooth, tunit, mean,
                              &a->q_tscale[(int64_t)b * Hq + h]);
            } else {
                float amax = centered_amax(x, n, (int64_t)Hq * ORC_D, mean);
                a->q_tscale[(int64_t)b * Hq + h] = tunit ? 1.0f : orc_tensor_scale(amax);
            }
        }
        if (stats) {
            for (int h = 0; h < Hkv; ++h) {
                const uint16_t* x = a->k + (t0 * Hkv + h) * ORC_D;
                orc_stats_one(x, n, (int64_t)Hkv * ORC_D, smooth, tunit,
                              a->k_mean + ((int64_t)b * Hkv + h) * ORC_D,
                              &a->k_tscale[(int64_t)b * Hkv + h]);
            }
        }
    }

    const int pv_bf16 = (a->flags & ORC_PV_BF16) != 0, pv_nv = (a->flags & ORC_PV_NVFP4) != 0;
    if (pv_bf16 && pv_nv) return -1;
    if ((pv_bf16 || pv_nv) && !a->v_aux) return -1;
    if (pv_nv) {   /* fresh-prefill layout: token i of a sequence at slot i % 64 of its page */
        for (int b = 0; b < B; ++b) {
            int64_t t0 = a->cu_seqlens[b], n = a->cu_seqlens[b + 1] - t0;
            for (int64_t i = 0; i < n; ++i) {
                int64_t first = a->slot_mapping[t0 + i - i % ORC_PAGE];
                if (first % ORC_PAGE != 0 || a->slot_mapping[t0 + i] != first + i % ORC_PAGE) return -2;
            }
        }
    }

    for (int b = 0; b < B; ++b) {
        int64_t t0 = a->cu_seqlens[b], t1 = a->cu_seqlens[b + 1];
#pragma omp parallel for schedule(static)
        for (int64_t tok = t0; tok < t1; ++tok) {
            float xc[ORC_D];
            float kc[ORC_D * 64];   /* up to 64 KV heads per call */
            int64_t slot = a->slot_mapping[tok];
            int64_t page = slot / ORC_PAGE, off = slot % ORC_PAGE;
            for (int h = 0; h < Hq; ++h) {
                const uint16_t* x = a->q + (tok * Hq + h) * ORC_D;
                const uint16_t* mean = a->q_mean + ((int64_t)b * Hq + h) * ORC_D;
                for (int c = 0; c < ORC_D; ++c)
                    xc[c] = orc_bf16_value(x[c]) - (smooth ? orc_bf16_value(mean[c]) : 0.0f);
                if (mx)
                    orc_mxfp4_row(xc, a->q_codes + (tok * Hq + h) * 64, a->q_scales + (tok * Hq + h) * 8);
                else
                    orc_nvfp4_row(xc, a->q_tscale[(int64_t)b * Hq + h],
                                  a->q_codes + (tok * Hq + h) * 64, a->q_scales + (tok * Hq + h) * 8);
            }
            for (int h = 0; h < Hkv; ++h) {
                const uint16_t* x = a->k + (tok * Hkv + h) * ORC_D;
                const uint16_t* mean = a->k_mean + ((int64_t)b * Hkv + h) * ORC_D;
                float* kch = kc + h * ORC_D;
                for (int c = 0; c < ORC_D; ++c)
                    kch[c] = orc_bf16_value(x[c]) - (smooth ? orc_bf16_value(mean[c]) : 0.0f);
                int64_t row = (page * Hkv + h) * ORC_PAGE + off;
                if (mx)
                    orc_mxfp4_row(kch, a->k_codes + row * 64, a->k_scales + row * 8);
                else
                    orc_nvfp4_row(kch, a->k_tscale[(int64_t)b * Hkv + h],
                                  a->k_codes + row * 64, a->k_scales + row * 8);
                const uint16_t* vx = a->v + (tok * Hkv + h) * ORC_D;
                for (int c = 0; c < ORC_D; ++c)
                    a->v_codes[((page * Hkv + h) * ORC_D + c) * ORC_PAGE + off] =
                        orc_e4m3_encode((double)orc_bf16_value(vx[c]));
                if (pv_bf16)
                    for (int c = 0; c < ORC_D; ++c)
                        ((uint16_t*)a->v_aux)[((page * Hkv + h) * ORC_D + c) * ORC_PAGE + off] = vx[c];
            }
            if (smooth) {
                for (int h = 0; h < Hq; ++h) {
                    const uint16_t* qm = a->q_mean + ((int64_t)b * Hq + h) * ORC_D;
                    const float* kch = kc + (h / grp) * ORC_D;
                    float d = 0.0f;
                    for (int c = 0; c < ORC_D; ++c) d = fmaf(orc_bf16_value(qm[c]), kch[c], d);
                    a->ds[(page * Hq + h) * ORC_PAGE + off] = orc_bf16_encode(d);
                }
            }
        }
    }
    if (pv_nv) nvfp4_v_pages(a, a->num_pages);
    return 0;
}

/* -------------------------------------------------------------------------- */
/* Attention core                                                              */
/* -------------------------------------------------------------------------- */

/* lambda = log2(e) / sqrt(d): the softmax scale folded into the base-2
 * exponent (Algorithm 1, P update; Sec. 5.1 last paragraph). */
static double lambda_d(void) { return 1.0 / (log(2.0) * sqrt((double)ORC_D)); }

void orc_state_init(orc_state* s)
{
    s->m = -INFINITY;
    s->l = 0.0;
    for (int c = 0; c < ORC_D; ++c) s->o[c] = 0.0;
}

/* Online softmax (Eqs. 3-6 in base 2, Algorithm 1 main loop) over one key
 * range, one KV tile at a time:
 *   S     = q . k (+ Delta_S[key]); keys after the query masked (after the
 *           compensation, before the maximum, Sec. 4.3)
 *   m'    = max(m, rowmax S)
 *   alpha = 2^(lambda (m - m'))      (0 while m is still -inf)
 *   P     = 2^(lambda (S - m'))
 *   l     = alpha l + sum P          (unquantized P)
 *   P_hat = E4M3(448 P)              (Sec. 4.1, fixed scale, relative to m')
 *   O     = alpha O + sum P_hat v
 * The tile order is reversed when ORC_REVERSE is set (Sec. 4.1, last
 * paragraph). */
void orc_visit(orc_state* st, const double* qd, const double* kd, const double* vd,
               const double* dsd, int64_t q_pos, int64_t key_lo, int64_t key_hi,
               int tile, int flags)
{
    if (key_hi <= key_lo) return;
    const double lam = lambda_d();
    const int quant_p = (flags & ORC_QUANT_P) != 0;
    const int p_bf16 = (flags & ORC_P_BF16) != 0, p_nv = (flags & ORC_P_NVFP4) != 0;
    int64_t first = key_lo / tile, last = (key_hi - 1) / tile;
    double* s = (double*)malloc(sizeof(double) * (size_t)tile);
    double* w_nv = (double*)malloc(sizeof(double) * (size_t)tile);
    for (int64_t it = 0; it <= last - first; ++it) {
        int64_t j = (flags & ORC_REVERSE) ? last - it : first + it;
        int64_t lo = j * tile > key_lo ? j * tile : key_lo;
        int64_t hi = (j + 1) * tile < key_hi ? (j + 1) * tile : key_hi;
        double tmax = -INFINITY;
        for (int64_t key = lo; key < hi; ++key) {
            double v = 0.0;
            const double* kr = kd + key * ORC_D;
            for (int c = 0; c < ORC_D; ++c) v += qd[c] * kr[c];
            if (dsd) v += dsd[key];
            if (key > q_pos) v = -INFINITY;
            s[key - lo] = v;
            if (v > tmax) tmax = v;
        }
        double m_new = st->m > tmax ? st->m : tmax;
        if (m_new == -INFINITY) continue;          /* nothing visible yet */
        double alpha = (st->m == -INFINITY) ? 0.0 : exp2(lam * (st->m - m_new));
        double l_add = 0.0;
        double o_add[ORC_D];
        for (int c = 0; c < ORC_D; ++c) o_add[c] = 0.0;
        if (p_nv) {
            /* P' = 2688 P (the largest P, 1, maps to 6 * 448), then one NVFP4
             * group per 16 keys aligned to multiples of 16 (Eq. 1, tensor scale
             * 1): scale = E4M3(amax / 6), weight = scale * E2M1(P' / scale). */
            for (int64_t key = lo; key < hi; ++key) {
                double v = s[key - lo];
                w_nv[key - lo] = v == -INFINITY ? 0.0 : 2688.0 * exp2(lam * (v - m_new));
            }
            for (int64_t g0 = lo - lo % 16; g0 < hi; g0 += 16) {
                int64_t a0 = g0 > lo ? g0 : lo, a1 = g0 + 16 < hi ? g0 + 16 : hi;
                double amax = 0.0;
                for (int64_t key = a0; key < a1; ++key)
                    if (w_nv[key - lo] > amax) amax = w_nv[key - lo];
                double sd = orc_e4m3_value(orc_e4m3_encode(amax / 6.0));
                for (int64_t key = a0; key < a1; ++key)
                    w_nv[key - lo] = sd == 0.0 ? 0.0 : sd * orc_e2m1_value(orc_e2m1_encode(w_nv[key - lo] / sd));
            }
        }
        for (int64_t key = lo; key < hi; ++key) {
            double v = s[key - lo];
            if (v == -INFINITY) continue;
            double p = exp2(lam * (v - m_new));
            l_add += p;
            double w = quant_p ? orc_e4m3_value(orc_e4m3_encode(448.0 * p))
                     : p_bf16  ? (double)orc_bf16_value(orc_bf16_encode_f64(p))
                     : p_nv    ? w_nv[key - lo]
                               : p;
            if (w == 0.0) continue;
            const double* vr = vd + key * ORC_D;
            for (int c = 0; c < ORC_D; ++c) o_add[c] += w * vr[c];
        }
        st->l = alpha * st->l + l_add;
        for (int c = 0; c < ORC_D; ++c) st->o[c] = alpha * st->o[c] + o_add[c];
        st->m = m_new;
    }
    free(s);
    free(w_nv);
}

/* Log-sum-exp merge of split-KV partition states (Sec. 5.3), then the final
 * normalisation O / l (O / (448 l) when O carries 448-scaled P codes). */
void orc_merge(const orc_state* parts, int n, double* out, double p_scale)
{
    const double lam = lambda_d();
    double M = -INFINITY;
    for (int p = 0; p < n; ++p) if (parts[p].m > M) M = parts[p].m;
    for (int c = 0; c < ORC_D; ++c) out[c] = 0.0;
    if (M == -INFINITY) return;
    double l = 0.0;
    double o[ORC_D];
    for (int c = 0; c < ORC_D; ++c) o[c] = 0.0;
    for (int p = 0; p < n; ++p) {
        if (parts[p].m == -INFINITY) continue;
        double f = exp2(lam * (parts[p].m - M));
        l += f * parts[p].l;
        for (int c = 0; c < ORC_D; ++c) o[c] += f * parts[p].o[c];
    }
    double denom = p_scale * l;
    for (int c = 0; c < ORC_D; ++c) out[c] = o[c] / denom;
}

void orc_attention_f64(const double* q, const double* k, const double* v,
                       const double* ds, const int64_t* q_pos, int64_t nq, int64_t nk,
                       int tile, int64_t partition, int flags, double* out)
{
    int64_t part = partition > 0 ? partition : (nk > 0 ? nk : 1);
    int64_t nparts = (nk + part - 1) / part;
    if (nparts < 1) nparts = 1;
#pragma omp parallel for schedule(dynamic)
    for (int64_t r = 0; r < nq; ++r) {
        orc_state* st = (orc_state*)malloc(sizeof(orc_state) * (size_t)nparts);
        for (int64_t p = 0; p < nparts; ++p) {
            orc_state_init(&st[p]);
            int64_t lo = p * part, hi = (p + 1) * part < nk ? (p + 1) * part : nk;
            orc_visit(&st[p], q + r * ORC_D, k, v, ds ? ds + r * nk : NULL, q_pos[r], lo, hi,
                      tile, flags);
        }
        orc_merge(st, (int)nparts, out + r * ORC_D,
                  (flags & ORC_QUANT_P) ? 448.0 : (flags & ORC_P_NVFP4) ? 2688.0 : 1.0);
        free(st);
    }
}

/* Eq. 2 as written: S = q k^T / sqrt(d), P = softmax(S) (natural base, max
 * subtracted for range), O = P V; keys after the query position masked. */
void orc_attention_textbook(const double* q, const double* k, const double* v,
                            const int64_t* q_pos, int64_t nq, int64_t nk, double* out)
{
#pragma omp parallel for schedule(dynamic)
    for (int64_t r = 0; r < nq; ++r) {
        int64_t n = q_pos[r] + 1 < nk ? q_pos[r] + 1 : nk;
        double* s = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
        double mx = -INFINITY;
        for (int64_t j = 0; j < n; ++j) {
            double acc = 0.0;
            for (int c = 0; c < ORC_D; ++c) acc += q[r * ORC_D + c] * k[j * ORC_D + c];
            s[j] = acc / sqrt((double)ORC_D);
            if (s[j] > mx) mx = s[j];
        }
        double den = 0.0;
        for (int64_t j = 0; j < n; ++j) { s[j] = exp(s[j] - mx); den += s[j]; }
        for (int c = 0; c < ORC_D; ++c) {
            double acc = 0.0;
            for (int64_t j = 0; j < n; ++j) acc += s[j] * v[j * ORC_D + c];
            out[r * ORC_D + c] = n > 0 ? acc / den : 0.0;
        }
        free(s);
    }
}

/* -------------------------------------------------------------------------- */
/* Attention over the quantized paged cache (prefill and split-KV decode)      */
/* -------------------------------------------------------------------------- */

/* Dequantize the whole key range of one (sequence, KV head) into FP64 rows. */
static void gather_kv(const orc_cache* c, int b, int hk, int64_t n, double* kd, double* vd)
{
    double tk = c->k_tscale[(int64_t)b * c->h_kv + hk];
#pragma omp parallel for schedule(static)
    for (int64_t key = 0; key < n; ++key) {
        int64_t page = c->page_table[(int64_t)b * c->max_pages + key / ORC_PAGE];
        int64_t off = key % ORC_PAGE;
        int64_t row = (page * c->h_kv + hk) * ORC_PAGE + off;
        if (c->flags & ORC_MXFP4)
            orc_mxfp4_dequant_row(c->k_codes + row * 64, c->k_scales + row * 8, kd + key * ORC_D);
        else
            orc_nvfp4_dequant_row(c->k_codes + row * 64, c->k_scales + row * 8, tk, kd + key * ORC_D);
        for (int d = 0; d < ORC_D; ++d) {
            int64_t vr = (page * c->h_kv + hk) * ORC_D + d;
            if (c->flags & ORC_PV_BF16) {
                vd[key * ORC_D + d] = orc_bf16_value(((const uint16_t*)c->v_aux)[vr * ORC_PAGE + off]);
            } else if (c->flags & ORC_PV_NVFP4) {
                const uint8_t* codes = (const uint8_t*)c->v_aux + vr * 32;
                const uint8_t* sc = (const uint8_t*)c->v_aux + c->num_pages * c->h_kv * ORC_D * 32 + vr * 4;
                uint8_t q = (uint8_t)((codes[off / 2] >> (4 * (off % 2))) & 15);
                vd[key * ORC_D + d] = orc_e4m3_value(sc[off / 16]) * orc_e2m1_value(q);
            } else {
                vd[key * ORC_D + d] = orc_e4m3_value(c->v_codes[vr * ORC_PAGE + off]);
            }
        }
    }
}

static void gather_ds(const orc_cache* c, int b, int h, int64_t n, double* dsd)
{
    for (int64_t key = 0; key < n; ++key) {
        int64_t page = c->page_table[(int64_t)b * c->max_pages + key / ORC_PAGE];
        dsd[key] = (double)orc_bf16_value(c->ds[(page * c->h_q + h) * ORC_PAGE + key % ORC_PAGE]);
    }
}

typedef struct { int32_t b, hk; int64_t idx; } item_key;

static int cmp_item(const void* x, const void* y)
{
    const item_key* a = (const item_key*)x;
    const item_key* b = (const item_key*)y;
    if (a->b != b->b) return a->b < b->b ? -1 : 1;
    if (a->hk != b->hk) return a->hk < b->hk ? -1 : 1;
    return a->idx < b->idx ? -1 : (a->idx > b->idx);
}

/* Shared driver: items grouped by (sequence, KV head) so that each key range
 * is dequantized once.  decode_part > 0 selects decode (query = sequence b,
 * position kv_len-1, partitions of decode_part keys); else prefill. */
static int run_items(const orc_cache* c, const int32_t* cu_seqlens, const int32_t* q_start,
                     int32_t decode_part, int64_t n_items, const int32_t* item_b,
                     const int32_t* item_row, const int32_t* item_h, uint16_t* out_bf16,
                     double* out_f64)
{
    const int grp = c->h_q / c->h_kv;
    const int smooth = (c->flags & ORC_SMOOTH) != 0;
    /* P quantizer of the cache's precision assignment (Sec. 3.1) */
    const int pmode = (c->flags & ORC_PV_BF16) ? ORC_P_BF16 : (c->flags & ORC_PV_NVFP4) ? ORC_P_NVFP4 : ORC_QUANT_P;
    const double p_scale = pmode == ORC_QUANT_P ? 448.0 : pmode == ORC_P_NVFP4 ? 2688.0 : 1.0;
    item_key* keys = (item_key*)malloc(sizeof(item_key) * (size_t)(n_items > 0 ? n_items : 1));
    for (int64_t i = 0; i < n_items; ++i) {
        keys[i].b = item_b[i];
        keys[i].hk = item_h[i] / grp;
        keys[i].idx = i;
    }
    qsort(keys, (size_t)n_items, sizeof(item_key), cmp_item);
    int64_t i0 = 0;
    while (i0 < n_items) {
        int64_t i1 = i0;
        while (i1 < n_items && keys[i1].b == keys[i0].b && keys[i1].hk == keys[i0].hk) ++i1;
        const int b = keys[i0].b, hk = keys[i0].hk;
        const int64_t n = c->kv_len[b];
        double* kd = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1) * ORC_D);
        double* vd = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1) * ORC_D);
        double* dsd = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1) * (size_t)grp);
        gather_kv(c, b, hk, n, kd, vd);
        if (smooth)
            for (int g = 0; g < grp; ++g) gather_ds(c, b, hk * grp + g, n, dsd + (int64_t)g * n);
#pragma omp parallel for schedule(dynamic)
        for (int64_t ii = i0; ii < i1; ++ii) {
            int64_t it = keys[ii].idx;
            int h = item_h[it];
            int64_t qtok, pos;
            if (decode_part > 0) {
                qtok = b;
                pos = n - 1;
            } else {
                qtok = (int64_t)cu_seqlens[b] + item_row[it];
                pos = (int64_t)q_start[b] + item_row[it];
            }
            double qd[ORC_D];
            if (c->flags & ORC_MXFP4)
                orc_mxfp4_dequant_row(c->q_codes + (qtok * c->h_q + h) * 64,
                                      c->q_scales + (qtok * c->h_q + h) * 8, qd);
            else
                orc_nvfp4_dequant_row(c->q_codes + (qtok * c->h_q + h) * 64,
                                      c->q_scales + (qtok * c->h_q + h) * 8,
                                      (double)c->q_tscale[(int64_t)b * c->h_q + h], qd);
            const double* dsh = smooth ? dsd + (int64_t)(h - hk * grp) * n : NULL;
            int64_t part = decode_part > 0 ? decode_part : (n > 0 ? n : 1);
            int64_t nparts = n > 0 ? (n + part - 1) / part : 1;
            orc_state* st = (orc_state*)malloc(sizeof(orc_state) * (size_t)nparts);
            for (int64_t p = 0; p < nparts; ++p) {
                orc_state_init(&st[p]);
                int64_t lo = p * part, hi = (p + 1) * part < n ? (p + 1) * part : n;
                orc_visit(&st[p], qd, kd, vd, dsh, pos, lo, hi, 128, pmode | ORC_REVERSE);
            }
            double o[ORC_D];
            orc_merge(st, (int)nparts, o, p_scale);
            free(st);
            for (int d = 0; d < ORC_D; ++d) {
                if (out_f64) out_f64[it * ORC_D + d] = o[d];
                if (out_bf16) out_bf16[it * ORC_D + d] = orc_bf16_encode_f64(o[d]);
            }
        }
        free(kd);
        free(vd);
        free(dsd);
        i0 = i1;
    }
    free(keys);
    return 0;
}

/* Algorithm 1 main loop for causal prefill: KV tiles of 128 keys visited from
 * the query's own tile down to tile 0; output rounded once from FP64 to
 * BF16 (R8). */
int orc_prefill(const orc_cache* c, const int32_t* cu_seqlens, const int32_t* q_start,
                int64_t n_items, const int32_t* item_b, const int32_t* item_row,
                const int32_t* item_h, uint16_t* out_bf16, double* out_f64)
{
    return run_items(c, cu_seqlens, q_start, 0, n_items, item_b, item_row, item_h, out_bf16,
                     out_f64);
}

/* Split-KV decode (Sec. 5.3): the key history is cut into fixed partitions,
 * each visited tile by tile in reverse with its own (m, l, O), merged by
 * log-sum-exp. */
int orc_decode(const orc_cache* c, int32_t partition_tokens, int64_t n_items,
               const int32_t* item_b, const int32_t* item_h, uint16_t* out_bf16, double* out_f64)
{
    if (partition_tokens <= 0 || partition_tokens % 128) return -1;
    return run_items(c, NULL, NULL, partition_tokens, n_items, item_b, NULL, item_h, out_bf16,
                     out_f64);
}

int orc_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
