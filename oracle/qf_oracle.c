/*
 * qf_oracle.c -- plain, slow CPU oracle for deployment-aligned fake quantization.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or call this
 * file; only the test suite, the smoke check and the benchmark's CPU-baseline leg do.
 * It shares no code, header, table or helper with the GPU library.
 *
 * What it computes (QATFactory, Sec. 3.2 "Deployment-aligned simulated quantization"):
 *   Q(X) -> (C, theta), Q^-1(C, theta) -> X_hat          (Eq. quantize-dequantize)
 * for three formats (Sec. 3.2.3, Tab. formats):
 *   NVFP4  E2M1 codes, E4M3 scale per 16, FP32 tensor scale   (Eqs. e2m1-values, nvfp4, nvfp4-dequant)
 *   MXFP4  E2M1 codes, E8M0 power-of-two scale per 32        (Eqs. mxfp4, mxfp4-dequant)
 *   Q4_K   uint4 codes, 6-bit scales/mins per 32 in 256,     (Eqs. q4k, q4k-dequant)
 *          FP16 super-block scale and min
 * Blocks run along the contiguous (K, in-features) axis of a row-major [R, K] tensor.
 *
 * Style: every step is written out one value at a time, in the order the format
 * definition states it.  Element and scale encoders are brute-force nearest-value
 * searches over the format's value table (ties to the even code); float16/bfloat16
 * rounding is "divide by the spacing of the binade, round half to even".  Where a
 * step is an FP32 operation of the reading (scale arithmetic of NVFP4 and Q4_K), it
 * is one binary32 operation on a `float` variable; build with -ffp-contract=off and
 * without fast-math so that each is a single IEEE operation.
 *
 * Readings where the paper is silent (operation order, zero blocks, saturation) are
 * stated at each function.  Parity pins: all codecs are pinned by the -m "not gpu"
 * tests (exhaustive code tables, library casts, brute force, closed forms).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

/* ------------------------------------------------------------------------- */
/* binary32 / bfloat16 / float16 helpers                                       */
/* ------------------------------------------------------------------------- */

static float f32_of_bits(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }

/* bfloat16 is the upper half of a binary32 word. */
float or_bf16_to_f32(uint16_t h) { return f32_of_bits((uint32_t)h << 16); }

/* Round a non-negative finite value to nearest, ties to even, on a binary format with
 * `mbits` stored fraction bits and exponent bias `bias` (subnormals kept, no upper
 * exponent limit: the caller handles overflow).  The spacing of representable values
 * in the binade of v is 2^(max(floor(log2 v), 1 - bias) - mbits). */
static double round_to_format(double v, int mbits, int bias) {
    if (v == 0.0) return 0.0;
    int e2;
    frexp(v, &e2);               /* v = f * 2^e2, f in [0.5, 1)  =>  floor(log2 v) = e2 - 1 */
    int ex = e2 - 1;
    if (ex < 1 - bias) ex = 1 - bias;
    double q = ldexp(1.0, ex - mbits);
    double n = v / q;            /* exact: q is a power of two */
    double lo = floor(n);
    double rem = n - lo;
    if (rem > 0.5 || (rem == 0.5 && fmod(lo, 2.0) != 0.0)) lo += 1.0;
    return lo * q;
}

/* Exponent/fraction fields of a positive value that the format represents exactly. */
static uint32_t fields_of_value(double r, int mbits, int bias) {
    int e2;
    frexp(r, &e2);
    int ex = e2 - 1;
    if (ex < 1 - bias) return (uint32_t)(r / ldexp(1.0, 1 - bias - mbits));     /* subnormal */
    uint32_t f = (uint32_t)(r / ldexp(1.0, ex - mbits)) - (1u << mbits);
    return ((uint32_t)(ex + bias) << mbits) | f;
}

/* binary32 -> bfloat16, round to nearest even; NaN -> 0x7FC0 (sign dropped). */
uint16_t or_bf16_from_f32(float v) {
    if (isnan(v)) return 0x7FC0;
    uint16_t s = signbit(v) ? 0x8000 : 0;
    double a = fabs((double)v);
    if (isinf(a)) return s | 0x7F80;
    double r = round_to_format(a, 7, 127);
    if (r >= ldexp(1.0, 128)) return s | 0x7F80;    /* rounds past the largest finite value */
    if (r == 0.0) return s;
    return s | (uint16_t)fields_of_value(r, 7, 127);
}

/* binary16 -> binary32. */
float or_f16_to_f32(uint16_t h) {
    int s = h >> 15, e = (h >> 10) & 31, f = h & 1023;
    double v;
    if (e == 0) v = ldexp((double)f, -24);
    else if (e == 31) v = f ? NAN : INFINITY;
    else v = ldexp((double)(1024 + f), e - 25);
    return (float)(s ? -v : v);
}

/* binary32 -> binary16, round to nearest even, subnormals kept; a result beyond the
 * largest finite value saturates to +-65504 (reading: the Q4_K super-block scales are
 * finite FP16 numbers).  NaN -> 0x7E00. */
uint16_t or_f16_from_f32(float v) {
    if (isnan(v)) return 0x7E00;
    uint16_t s = signbit(v) ? 0x8000 : 0;
    double a = fabs((double)v);
    if (isinf(a)) return s | 0x7BFF;
    double r = round_to_format(a, 10, 15);
    if (r > 65504.0) return s | 0x7BFF;
    if (r == 0.0) return s;
    return s | (uint16_t)fields_of_value(r, 10, 15);
}

/* ------------------------------------------------------------------------- */
/* E2M1 element code (Eq. e2m1-values)                                          */
/* ------------------------------------------------------------------------- */

/* The eight E2M1 magnitudes, indexed by the 3-bit magnitude code (sign is bit 3). */
static const double kE2M1[8] = {0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0};

double or_e2m1_value(int code) {            /* code 0..15, bit 3 = sign */
    double v = kE2M1[code & 7];
    return (code & 8) ? -v : v;
}

/* Nearest E2M1 magnitude to v >= 0, ties to the even code; anything above 6 (incl. +inf)
 * saturates to 6 (code 7). */
int or_e2m1_encode(double v) {
    if (v > 6.0) return 7;
    int best = 0;
    double bd = fabs(v - kE2M1[0]);
    for (int m = 1; m < 8; ++m) {
        double d = fabs(v - kE2M1[m]);
        if (d < bd || (d == bd && (m % 2) == 0)) { best = m; bd = d; }
    }
    return best;
}

/* ------------------------------------------------------------------------- */
/* E4M3 (OCP "FN": bias 7, no infinity, 0x7F/0xFF NaN, max 448) and E8M0        */
/* ------------------------------------------------------------------------- */

double or_e4m3_decode(int code) {
    int s = (code >> 7) & 1, e = (code >> 3) & 15, m = code & 7;
    double v;
    if (e == 15 && m == 7) return NAN;
    if (e == 0) v = ldexp((double)m, -9);
    else v = ldexp(1.0 + m / 8.0, e - 7);
    return s ? -v : v;
}

/* Nearest non-negative finite E4M3 value to t >= 0, ties to the even code; values at or
 * beyond 448 give 0x7E (saturating, never NaN).  NaN input -> 0x7F. */
int or_e4m3_encode(double t) {
    if (isnan(t)) return 0x7F;
    if (t >= 448.0) return 0x7E;
    int best = 0;
    double bd = fabs(t - or_e4m3_decode(0));
    for (int c = 1; c <= 0x7E; ++c) {
        double d = fabs(t - or_e4m3_decode(c));
        if (d < bd || (d == bd && (c % 2) == 0)) { best = c; bd = d; }
    }
    return best;
}

/* E8M0: code e means 2^(e-127); 0xFF is NaN (Eq. mxfp4-dequant: scales are powers of two). */
double or_e8m0_decode(int code) {
    if ((code & 0xFF) == 0xFF) return NAN;
    return ldexp(1.0, (code & 0xFF) - 127);
}

/* ------------------------------------------------------------------------- */
/* Tensor amax (Sec. 3.2.1: scales derive from the maximum absolute value)        */
/* ------------------------------------------------------------------------- */

float or_amax(const uint16_t* x, int64_t R, int64_t K, int64_t ldx) {
    float g = 0.0f;
    for (int64_t r = 0; r < R; ++r)
        for (int64_t k = 0; k < K; ++k) {
            float a = fabsf(or_bf16_to_f32(x[r * ldx + k]));
            if (a > g || isnan(a)) g = a;
        }
    return g;
}

/* ------------------------------------------------------------------------- */
/* NVFP4 (Eqs. nvfp4, nvfp4-dequant): W_hat_i = s_FP32 * s_E4M3,b * C_i          */
/* ------------------------------------------------------------------------- */
/*
 * Reading (the paper fixes the representation and the decode, not the encoder):
 *  1. g = tensor amax (or a caller-supplied running / tied-group amax).
 *  2. s_FP32 = S = fl(g / 2688), 2688 = 6 * 448: the tensor amax maps to the largest
 *     E2M1 value times the largest E4M3 value.  g = 0 gives S = 0.
 *  3. Per block of 16: a_b = max|x|; t_b = fl(a_b / fl(6 S)); s_E4M3,b = nearest E4M3 to
 *     t_b, saturating at 448.  S = 0 gives scale code 0.
 *  4. D_b = fl(S * s_E4M3,b)  (the block's decode scale, the product in Eq. nvfp4-dequant).
 *  5. C_i = nearest E2M1 to fl(|x_i| * fl(1 / D_b)), sign copied from x_i; D_b = 0 gives +-0.
 *  6. x_hat_i = bf16(fl(+-V(C_i) * D_b)).
 * Outputs: codes [R][K/2] (element 2i in the low nibble), scales [R][K/16] E4M3 bytes,
 * S, x_hat [R][K] bf16.  Any output pointer may be NULL.
 */
void or_nvfp4_quant(const uint16_t* x, int64_t R, int64_t K, int64_t ldx,
                    const float* amax_in, uint8_t* codes, uint8_t* scales,
                    float* s_out, uint16_t* xhat) {
    float g = amax_in ? *amax_in : or_amax(x, R, K, ldx);
    float S = g / 2688.0f;
    float six_s = 6.0f * S;
    if (s_out) *s_out = S;
    for (int64_t r = 0; r < R; ++r) {
        for (int64_t b = 0; b < K / 16; ++b) {
            const uint16_t* xb = x + r * ldx + b * 16;
            float ab = 0.0f;
            for (int i = 0; i < 16; ++i) {
                float a = fabsf(or_bf16_to_f32(xb[i]));
                if (a > ab) ab = a;
            }
            int sc = 0;
            if (S != 0.0f) {
                float t = ab / six_s;
                sc = or_e4m3_encode((double)t);
            }
            float D = S * (float)or_e4m3_decode(sc);
            float rcp = (D != 0.0f) ? 1.0f / D : 0.0f;
            if (scales) scales[r * (K / 16) + b] = (uint8_t)sc;
            for (int i = 0; i < 16; ++i) {
                float v = or_bf16_to_f32(xb[i]);
                int sign = (xb[i] >> 15) & 1;
                int m = 0;
                if (D != 0.0f) {
                    float u = fabsf(v) * rcp;
                    m = or_e2m1_encode((double)u);
                }
                int code = (sign << 3) | m;
                int64_t k = b * 16 + i;
                if (codes) {
                    uint8_t* p = &codes[r * (K / 2) + k / 2];
                    if ((k & 1) == 0) *p = (uint8_t)((*p & 0xF0) | code);
                    else *p = (uint8_t)((*p & 0x0F) | (code << 4));
                }
                if (xhat) {
                    float mag = (float)kE2M1[m] * D;
                    xhat[r * K + k] = or_bf16_from_f32(sign ? -mag : mag);
                }
            }
        }
    }
}

/* Decode NVFP4 codes + scales + S back to bf16 (Eq. nvfp4-dequant, same rounding as above). */
void or_nvfp4_dequant(const uint8_t* codes, const uint8_t* scales, float S,
                      int64_t R, int64_t K, uint16_t* xhat) {
    for (int64_t r = 0; r < R; ++r)
        for (int64_t k = 0; k < K; ++k) {
            uint8_t byte = codes[r * (K / 2) + k / 2];
            int code = (k & 1) ? (byte >> 4) : (byte & 15);
            float D = S * (float)or_e4m3_decode(scales[r * (K / 16) + k / 16]);
            float mag = (float)kE2M1[code & 7] * D;
            xhat[r * K + k] = or_bf16_from_f32((code & 8) ? -mag : mag);
        }
}

/* ------------------------------------------------------------------------- */
/* MXFP4 (Eqs. mxfp4, mxfp4-dequant): W_hat_i = 2^p_b * C_i                      */
/* ------------------------------------------------------------------------- */
/*
 * Reading (OCP microscaling rule; the paper fixes only the power-of-two block scale):
 *  - a = max|x| over the block of 32.
 *  - Non-finite value in the block: scale code 0xFF (NaN), element codes 0, x_hat NaN.
 *  - a = 0: scale code 0 (2^-127), codes carry only the sign.
 *  - otherwise p = floor(log2 a) - 2 (2 = exponent of the largest E2M1 value, 6 = 1.5*2^2),
 *    clamped to [-127, 127]; scale code p + 127.
 *  - C_i = nearest E2M1 to |x_i| / 2^p (saturating at 6), sign copied.
 *  - x_hat_i = +-V(C_i) * 2^p, which bf16 represents exactly.
 */
void or_mxfp4_quant(const uint16_t* x, int64_t R, int64_t K, int64_t ldx,
                    uint8_t* codes, uint8_t* scales, uint16_t* xhat) {
    for (int64_t r = 0; r < R; ++r) {
        for (int64_t b = 0; b < K / 32; ++b) {
            const uint16_t* xb = x + r * ldx + b * 32;
            double a = 0.0;
            int nonfinite = 0;
            for (int i = 0; i < 32; ++i) {
                double v = fabs((double)or_bf16_to_f32(xb[i]));
                if (!isfinite(v)) nonfinite = 1;
                else if (v > a) a = v;
            }
            int sc;
            int p = 0;
            if (nonfinite) sc = 0xFF;
            else if (a == 0.0) { sc = 0; p = -127; }
            else {
                int e2;
                frexp(a, &e2);
                p = (e2 - 1) - 2;
                if (p < -127) p = -127;
                if (p > 127) p = 127;
                sc = p + 127;
            }
            if (scales) scales[r * (K / 32) + b] = (uint8_t)sc;
            for (int i = 0; i < 32; ++i) {
                int64_t k = b * 32 + i;
                int sign = (xb[i] >> 15) & 1;
                int code = 0;
                uint16_t h;
                if (sc == 0xFF) { code = 0; h = 0x7FC0; }
                else {
                    double v = fabs((double)or_bf16_to_f32(xb[i]));
                    int m = or_e2m1_encode(v / ldexp(1.0, p));
                    code = (sign << 3) | m;
                    double mag = kE2M1[m] * ldexp(1.0, p);
                    h = or_bf16_from_f32((float)(sign ? -mag : mag));
                }
                if (codes) {
                    uint8_t* q = &codes[r * (K / 2) + k / 2];
                    if ((k & 1) == 0) *q = (uint8_t)((*q & 0xF0) | code);
                    else *q = (uint8_t)((*q & 0x0F) | (code << 4));
                }
                if (xhat) xhat[r * K + k] = h;
            }
        }
    }
}

void or_mxfp4_dequant(const uint8_t* codes, const uint8_t* scales,
                      int64_t R, int64_t K, uint16_t* xhat) {
    for (int64_t r = 0; r < R; ++r)
        for (int64_t k = 0; k < K; ++k) {
            uint8_t byte = codes[r * (K / 2) + k / 2];
            int code = (k & 1) ? (byte >> 4) : (byte & 15);
            int sc = scales[r * (K / 32) + k / 32];
            if (sc == 0xFF) { xhat[r * K + k] = 0x7FC0; continue; }
            double mag = kE2M1[code & 7] * or_e8m0_decode(sc);
            xhat[r * K + k] = or_bf16_from_f32((float)((code & 8) ? -mag : mag));
        }
}

/* ------------------------------------------------------------------------- */
/* Q4_K (Eqs. q4k, q4k-dequant): W_hat_i = (s_FP16 s_6,b) C_i - (m_FP16 m_6,b)   */
/* ------------------------------------------------------------------------- */

/* Round a binary32 value to the nearest integer, ties to even. */
static double rne_int(float v) {
    double d = (double)v;
    double lo = floor(d);
    double rem = d - lo;
    if (rem > 0.5 || (rem == 0.5 && fmod(lo, 2.0) != 0.0)) lo += 1.0;
    return lo;
}

static int clampi(double v, int lo, int hi) {
    if (!(v >= lo)) return lo;     /* also maps NaN to lo */
    if (v > hi) return hi;
    return (int)v;
}

/* Pack one super-block: d, dmin (FP16 little-endian), 12 bytes of 6-bit scales and mins,
 * 128 bytes of codes (byte 32c+l: q[64c+l] low nibble, q[64c+32+l] high nibble). */
static void q4k_pack(uint8_t* out, uint16_t dh, uint16_t mh, const int ls[8],
                     const int lm[8], const int q[256]) {
    out[0] = dh & 0xFF; out[1] = dh >> 8;
    out[2] = mh & 0xFF; out[3] = mh >> 8;
    uint8_t* sc = out + 4;
    for (int j = 0; j < 4; ++j) {
        sc[j]     = (uint8_t)((ls[j] & 63) | ((ls[j + 4] >> 4) << 6));
        sc[j + 4] = (uint8_t)((lm[j] & 63) | ((lm[j + 4] >> 4) << 6));
        sc[j + 8] = (uint8_t)((ls[j + 4] & 15) | ((lm[j + 4] & 15) << 4));
    }
    uint8_t* qs = out + 16;
    for (int c = 0; c < 4; ++c)
        for (int l = 0; l < 32; ++l)
            qs[32 * c + l] = (uint8_t)((q[64 * c + l] & 15) | ((q[64 * c + 32 + l] & 15) << 4));
}

static void q4k_unpack(const uint8_t* in, uint16_t* dh, uint16_t* mh, int ls[8],
                       int lm[8], int q[256]) {
    *dh = (uint16_t)(in[0] | (in[1] << 8));
    *mh = (uint16_t)(in[2] | (in[3] << 8));
    const uint8_t* sc = in + 4;
    for (int j = 0; j < 4; ++j) {
        ls[j] = sc[j] & 63;
        lm[j] = sc[j + 4] & 63;
        ls[j + 4] = (sc[j + 8] & 15) | ((sc[j] >> 6) << 4);
        lm[j + 4] = (sc[j + 8] >> 4) | ((sc[j + 4] >> 6) << 4);
    }
    const uint8_t* qs = in + 16;
    for (int c = 0; c < 4; ++c)
        for (int l = 0; l < 32; ++l) {
            q[64 * c + l] = qs[32 * c + l] & 15;
            q[64 * c + 32 + l] = qs[32 * c + l] >> 4;
        }
}

void or_q4k_pack_block(uint8_t* out, uint16_t dh, uint16_t mh, const int* ls,
                       const int* lm, const int* q) { q4k_pack(out, dh, mh, ls, lm, q); }
void or_q4k_unpack_block(const uint8_t* in, uint16_t* dh, uint16_t* mh, int* ls,
                         int* lm, int* q) { q4k_unpack(in, dh, mh, ls, lm, q); }

/*
 * Reading ("min-max"; the paper fixes the representation and the decode equation, not the
 * scale search):
 *  per sub-block j of 32: lo_j = min(0, min x), hi_j = max x, signed zeros counted as +0
 *     (the sign of a zero plays no part in an unsigned-code format, and this keeps the
 *     extremes independent of element order),
 *     a_j = fl(fl(hi_j - lo_j) / 15), mu_j = fl(0 - lo_j)   (the unsigned min m_6 is
 *     subtracted, so the offset is never positive)
 *  per super-block of 256: s_FP16 = h(fl(max a_j / 63)), m_FP16 = h(fl(max mu_j / 63))
 *  s_6,j = clamp(rne(fl(a_j / s_FP16)), 0, 63), m_6,j = clamp(rne(fl(mu_j / m_FP16)), 0, 63)
 *     (0 when the FP16 value is 0)
 *  t1 = fl(s_FP16 s_6,j), t2 = fl(m_FP16 m_6,j)
 *  C_i = clamp(rne(fl(fl(x_i + t2) / t1)), 0, 15)   (0 when t1 = 0)
 *  x_hat_i = bf16(fl(t1 C_i - t2))                  (t1 C_i is exact)
 * Output: packed [R][K/256][144] bytes, x_hat [R][K].
 */
void or_q4k_quant(const uint16_t* x, int64_t R, int64_t K, int64_t ldx,
                  uint8_t* packed, uint16_t* xhat) {
    for (int64_t r = 0; r < R; ++r) {
        for (int64_t sb = 0; sb < K / 256; ++sb) {
            const uint16_t* xs = x + r * ldx + sb * 256;
            float a[8], mu[8];
            for (int j = 0; j < 8; ++j) {
                float lo = 0.0f, hi = or_bf16_to_f32(xs[32 * j]) + 0.0f;   /* -0 -> +0 */
                for (int i = 0; i < 32; ++i) {
                    float v = or_bf16_to_f32(xs[32 * j + i]) + 0.0f;
                    if (v < lo) lo = v;
                    if (v > hi) hi = v;
                }
                float range = hi - lo;
                a[j] = range / 15.0f;
                mu[j] = 0.0f - lo;
            }
            float amx = a[0], mmx = mu[0];
            for (int j = 1; j < 8; ++j) {
                if (a[j] > amx) amx = a[j];
                if (mu[j] > mmx) mmx = mu[j];
            }
            uint16_t dh = or_f16_from_f32(amx / 63.0f);
            uint16_t mh = or_f16_from_f32(mmx / 63.0f);
            float d = or_f16_to_f32(dh), dmin = or_f16_to_f32(mh);
            int ls[8], lm[8], q[256];
            for (int j = 0; j < 8; ++j) {
                ls[j] = (d != 0.0f) ? clampi(rne_int(a[j] / d), 0, 63) : 0;
                lm[j] = (dmin != 0.0f) ? clampi(rne_int(mu[j] / dmin), 0, 63) : 0;
                float t1 = d * (float)ls[j];
                float t2 = dmin * (float)lm[j];
                for (int i = 0; i < 32; ++i) {
                    float v = or_bf16_to_f32(xs[32 * j + i]);
                    int c = 0;
                    if (t1 != 0.0f) {
                        float sh = v + t2;
                        c = clampi(rne_int(sh / t1), 0, 15);
                    }
                    q[32 * j + i] = c;
                    if (xhat) {
                        float prod = t1 * (float)c;
                        xhat[r * K + sb * 256 + 32 * j + i] = or_bf16_from_f32(prod - t2);
                    }
                }
            }
            if (packed) q4k_pack(packed + (r * (K / 256) + sb) * 144, dh, mh, ls, lm, q);
        }
    }
}

/* Dequantize packed Q4_K super-blocks straight from Eq. q4k-dequant. */
void or_q4k_dequant(const uint8_t* packed, int64_t R, int64_t K, uint16_t* xhat) {
    for (int64_t r = 0; r < R; ++r)
        for (int64_t sb = 0; sb < K / 256; ++sb) {
            uint16_t dh, mh;
            int ls[8], lm[8], q[256];
            q4k_unpack(packed + (r * (K / 256) + sb) * 144, &dh, &mh, ls, lm, q);
            float d = or_f16_to_f32(dh), dmin = or_f16_to_f32(mh);
            for (int i = 0; i < 256; ++i) {
                float t1 = d * (float)ls[i / 32];
                float t2 = dmin * (float)lm[i / 32];
                float prod = t1 * (float)q[i];
                xhat[r * K + sb * 256 + i] = or_bf16_from_f32(prod - t2);
            }
        }
}

/* ------------------------------------------------------------------------- */
/* LoRA merge (Sec. 3.3, Eqs. qad-lora and export-lora): W + s * B A            */
/* ------------------------------------------------------------------------- */
/*
 * The merged weight that LoRA-QAD quantizes in the forward pass and that the exporter
 * quantizes into the checkpoint.  W is bf16 [N, K] (nn.Linear layout), B is FP32 [N, r],
 * A is FP32 [r, K] (the trainable low-rank factors), s a scalar multiplier (1 for the
 * paper's W + BA; LoRA's alpha / r otherwise).
 * Reading (the paper fixes neither the precision nor the order of the merge):
 *  1. acc = sum over j = 0, 1, ..., r-1 of B[n][j] * A[j][k] in binary32, one fused
 *     multiply-add (a single rounding) per rank term, starting from +0;
 *  2. t = fl(s * acc);  m = fl(W[n][k] + t);
 *  3. the merged element is bf16(m) (round to nearest even): the merged weight has the
 *     base weight's type, so the quantizer sees the same input type as without adapters.
 * IEEE rules apply throughout: W = -0 with t = +0 merges to +0; NaN and Inf propagate.
 */
void or_lora_merge(const uint16_t* w, int64_t N, int64_t K, int64_t ldw, const float* B,
                   const float* A, int64_t r, float s, uint16_t* out) {
    for (int64_t n = 0; n < N; ++n)
        for (int64_t k = 0; k < K; ++k) {
            float acc = 0.0f;
            for (int64_t j = 0; j < r; ++j) acc = fmaf(B[n * r + j], A[j * K + k], acc);
            float t = s * acc;
            float m = or_bf16_to_f32(w[n * ldw + k]) + t;
            out[n * K + k] = or_bf16_from_f32(m);
        }
}

/* ------------------------------------------------------------------------- */
/* Q4_K with an MSE search of the sub-block scales (Sec. 4: PTQ searching for   */
/* scales that minimize ||W - W_q||^2; the search below is this library's own)  */
/* ------------------------------------------------------------------------- */
/*
 * FP32 sums over a 32-element sub-block are taken in one fixed order: four groups of 8
 * consecutive elements, each summed from +0 in index order, then (g0 + g1) + (g2 + g3);
 * super-block totals add the 8 sub-block sums as ((s0 + s1) + (s2 + s3)) + ((s4 + s5) +
 * (s6 + s7)).  (The comparisons between candidates depend on the rounding of these sums, so
 * the reading fixes their order.)
 */
static float sb_sum(const float* f) {
    float g[4];
    for (int c = 0; c < 4; ++c) {
        float s = 0.0f;
        for (int i = 0; i < 8; ++i) s += f[8 * c + i];
        g[c] = s;
    }
    return (g[0] + g[1]) + (g[2] + g[3]);
}

static float clampf15(float v) { return v < 0.0f ? 0.0f : (v > 15.0f ? 15.0f : v); }

/*
 * One sub-block (x[32], signed zeros as +0): min-max anchors lo = min(0, min x), hi = max x,
 * mu0 = 0 - lo.  Candidate k = 0..16 takes the step a_k = (hi - lo) / (14 + k/4), codes
 * q = clamp(rne((x + mu0) * fl(1 / a_k)), 0, 15), then refits the step and offset to those
 * codes by least squares (minimizing sum (x - (a q - mu))^2):
 *     den = 32 Sqq - Sq^2,  a* = (32 Sqx - Sq Sx) / den,  mu* = (a* Sq - Sx) / 32
 * (den = 0: keep a_k, mu0); mu* < 0 is moved to the constraint mu = 0 with a* = Sqx / Sqq; a
 * refit with a* <= 0 keeps a_k, mu0.  a_k = 0 (a constant sub-block at lo) keeps (0, mu0).
 * The candidate with the smallest error sum (x - fl(fl(a* q) - mu*))^2 wins (the first one
 * on ties).  Outputs the winning (a, mu) and its codes.
 */
static void q4k_mse_subblock(const float* x, float* a_out, float* mu_out, int* q_out) {
    float lo = 0.0f, hi = x[0];
    for (int i = 0; i < 32; ++i) {
        if (x[i] < lo) lo = x[i];
        if (x[i] > hi) hi = x[i];
    }
    const float range = hi - lo, mu0 = 0.0f - lo;
    const float sx = sb_sum(x);
    float best_e = INFINITY, best_a = range / 15.0f, best_mu = mu0;
    for (int i = 0; i < 32; ++i) q_out[i] = 0;
    for (int k = 0; k <= 16; ++k) {
        const float Dk = 14.0f + 0.25f * (float)k;
        const float ak = range / Dk;
        float q[32], ac = ak, mc = mu0;
        if (ak == 0.0f) {
            for (int i = 0; i < 32; ++i) q[i] = 0.0f;
        } else {
            const float r = 1.0f / ak;
            float qq[32], qx[32];
            for (int i = 0; i < 32; ++i) {
                q[i] = clampf15((float)rne_int((x[i] + mu0) * r));
                qq[i] = q[i] * q[i];
                qx[i] = q[i] * x[i];
            }
            const float sq = sb_sum(q), sqq = sb_sum(qq), sqx = sb_sum(qx);
            const float den = 32.0f * sqq - sq * sq;
            if (den > 0.0f) {
                ac = (32.0f * sqx - sq * sx) / den;
                mc = (ac * sq - sx) / 32.0f;
                if (mc < 0.0f) {
                    mc = 0.0f;
                    ac = sqx / sqq;
                }
                if (!(ac > 0.0f)) {
                    ac = ak;
                    mc = mu0;
                }
            }
        }
        float e2[32];
        for (int i = 0; i < 32; ++i) {
            const float e = x[i] - (ac * q[i] - mc);
            e2[i] = e * e;
        }
        const float err = sb_sum(e2);
        if (err < best_e) {
            best_e = err;
            best_a = ac;
            best_mu = mc;
            for (int i = 0; i < 32; ++i) q_out[i] = (int)q[i];
        }
    }
    *a_out = best_a;
    *mu_out = best_mu;
}

void or_q4k_mse_subblock(const float* x, float* a, float* mu, int* q) {
    q4k_mse_subblock(x, a, mu, q);
}

/* Super-block from per-sub-block (a_j, mu_j): the 6-bit scale / min quantization and the
 * final codes of the min-max reading (or_q4k_quant), plus the super-block's error sum of
 * (x - fl(fl(t1 C) - t2))^2 in the fixed order. */
static float q4k_finish(const float* x, const float* a, const float* mu, uint16_t* dh,
                        uint16_t* mh, int* ls, int* lm, int* q, float* xf) {
    float amx = a[0], mmx = mu[0];
    for (int j = 1; j < 8; ++j) {
        if (a[j] > amx) amx = a[j];
        if (mu[j] > mmx) mmx = mu[j];
    }
    *dh = or_f16_from_f32(amx / 63.0f);
    *mh = or_f16_from_f32(mmx / 63.0f);
    const float d = or_f16_to_f32(*dh), dmin = or_f16_to_f32(*mh);
    float s8[8];
    for (int j = 0; j < 8; ++j) {
        ls[j] = (d != 0.0f) ? clampi(rne_int(a[j] / d), 0, 63) : 0;
        lm[j] = (dmin != 0.0f) ? clampi(rne_int(mu[j] / dmin), 0, 63) : 0;
        const float t1 = d * (float)ls[j], t2 = dmin * (float)lm[j];
        float e2[32];
        for (int i = 0; i < 32; ++i) {
            const float v = x[32 * j + i];
            int c = 0;
            if (t1 != 0.0f) c = clampi(rne_int((v + t2) / t1), 0, 15);
            q[32 * j + i] = c;
            xf[32 * j + i] = t1 * (float)c - t2;
            const float e = v - xf[32 * j + i];
            e2[i] = e * e;
        }
        s8[j] = sb_sum(e2);
    }
    return ((s8[0] + s8[1]) + (s8[2] + s8[3])) + ((s8[4] + s8[5]) + (s8[6] + s8[7]));
}

/*
 * or_q4k_mse_quant -- Q4_K with the searched sub-block steps: per super-block, the search
 * above gives (a_j, mu_j), q4k_finish quantizes them to 6 bits and recomputes the codes; the
 * min-max reading does the same from its own (a_j, mu_j); the super-block keeps the search's
 * result when its error sum is smaller, else the min-max one (so it is never worse).
 */
void or_q4k_mse_quant(const uint16_t* x, int64_t R, int64_t K, int64_t ldx, uint8_t* packed,
                      uint16_t* xhat) {
    for (int64_t r = 0; r < R; ++r)
        for (int64_t sb = 0; sb < K / 256; ++sb) {
            const uint16_t* xs = x + r * ldx + sb * 256;
            float xv[256];
            for (int i = 0; i < 256; ++i) xv[i] = or_bf16_to_f32(xs[i]) + 0.0f;   /* -0 -> +0 */
            float as[8], ms[8], am[8], mm[8];
            int qtmp[32];
            for (int j = 0; j < 8; ++j) {
                q4k_mse_subblock(xv + 32 * j, &as[j], &ms[j], qtmp);
                float lo = 0.0f, hi = xv[32 * j];
                for (int i = 0; i < 32; ++i) {
                    if (xv[32 * j + i] < lo) lo = xv[32 * j + i];
                    if (xv[32 * j + i] > hi) hi = xv[32 * j + i];
                }
                am[j] = (hi - lo) / 15.0f;
                mm[j] = 0.0f - lo;
            }
            uint16_t dh1, mh1, dh2, mh2;
            int ls1[8], lm1[8], q1[256], ls2[8], lm2[8], q2[256];
            float xf1[256], xf2[256];
            const float e1 = q4k_finish(xv, as, ms, &dh1, &mh1, ls1, lm1, q1, xf1);
            const float e2 = q4k_finish(xv, am, mm, &dh2, &mh2, ls2, lm2, q2, xf2);
            const int use1 = e1 < e2;
            if (packed)
                q4k_pack(packed + (r * (K / 256) + sb) * 144, use1 ? dh1 : dh2, use1 ? mh1 : mh2,
                         use1 ? ls1 : ls2, use1 ? lm1 : lm2, use1 ? q1 : q2);
            if (xhat)
                for (int i = 0; i < 256; ++i)
                    xhat[r * K + sb * 256 + i] = or_bf16_from_f32(use1 ? xf1[i] : xf2[i]);
        }
}

int or_version(void) { return 1; }
