/*
 * CPU oracle for the M+Adam optimizer step.  TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, scalar C.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load this library; the product path (the HIP
 * library) never does, and the two share no source, header or table.
 *
 * What it computes, by the paper's section / algorithm / equation:
 *
 *   Algorithm 1 (M+Adam: additive-multiplicative update), restated in
 *   Section 3.1 (Additive-Multiplicative Updates):
 *     additive branch        u <- b1 u + (1-b1) g ;  v <- b2 v + (1-b2) g^2
 *                            u^ = u/(1-b1^t), v^ = v/(1-b2^t)
 *                            u_a = -eta_a u^/(sqrt(v^)+eps)
 *     multiplicative branch  g_e = ln2 * w * g        (gradient w.r.t. the exponent)
 *                            v_e <- b2 v_e + (1-b2) g_e^2 ;  v_e^ = v_e/(1-b2^t)
 *                            ut_m = -eta_m g_e/(sqrt(v_e^)+eps)
 *                            rho = max(|w|, tau) ;  u_m = clip(ut_m/rho)
 *     combine                w <- w + w u_m + u_a
 *
 *   Algorithm 2 (Appendix A, detailed algorithm) adds the optional clamps used
 *   here as options: clamp_{g_max} of the normalised multiplicative direction,
 *   the clip of u_m to [-(0.75-eps0), 0.75], the exponent-step cap
 *   clamp_{d_mult,max}(log2(1+u_m)) followed by u_m = 2^de - 1, and the final
 *   weight clamp clamp_{w_max}(w).  Algorithm 2 is printed without bias
 *   correction; bias_correction = 0 reproduces it, 1 gives Algorithm 1.
 *
 *   Appendix B (BF16-stored matrix fitting) also defines moment-free rules
 *   used by its diagnostic (oracle_plain_step): additive -eta_a g,
 *   multiplicative clip(-eta_m ln2 w g / max(|w|, tau), +-r_max), and their
 *   sum, each followed by the round trip into the storage format.
 *
 *   Appendix B (BF16-stored matrix fitting) fixes the precision: the step is
 *   computed in FP32 and the weight is rounded into the storage format before
 *   the next step.  This oracle generalises that round trip from BF16 to the
 *   FP8 storage of Section 4.2 (FP8 payload with FP16 block scales).
 *
 * Readings where the paper is silent (each is listed in the design notes):
 *   - FP32 operation order: one fixed sequence (oracle_step_elem below); every
 *     line is one IEEE binary32 operation with round-to-nearest-even, fmaf is
 *     one rounding, division and square root are correctly rounded.
 *   - The hyper-parameter scalars are evaluated in double and rounded once to
 *     float: B1, B2, 1-B1, 1-B2, SA = eta_a/(1-b1^t), IBC2 = 1/(1-b2^t), and
 *     the u_m clip bounds.
 *   - The exponent-step cap is applied as the equivalent clamp of u_m to
 *     [2^-d - 1, 2^d - 1] (log2 is monotone), so no transcendental is
 *     evaluated per element.
 *   - Stochastic rounding (cited, not defined, in the paper): on the
 *     magnitude a = |x| with grid neighbours lo <= a < hi,
 *     k = floor((a-lo)/(hi-lo) * 2^16), round up iff k + r16 >= 2^16, where
 *     r16 is a 16-bit draw.  For BF16 this is exact: P(up) = (a-lo)/(hi-lo).
 *   - The 16-bit draw for global element index i at step t is a 16-bit lane
 *     of Philox4x32-10 (Salmon, Moraes, Dror and Shaw, SC'11) with key
 *     (seed lo32, seed hi32) and counter (j lo32, j hi32, t, stream), j = i>>3:
 *     lane (i & 7) = bits 16*(i&1) .. +15 of output word (i&7)>>1.
 *   - FP8 formats: OCP E4M3 (bias 7, no Inf, NaN = S.1111.111, max 448) and
 *     E5M2 (bias 15, IEEE specials, max 57344), both saturating finite
 *     overflow (and Inf) to +-max; NaN encodes as the positive code 0x7F
 *     (0.1111.111 / 0.11111.11) in both.
 *   - BF16 / FP16 follow IEEE: overflow under RNE rounds to Inf, NaN encodes
 *     as the positive quiet NaN 0x7FC0 / 0x7E00 (a NaN's sign is not
 *     meaningful, so it is dropped).
 *   - FP32 "storage" (test passthrough) keeps the float bits; a NaN is stored
 *     as 0x7FC00000.
 *   - Compute copy (optional): after the update, the BF16 value of each stored
 *     weight (payload x scale for block-scaled FP8), rounded to nearest-even,
 *     for the GEMMs of the next step (in the FP8-master dataflow figure the
 *     BF16 copy the GEMMs read is rebuilt from the stored FP8 weights after
 *     every step).
 *   - Moments m, v, v_e are stored in fp32, or in bf16 (the precision of the
 *     optimizer states in the paper's memory accounting table).  With bf16
 *     storage the step decodes them exactly, computes in fp32 as above, uses
 *     the fp32 results within the step and stores them rounded to nearest
 *     (ties to even), or stochastically by the rule above with the draws of
 *     streams 1 (m), 2 (v) and 3 (v_e) of the same generator.
 *   - Block-scaled FP8: contiguous blocks of 128 elements, one FP16 scale s
 *     per block, weight = q * s (fp32 product).  After the update,
 *     amax = max|w'| over the block; s' = RNE_fp16(amax / FMAX) with
 *     s' = 1 when amax = 0, the smallest FP16 subnormal when it underflows to
 *     0, the largest finite FP16 when it overflows, and FP16 NaN when any w'
 *     of the block is not finite; q' = encode(w'/s') with the block's
 *     rounding mode.
 *   - 4-bit storage (the NVFP4/FP8 setting of Section 4.2; the paper does not
 *     define the format): the OCP MX block format MXFP4 -- 32-element blocks
 *     of E2M1 values with one E8M0 power-of-two scale; rule at oracle_step_mx
 *     -- and NVFP4 (16-element blocks, E4M3 block scales, one fp32 scale per
 *     tensor), either held fixed by the step (oracle_step_nv) or derived
 *     anew from the updated tensor every step (oracle_step_nv_current).
 *
 * Pin status (tests/test_oracle_*.py; a mutation test checks the pins catch
 * planted mistakes): the real-number update is pinned by closed forms, the
 * Adam limit, limits and invariants; the codecs by library conversions, the
 * OCP value tables and brute force; Philox by published known-answer vectors.
 * Parity unpinned against the paper, because the paper does not fix them:
 * the exact fp32 operation order (a contract shared with the kernel), the
 * block-scaled FP8 block length and scale rule, the 4-bit formats (MXFP4
 * and NVFP4, pinned to their published definitions instead; when NVFP4's
 * tensor scale is refreshed is a choice, and both are built: at encoding
 * only, or at every step), and the
 * stochastic-rounding rule and its generator (pinned to their own
 * definitions).
 *
 * Codec implementation: values are decoded from the (sign, exponent,
 * mantissa) definition of each format; encoding searches the sorted table of
 * decoded grid values for the neighbours of |x| and decides with exact double
 * arithmetic (no bit manipulation of the float representation).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* OF_E2M1 is the 4-bit MXFP4 element format; OF_E8M0 the MX block scale
 * (a power of two, not a sign/exponent/mantissa format: decoded separately). */
enum { OF_BF16 = 0, OF_E4M3 = 1, OF_E5M2 = 2, OF_FP32 = 3, OF_FP16 = 4, OF_E2M1 = 5, OF_NFMT = 6,
       OF_E8M0 = 6 };
enum { OG_FP32 = 0, OG_BF16 = 1 };
/* storage of the moments m, v, v_e: fp32, bf16 rounded to nearest-even, or
 * bf16 rounded stochastically (draws on streams 1, 2, 3 for m, v, v_e) */
enum { OS_FP32 = 0, OS_BF16 = 1, OS_BF16_SR = 2 };
enum { OR_RNE = 0, OR_SR = 1 };

enum {
  ORACLE_OK = 0,
  ORACLE_EINVAL = -1,
};

/* ------------------------------------------------------------------------ */
/* Storage formats, from their definitions                                   */
/* ------------------------------------------------------------------------ */

typedef struct {
  int ebits, mbits, bias;
  int specials;     /* SPEC_IEEE: all-ones exponent = Inf / NaN; SPEC_E4M3: only
                       S.1111.111 is NaN; SPEC_NONE: every code is finite      */
  int satfinite;    /* finite overflow and Inf saturate to +-max                */
  uint32_t nan_code;
  uint32_t inf_code;
  /* sorted non-negative finite grid */
  int nval;
  double *val;
  uint32_t *code;
  double max;
  uint32_t max_code;
  double beyond; /* next grid point above max if the exponent were unbounded */
} ofmt;

enum { SPEC_E4M3 = 0, SPEC_IEEE = 1, SPEC_NONE = 2 };

static ofmt g_fmt[OF_NFMT];
static int g_ready = 0;

static double decode_def(const ofmt *f, uint32_t c) {
  const int nb = f->ebits + f->mbits;
  const uint32_t s = (c >> nb) & 1u;
  const uint32_t e = (c >> f->mbits) & ((1u << f->ebits) - 1u);
  const uint32_t m = c & ((1u << f->mbits) - 1u);
  const uint32_t eall = (1u << f->ebits) - 1u, mall = (1u << f->mbits) - 1u;
  double mag;
  if (f->specials == SPEC_IEEE && e == eall) {
    mag = m ? NAN : INFINITY;
  } else if (f->specials == SPEC_E4M3 && e == eall && m == mall) {
    mag = NAN; /* E4M3: only S.1111.111 is special */
  } else if (e == 0) {
    mag = ldexp((double)m, 1 - f->bias - f->mbits); /* subnormal */
  } else {
    mag = ldexp((double)((1u << f->mbits) + m), (int)e - f->bias - f->mbits);
  }
  return s ? -mag : mag;
}

typedef struct {
  double v;
  uint32_t c;
} vc_pair;

static int cmp_vc(const void *a, const void *b) {
  const double x = ((const vc_pair *)a)->v, y = ((const vc_pair *)b)->v;
  return (x > y) - (x < y);
}

static void fmt_init(ofmt *f, int ebits, int mbits, int bias, int specials, int sat) {
  f->ebits = ebits;
  f->mbits = mbits;
  f->bias = bias;
  f->specials = specials;
  f->inf_code = 0u;
  f->satfinite = sat;
  const int nb = ebits + mbits;
  const uint32_t ncodes = 1u << nb; /* codes with the sign bit clear */
  vc_pair *tmp = (vc_pair *)malloc(sizeof(vc_pair) * ncodes);
  int n = 0;
  for (uint32_t c = 0; c < ncodes; ++c) {
    const double x = decode_def(f, c);
    if (isfinite(x)) {
      tmp[n].v = x;
      tmp[n].c = c;
      ++n;
    } else if (isinf(x)) {
      f->inf_code = c;
    }
  }
  qsort(tmp, (size_t)n, sizeof(vc_pair), cmp_vc);
  f->nval = n;
  f->val = (double *)malloc(sizeof(double) * (size_t)n);
  f->code = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)n);
  for (int i = 0; i < n; ++i) {
    f->val[i] = tmp[i].v;
    f->code[i] = tmp[i].c;
  }
  free(tmp);
  f->max = f->val[n - 1];
  f->max_code = f->code[n - 1];
  /* spacing at the top binade, continued one more step */
  f->beyond = f->max + (f->val[n - 1] - f->val[n - 2]);
}

static void init_formats(void) {
  if (g_ready) return;
  fmt_init(&g_fmt[OF_BF16], 8, 7, 127, SPEC_IEEE, 0);
  fmt_init(&g_fmt[OF_E4M3], 4, 3, 7, SPEC_E4M3, 1);
  fmt_init(&g_fmt[OF_E5M2], 5, 2, 15, SPEC_IEEE, 1);
  fmt_init(&g_fmt[OF_FP16], 5, 10, 15, SPEC_IEEE, 0);
  /* OCP MX E2M1: bias 1, no Inf or NaN, largest magnitude 6 */
  fmt_init(&g_fmt[OF_E2M1], 2, 1, 1, SPEC_NONE, 1);
  /* canonical NaN codes (positive) */
  g_fmt[OF_BF16].nan_code = 0x7FC0u;
  g_fmt[OF_FP16].nan_code = 0x7E00u;
  g_fmt[OF_E4M3].nan_code = 0x7Fu;
  g_fmt[OF_E5M2].nan_code = 0x7Fu;
  g_fmt[OF_E2M1].nan_code = 0x0u; /* no NaN code: an MX block carries NaN in its scale */
  /* OF_FP32 is a passthrough and has no grid */
  g_ready = 1;
}

static int fmt_bits(int fmt) {
  switch (fmt) {
  case OF_BF16: return 16;
  case OF_FP16: return 16;
  case OF_E4M3: return 8;
  case OF_E5M2: return 8;
  case OF_FP32: return 32;
  case OF_E2M1: return 4;
  case OF_E8M0: return 8;
  default: return 0;
  }
}

static uint32_t f32_bits(float x) {
  uint32_t u;
  memcpy(&u, &x, 4);
  return u;
}

static float f32_from_bits(uint32_t u) {
  float x;
  memcpy(&x, &u, 4);
  return x;
}

/* E8M0: the value 2^(code - 127); code 255 is NaN (OCP MX scale format). */
static double decode_e8m0(uint32_t code) {
  code &= 0xFFu;
  return code == 0xFFu ? NAN : ldexp(1.0, (int)code - 127);
}

/* Value of a stored code, as a double (exact). */
static double decode(int fmt, uint32_t code) {
  if (fmt == OF_FP32) return (double)f32_from_bits(code);
  if (fmt == OF_E8M0) return decode_e8m0(code);
  return decode_def(&g_fmt[fmt], code);
}

/* Round the value x (exact, as a double) onto the grid of format fmt.
 * mode = OR_RNE (nearest, ties to the code with an even last mantissa bit) or
 * OR_SR (stochastic, draw r16). */
static uint32_t encode_val(int fmt, double x, int mode, uint32_t r16) {
  const ofmt *f = &g_fmt[fmt];
  const int nb = f->ebits + f->mbits;
  const uint32_t sign = signbit(x) ? (1u << nb) : 0u;
  if (isnan(x)) return f->nan_code; /* the sign of a NaN carries no meaning */
  const double a = fabs(x);
  if (f->satfinite && a >= f->max) return sign | f->max_code;
  if (!f->satfinite && isinf(a)) return sign | f->inf_code;

  /* largest grid index i with val[i] <= a */
  int lo_i = 0, hi_i = f->nval - 1;
  while (lo_i < hi_i) {
    const int mid = (lo_i + hi_i + 1) / 2;
    if (f->val[mid] <= a) lo_i = mid;
    else hi_i = mid - 1;
  }
  const double lo = f->val[lo_i];
  if (lo == a) return sign | f->code[lo_i];
  double hi;
  uint32_t hi_code;
  if (lo_i + 1 < f->nval) {
    hi = f->val[lo_i + 1];
    hi_code = f->code[lo_i + 1];
  } else {
    /* above the largest finite value of an IEEE format: the next point of
     * the unbounded grid stands for Inf */
    hi = f->beyond;
    hi_code = f->inf_code;
  }
  const uint32_t lo_code = f->code[lo_i];
  uint32_t out;
  if (mode == OR_RNE) {
    const double dlo = a - lo, dhi = hi - a; /* exact */
    if (dlo < dhi) out = lo_code;
    else if (dhi < dlo) out = hi_code;
    else out = (lo_code & 1u) ? hi_code : lo_code;
  } else {
    const double frac = (a - lo) / (hi - lo); /* exact: spacing is a power of two */
    const double k = floor(frac * 65536.0);
    out = (k + (double)r16 >= 65536.0) ? hi_code : lo_code;
  }
  return sign | out;
}

/* Round the fp32 value xf into format fmt (FP32 is a passthrough). */
static uint32_t encode(int fmt, float xf, int mode, uint32_t r16) {
  if (fmt == OF_FP32) return isnan(xf) ? 0x7FC00000u : f32_bits(xf);
  return encode_val(fmt, (double)xf, mode, r16);
}

/* ------------------------------------------------------------------------ */
/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw; SC'11)                         */
/* ------------------------------------------------------------------------ */

static void philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
  uint32_t c[4] = {ctr_in[0], ctr_in[1], ctr_in[2], ctr_in[3]};
  uint32_t k0 = key_in[0], k1 = key_in[1];
  for (int round = 0; round < 10; ++round) {
    if (round > 0) {
      k0 += 0x9E3779B9u; /* golden ratio */
      k1 += 0xBB67AE85u; /* sqrt(3) - 1 */
    }
    const uint64_t p0 = (uint64_t)0xD2511F53u * (uint64_t)c[0];
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * (uint64_t)c[2];
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c[1] ^ k0;
    const uint32_t n1 = (uint32_t)p1;
    const uint32_t n2 = (uint32_t)(p0 >> 32) ^ c[3] ^ k1;
    const uint32_t n3 = (uint32_t)p0;
    c[0] = n0;
    c[1] = n1;
    c[2] = n2;
    c[3] = n3;
  }
  out[0] = c[0];
  out[1] = c[1];
  out[2] = c[2];
  out[3] = c[3];
}

/* 16-bit draw for global element index idx at step t on stream `stream`. */
static uint32_t draw16(uint64_t seed, int64_t t, uint32_t stream, int64_t idx) {
  const uint64_t j = (uint64_t)idx >> 3;
  const uint32_t ctr[4] = {(uint32_t)j, (uint32_t)(j >> 32), (uint32_t)t, stream};
  const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  uint32_t out[4];
  philox4x32_10(ctr, key, out);
  const uint32_t lane = (uint32_t)((uint64_t)idx & 7u);
  const uint32_t word = out[lane >> 1];
  return (lane & 1u) ? (word >> 16) : (word & 0xFFFFu);
}

/* ------------------------------------------------------------------------ */
/* The step                                                                  */
/* ------------------------------------------------------------------------ */

typedef struct {
  double lr_add, lr_mul, beta1, beta2, eps, tau, r_max, eps0, g_max, d_mult_max, w_max;
  int bias_correction, rounding;
  uint64_t seed;
  int64_t step;
} ohp;

typedef struct {
  float B1, B2, OMB1, OMB2, SA, IBC2, LRM, EPS, TAU, GMAX, ULO, UHI, WMAX;
} oscal;

static int check_hp(const ohp *h) {
  if (!(h->beta1 >= 0.0 && h->beta1 < 1.0)) return ORACLE_EINVAL;
  if (!(h->beta2 >= 0.0 && h->beta2 < 1.0)) return ORACLE_EINVAL;
  if (!(h->eps >= 0.0)) return ORACLE_EINVAL;
  if (!(h->tau > 0.0)) return ORACLE_EINVAL;
  if (!(h->r_max > 0.0 && h->r_max < 1.0)) return ORACLE_EINVAL;
  if (!(h->eps0 >= 0.0 && h->eps0 < h->r_max)) return ORACLE_EINVAL;
  if (!(h->g_max > 0.0) || !(h->d_mult_max > 0.0) || !(h->w_max > 0.0)) return ORACLE_EINVAL;
  if (h->step < 1 || h->step > 0xFFFFFFFFll) return ORACLE_EINVAL;
  if (h->rounding != OR_RNE && h->rounding != OR_SR) return ORACLE_EINVAL;
  if (h->bias_correction != 0 && h->bias_correction != 1) return ORACLE_EINVAL;
  return ORACLE_OK;
}

static void make_scalars(const ohp *h, oscal *s) {
  const double t = (double)h->step;
  s->B1 = (float)h->beta1;
  s->B2 = (float)h->beta2;
  s->OMB1 = (float)(1.0 - h->beta1);
  s->OMB2 = (float)(1.0 - h->beta2);
  if (h->bias_correction) {
    s->SA = (float)(h->lr_add / (1.0 - pow(h->beta1, t)));
    s->IBC2 = (float)(1.0 / (1.0 - pow(h->beta2, t)));
  } else {
    s->SA = (float)h->lr_add;
    s->IBC2 = 1.0f;
  }
  s->LRM = (float)h->lr_mul;
  s->EPS = (float)h->eps;
  s->TAU = (float)h->tau;
  s->GMAX = (float)h->g_max;
  double ulo = -(h->r_max - h->eps0), uhi = h->r_max;
  if (isfinite(h->d_mult_max)) {
    /* |log2(1+u)| <= d  <=>  2^-d - 1 <= u <= 2^d - 1 */
    const double lo_cap = exp2(-h->d_mult_max) - 1.0, hi_cap = exp2(h->d_mult_max) - 1.0;
    if (lo_cap > ulo) ulo = lo_cap;
    if (hi_cap < uhi) uhi = hi_cap;
  }
  s->ULO = (float)ulo;
  s->UHI = (float)uhi;
  s->WMAX = (float)h->w_max;
}

/* NaN passes through: both comparisons are false. */
static float clampf(float x, float lo, float hi) { return x < lo ? lo : (x > hi ? hi : x); }

/* One element of the step in the fixed FP32 order; returns the unrounded new
 * weight and updates the three moments in place. */
static float oracle_step_elem(float w, float g, float *pm, float *pv, float *pve, const oscal *s) {
  const float LN2 = (float)0.69314718055994530942; /* fp32(ln 2) */
  /* additive branch (Algorithm 1; Algorithm 2 without bias correction) */
  const float m = fmaf(s->B1, *pm, s->OMB1 * g);
  const float v = fmaf(s->B2, *pv, s->OMB2 * (g * g));
  const float den_a = sqrtf(v * s->IBC2) + s->EPS;
  const float ua = -((s->SA * m) / den_a);
  /* multiplicative branch: gradient w.r.t. the exponent, second moment */
  const float ge = (LN2 * w) * g;
  const float ve = fmaf(s->B2, *pve, s->OMB2 * (ge * ge));
  const float den_m = sqrtf(ve * s->IBC2) + s->EPS;
  const float r = clampf(ge / den_m, -s->GMAX, s->GMAX);
  const float ut = -(s->LRM * r);
  /* relative conversion: rho = max(|w|, tau), then the u_m clip and cap */
  const float aw = fabsf(w);
  const float rho = aw > s->TAU ? aw : s->TAU;
  const float um = clampf(ut / rho, s->ULO, s->UHI);
  /* combine: w + w u_m + u_a, then the optional final weight clamp */
  float wn = fmaf(w, um, w) + ua;
  wn = clampf(wn, -s->WMAX, s->WMAX);
  *pm = m;
  *pv = v;
  *pve = ve;
  return wn;
}

static float load_grad(int gfmt, const void *g, int64_t i) {
  if (gfmt == OG_FP32) return ((const float *)g)[i];
  return (float)decode(OF_BF16, ((const uint16_t *)g)[i]);
}

/* A moment as stored: fp32, or a bf16 code decoded exactly. */
static float load_state(int sfmt, const void *a, int64_t i) {
  if (sfmt == OS_FP32) return ((const float *)a)[i];
  return (float)decode(OF_BF16, ((const uint16_t *)a)[i]);
}

/* Store a moment: fp32 as is, or rounded to bf16 -- to nearest (ties to
 * even), or stochastically with the 16-bit draw r16. */
static void store_state(int sfmt, void *a, int64_t i, float x, uint32_t r16) {
  if (sfmt == OS_FP32) ((float *)a)[i] = x;
  else if (sfmt == OS_BF16) ((uint16_t *)a)[i] = (uint16_t)encode(OF_BF16, x, OR_RNE, 0u);
  else ((uint16_t *)a)[i] = (uint16_t)encode(OF_BF16, x, OR_SR, r16);
}

/* One element: load the three moments, step, store them back.  With
 * stochastically rounded bf16 moments, moment k (m, v, v_e) of the element
 * with global index idx draws from stream 1 + k at the step's (seed, t). */
static float step_stored(float w, float g, int sfmt, void *m, void *v, void *ve, int64_t i,
                         const oscal *s, const ohp *h, int64_t idx) {
  float mi = load_state(sfmt, m, i), vi = load_state(sfmt, v, i), vei = load_state(sfmt, ve, i);
  const float wn = oracle_step_elem(w, g, &mi, &vi, &vei, s);
  const int sr = sfmt == OS_BF16_SR;
  store_state(sfmt, m, i, mi, sr ? draw16(h->seed, h->step, 1u, idx) : 0u);
  store_state(sfmt, v, i, vi, sr ? draw16(h->seed, h->step, 2u, idx) : 0u);
  store_state(sfmt, ve, i, vei, sr ? draw16(h->seed, h->step, 3u, idx) : 0u);
  return wn;
}

static uint32_t load_code(int fmt, const void *w, int64_t i) {
  switch (fmt_bits(fmt)) {
  case 8: return ((const uint8_t *)w)[i];
  case 16: return ((const uint16_t *)w)[i];
  default: return ((const uint32_t *)w)[i];
  }
}

static void store_code(int fmt, void *w, int64_t i, uint32_t c) {
  switch (fmt_bits(fmt)) {
  case 8: ((uint8_t *)w)[i] = (uint8_t)c; break;
  case 16: ((uint16_t *)w)[i] = (uint16_t)c; break;
  default: ((uint32_t *)w)[i] = c; break;
  }
}

static int fill_hp(ohp *h, double lr_add, double lr_mul, double beta1, double beta2, double eps,
                   double tau, double r_max, double eps0, double g_max, double d_mult_max,
                   double w_max, int bias_correction, int rounding, uint64_t seed, int64_t step) {
  h->lr_add = lr_add;
  h->lr_mul = lr_mul;
  h->beta1 = beta1;
  h->beta2 = beta2;
  h->eps = eps;
  h->tau = tau;
  h->r_max = r_max;
  h->eps0 = eps0;
  h->g_max = g_max;
  h->d_mult_max = d_mult_max;
  h->w_max = w_max;
  h->bias_correction = bias_correction;
  h->rounding = rounding;
  h->seed = seed;
  h->step = step;
  return check_hp(h);
}

/* The BF16 compute copy of a stored weight value: the value the forward and
 * backward GEMMs read, refreshed from the master storage after each update
 * (the FP8-master dataflow figure), rounded to nearest-even. */
static uint16_t compute_copy(float stored) { return (uint16_t)encode(OF_BF16, stored, OR_RNE, 0u); }

/* Per-element M+Adam step on an unscaled storage format.
 * Element i has global index gidx[i] (or index_base + i when gidx is NULL),
 * which keys its stochastic-rounding draw. */
int oracle_step(int wfmt, void *w, uint16_t *copy, int gfmt, const void *g, int sfmt, void *m,
                void *v, void *ve, int64_t n, const int64_t *gidx, int64_t index_base, double lr_add, double lr_mul,
                double beta1, double beta2, double eps, double tau, double r_max, double eps0,
                double g_max, double d_mult_max, double w_max, int bias_correction, int rounding,
                uint64_t seed, int64_t step) {
  init_formats();
  ohp h;
  if (fill_hp(&h, lr_add, lr_mul, beta1, beta2, eps, tau, r_max, eps0, g_max, d_mult_max,
              w_max, bias_correction, rounding, seed, step) != ORACLE_OK)
    return ORACLE_EINVAL;
  if (wfmt != OF_BF16 && wfmt != OF_E4M3 && wfmt != OF_E5M2 && wfmt != OF_FP32) return ORACLE_EINVAL;
  if (gfmt != OG_FP32 && gfmt != OG_BF16) return ORACLE_EINVAL;
  if (sfmt != OS_FP32 && sfmt != OS_BF16 && sfmt != OS_BF16_SR) return ORACLE_EINVAL;
  if (n < 0) return ORACLE_EINVAL;
  oscal s;
  make_scalars(&h, &s);
  for (int64_t i = 0; i < n; ++i) {
    const float wv = (float)decode(wfmt, load_code(wfmt, w, i));
    const float gv = load_grad(gfmt, g, i);
    const int64_t idx = gidx ? gidx[i] : index_base + i;
    const float wn = step_stored(wv, gv, sfmt, m, v, ve, i, &s, &h, idx);
    const uint32_t r16 = (h.rounding == OR_SR) ? draw16(h.seed, h.step, 0u, idx) : 0u;
    const uint32_t code = encode(wfmt, wn, h.rounding, r16);
    store_code(wfmt, w, i, code);
    if (copy) copy[i] = compute_copy((float)decode(wfmt, code));
  }
  return ORACLE_OK;
}

#define BLOCK 128

static float fp8_max(int fmt) { return (float)g_fmt[fmt].max; }

/* FP16 scale for one block of updated weights (rule in the file header). */
static uint16_t block_scale(int fmt, const float *wn) {
  double amax = 0.0;
  int nonfinite = 0;
  for (int i = 0; i < BLOCK; ++i) {
    if (!isfinite(wn[i])) nonfinite = 1;
    else if (fabs((double)wn[i]) > amax) amax = fabs((double)wn[i]);
  }
  if (nonfinite) return 0x7E00u;
  if (amax == 0.0) return 0x3C00u; /* 1.0 */
  const float ratio = (float)amax / fp8_max(fmt);
  uint32_t sc = encode(OF_FP16, ratio, OR_RNE, 0u);
  if (sc == 0u) sc = 0x0001u;       /* underflow: smallest subnormal */
  if (sc == 0x7C00u) sc = 0x7BFFu;  /* overflow: largest finite */
  return (uint16_t)sc;
}

/* Block-scaled FP8 M+Adam step.  n must be a multiple of 128; elements
 * [128 b, 128 b + 128) form block b with scale scales[b]. */
int oracle_step_block(int wfmt, uint8_t *q, uint16_t *scales, uint16_t *copy, int gfmt,
                      const void *g, int sfmt, void *m, void *v, void *ve, int64_t n, const int64_t *gidx, int64_t index_base,
                      double lr_add, double lr_mul, double beta1, double beta2, double eps,
                      double tau, double r_max, double eps0, double g_max, double d_mult_max,
                      double w_max, int bias_correction, int rounding, uint64_t seed,
                      int64_t step) {
  init_formats();
  ohp h;
  if (fill_hp(&h, lr_add, lr_mul, beta1, beta2, eps, tau, r_max, eps0, g_max, d_mult_max,
              w_max, bias_correction, rounding, seed, step) != ORACLE_OK)
    return ORACLE_EINVAL;
  if (wfmt != OF_E4M3 && wfmt != OF_E5M2) return ORACLE_EINVAL;
  if (gfmt != OG_FP32 && gfmt != OG_BF16) return ORACLE_EINVAL;
  if (sfmt != OS_FP32 && sfmt != OS_BF16 && sfmt != OS_BF16_SR) return ORACLE_EINVAL;
  if (n < 0 || n % BLOCK != 0) return ORACLE_EINVAL;
  oscal s;
  make_scalars(&h, &s);
  float wn[BLOCK];
  for (int64_t b = 0; b < n / BLOCK; ++b) {
    const float sold = (float)decode(OF_FP16, scales[b]);
    for (int k = 0; k < BLOCK; ++k) {
      const int64_t i = b * BLOCK + k;
      const float wv = (float)decode(wfmt, q[i]) * sold;
      const float gv = load_grad(gfmt, g, i);
      wn[k] = step_stored(wv, gv, sfmt, m, v, ve, i, &s, &h, gidx ? gidx[i] : index_base + i);
    }
    const uint16_t snew = block_scale(wfmt, wn);
    const float sf = (float)decode(OF_FP16, snew);
    for (int k = 0; k < BLOCK; ++k) {
      const int64_t i = b * BLOCK + k;
      const int64_t idx = gidx ? gidx[i] : index_base + i;
      const uint32_t r16 = (h.rounding == OR_SR) ? draw16(h.seed, h.step, 0u, idx) : 0u;
      q[i] = (uint8_t)encode(wfmt, wn[k] / sf, h.rounding, r16);
      if (copy) copy[i] = compute_copy((float)decode(wfmt, q[i]) * sf);
    }
    scales[b] = snew;
  }
  return ORACLE_OK;
}

/* Round fp32 values into a storage format with round-to-nearest-even. */
int oracle_encode_array(int fmt, const float *x, void *codes, int64_t n) {
  init_formats();
  if (fmt < 0 || fmt >= OF_NFMT || fmt == OF_E2M1 || n < 0) return ORACLE_EINVAL;
  for (int64_t i = 0; i < n; ++i) store_code(fmt, codes, i, encode(fmt, x[i], OR_RNE, 0u));
  return ORACLE_OK;
}

/* Block-scaled FP8 encoding of fp32 values with round-to-nearest-even. */
int oracle_encode_block(int fmt, const float *x, uint8_t *q, uint16_t *scales, int64_t n) {
  init_formats();
  if ((fmt != OF_E4M3 && fmt != OF_E5M2) || n < 0 || n % BLOCK != 0) return ORACLE_EINVAL;
  for (int64_t b = 0; b < n / BLOCK; ++b) {
    const uint16_t sc = block_scale(fmt, x + b * BLOCK);
    const float sf = (float)decode(OF_FP16, sc);
    for (int k = 0; k < BLOCK; ++k)
      q[b * BLOCK + k] = (uint8_t)encode(fmt, x[b * BLOCK + k] / sf, OR_RNE, 0u);
    scales[b] = sc;
  }
  return ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* MXFP4 storage (OCP Microscaling Formats v1.0)                             */
/* ------------------------------------------------------------------------ */

/* The paper trains with 4-bit block-scaled master weights (Section 4.2, its
 * NVFP4/FP8 setting) without defining the format.  This oracle uses the MX
 * block format of the OCP specification: blocks of 32 contiguous elements,
 * each an E2M1 value, sharing one E8M0 scale X = 2^s; the weight is q * X.
 * Two elements per byte, element 2k in the low nibble.
 *
 * Scale of a block of new weights w' (the specification's conversion rule):
 *   s = floor(log2(max|w'|)) - emax, emax = exponent of E2M1's largest value
 *   (6 = 1.5 * 2^2, so emax = 2), clamped to E8M0's range [-127, 127];
 *   an all-zero block takes s = 0 (any scale represents it); a block holding
 *   a non-finite w' takes the NaN scale and zero payloads.
 * Payloads: q = round(w' / X) on the E2M1 grid with the step's rounding mode,
 * saturating at +-6 (w' / X is exact: X is a power of two). */
#define MX_BLOCK 32

static uint32_t mx_get(const uint8_t *q, int64_t i) { return (q[i >> 1] >> (4 * (i & 1))) & 0xFu; }

static void mx_put(uint8_t *q, int64_t i, uint32_t c) {
  const int sh = 4 * (int)(i & 1);
  q[i >> 1] = (uint8_t)((q[i >> 1] & ~(0xFu << sh)) | ((c & 0xFu) << sh));
}

/* Exponent s of the block scale for the values wn[0..31]; 128 marks NaN. */
static int mx_scale_exp(const float *wn) {
  double amax = 0.0;
  for (int i = 0; i < MX_BLOCK; ++i) {
    if (!isfinite(wn[i])) return 128;
    if (fabs((double)wn[i]) > amax) amax = fabs((double)wn[i]);
  }
  if (amax == 0.0) return 0;
  int e_amax, e_top;
  (void)frexp(amax, &e_amax);                 /* amax = f 2^e, f in [0.5, 1) */
  (void)frexp(g_fmt[OF_E2M1].max, &e_top);
  int s = (e_amax - 1) - (e_top - 1);         /* floor(log2 amax) - emax */
  if (s < -127) s = -127;
  if (s > 127) s = 127;
  return s;
}

static uint32_t mx_scale_code(int s) { return s == 128 ? 0xFFu : (uint32_t)(s + 127); }

/* Payload code of w' in a block of scale exponent s. */
static uint32_t mx_payload(float wn, int s, int mode, uint32_t r16) {
  if (s == 128) return 0u;
  return encode_val(OF_E2M1, ldexp((double)wn, -s), mode, r16);
}

/* The stored value q * X as the fp32 the step reads. */
static float mx_value(uint32_t qcode, uint32_t scode) {
  return (float)(decode(OF_E2M1, qcode) * decode_e8m0(scode));
}

/* M+Adam step on MXFP4 storage.  n must be a multiple of 32; q holds n/2
 * bytes, scales n/32 E8M0 codes. */
int oracle_step_mx(uint8_t *q, uint8_t *scales, uint16_t *copy, int gfmt, const void *g, int sfmt,
                   void *m, void *v, void *ve, int64_t n, const int64_t *gidx, int64_t index_base,
                   double lr_add, double lr_mul, double beta1, double beta2, double eps, double tau,
                   double r_max, double eps0, double g_max, double d_mult_max, double w_max,
                   int bias_correction, int rounding, uint64_t seed, int64_t step) {
  init_formats();
  ohp h;
  if (fill_hp(&h, lr_add, lr_mul, beta1, beta2, eps, tau, r_max, eps0, g_max, d_mult_max,
              w_max, bias_correction, rounding, seed, step) != ORACLE_OK)
    return ORACLE_EINVAL;
  if (gfmt != OG_FP32 && gfmt != OG_BF16) return ORACLE_EINVAL;
  if (sfmt != OS_FP32 && sfmt != OS_BF16 && sfmt != OS_BF16_SR) return ORACLE_EINVAL;
  if (n < 0 || n % MX_BLOCK != 0) return ORACLE_EINVAL;
  oscal s;
  make_scalars(&h, &s);
  float wn[MX_BLOCK];
  for (int64_t b = 0; b < n / MX_BLOCK; ++b) {
    for (int k = 0; k < MX_BLOCK; ++k) {
      const int64_t i = b * MX_BLOCK + k;
      const float wv = mx_value(mx_get(q, i), scales[b]);
      wn[k] = step_stored(wv, load_grad(gfmt, g, i), sfmt, m, v, ve, i, &s, &h,
                          gidx ? gidx[i] : index_base + i);
    }
    const int se = mx_scale_exp(wn);
    const uint32_t sc = mx_scale_code(se);
    for (int k = 0; k < MX_BLOCK; ++k) {
      const int64_t i = b * MX_BLOCK + k;
      const int64_t idx = gidx ? gidx[i] : index_base + i;
      const uint32_t r16 = (h.rounding == OR_SR) ? draw16(h.seed, h.step, 0u, idx) : 0u;
      const uint32_t c = mx_payload(wn[k], se, h.rounding, r16);
      mx_put(q, i, c);
      if (copy) copy[i] = compute_copy(mx_value(c, sc));
    }
    scales[b] = (uint8_t)sc;
  }
  return ORACLE_OK;
}

/* MXFP4 encoding of fp32 values with round-to-nearest-even. */
int oracle_encode_mx(const float *x, uint8_t *q, uint8_t *scales, int64_t n) {
  init_formats();
  if (n < 0 || n % MX_BLOCK != 0) return ORACLE_EINVAL;
  for (int64_t b = 0; b < n / MX_BLOCK; ++b) {
    const int se = mx_scale_exp(x + b * MX_BLOCK);
    for (int k = 0; k < MX_BLOCK; ++k)
      mx_put(q, b * MX_BLOCK + k, mx_payload(x[b * MX_BLOCK + k], se, OR_RNE, 0u));
    scales[b] = (uint8_t)mx_scale_code(se);
  }
  return ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* NVFP4 storage (NVIDIA's two-level 4-bit block format)                     */
/* ------------------------------------------------------------------------ */

/* NVFP4 (the format the paper's 4-bit runs name, Section 4.2): blocks of 16
 * contiguous E2M1 values, each block with an E4M3 scale code c_b, and one
 * fp32 scale s_t per tensor.  The weight is q * D_b with D_b = fp32(E4M3(c_b)
 * * s_t).  The scale array holds s_t (4 bytes) followed by one c_b per block.
 *
 * Encoding: s_t = fp32(amax / 2688) over the finite |x| of the tensor
 * (2688 = 6 * 448: E2M1's largest value times E4M3's), 1 when there is no
 * finite nonzero value.  A step keeps s_t (the caller re-encodes to refresh
 * it) and recomputes every block: c_b = RNE_E4M3(fp32(amax_b / fp32(6 s_t)))
 * (saturating at 448), the NaN code 0x7F when the block holds a non-finite
 * value; payloads q = round(fp32(w' / D_b)) onto E2M1 with the step's
 * rounding, saturating at +-6, and 0 when D_b is 0 or the block is NaN. */
#define NV_BLOCK 16

static float nv_get_st(const uint8_t *scales) {
  float st;
  memcpy(&st, scales, 4);
  return st;
}

/* D_b: the block's dequantization factor, fp32(E4M3 value * s_t). */
static float nv_den(uint32_t code, float st) { return (float)decode(OF_E4M3, code) * st; }

static uint32_t nv_block_code(const float *wn, float st) {
  float amax = 0.0f;
  for (int i = 0; i < NV_BLOCK; ++i) {
    if (!isfinite(wn[i])) return 0x7Fu;
    if (fabsf(wn[i]) > amax) amax = fabsf(wn[i]);
  }
  const float six_st = 6.0f * st;
  return encode(OF_E4M3, amax / six_st, OR_RNE, 0u);
}

static uint32_t nv_payload(float wn, uint32_t code, float den, int mode, uint32_t r16) {
  if (code == 0x7Fu || den == 0.0f) return 0u;
  return encode(OF_E2M1, wn / den, mode, r16);
}

/* M+Adam step on NVFP4 storage.  n must be a multiple of 16; q holds n/2
 * bytes, scales 4 + n/16 bytes (s_t, then the block codes). */
int oracle_step_nv(uint8_t *q, uint8_t *scales, uint16_t *copy, int gfmt, const void *g, int sfmt,
                   void *m, void *v, void *ve, int64_t n, const int64_t *gidx, int64_t index_base,
                   double lr_add, double lr_mul, double beta1, double beta2, double eps, double tau,
                   double r_max, double eps0, double g_max, double d_mult_max, double w_max,
                   int bias_correction, int rounding, uint64_t seed, int64_t step) {
  init_formats();
  ohp h;
  if (fill_hp(&h, lr_add, lr_mul, beta1, beta2, eps, tau, r_max, eps0, g_max, d_mult_max,
              w_max, bias_correction, rounding, seed, step) != ORACLE_OK)
    return ORACLE_EINVAL;
  if (gfmt != OG_FP32 && gfmt != OG_BF16) return ORACLE_EINVAL;
  if (sfmt != OS_FP32 && sfmt != OS_BF16 && sfmt != OS_BF16_SR) return ORACLE_EINVAL;
  if (n < 0 || n % NV_BLOCK != 0) return ORACLE_EINVAL;
  oscal s;
  make_scalars(&h, &s);
  const float st = nv_get_st(scales);
  uint8_t *codes = scales + 4;
  float wn[NV_BLOCK];
  for (int64_t b = 0; b < n / NV_BLOCK; ++b) {
    const float dold = nv_den(codes[b], st);
    for (int k = 0; k < NV_BLOCK; ++k) {
      const int64_t i = b * NV_BLOCK + k;
      const float wv = (float)decode(OF_E2M1, mx_get(q, i)) * dold;
      wn[k] = step_stored(wv, load_grad(gfmt, g, i), sfmt, m, v, ve, i, &s, &h,
                          gidx ? gidx[i] : index_base + i);
    }
    const uint32_t c = nv_block_code(wn, st);
    const float dnew = nv_den(c, st);
    for (int k = 0; k < NV_BLOCK; ++k) {
      const int64_t i = b * NV_BLOCK + k;
      const int64_t idx = gidx ? gidx[i] : index_base + i;
      const uint32_t r16 = (h.rounding == OR_SR) ? draw16(h.seed, h.step, 0u, idx) : 0u;
      const uint32_t pc = nv_payload(wn[k], c, dnew, h.rounding, r16);
      mx_put(q, i, pc);
      if (copy) copy[i] = compute_copy((float)decode(OF_E2M1, pc) * dnew);
    }
    codes[b] = (uint8_t)c;
  }
  return ORACLE_OK;
}

/* NVFP4 with current scaling: the per-tensor scale is derived anew from the
 * updated tensor at every step.  Section 4.2's prototype keeps its master
 * weights in NVFP4 by dequantizing, taking the FP32 step and quantizing the
 * result again (the quantize/dequantize simulation its overhead discussion
 * and Appendix G describe); a quantizer that sees the whole updated tensor
 * derives its per-tensor scale from that tensor's amax.  This step does the
 * same: every w' of the tensor first (moments updated as in every step),
 * then s_t' = fp32(amax / 2688) over the finite |w'| (1 when none is
 * nonzero), then every block by the NVFP4 rule above with s_t'.
 * State: q (n/2 packed payload bytes), st (4 bytes: the fp32 per-tensor
 * scale) and codes (n/16 E4M3 block codes), all updated in place; g (fp32)
 * is only read.  wn (n floats, output) receives the FP32 step's w' of every element,
 * the values the re-quantization starts from. */
int oracle_step_nv_current(uint8_t *q, uint8_t *st, uint8_t *codes, uint16_t *copy,
                           const float *g, int sfmt, void *m, void *v, void *ve, int64_t n,
                           const int64_t *gidx, int64_t index_base, float *wn, double lr_add,
                           double lr_mul, double beta1, double beta2, double eps, double tau,
                           double r_max, double eps0, double g_max, double d_mult_max,
                           double w_max, int bias_correction, int rounding, uint64_t seed,
                           int64_t step) {
  init_formats();
  ohp h;
  if (fill_hp(&h, lr_add, lr_mul, beta1, beta2, eps, tau, r_max, eps0, g_max, d_mult_max,
              w_max, bias_correction, rounding, seed, step) != ORACLE_OK)
    return ORACLE_EINVAL;
  if (sfmt != OS_FP32 && sfmt != OS_BF16 && sfmt != OS_BF16_SR) return ORACLE_EINVAL;
  if (n < 0 || n % NV_BLOCK != 0 || !st || !wn) return ORACLE_EINVAL;
  oscal s;
  make_scalars(&h, &s);
  const float sto = nv_get_st(st);
  /* the FP32 step on every dequantized weight */
  float amax = 0.0f;
  for (int64_t i = 0; i < n; ++i) {
    const float wv = (float)decode(OF_E2M1, mx_get(q, i)) * nv_den(codes[i / NV_BLOCK], sto);
    wn[i] = step_stored(wv, g[i], sfmt, m, v, ve, i, &s, &h, gidx ? gidx[i] : index_base + i);
    if (isfinite(wn[i]) && fabsf(wn[i]) > amax) amax = fabsf(wn[i]);
  }
  /* the new per-tensor scale, then every block with it */
  const float stn = amax > 0.0f ? amax / 2688.0f : 1.0f;
  memcpy(st, &stn, 4);
  for (int64_t b = 0; b < n / NV_BLOCK; ++b) {
    const float *wb = wn + b * NV_BLOCK;
    const uint32_t c = nv_block_code(wb, stn);
    const float den = nv_den(c, stn);
    for (int k = 0; k < NV_BLOCK; ++k) {
      const int64_t i = b * NV_BLOCK + k;
      const int64_t idx = gidx ? gidx[i] : index_base + i;
      const uint32_t r16 = (h.rounding == OR_SR) ? draw16(h.seed, h.step, 0u, idx) : 0u;
      const uint32_t pc = nv_payload(wb[k], c, den, h.rounding, r16);
      mx_put(q, i, pc);
      if (copy) copy[i] = compute_copy((float)decode(OF_E2M1, pc) * den);
    }
    codes[b] = (uint8_t)c;
  }
  return ORACLE_OK;
}

int oracle_encode_nv(const float *x, uint8_t *q, uint8_t *scales, int64_t n) {
  init_formats();
  if (n < 0 || n % NV_BLOCK != 0) return ORACLE_EINVAL;
  float amax = 0.0f;
  for (int64_t i = 0; i < n; ++i)
    if (isfinite(x[i]) && fabsf(x[i]) > amax) amax = fabsf(x[i]);
  const float st = amax > 0.0f ? amax / 2688.0f : 1.0f;
  memcpy(scales, &st, 4);
  for (int64_t b = 0; b < n / NV_BLOCK; ++b) {
    const uint32_t c = nv_block_code(x + b * NV_BLOCK, st);
    const float den = nv_den(c, st);
    for (int k = 0; k < NV_BLOCK; ++k)
      mx_put(q, b * NV_BLOCK + k, nv_payload(x[b * NV_BLOCK + k], c, den, OR_RNE, 0u));
    scales[4 + b] = (uint8_t)c;
  }
  return ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* The moment-free update rules of Appendix B                               */
/* ------------------------------------------------------------------------ */

/* One element of Appendix B's rules: additive u_a = -eta_a g; multiplicative
 * g_e = ln2 w g, ut = -eta_m g_e, u_m = clip(ut / max(|w|, tau)); combined
 * w + w u_m + u_a (eta_m = 0 gives the additive rule, eta_a = 0 the
 * multiplicative one).  Same FP32 conventions as the M+Adam step. */
static float plain_step_elem(float w, float g, float lra, const oscal *s) {
  const float LN2 = (float)0.69314718055994530942;
  const float ua = -(lra * g);
  const float ge = (LN2 * w) * g;
  const float ut = -(s->LRM * ge);
  const float aw = fabsf(w);
  const float rho = aw > s->TAU ? aw : s->TAU;
  const float um = clampf(ut / rho, s->ULO, s->UHI);
  const float wn = fmaf(w, um, w) + ua;
  return clampf(wn, -s->WMAX, s->WMAX);
}

int oracle_plain_step(int wfmt, void *w, int gfmt, const void *g, int64_t n, const int64_t *gidx,
                      int64_t index_base, double lr_add, double lr_mul, double tau, double r_max,
                      double eps0, double d_mult_max, double w_max, int rounding, uint64_t seed,
                      int64_t step) {
  init_formats();
  ohp h;
  /* moment hyper-parameters are unused by these rules; fixed valid values */
  if (fill_hp(&h, lr_add, lr_mul, 0.9, 0.999, 1e-8, tau, r_max, eps0, INFINITY, d_mult_max, w_max,
              1, rounding, seed, step) != ORACLE_OK)
    return ORACLE_EINVAL;
  if (wfmt != OF_BF16 && wfmt != OF_E4M3 && wfmt != OF_E5M2 && wfmt != OF_FP32) return ORACLE_EINVAL;
  if (gfmt != OG_FP32 && gfmt != OG_BF16) return ORACLE_EINVAL;
  if (n < 0) return ORACLE_EINVAL;
  oscal s;
  make_scalars(&h, &s);
  const float lra = (float)lr_add;
  for (int64_t i = 0; i < n; ++i) {
    const float wv = (float)decode(wfmt, load_code(wfmt, w, i));
    const float wn = plain_step_elem(wv, load_grad(gfmt, g, i), lra, &s);
    const int64_t idx = gidx ? gidx[i] : index_base + i;
    const uint32_t r16 = (h.rounding == OR_SR) ? draw16(h.seed, h.step, 0u, idx) : 0u;
    store_code(wfmt, w, i, encode(wfmt, wn, h.rounding, r16));
  }
  return ORACLE_OK;
}

/* --- small exports used by the tests ------------------------------------ */

double oracle_decode(int fmt, uint32_t code) {
  init_formats();
  return decode(fmt, code);
}

uint32_t oracle_encode(int fmt, float x, int rounding, uint32_t r16) {
  init_formats();
  if (fmt < 0 || fmt >= OF_NFMT) return 0xFFFFFFFFu;
  return encode(fmt, x, rounding, r16 & 0xFFFFu);
}

void oracle_philox4x32_10(const uint32_t *ctr, const uint32_t *key, uint32_t *out) {
  philox4x32_10(ctr, key, out);
}

uint32_t oracle_draw16(uint64_t seed, int64_t step, uint32_t stream, int64_t idx) {
  return draw16(seed, step, stream, idx);
}

/* The fp32 scalars of one step, in the order of oscal. */
int oracle_scalars(double lr_add, double lr_mul, double beta1, double beta2, double eps,
                   double tau, double r_max, double eps0, double g_max, double d_mult_max,
                   double w_max, int bias_correction, int64_t step, float *out13) {
  ohp h;
  if (fill_hp(&h, lr_add, lr_mul, beta1, beta2, eps, tau, r_max, eps0, g_max, d_mult_max, w_max,
              bias_correction, OR_RNE, 0u, step) != ORACLE_OK)
    return ORACLE_EINVAL;
  oscal s;
  make_scalars(&h, &s);
  memcpy(out13, &s, sizeof(oscal));
  return ORACLE_OK;
}
