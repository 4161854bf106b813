"""The oracle's pins must catch plausible mistakes (CPU, mutation analysis).

Each case plants one mistake in a copy of the oracle's C source (a dropped
term, a flipped sign, a wrong index or constant, a missing clamp), builds the
copy, and runs the pin tests against it; at least one pin must fail.  The
real oracle is never modified.
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "madd_oracle.c")
PINS = ["tests/test_oracle_step.py", "tests/test_oracle_block.py", "tests/test_oracle_sr_rng.py",
        "tests/test_oracle_formats.py", "tests/test_oracle_mx.py", "tests/test_oracle_nv.py",
        "tests/test_oracle_hypothesis.py"]

MUTANTS = {
    "additive sign": ("const float ua = -((s->SA * m) / den_a);",
                      "const float ua = ((s->SA * m) / den_a);"),
    "ln2 dropped": ("const float ge = (LN2 * w) * g;", "const float ge = w * g;"),
    "g not squared": ("s->OMB2 * (g * g)", "s->OMB2 * g"),
    "v_e bias correction dropped": ("sqrtf(ve * s->IBC2)", "sqrtf(ve)"),
    "v bias correction dropped": ("sqrtf(v * s->IBC2)", "sqrtf(v)"),
    "w term dropped": ("fmaf(w, um, w) + ua", "w * um + ua"),
    "multiplicative term dropped": ("fmaf(w, um, w) + ua", "w + ua"),
    "multiplicative sign": ("const float ut = -(s->LRM * r);", "const float ut = (s->LRM * r);"),
    "rho without abs": ("const float rho = aw > s->TAU ? aw : s->TAU;",
                        "const float rho = w > s->TAU ? w : s->TAU;"),
    "lower clip dropped": ("clampf(ut / rho, s->ULO, s->UHI)", "clampf(ut / rho, -1e30f, s->UHI)"),
    "g_max ignored": ("clampf(ge / den_m, -s->GMAX, s->GMAX)", "(ge / den_m)"),
    "w_max ignored": ("wn = clampf(wn, -s->WMAX, s->WMAX);", ""),
    "SR threshold off by one": ("(k + (double)r16 >= 65536.0)", "(k + (double)r16 > 65536.0)"),
    "RNE ties to odd": ("(lo_code & 1u) ? hi_code : lo_code", "(lo_code & 1u) ? lo_code : hi_code"),
    "Philox multiplier": ("0xD2511F53u", "0xD2511F55u"),
    "draw lanes swapped": ("(lane & 1u) ? (word >> 16) : (word & 0xFFFFu)",
                           "(lane & 1u) ? (word & 0xFFFFu) : (word >> 16)"),
    "first-moment bias correction dropped": (
        "s->SA = (float)(h->lr_add / (1.0 - pow(h->beta1, t)));", "s->SA = (float)h->lr_add;"),
    "beta2 in first moment": ("fmaf(s->B1, *pm, s->OMB1 * g)", "fmaf(s->B2, *pm, s->OMB2 * g)"),
    "eps inside sqrt": ("sqrtf(v * s->IBC2) + s->EPS", "sqrtf(v * s->IBC2 + s->EPS)"),
    "exponent cap symmetric in u": (
        "const double lo_cap = exp2(-h->d_mult_max) - 1.0, hi_cap = exp2(h->d_mult_max) - 1.0;",
        "const double lo_cap = -(exp2(h->d_mult_max) - 1.0), hi_cap = exp2(h->d_mult_max) - 1.0;"),
    "eps0 sign": ("double ulo = -(h->r_max - h->eps0)", "double ulo = -(h->r_max + h->eps0)"),
    "block scale constant": ("const float ratio = (float)amax / fp8_max(fmt);",
                             "const float ratio = (float)amax / 256.0f;"),
    "bf16 moments truncated": (
        "else if (sfmt == OS_BF16) ((uint16_t *)a)[i] = (uint16_t)encode(OF_BF16, x, OR_RNE, 0u);",
        "else if (sfmt == OS_BF16) ((uint16_t *)a)[i] = (uint16_t)encode(OF_BF16, x, OR_SR, 0u);"),
    "stochastic bf16 moments rounded to nearest": (
        "else ((uint16_t *)a)[i] = (uint16_t)encode(OF_BF16, x, OR_SR, r16);",
        "else ((uint16_t *)a)[i] = (uint16_t)encode(OF_BF16, x, OR_RNE, r16);"),
    "compute copy of the unrounded weight": (
        "    if (copy) copy[i] = compute_copy((float)decode(wfmt, code));",
        "    if (copy) copy[i] = compute_copy(wn);"),
    "block compute copy without the scale": (
        "      if (copy) copy[i] = compute_copy((float)decode(wfmt, q[i]) * sf);",
        "      if (copy) copy[i] = compute_copy((float)decode(wfmt, q[i]));"),
    "plain additive sign": ("  const float ua = -(lra * g);", "  const float ua = (lra * g);"),
    "plain multiplicative without rho": ("  const float um = clampf(ut / rho, s->ULO, s->UHI);\n  const float wn = fmaf(w, um, w) + ua;\n  return",
                                         "  const float um = clampf(ut, s->ULO, s->UHI);\n  const float wn = fmaf(w, um, w) + ua;\n  return"),
    "MX scale exponent off by one": ("int s = (e_amax - 1) - (e_top - 1);",
                                     "int s = (e_amax - 1) - (e_top - 2);"),
    "MX nibble order": ("const int sh = 4 * (int)(i & 1);", "const int sh = 4 * (int)(1 - (i & 1));"),
    "MX zero block scale": ("if (amax == 0.0) return 0;", "if (amax == 0.0) return -127;"),
    "MX NaN block payload": ("if (s == 128) return 0u;", "if (s == 128) return 7u;"),
    "MX scale exponent unclamped": ("  if (s < -127) s = -127;\n", ""),
    "MX dequantize without the scale": (
        "const float wv = mx_value(mx_get(q, i), scales[b]);",
        "const float wv = (float)decode(OF_E2M1, mx_get(q, i));"),
    "MX compute copy without the scale": ("if (copy) copy[i] = compute_copy(mx_value(c, sc));",
                                          "if (copy) copy[i] = compute_copy((float)decode(OF_E2M1, c));"),
    "moment draws on the weight stream": ("sr ? draw16(h->seed, h->step, 1u, idx) : 0u",
                                          "sr ? draw16(h->seed, h->step, 0u, idx) : 0u"),
    "v and v_e share a stream": ("sr ? draw16(h->seed, h->step, 3u, idx) : 0u",
                                 "sr ? draw16(h->seed, h->step, 2u, idx) : 0u"),
    "NV block scale without the factor 6": ("const float six_st = 6.0f * st;",
                                            "const float six_st = st;"),
    "NV divisor ignores the tensor scale": (
        "static float nv_den(uint32_t code, float st) { return (float)decode(OF_E4M3, code) * st; }",
        "static float nv_den(uint32_t code, float st) { return (float)decode(OF_E4M3, code); }"),
    "NV tensor scale from 448 alone": ("amax > 0.0f ? amax / 2688.0f : 1.0f", "amax > 0.0f ? amax / 448.0f : 1.0f"),
    "NV NaN block payload": ("if (code == 0x7Fu || den == 0.0f) return 0u;",
                             "if (code == 0x7Fu || den == 0.0f) return 7u;"),
    "NV current scale over non-finite values too": (
        "    if (isfinite(wn[i]) && fabsf(wn[i]) > amax) amax = fabsf(wn[i]);",
        "    if (fabsf(wn[i]) > amax) amax = fabsf(wn[i]);"),
    "NV current scaling keeps the old scale": (
        "  const float stn = amax > 0.0f ? amax / 2688.0f : 1.0f;\n  memcpy(st, &stn, 4);",
        "  const float stn = sto;\n  memcpy(st, &stn, 4);"),
    "tau replaced by eps in the relative update": (
        "const float rho = aw > s->TAU ? aw : s->TAU;", "const float rho = aw > s->EPS ? aw : s->EPS;"),
    "eps replaced by tau in the multiplicative denominator": (
        "const float den_m = sqrtf(ve * s->IBC2) + s->EPS;",
        "const float den_m = sqrtf(ve * s->IBC2) + s->TAU;"),
    "no FP8 saturation": ("if (f->satfinite && a >= f->max) return sign | f->max_code;",
                          "if (f->satfinite && a > 2 * f->max) return sign | f->max_code;"),
}


def _killed(name, tmpdir):
    a, b = MUTANTS[name]
    src = open(SRC).read()
    assert a in src, f"mutation site of {name!r} not found"
    d = os.path.join(tmpdir, str(abs(hash(name))))
    os.makedirs(d, exist_ok=True)
    c, so = os.path.join(d, "m.c"), os.path.join(d, "m.so")
    with open(c, "w") as f:
        f.write(src.replace(a, b))
    subprocess.run(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fPIC", "-shared", "-o", so, c,
                    "-lm"], check=True)
    env = dict(os.environ, MADD_ORACLE_LIB=so)
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", *PINS],
                       cwd=ROOT, env=env, capture_output=True, text=True)
    return r.returncode != 0


def test_every_planted_mistake_fails_a_pin(tmp_path):
    names = list(MUTANTS)
    with ThreadPoolExecutor(max_workers=4) as ex:
        results = list(ex.map(lambda n: _killed(n, str(tmp_path)), names))
    survivors = [n for n, k in zip(names, results) if not k]
    assert not survivors, f"mistakes no pin catches: {survivors}"
