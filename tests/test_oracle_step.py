"""Pins of the oracle's M+Adam step (CPU).

The step is an iteration without a closed-form end result, so the oracle
follows Algorithm 1 (and Algorithm 2's clamps) step by step in FP32.  These
tests tie it to what the paper and the mathematics fix:

  * additive limit (eta_m = 0): exactly Adam (Kingma & Ba), written here
    independently in fp64 -- per step and along a 100-step trajectory;
  * constant-gradient closed forms for the additive branch (Adam moves by
    eta_a * |g|/(|g|+eps) per step) and, with beta2 = 0, for the
    multiplicative branch (|w| moves by eta_m per step, or by the 0.75 clip);
  * step-1 closed forms with and without bias correction (Algorithms 1, 2);
  * multiplicative limit (eta_a = 0): sign preserving and zero absorbing in
    every storage format and rounding mode (Section 3.1, Figure 1);
  * zero revival and sign change need the additive branch (Section 3.1);
  * descent on a convex quadratic (Theorem 3.1 setting, small steps);
  * each optional clamp of Algorithm 2 (g_max, the u_m clip with eps0,
    the exponent-step cap, w_max);
  * brute force over every finite FP8 weight code against an fp64
    evaluation of the same formulas, rounded with the library RNE;
  * index keying: shards, subsets and resumption are bit-identical.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2607_10611_amd.workloads import DEFAULT_HPARAMS

LN2 = math.log(2.0)


def hp(**kw):
    h = dict(DEFAULT_HPARAMS)
    h["rounding"] = "rne"
    h.update(kw)
    return h


def run_fp32(w, g, m=None, v=None, ve=None, **kw):
    """One oracle step in the FP32 passthrough format; returns new (w, m, v, ve)."""
    w = np.ascontiguousarray(w, dtype=np.float32).copy()
    n = w.size
    m = np.zeros(n, np.float32) if m is None else m.astype(np.float32).copy()
    v = np.zeros(n, np.float32) if v is None else v.astype(np.float32).copy()
    ve = np.zeros(n, np.float32) if ve is None else ve.astype(np.float32).copy()
    codes = w.view(np.uint32)
    oracle.step("fp32", codes, np.ascontiguousarray(g, dtype=np.float32), m, v, ve, hp(**kw))
    return codes.view(np.float32), m, v, ve


def ulp32(x):
    x = np.abs(np.asarray(x, dtype=np.float32))
    return np.spacing(np.maximum(x, np.float32(np.finfo(np.float32).tiny)))


# --------------------------------------------------------------------------
# additive limit: Adam
# --------------------------------------------------------------------------

def adam_fp64(w, g, m, v, t, lr, b1, b2, eps, bias_correction=True):
    """Adam, Kingma & Ba (ICLR 2015), Algorithm 1, in float64."""
    m = b1 * m + (1 - b1) * g
    v = b2 * v + (1 - b2) * g * g
    if bias_correction:
        mh, vh = m / (1 - b1 ** t), v / (1 - b2 ** t)
    else:
        mh, vh = m, v
    return w - lr * mh / (np.sqrt(vh) + eps), m, v


@pytest.mark.parametrize("bc", [1, 0])
def test_additive_limit_is_adam_each_step(bc):
    rng = np.random.default_rng(0)
    n = 4096
    w = rng.normal(0, 0.02, n).astype(np.float32)
    m = np.zeros(n, np.float32)
    v = np.zeros(n, np.float32)
    ve = np.zeros(n, np.float32)
    for t in range(1, 31):
        g = (rng.normal(0, 1, n) * 10.0 ** rng.uniform(-5, -2, n)).astype(np.float32)
        w64, m64, v64 = adam_fp64(w.astype(np.float64), g.astype(np.float64),
                                  m.astype(np.float64), v.astype(np.float64), t, 1e-3, 0.9, 0.999,
                                  1e-8, bool(bc))
        # scale of the two terms of each moment update (bounds the fp32 error,
        # including the rounding of b1, b2 to float)
        msc = 0.9 * np.abs(m.astype(np.float64)) + 0.1 * np.abs(g.astype(np.float64))
        vsc = 0.999 * v.astype(np.float64) + 1e-3 * g.astype(np.float64) ** 2
        w, m, v, ve = run_fp32(w, g, m, v, ve, lr_mul=0.0, step=t, bias_correction=bc)
        err = np.abs(w64 - w.astype(np.float64))  # compare the new weight
        tol = ulp32(w64) * 0.5 + 1e-5 * 1e-3 * (1 + 3 * (1 - bc))
        assert (err <= tol).all()
        assert (np.abs(m - m64) <= 4 * 2 ** -24 * msc).all()
        assert (np.abs(v - v64) <= 6 * 2 ** -24 * vsc + 1e-45).all()


def test_additive_limit_trajectory_100_steps():
    rng = np.random.default_rng(1)
    n = 2048
    w0 = rng.normal(0, 0.02, n)
    w, m, v, ve = w0.astype(np.float32), None, None, None
    w64, m64, v64 = w0.copy(), np.zeros(n), np.zeros(n)
    for t in range(1, 101):
        g = (rng.normal(0, 1e-3, n)).astype(np.float32)
        w, m, v, ve = run_fp32(w, g, m, v, ve, lr_mul=0.0, step=t)
        w64, m64, v64 = adam_fp64(w64, g.astype(np.float64), m64, v64, t, 1e-3, 0.9, 0.999, 1e-8)
    drift = np.abs(w.astype(np.float64) - w64)
    assert drift.max() <= 1e-5 * np.abs(w64).max()


def test_additive_constant_gradient_closed_form():
    # m^ = g and v^ = g^2 at every step for a constant gradient, so each step
    # moves w by -eta_a g / (|g| + eps).
    g = np.array([3e-4, -2e-2, 1e-6, -5e-3], np.float32)
    w0 = np.array([0.5, -0.25, 1e-3, 2.0], np.float32)
    w, m, v, ve = w0, None, None, None
    for t in range(1, 21):
        w, m, v, ve = run_fp32(w, g, m, v, ve, lr_mul=0.0, step=t)
    g64 = g.astype(np.float64)
    want = w0.astype(np.float64) - 20 * 1e-3 * g64 / (np.abs(g64) + 1e-8)
    assert np.allclose(w, want, rtol=0, atol=40 * ulp32(want).max())


# --------------------------------------------------------------------------
# multiplicative branch
# --------------------------------------------------------------------------

def test_multiplicative_beta2_zero_closed_form():
    # beta2 = 0 makes v_e^ = g_e^2, so r = g_e/(|g_e|+eps) ~ sign(w g) and the
    # relative step is u_m = clip(-eta_m sign(w g) / |w|): |w| moves by eta_m,
    # or by the factor 0.25 / 1.75 once eta_m / |w| exceeds 0.75.
    lr_m = 1e-3
    w0 = np.array([0.02, -0.5, 0.004, -0.003, 1e-4, 0.3], np.float32)
    g = np.array([1e-3, 2e-4, 5e-2, -1e-5, 1e-3, -7e-4], np.float32)
    w, m, v, ve = w0, None, None, None
    w64 = w0.astype(np.float64)
    for t in range(1, 11):
        w, m, v, ve = run_fp32(w, g, m, v, ve, lr_add=0.0, lr_mul=lr_m, beta2=0.0, step=t)
        ge = LN2 * w64 * g
        r = ge / (np.abs(ge) + 1e-8)
        um = np.clip(-lr_m * r / np.maximum(np.abs(w64), 1e-8), -0.75, 0.75)
        w64 = w64 + w64 * um
        assert np.allclose(w, w64, rtol=1e-5, atol=0)
    assert (np.sign(w) == np.sign(w0)).all()


def test_step1_closed_form_bias_corrected():
    # Algorithm 1 at t = 1 from zero state: m^ = g, v^ = g^2, v_e^ = g_e^2.
    rng = np.random.default_rng(2)
    n = 20000
    w = np.concatenate([rng.normal(0, 0.02, n - 4), [0.0, 1e-9, -2e-4, 1.0]]).astype(np.float32)
    g = (rng.normal(0, 1, n) * 10.0 ** rng.uniform(-6, -1, n)).astype(np.float32)
    lr_a, lr_m = 1e-3, 2e-3
    wn, *_ = run_fp32(w, g, lr_add=lr_a, lr_mul=lr_m)
    w64, g64 = w.astype(np.float64), g.astype(np.float64)
    ua = -lr_a * g64 / (np.abs(g64) + 1e-8)
    ge = LN2 * w64 * g64
    um = np.clip(-lr_m * ge / (np.abs(ge) + 1e-8) / np.maximum(np.abs(w64), 1e-8), -0.75, 0.75)
    want = w64 + w64 * um + ua
    # two roundings of the result (fmaf, final add) plus fp32 error of the terms
    tol = ulp32(want) + 1e-6 * (np.abs(ua) + np.abs(w64 * um))
    assert (np.abs(wn - want) <= tol).all()
    # where the clip is inactive, w u_m = -eta_m sign(g) up to eps terms
    big = (np.abs(w64) > lr_m / 0.75 * 1.01) & (np.abs(ge) > 1e-5)
    assert np.allclose((wn - w64 - ua)[big], -lr_m * np.sign(g64[big]), rtol=2e-3)


def test_step1_closed_form_algorithm2_without_bias_correction():
    # Algorithm 2 (no bias correction) at t = 1: m = (1-b1) g, v = (1-b2) g^2,
    # so u_a = -eta_a (1-b1) g / (sqrt(1-b2)|g| + eps) ~ -3.16 eta_a sign(g).
    g = np.array([1e-2, -3e-3, 5e-4], np.float32)
    w = np.array([0.5, 0.5, -0.5], np.float32)
    wn, *_ = run_fp32(w, g, lr_add=1e-3, lr_mul=1e-4, bias_correction=0)
    g64, w64 = g.astype(np.float64), w.astype(np.float64)
    ua = -1e-3 * 0.1 * g64 / (math.sqrt(1e-3) * np.abs(g64) + 1e-8)
    ge = LN2 * w64 * g64
    um = np.clip(-1e-4 * ge / (math.sqrt(1e-3) * np.abs(ge) + 1e-8) / np.abs(w64), -0.75, 0.75)
    want = w64 + w64 * um + ua
    assert np.allclose(wn, want, rtol=2e-6)
    assert np.allclose(ua, -1e-3 * np.sign(g64) * 0.1 / math.sqrt(1e-3), rtol=1e-3)


@pytest.mark.parametrize("wfmt", ["bf16", "e4m3", "e5m2", "fp32"])
@pytest.mark.parametrize("rounding", ["rne", "sr"])
def test_multiplicative_limit_preserves_sign_and_zero(wfmt, rounding):
    rng = np.random.default_rng(3)
    n = 8192
    x = rng.normal(0, 0.02, n).astype(np.float32)
    x[::17] = 0.0
    x[1::17] = -0.0
    codes = oracle.encode_array(wfmt, x)
    w0 = oracle.decode_array(wfmt, codes)
    m, v, ve = (np.zeros(n, np.float32) for _ in range(3))
    for t in range(1, 21):
        g = (rng.normal(0, 1, n) * 10.0 ** rng.uniform(-5, 0, n)).astype(np.float32)
        oracle.step(wfmt, codes, g, m, v, ve, hp(lr_add=0.0, lr_mul=5e-2, rounding=rounding,
                                                 step=t, seed=42))
    w = oracle.decode_array(wfmt, codes)
    assert (w[w0 == 0] == 0).all()
    nz = w != 0
    assert (np.sign(w[nz]) == np.sign(w0[nz])).all()


def test_zero_revival_and_sign_change_need_the_additive_branch():
    n = 256
    g = np.full(n, 2e-3, np.float32)  # pushes every weight down
    for lr_add, expect_move in ((1e-3, True), (0.0, False)):
        x = np.concatenate([np.zeros(n // 2), np.full(n // 2, 0.004)]).astype(np.float32)
        codes = oracle.encode_array("bf16", x)
        m, v, ve = (np.zeros(n, np.float32) for _ in range(3))
        for t in range(1, 41):
            oracle.step("bf16", codes, g, m, v, ve, hp(lr_add=lr_add, lr_mul=1e-3, step=t))
        w = oracle.decode_array("bf16", codes)
        if expect_move:
            assert (w[: n // 2] < 0).all()   # revived from exact zero
            assert (w[n // 2:] < 0).all()    # crossed zero
        else:
            assert (w[: n // 2] == 0).all()
            assert (w[n // 2:] > 0).all()


# --------------------------------------------------------------------------
# descent (Theorem 3.1 setting)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("lr_add,lr_mul", [(1e-4, 1e-4), (1e-4, 0.0), (0.0, 1e-4)])
def test_descent_on_convex_quadratic(lr_add, lr_mul):
    rng = np.random.default_rng(5)
    n = 1000
    a = rng.uniform(0.5, 2.0, n)
    c = rng.normal(0, 0.05, n)
    loss = lambda w: 0.5 * float((a * (w.astype(np.float64) - c) ** 2).sum())  # noqa: E731
    w = rng.normal(0, 0.05, n).astype(np.float32)
    m = v = ve = None
    losses = [loss(w)]
    for t in range(1, 51):
        g = (a * (w.astype(np.float64) - c)).astype(np.float32)
        w, m, v, ve = run_fp32(w, g, m, v, ve, lr_add=lr_add, lr_mul=lr_mul, step=t)
        losses.append(loss(w))
    assert losses[1] < losses[0]
    assert losses[-1] < 0.9 * losses[0]


# --------------------------------------------------------------------------
# clamps of Algorithm 2
# --------------------------------------------------------------------------

def test_g_max_clamps_normalised_direction():
    # bias-corrected step 1: g_e/(sqrt(v_e^)+eps) ~ sign(g_e); g_max = 0.5 halves it
    w = np.array([0.5, -0.5], np.float32)
    g = np.array([1e-2, 1e-2], np.float32)
    wn, *_ = run_fp32(w, g, lr_add=0.0, lr_mul=1e-3, g_max=0.5)
    assert np.allclose(wn - w, [-0.5e-3, -0.5e-3], rtol=1e-4)


def test_u_m_clip_with_eps0():
    # |w| tiny: the relative step saturates at the clip bounds
    w = np.array([1e-5, 1e-5], np.float32)
    g = np.array([1.0, -1.0], np.float32)
    wn, *_ = run_fp32(w, g, lr_add=0.0, lr_mul=1e-2)
    assert np.allclose(wn / w, [0.25, 1.75], rtol=1e-6)
    wn, *_ = run_fp32(w, g, lr_add=0.0, lr_mul=1e-2, eps0=0.25)
    assert np.allclose(wn / w, [0.5, 1.75], rtol=1e-6)


def test_exponent_step_cap():
    # |log2(1+u)| <= d  <=>  u in [2^-d - 1, 2^d - 1]
    d = 0.1
    w = np.array([1e-4, 1e-4, 0.5], np.float32)
    g = np.array([1.0, -1.0, 1e-3], np.float32)
    wn, *_ = run_fp32(w, g, lr_add=0.0, lr_mul=1e-2, d_mult_max=d)
    ratio = wn.astype(np.float64) / w
    assert abs(ratio[0] - 2 ** -d) < 1e-6 and abs(ratio[1] - 2 ** d) < 1e-6
    assert abs(np.log2(ratio[2])) < d  # not capped
    assert abs(wn[2] - (0.5 - 1e-2)) < 1e-6


def test_w_max_clamps_final_weight():
    w = np.array([0.999, -0.999, 0.5], np.float32)
    g = np.array([-1.0, 1.0, -1.0], np.float32)
    wn, *_ = run_fp32(w, g, lr_add=1e-2, lr_mul=1e-2, w_max=1.0)
    assert wn[0] == 1.0 and wn[1] == -1.0 and 0.5 < wn[2] < 1.0


# --------------------------------------------------------------------------
# brute force over every finite FP8 code
# --------------------------------------------------------------------------

def step_fp64(w, g, m, v, ve, t, lr_a=1e-3, lr_m=1e-3, b1=0.9, b2=0.999, eps=1e-8, tau=1e-8):
    """Algorithm 1 with the 0.75 clip, evaluated in float64."""
    m = b1 * m + (1 - b1) * g
    v = b2 * v + (1 - b2) * g * g
    ua = -lr_a * (m / (1 - b1 ** t)) / (np.sqrt(v / (1 - b2 ** t)) + eps)
    ge = LN2 * w * g
    ve = b2 * ve + (1 - b2) * ge * ge
    um = -lr_m * ge / (np.sqrt(ve / (1 - b2 ** t)) + eps) / np.maximum(np.abs(w), tau)
    um = np.clip(um, -0.75, 0.75)
    return w + w * um + ua


@pytest.mark.parametrize("fmt,dtype", [("e4m3", torch.float8_e4m3fn), ("e5m2", torch.float8_e5m2)])
def test_bruteforce_every_fp8_code(fmt, dtype):
    codes_all = np.arange(256, dtype=np.uint8)
    wv = oracle.decode_array(fmt, codes_all)
    codes_all = codes_all[np.isfinite(wv)]
    gs = np.array([-3.0, -0.2, -1e-2, -7e-4, -3e-5, -1e-7, 0.0, 2e-8, 4e-5, 9e-4, 3e-2, 0.7, 5.0],
                  np.float32)
    states = [(0.0, 0.0, 0.0, 1), (1e-3, 2e-6, 5e-9, 4), (-2e-2, 1e-4, 3e-3, 9),
              (5e-4, 3e-8, 1e-12, 2)]
    total = mismatch = 0
    for (m0, v0, ve0, t) in states:
        W, G = np.meshgrid(codes_all, gs, indexing="ij")
        W, G = W.ravel().copy(), G.ravel().copy()
        n = W.size
        m = np.full(n, m0, np.float32)
        v = np.full(n, v0, np.float32)
        ve = np.full(n, ve0, np.float32)
        wf = oracle.decode_array(fmt, W)
        ref64 = step_fp64(wf, G.astype(np.float64), np.float64(np.float32(m0)),
                          np.float64(np.float32(v0)), np.float64(np.float32(ve0)), t)
        oracle.step(fmt, W, G, m, v, ve, hp(step=t))
        want = torch.from_numpy(np.clip(ref64, -448.0 if fmt == "e4m3" else -57344.0,
                                        448.0 if fmt == "e4m3" else 57344.0).astype(np.float32)
                                ).to(dtype).view(torch.uint8).numpy()
        bad = W != want
        # tolerated only next to a rounding boundary of the target grid
        if bad.any():
            lo = oracle.decode_array(fmt, np.minimum(W[bad], want[bad]))
            hi = oracle.decode_array(fmt, np.maximum(W[bad], want[bad]))
            mid = (lo + hi) / 2
            near = np.abs(ref64[bad] - mid) <= 2 ** -20 * np.abs(mid) + 1e-30
            assert near.all(), (ref64[bad][~near][:5], W[bad][~near][:5], want[bad][~near][:5])
        total += n
        mismatch += int(bad.sum())
    assert mismatch <= 0.001 * total


# --------------------------------------------------------------------------
# keying: sharding, subsets, resumption
# --------------------------------------------------------------------------

def _state(n, seed):
    rng = np.random.default_rng(seed)
    x = rng.normal(0, 0.02, n).astype(np.float32)
    return (oracle.encode_array("bf16", x), rng.normal(0, 1e-3, n).astype(np.float32),
            *(np.zeros(n, np.float32) for _ in range(3)))


def test_shard_subset_and_resume_are_bit_identical():
    n, base = 10_000, 123_457
    h = hp(rounding="sr", seed=9)
    w, g, m, v, ve = _state(n, 1)
    ref = [a.copy() for a in (w, m, v, ve)]
    for t in (1, 2, 3):
        oracle.step("bf16", ref[0], g, *ref[1:], dict(h, step=t), index_base=base)
    # shards with their own index bases
    parts = [a.copy() for a in (w, m, v, ve)]
    cut = 3_333
    for t in (1, 2, 3):
        for s0, s1 in ((0, cut), (cut, n)):
            sl = [p[s0:s1] for p in parts]
            sl = [np.ascontiguousarray(x) for x in sl]
            oracle.step("bf16", sl[0], np.ascontiguousarray(g[s0:s1]), *sl[1:], dict(h, step=t),
                        index_base=base + s0)
            for p, x in zip(parts, sl):
                p[s0:s1] = x
    for a, b in zip(ref, parts):
        assert a.tobytes() == b.tobytes()
    # a strided subset with explicit global indices
    idx = np.arange(5, n, 97)
    sub = [np.ascontiguousarray(a[idx]) for a in (w, m, v, ve)]
    for t in (1, 2, 3):
        oracle.step("bf16", sub[0], np.ascontiguousarray(g[idx]), *sub[1:], dict(h, step=t),
                    gidx=idx + base)
    for a, b in zip(ref, sub):
        assert a[idx].tobytes() == b.tobytes()


def test_nan_gradient_gives_canonical_nan_codes():
    for fmt, nan_code in (("bf16", 0x7FC0), ("e4m3", 0x7F), ("e5m2", 0x7F)):
        x = np.array([0.01, -0.01, 0.0], np.float32)
        codes = oracle.encode_array(fmt, x)
        g = np.array([np.nan, np.inf, -np.nan], np.float32)
        z = [np.zeros(3, np.float32) for _ in range(3)]
        oracle.step(fmt, codes, g, *z, hp())
        assert (codes == nan_code).all()
        assert np.isnan(z[0]).sum() >= 2


def test_validation():
    w, g, m, v, ve = _state(8, 2)
    for bad in (dict(beta1=1.0), dict(beta2=-0.1), dict(tau=0.0), dict(r_max=1.0), dict(step=0),
                dict(eps0=0.75), dict(g_max=0.0)):
        with pytest.raises(oracle.OracleError):
            oracle.step("bf16", w, g, m, v, ve, hp(**bad))


# --------------------------------------------------------------------------
# moments stored in bf16
# --------------------------------------------------------------------------

@pytest.mark.parametrize("wfmt", ["bf16", "e4m3"])
def test_bf16_moments_are_fp32_step_then_nearest_rounding(wfmt):
    # With bf16 moments a step is the fp32-moment step on the decoded moments,
    # the new moments then rounded to bf16 by the library conversion.
    rng = np.random.default_rng(8)
    n = 5000
    codes = oracle.encode_array(wfmt, rng.normal(0, 0.02, n).astype(np.float32))
    to_bf16 = lambda x: torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(  # noqa: E731
        torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    ms = [to_bf16(rng.normal(0, s, n)) for s in (1e-3, 1e-6, 1e-6)]
    ms[1] = to_bf16(np.abs(oracle.decode_array("bf16", ms[1])))
    ms[2] = to_bf16(np.abs(oracle.decode_array("bf16", ms[2])))
    for t in range(1, 4):
        g = (rng.normal(0, 1, n) * 10.0 ** rng.uniform(-5, -2, n)).astype(np.float32)
        h = hp(step=t, rounding="sr", seed=3)
        w32, c32 = codes.copy(), codes.copy()
        f32 = [oracle.decode_array("bf16", a).astype(np.float32) for a in ms]
        oracle.step(wfmt, c32, g, *f32, h)
        oracle.step(wfmt, codes, g, *ms, h, sfmt="bf16")
        assert (codes == c32).all()
        for a, b in zip(ms, f32):
            assert (a == to_bf16(b)).all()
        del w32


def _bf16_sr_bits(x: np.ndarray, r16: np.ndarray) -> np.ndarray:
    """bf16 stochastic rounding at the bit level: add the 16-bit draw to the
    16 bits that are cut off, then truncate (finite inputs)."""
    u = np.ascontiguousarray(x, np.float32).view(np.uint32).astype(np.uint64)
    return ((u + r16.astype(np.uint64)) >> 16).astype(np.uint16)


def test_bf16_sr_moments_use_streams_1_2_3_and_the_bit_level_rule():
    # Weights as with fp32 moments; each new moment is the fp32 moment rounded
    # stochastically with the draw of stream 1 (m), 2 (v), 3 (v_e) at the
    # element's global index.
    rng = np.random.default_rng(9)
    n, base, seed = 4000, 777, 12345
    codes = oracle.encode_array("bf16", rng.normal(0, 0.02, n).astype(np.float32))
    ms = [np.zeros(n, np.uint16) for _ in range(3)]
    for t in range(1, 4):
        g = (rng.normal(0, 1, n) * 10.0 ** rng.uniform(-5, -2, n)).astype(np.float32)
        h = hp(step=t, rounding="sr", seed=seed)
        c32 = codes.copy()
        f32 = [oracle.decode_array("bf16", a).astype(np.float32) for a in ms]
        oracle.step("bf16", c32, g, *f32, h, index_base=base)
        oracle.step("bf16", codes, g, *ms, h, sfmt="bf16_sr", index_base=base)
        assert (codes == c32).all()
        for k, (a, b) in enumerate(zip(ms, f32)):
            r16 = np.array([oracle.draw16(seed, t, 1 + k, base + i) for i in range(n)], np.uint32)
            assert (a == _bf16_sr_bits(b, r16)).all(), (t, k)


def test_bf16_sr_moments_are_unbiased_and_independent_across_streams():
    rng = np.random.default_rng(10)
    n = 60000
    codes = oracle.encode_array("bf16", rng.normal(0, 0.02, n).astype(np.float32))
    g = (rng.normal(0, 1, n) * 1e-3).astype(np.float32)
    ms = [np.zeros(n, np.uint16) for _ in range(3)]
    f32 = [np.zeros(n, np.float32) for _ in range(3)]
    oracle.step("bf16", codes.copy(), g, *f32, hp(rounding="sr", seed=4))
    oracle.step("bf16", codes, g, *ms, hp(rounding="sr", seed=4), sfmt="bf16_sr")
    ups = []
    for a, b in zip(ms, f32):
        lo = b.view(np.uint32) >> 16                        # truncation (finite, >= 0 here)
        frac = (b.view(np.uint32) & 0xFFFF) / 65536.0       # position between the neighbours
        up = a.astype(np.uint32) == lo + 1
        assert ((a == lo) | up).all()
        inexact = frac > 0
        # E[up] = frac: the mean of (up - frac) is within 5 sigma of 0
        d = up[inexact] - frac[inexact]
        sd = np.sqrt(np.sum(frac[inexact] * (1 - frac[inexact]))) / inexact.sum()
        assert abs(d.mean()) < 5 * sd
        ups.append(up)
    # the three streams make different decisions
    assert (ups[0] != ups[1]).mean() > 0.2 and (ups[1] != ups[2]).mean() > 0.2


@pytest.mark.parametrize("wfmt", ["bf16", "e4m3", "e5m2"])
@pytest.mark.parametrize("rounding", ["rne", "sr"])
def test_zero_learning_rates_keep_every_finite_weight(wfmt, rounding):
    # eta_a = eta_m = 0: both updates are zero, w' = w exactly (a stored
    # value is on the grid, so either rounding returns it); the moments still
    # follow the gradients.
    rng = np.random.default_rng(11)
    n = 4000
    x = rng.normal(0, 0.5, n).astype(np.float32)
    x[:5] = [0.0, -0.0, 1e-30, -3.0, 2.0 ** -20]
    codes = oracle.encode_array(wfmt, x)
    before = oracle.decode_array(wfmt, codes)
    m, v, ve = (np.zeros(n, np.float32) for _ in range(3))
    g = rng.normal(0, 1e-2, n).astype(np.float32)
    oracle.step(wfmt, codes, g, m, v, ve, hp(lr_add=0.0, lr_mul=0.0, rounding=rounding, seed=3))
    assert (oracle.decode_array(wfmt, codes) == before).all()
    assert np.allclose(m, np.float32(0.1) * g, rtol=1e-6) and (v > 0).mean() > 0.99


# --------------------------------------------------------------------------
# Appendix B's moment-free rules
# --------------------------------------------------------------------------

def test_plain_additive_rule_is_sgd_then_bf16_rounding():
    rng = np.random.default_rng(20)
    n = 8192
    codes = oracle.encode_array("bf16", rng.normal(0, 0.5, n).astype(np.float32))
    g = (rng.normal(0, 1, n) * 10.0 ** rng.uniform(-4, 1, n)).astype(np.float32)
    w = oracle.decode_array("bf16", codes).astype(np.float32)
    oracle.plain_step("bf16", codes, g, hp(lr_add=0.01, lr_mul=0.0))
    want = w + (-(np.float32(0.01) * g))  # fp32, as the rule is written
    ref = torch.from_numpy(want.astype(np.float32)).to(torch.bfloat16).view(torch.int16)
    assert (codes == ref.numpy().view(np.uint16)).all()


def test_plain_multiplicative_rule_closed_form():
    # u_m = clip(-eta_m ln2 w g / |w|) = clip(-eta_m ln2 g sign(w)) for |w| > tau
    rng = np.random.default_rng(21)
    n = 4096
    w = rng.normal(0, 1, n).astype(np.float32)
    w[:5] = [0.0, 1e-9, -2.0, 50.0, -1e-3]
    g = rng.normal(0, 2, n).astype(np.float32)
    codes = w.view(np.uint32).copy()
    oracle.plain_step("fp32", codes, g, hp(lr_add=0.0, lr_mul=0.3))
    wn = codes.view(np.float32).astype(np.float64)
    w64, g64 = w.astype(np.float64), g.astype(np.float64)
    um = np.clip(-0.3 * LN2 * w64 * g64 / np.maximum(np.abs(w64), 1e-8), -0.75, 0.75)
    want = w64 * (1 + um)
    assert np.allclose(wn, want, rtol=4e-7, atol=0)
    assert wn[0] == 0.0 and (np.sign(wn) == np.sign(w64)).all()


def test_plain_rules_on_appendix_b_regimes():
    # Section 3.1 / Appendix B: the multiplicative rule cannot change a sign
    # or leave exact zero; the additive rule can; at large magnitudes an
    # additive step below half the BF16 spacing is rounded away while the
    # multiplicative step, relative to |w|, is not.
    from paper_2607_10611_amd import diagnostic as D
    from paper_2607_10611_amd import workloads as W

    def run(regime, rule, lr, steps=60):
        ws, w0, c = W.toy_regime(regime)
        codes = oracle.encode_array("bf16", w0)
        rng = np.random.default_rng(0)
        for t in range(1, steps + 1):
            w = oracle.decode_array("bf16", codes).astype(np.float32)
            idx = rng.integers(0, W.TOY_N, W.TOY_N)
            g = oracle.toy_gradient(w, ws, c, idx, W.TOY_N)
            oracle.plain_step("bf16", codes, g, D.rule_hparams(rule, lr, t))
        return oracle.decode_array("bf16", codes), ws, w0

    w, ws, w0 = run("sign_flip", "multiplicative", 10.0)
    assert (np.sign(w) == np.sign(w0)).all()
    w, ws, w0 = run("sign_flip", "combined", 10.0)
    assert np.mean(np.sign(w) == np.sign(ws)) > 0.99
    w, ws, w0 = run("zero_revival", "multiplicative", 10.0)
    assert (w == 0).all()
    w, ws, w0 = run("zero_revival", "additive", 10.0)
    assert (w != 0).all()
    w, ws, w0 = run("large", "additive", 1.0)
    wm, _, _ = run("large", "multiplicative", 1.0)
    assert np.mean(w == w0) > 0.5 > np.mean(wm == w0)
