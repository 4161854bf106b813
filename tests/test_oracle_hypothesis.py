"""The oracle against the update rule over the hyper-parameter space (CPU,
property-based).

The fixed-value pins run at the defaults, where eps and tau are both 1e-8;
here hypothesis draws the learning rates, betas, eps, tau, the clip, the
step and the moment state, so that a mistake that coincides at the defaults
(eps for tau, one beta for the other) fails.  Each example is one step in
the FP32 passthrough format, compared with the rule evaluated in float64 on
the same fp32 inputs: the additive limit (eta_m = 0) is Adam (Algorithm 1),
the multiplicative limit (eta_a = 0) is w (1 + u_m) with
u_m = clip(-eta_m r / max(|w|, tau)), r = g_e / (sqrt(v_e^) + eps),
g_e = ln2 w g (Section 3.1).  The bounds allow the fp32 roundings of the
canonical sequence: a few units of 2^-24 on each operation's inputs."""
import math

import numpy as np
from hypothesis import given, settings
from hypothesis import strategies as st

import oracle
from paper_2607_10611_amd.workloads import DEFAULT_HPARAMS

N = 64
U = 2.0 ** -24
LN2 = math.log(2.0)

hparams = st.fixed_dictionaries(dict(
    lr=st.floats(1e-6, 1e-1), b1=st.floats(0.0, 0.99), b2=st.floats(0.5, 0.9999),
    eps=st.floats(1e-12, 1e-3), tau=st.floats(1e-10, 1e-2), t=st.integers(1, 2000),
    bc=st.sampled_from([0, 1]), seed=st.integers(0, 2 ** 32 - 1)))


def inputs(seed):
    rng = np.random.default_rng(seed)
    w = (rng.normal(0, 0.05, N) * 10.0 ** rng.uniform(-3, 0, N)).astype(np.float32)
    g = (rng.normal(0, 1, N) * 10.0 ** rng.uniform(-6, -1, N)).astype(np.float32)
    m = (rng.normal(0, 1, N) * 10.0 ** rng.uniform(-6, -2, N)).astype(np.float32)
    v = (10.0 ** rng.uniform(-14, -3, N)).astype(np.float32)
    ve = (10.0 ** rng.uniform(-16, -5, N)).astype(np.float32)
    return w, g, m, v, ve


def step(w, g, m, v, ve, **kw):
    h = dict(DEFAULT_HPARAMS, rounding="rne")
    h.update(kw)
    w, m, v, ve = (a.copy() for a in (w, m, v, ve))
    codes = w.view(np.uint32)
    oracle.step("fp32", codes, g.copy(), m, v, ve, h)
    return codes.view(np.float32), m, v, ve


@settings(max_examples=150, deadline=None)
@given(hparams)
def test_additive_limit_is_adam(p):
    w, g, m, v, ve = inputs(p["seed"])
    wn, mn, vn, _ = step(w, g, m, v, ve, lr_add=p["lr"], lr_mul=0.0, beta1=p["b1"],
                         beta2=p["b2"], eps=p["eps"], tau=p["tau"], step=p["t"],
                         bias_correction=p["bc"])
    W, G, M, V = (a.astype(np.float64) for a in (w, g, m, v))
    b1, b2, t = p["b1"], p["b2"], p["t"]
    m64 = b1 * M + (1 - b1) * G
    v64 = b2 * V + (1 - b2) * G * G
    mh = m64 / (1 - b1 ** t) if p["bc"] else m64
    vh = v64 / (1 - b2 ** t) if p["bc"] else v64
    den = np.sqrt(vh) + p["eps"]
    u64 = -p["lr"] * mh / den
    # error bound: each moment to a few ulp of its two terms, then the
    # quotient and the final rounding of w + u
    msc = b1 * np.abs(M) + (1 - b1) * np.abs(G)
    vsc = b2 * V + (1 - b2) * G * G
    assert (np.abs(mn - m64) <= 4 * U * msc).all()
    assert (np.abs(vn - v64) <= 6 * U * vsc + 1e-45).all()
    sa = p["lr"] / (1 - b1 ** t) if p["bc"] else p["lr"]
    du = sa * (8 * U * msc / den + np.abs(mh) * 8 * U * np.sqrt(vh) / den ** 2)
    err = np.abs(wn.astype(np.float64) - (W + u64))
    tol = 0.5 * np.spacing(np.abs(W + u64).astype(np.float32)) + 16 * U * np.abs(u64) + du
    assert (err <= tol).all(), (err / tol).max()


@settings(max_examples=150, deadline=None)
@given(hparams, st.floats(0.05, 0.9), st.floats(0.0, 0.04))
def test_multiplicative_limit_is_the_relative_exponent_step(p, r_max, eps0):
    w, g, m, v, ve = inputs(p["seed"])
    wn, _, _, ven = step(w, g, m, v, ve, lr_add=0.0, lr_mul=p["lr"], beta1=p["b1"],
                         beta2=p["b2"], eps=p["eps"], tau=p["tau"], step=p["t"],
                         bias_correction=p["bc"], r_max=r_max, eps0=eps0)
    W, G, VE = (a.astype(np.float64) for a in (w, g, ve))
    b2, t = p["b2"], p["t"]
    ge = LN2 * W * G
    ve64 = b2 * VE + (1 - b2) * ge * ge
    veh = ve64 / (1 - b2 ** t) if p["bc"] else ve64
    r = ge / (np.sqrt(veh) + p["eps"])
    ut = -p["lr"] * r
    um = np.clip(ut / np.maximum(np.abs(W), p["tau"]), -(r_max - eps0), r_max)
    w64 = W * (1 + um)
    assert (np.abs(ven - ve64) <= 8 * U * (b2 * VE + (1 - b2) * ge * ge) + 1e-45).all()
    # u_m to ~16 ulp of its own size (the clip bounds are exact), then w u_m + w
    clipped = np.abs(ut / np.maximum(np.abs(W), p["tau"])) >= np.where(um < 0, r_max - eps0,
                                                                        r_max)
    dum = np.where(clipped, 2 * U * np.abs(um), 16 * U * np.abs(um))
    err = np.abs(wn.astype(np.float64) - w64)
    tol = 0.5 * np.spacing(np.abs(w64).astype(np.float32)) + np.abs(W) * dum + 4 * U * np.abs(W * um)
    assert (err <= tol).all(), (err / tol).max()
    # the sign never changes (1 + u_m > 0) and zero stays zero
    assert (np.sign(wn) == np.sign(w)).all()
