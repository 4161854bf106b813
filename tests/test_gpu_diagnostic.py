"""Appendix B's diagnostic on the GPU: the moment-free rules
(madd_plain_step) and the gradient of the sampled quartic loss
(madd_toy_gradient) against the oracle, bit-exact trajectories of the
diagnostic regimes computed entirely on the GPU, and the qualitative
outcomes of the paper's diagnostic figure."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_10611_amd import binding as B
from paper_2607_10611_amd import diagnostic as D
from paper_2607_10611_amd import workloads as W
from gpu_parity_util import CODE_NP, to_dev, to_host

pytestmark = pytest.mark.gpu


def hp(**kw):
    h = dict(W.DEFAULT_HPARAMS)
    h.update(kw)
    return h


@pytest.mark.parametrize("wfmt", ["bf16", "e4m3", "e5m2", "fp32"])
@pytest.mark.parametrize("rounding", ["rne", "sr"])
@pytest.mark.parametrize("n", [1, 1023, 4096 + 5])
def test_plain_step_parity(wfmt, rounding, n):
    rng = np.random.default_rng(n)
    x = rng.normal(0, 0.5, n).astype(np.float32)
    x[::11] = 0.0
    if wfmt in ("e4m3", "e5m2"):
        x = np.clip(x, -448, 448)
    codes = oracle.encode_array(wfmt, x)
    wd = to_dev(codes)
    for t, (la, lm) in enumerate([(0.01, 0.0), (0.0, 0.05), (0.02, 0.03)], start=1):
        g = (rng.normal(0, 1, n) * 10.0 ** rng.uniform(-5, 1, n)).astype(np.float32)
        h = hp(lr_add=la, lr_mul=lm, rounding=rounding, step=t, seed=11)
        B.madd_plain_step(wd, wfmt, to_dev(g), h, index_base=77)
        oracle.plain_step(wfmt, codes, g, h, index_base=77)
        torch.cuda.synchronize()
        got = to_host(wd, CODE_NP[wfmt])
        assert (got == codes).all(), (wfmt, rounding, n, t, np.nonzero(got != codes)[0][:5])


def test_plain_step_bf16_gradients():
    rng = np.random.default_rng(5)
    n = 3000
    codes = oracle.encode_array("bf16", rng.normal(0, 1, n).astype(np.float32))
    g = oracle.encode_array("bf16", rng.normal(0, 1e-2, n).astype(np.float32))
    wd = to_dev(codes)
    h = hp(lr_add=0.1, lr_mul=0.1, rounding="sr")
    B.madd_plain_step(wd, "bf16", to_dev(g), h, gfmt="bf16")
    oracle.plain_step("bf16", codes, g, h, gfmt="bf16")
    torch.cuda.synchronize()
    assert (to_host(wd, np.uint16) == codes).all()


@pytest.mark.parametrize("wfmt", ["bf16", "e4m3", "e5m2", "fp32"])
def test_toy_gradient_kernel_matches_the_oracle(wfmt):
    """madd_toy_gradient against oracle.toy_gradient bit for bit: entries
    drawn several times, never drawn, out of range, zero differences."""
    rng = np.random.default_rng(7)
    n, batch = 5000, 7000
    x = rng.normal(0, 2, n).astype(np.float32)
    if wfmt in ("e4m3", "e5m2"):
        x = np.clip(x, -448, 448)
    codes = oracle.encode_array(wfmt, x)
    w = oracle.decode_array(wfmt, codes).astype(np.float32)
    target = rng.normal(0, 2, n).astype(np.float32)
    target[::13] = w[::13]
    c = (10.0 ** rng.uniform(-7, 8, n)).astype(np.float32)
    idx = rng.integers(0, n, batch)
    idx[:5] = [n, -1, n + 7, 3, 3]
    counts = torch.full((n,), 77, dtype=torch.int32, device="cuda")
    g = torch.full((n,), 1.0, device="cuda")
    B.madd_toy_gradient(to_dev(codes), wfmt, to_dev(target), to_dev(c),
                        torch.from_numpy(idx).cuda(), counts, g)
    want = oracle.toy_gradient(w, target, c, idx, batch)
    torch.cuda.synchronize()
    got = to_host(g)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
    ok = (idx >= 0) & (idx < n)
    assert np.array_equal(to_host(counts), np.bincount(idx[ok], minlength=n))


@pytest.mark.parametrize("regime", W.TOY_REGIMES)
def test_diagnostic_trajectory_bit_exact(regime):
    """Combined rule, 100 steps, everything on the GPU (madd_toy_gradient,
    then madd_plain_step) against the oracle (toy_gradient, plain_step) on the
    same sampled entries."""
    ws, w0, c = W.toy_regime(regime)
    codes = oracle.encode_array("bf16", w0)
    wd = to_dev(codes)
    td, cd = to_dev(ws), to_dev(c)
    g = torch.empty(W.TOY_N, device="cuda")
    counts = torch.empty(W.TOY_N, dtype=torch.int32, device="cuda")
    rng = np.random.default_rng(1)
    for t in range(1, 101):
        idx = rng.integers(0, W.TOY_N, W.TOY_N)
        h = D.rule_hparams("combined", 10.0, t)
        B.madd_toy_gradient(wd, "bf16", td, cd, torch.from_numpy(idx).cuda(), counts, g)
        B.madd_plain_step(wd, "bf16", g, h)
        w = oracle.decode_array("bf16", codes).astype(np.float32)
        oracle.plain_step("bf16", codes, oracle.toy_gradient(w, ws, c, idx, W.TOY_N), h)
    torch.cuda.synchronize()
    assert (to_host(wd, np.uint16) == codes).all()


def test_diagnostic_figure_outcomes():
    """One shared learning rate (10) for every rule and regime, 200 steps."""
    res = D.figure3(lr=10.0, steps=200)
    rel = {k: v["rel_err"] for k, v in res.items()}
    # multiplicative-only: structural failures at sign changes and exact zero
    assert res[("sign_flip", "multiplicative")]["sign_agree"] == 0.0
    assert res[("zero_revival", "multiplicative")]["unchanged"] == 1.0
    assert res[("small", "multiplicative")]["unchanged"] == 1.0
    # additive-only: sign changes and revival work, large magnitudes stall
    assert res[("sign_flip", "additive")]["sign_agree"] > 0.99
    assert res[("zero_revival", "additive")]["unchanged"] == 0.0
    assert rel[("large", "additive")] > 2 * rel[("large", "multiplicative")]
    # combined: never worse than the better branch by more than 5%, every regime
    for r in W.TOY_REGIMES:
        best = min(rel[(r, "additive")], rel[(r, "multiplicative")])
        assert rel[(r, "combined")] <= 1.05 * best, (r, rel[(r, "combined")], best)
    # mixed scales: only the combined rule serves both halves -- it revives the
    # small half (the multiplicative rule leaves it at zero) and fits the large
    # half far better than the additive rule, whose steps there are rounded away
    h = W.TOY_N // 2

    def half_err(rule, sl):
        m = res[("mixed", rule)]
        return np.linalg.norm(m["w"][sl] - m["target"][sl]) / np.linalg.norm(m["target"][sl])

    assert np.all(res[("mixed", "combined")]["w"][:h] != 0)
    assert np.all(res[("mixed", "multiplicative")]["w"][:h] == 0)
    assert half_err("combined", slice(h, None)) < 0.5 * half_err("additive", slice(h, None))
