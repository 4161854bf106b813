"""Parity of the HIP step with the CPU oracle over the whole fp32 range of the
step's operands (GPU, through the C ABI).

Algorithm 1 divides the first moments by sqrt of the bias-corrected second
moments plus eps, divides the multiplicative step by rho = max(|w|, tau) and
squares the gradients; trajectories that start from zero moments with small
gradients only reach a narrow band of those operands.  Here the weights, the
three moments and the gradients are drawn with their exponent field uniform
over every finite binade (subnormals included) plus fixed special values
(signed zeros, the smallest and largest subnormals, the smallest normal,
the largest finite values), so that the square roots see subnormal, zero and
near-overflow inputs, g*g and (ln2 w g)^2 overflow and underflow, the
divisions see zero, subnormal and infinite divisors (eps = 0 included), and
the results cover Inf and NaN.  Bar: weight codes bit-exact, fp32 moments
within 2 ulp with the same NaN pattern, bf16 moment codes bit-exact.
"""
import zlib

import numpy as np
import pytest
import torch

from paper_2607_10611_amd import binding as B
from paper_2607_10611_amd import workloads as W
from gpu_parity_util import (DevState, HostState, assert_state_equal, gpu_step, oracle_step,
                             to_dev)

pytestmark = pytest.mark.gpu

# special fp32 bit patterns placed at the start of every array
SPECIAL_F32 = np.array([
    0x00000000, 0x80000000,            # +0, -0
    0x00000001, 0x80000001,            # smallest subnormal
    0x00000002, 0x00400000,            # small and mid subnormals
    0x007FFFFF, 0x807FFFFF,            # largest subnormal
    0x00800000, 0x80800000,            # smallest normal
    0x7F7FFFFF, 0xFF7FFFFF,            # largest finite
    0x7F7FFFFE, 0x7F000000,            # near overflow
    0x7E967699, 0xFE967699,            # 1e38
    0x00E2E6C3, 0x0A4FB11F,            # 2.08e-38, ~1e-32
    0x3F800000, 0xBF800000,            # +-1
    0x322BCC77, 0x1E3CE508,            # 1e-8, ~1e-20
], dtype=np.uint32)


def full_range_f32(rng, n, nonneg=False):
    """fp32 values with the exponent field uniform over 0..254 (every finite
    binade, subnormals included), random mantissas and signs; the special
    values first."""
    e = rng.integers(0, 255, n).astype(np.uint32)
    mant = rng.integers(0, 1 << 23, n).astype(np.uint32)
    sign = np.zeros(n, np.uint32) if nonneg else rng.integers(0, 2, n).astype(np.uint32)
    bits = (sign << 31) | (e << 23) | mant
    k = min(n, SPECIAL_F32.size)
    bits[:k] = SPECIAL_F32[:k]
    if nonneg:
        bits &= np.uint32(0x7FFFFFFF)
    return bits.view(np.float32)


def full_range_bf16(rng, n, nonneg=False):
    """bf16 codes of full_range_f32 values, truncated (every finite binade)."""
    return (full_range_f32(rng, n, nonneg).view(np.uint32) >> 16).astype(np.uint16)


def hp(**kw):
    h = dict(W.DEFAULT_HPARAMS)
    h.update(kw)
    return h


def start_state(rng, wfmt, sfmt, n, state):
    """Weight codes and the three moments; `state` is "full" (moments over
    the whole range, v and v_e non-negative as every reachable state is),
    "zero" (zero moments) or "zero_v" (m over the whole range, v = v_e = 0:
    with eps = 0 the additive division is m / 0)."""
    if wfmt == "fp32":
        codes = full_range_f32(rng, n).view(np.uint32).copy()
    else:
        codes = full_range_bf16(rng, n)
    if sfmt == "fp32":
        full = lambda nn: full_range_f32(rng, n, nonneg=nn)  # noqa: E731
        zero = lambda: np.zeros(n, np.float32)  # noqa: E731
    else:
        full = lambda nn: full_range_bf16(rng, n, nonneg=nn)  # noqa: E731
        zero = lambda: np.zeros(n, np.uint16)  # noqa: E731
    if state == "full":
        mom = (full(False), full(True), full(True))
    elif state == "zero_v":
        mom = (full(False), zero(), zero())
    else:
        mom = (zero(), zero(), zero())
    return codes, mom


def run(wfmt, sfmt, state, grads, h_list, n=4 * 2048 + 1000 + 5, index_base=0, seed=0):
    rng = np.random.default_rng(seed)
    codes, mom = start_state(rng, wfmt, sfmt, n, state)
    ds = DevState(wfmt, codes, n, sfmt=sfmt)
    hs = HostState(codes, n, sfmt=sfmt)
    for t_dev, t_host, a in zip((ds.m, ds.v, ds.ve), ("m", "v", "ve"), mom):
        t_dev.copy_(to_dev(a))
        setattr(hs, t_host, a.copy())
    for k, h in enumerate(h_list):
        if grads == "full":
            g = full_range_f32(rng, n)
        else:
            g = (rng.normal(0, 1, n) * 10.0 ** rng.uniform(-6, -1, n)).astype(np.float32)
        gpu_step(ds, to_dev(g), h, index_base=index_base)
        oracle_step(wfmt, hs, g.copy(), h, index_base=index_base)
        torch.cuda.synchronize()
        w_g, m_g, v_g, ve_g = ds.host()
        assert_state_equal(f"{wfmt}/{sfmt} {state} state, {grads} grads, step {k + 1} {h}",
                           w_g, hs.w, m_g, hs.m, v_g, hs.v, ve_g, hs.ve)


HPARAM_SETS = {
    "default": [hp(step=t) for t in (1, 2, 3)],
    "eps0": [hp(step=t, eps=0.0) for t in (1, 2, 3)],
    "eps0_no_bias_correction": [hp(step=t, eps=0.0, bias_correction=0) for t in (1, 2)],
    "late_step_sr": [hp(step=t, rounding="sr", seed=77) for t in (1000, 1001)],
    "large_rates_clamps": [hp(step=t, lr_add=10.0, lr_mul=0.5, g_max=4.0, w_max=1e30,
                              rounding="sr", seed=5) for t in (1, 2)],
}


@pytest.mark.parametrize("wfmt", ["fp32", "bf16"])
@pytest.mark.parametrize("hset", list(HPARAM_SETS))
@pytest.mark.parametrize("state,grads", [("full", "normal"), ("zero", "full"),
                                         ("full", "full"), ("zero_v", "normal")])
def test_full_range_fp32_moments(wfmt, hset, state, grads):
    seed = zlib.crc32(f"{wfmt} {hset} {state}".encode())
    run(wfmt, "fp32", state, grads, HPARAM_SETS[hset], seed=seed)


@pytest.mark.parametrize("wfmt", ["fp32", "bf16"])
@pytest.mark.parametrize("sfmt", ["bf16", "bf16_sr"])
@pytest.mark.parametrize("state,grads", [("full", "normal"), ("full", "full")])
def test_full_range_bf16_moments(wfmt, sfmt, state, grads):
    run(wfmt, sfmt, state, grads, HPARAM_SETS["default"] + HPARAM_SETS["eps0"][:1], seed=31)


def test_full_range_unaligned_index_base_per_element_path():
    """The per-element path (index base not a multiple of 8)."""
    run("bf16", "fp32", "full", "full", HPARAM_SETS["eps0"], index_base=5, seed=32)
    run("fp32", "fp32", "zero_v", "normal", HPARAM_SETS["late_step_sr"], index_base=3, seed=33)


def test_multi_tensor_list_full_range():
    """One multi-tensor call over full-range tensors of both formats."""
    rng = np.random.default_rng(34)
    layout = [("fp32", 4096 + 24), ("bf16", 2048 + 7), ("fp32", 64), ("bf16", 3 * 2048)]
    devs, hosts = [], []
    for wfmt, n in layout:
        codes, mom = start_state(rng, wfmt, "fp32", n, "full")
        ds, hs = DevState(wfmt, codes, n), HostState(codes, n)
        for t_dev, name, a in zip((ds.m, ds.v, ds.ve), ("m", "v", "ve"), mom):
            t_dev.copy_(to_dev(a))
            setattr(hs, name, a.copy())
        devs.append(ds)
        hosts.append(hs)
    for t in (1, 2):
        gs = [full_range_f32(rng, n) for _, n in layout]
        h = hp(step=t, eps=0.0, rounding="sr", seed=8)
        tl = B.TensorList([d.w for d in devs], [w for w, _ in layout], [to_dev(g) for g in gs],
                          [d.m for d in devs], [d.v for d in devs], [d.ve for d in devs])
        B.madd_multi_tensor_step(tl, h, index_base=64)
        off = 64
        for (wfmt, n), hs, g in zip(layout, hosts, gs):
            oracle_step(wfmt, hs, g.copy(), h, index_base=off)
            off += n
        torch.cuda.synchronize()
        for (wfmt, n), ds, hs in zip(layout, devs, hosts):
            w_g, m_g, v_g, ve_g = ds.host()
            assert_state_equal(f"list {wfmt} n={n} t={t}", w_g, hs.w, m_g, hs.m, v_g, hs.v,
                               ve_g, hs.ve)
