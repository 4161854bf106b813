"""Seeded random configurations of the whole step (CPU oracle vs HIP, through
the C ABI): every weight format (unscaled, block-scaled FP8, MXFP4, NVFP4
with the tensor scale kept or derived anew), moment storage, gradient
format, rounding, compute copy, index base and size drawn at random, with
hyper-parameters spanning several orders of magnitude and the optional
clamps switched on at random.  Same bar as the other parity tests: codes,
scales and copies bit-exact, fp32 moments within 2 ulp.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_10611_amd import binding as B
from paper_2607_10611_amd import workloads as W
from gpu_parity_util import (DevState, HostState, assert_copy_equal, assert_state_equal,
                             encode_nv_current, gpu_step, oracle_step, to_dev, to_host)

pytestmark = pytest.mark.gpu

FORMATS = [("bf16", None), ("e4m3", None), ("e5m2", None), ("fp32", None), ("e4m3", "block"),
           ("e5m2", "block"), ("mxfp4", "mx"), ("nvfp4", "nv"), ("nvfp4_current", "nvcs")]
BLOCK = {None: 8, "block": 128, "mx": 32, "nv": 16, "nvcs": 16}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    B.lib()
    yield
    torch.cuda.synchronize()


def random_case(rng):
    wfmt, kind = FORMATS[rng.integers(len(FORMATS))]
    blk = BLOCK[kind]
    n = int(rng.integers(1, 40)) * blk * int(rng.choice([1, 4, 37])) + (
        int(rng.integers(0, 8)) if kind is None else 0)
    h = dict(W.DEFAULT_HPARAMS)
    h.update(lr_add=float(10.0 ** rng.uniform(-5, -0.5)), lr_mul=float(10.0 ** rng.uniform(-5, -0.5)),
             beta1=float(rng.choice([0.0, 0.5, 0.9, 0.99])), beta2=float(rng.choice([0.0, 0.9, 0.999, 0.99999])),
             eps=float(rng.choice([0.0, 1e-12, 1e-8, 1e-4])), tau=float(rng.choice([1e-12, 1e-8, 1e-3])),
             r_max=float(rng.uniform(0.1, 0.95)), bias_correction=int(rng.integers(2)),
             rounding=str(rng.choice(["rne", "sr"])), seed=int(rng.integers(2**63)))
    h["eps0"] = float(rng.uniform(0, h["r_max"] * 0.9)) if rng.random() < 0.3 else 0.0
    if rng.random() < 0.3:
        h["g_max"] = float(10.0 ** rng.uniform(-1, 1))
    if rng.random() < 0.3:
        h["d_mult_max"] = float(rng.uniform(0.01, 2))
    if rng.random() < 0.3:
        h["w_max"] = float(10.0 ** rng.uniform(-2, 1))
    gfmt = "fp32" if kind == "nvcs" else str(rng.choice(["fp32", "bf16"]))
    sfmt = str(rng.choice(["fp32", "bf16", "bf16_sr"]))
    copy = kind is not None and rng.random() < 0.7
    base = int(rng.integers(0, 2**40)) if rng.random() < 0.5 else 0
    scale = float(10.0 ** rng.uniform(-4, 1))
    return wfmt, kind, n, h, gfmt, sfmt, copy, base, scale


def encode(wfmt, kind, x):
    if kind is None:
        return oracle.encode_array(wfmt, x), None
    if kind == "block":
        return oracle.encode_block(wfmt, x)
    if kind == "mx":
        return oracle.encode_mx(x)
    if kind == "nv":
        return oracle.encode_nv(x)
    return encode_nv_current(x)


@pytest.mark.parametrize("case", range(160))
def test_random_configuration(case):
    rng = np.random.default_rng(10_000 + case)
    wfmt, kind, n, h, gfmt, sfmt, copy, base, scale = random_case(rng)
    x = (rng.normal(0, 1, n) * scale).astype(np.float32)
    x[rng.random(n) < 0.03] = 0.0
    if wfmt in ("e4m3", "e5m2") and kind is None:
        lim = 448.0 if wfmt == "e4m3" else 57344.0
        x = np.clip(x, -lim, lim)
    codes, scales = encode(wfmt, kind, x)
    ds = DevState(wfmt, codes, n, scales, sfmt=sfmt, copy=copy)
    hs = HostState(codes, n, scales, sfmt=sfmt, copy=copy)
    tag = (f"case {case}: {wfmt}/{kind} n={n} gfmt={gfmt} sfmt={sfmt} copy={copy} base={base} "
           f"hp={h}")
    for t in range(1, int(rng.integers(1, 4)) + 1):
        g = (rng.normal(0, 1, n) * 10.0 ** rng.uniform(-6, 0, n)).astype(np.float32)
        g[rng.random(n) < 0.05] = 0.0
        if gfmt == "bf16":
            g = oracle.encode_array("bf16", g)
        hh = dict(h, step=t)
        g_dev = to_dev(g)
        gpu_step(ds, g_dev, hh, gfmt=gfmt, index_base=base)
        oracle_step(wfmt, hs, g, hh, gfmt=gfmt, index_base=base)
        torch.cuda.synchronize()
        w_g, m_g, v_g, ve_g = ds.host()
        assert_state_equal(f"{tag} t={t}", w_g, hs.w, m_g, hs.m, v_g, hs.v, ve_g, hs.ve)
        assert_copy_equal(f"{tag} t={t}", ds, hs)
        if scales is not None:
            sn = np.uint16 if kind == "block" else np.uint8
            assert (to_host(ds.scales, sn) == hs.scales).all(), f"{tag} t={t}: scales"
        if kind == "nvcs":
            a, b = to_host(g_dev), g
            nan = np.isnan(a) & np.isnan(b)
            assert ((a.view(np.uint32) == b.view(np.uint32)) | nan).all(), f"{tag} t={t}: w'"
