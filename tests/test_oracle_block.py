"""Pins of the oracle's block-scaled FP8 storage (CPU).

The paper stores selected weight matrices as FP8 payloads with FP16 block
scales and re-quantizes them after every update (Section 4.2; the FP8-master
dataflow figure).  Block length and scale rule are not given; the reading is
128 contiguous elements and scale = RNE_fp16(max|w| / FMAX).  Pins:
  * the scale is numpy's float16 rounding of the fp32 ratio; the payloads
    are torch's float8 rounding of w / scale; special blocks follow the rule;
  * the block step equals the unscaled step (FP32 passthrough format) on the
    dequantized weights followed by block encoding -- the update itself is
    the same M+Adam step;
  * with stochastic rounding every new weight lies on one of the two grid
    points around the unrounded update.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_10611_amd.workloads import DEFAULT_HPARAMS

FMAX = {"e4m3": 448.0, "e5m2": 57344.0}
TDT = {"e4m3": torch.float8_e4m3fn, "e5m2": torch.float8_e5m2}


def hp(**kw):
    h = dict(DEFAULT_HPARAMS)
    h["rounding"] = "rne"
    h.update(kw)
    return h


def dequant(fmt, q, s):
    qv = oracle.decode_array(fmt, q).astype(np.float32)
    sv = oracle.decode_array("fp16", s).astype(np.float32)
    return (qv.reshape(-1, 128) * sv[:, None]).ravel().astype(np.float32)


def blocks(rng, nb):
    scales = 10.0 ** rng.uniform(-6, 1, nb)
    x = rng.normal(0, 1, (nb, 128)) * scales[:, None]
    x[0] = 0.0                      # all-zero block
    x[1, 5] = 3e-9                  # tiny block: scale underflows
    x[1, :5] = 0.0
    x[1, 6:] = 0.0
    return x.astype(np.float32).ravel()


@pytest.mark.parametrize("fmt", ["e4m3", "e5m2"])
def test_encode_block_rule(fmt):
    rng = np.random.default_rng(0)
    x = blocks(rng, 64)
    q, s = oracle.encode_block(fmt, x)
    xb = x.reshape(-1, 128)
    amax = np.abs(xb).max(axis=1).astype(np.float32)
    ratio = (amax / np.float32(FMAX[fmt])).astype(np.float32)
    want = ratio.astype(np.float16).view(np.uint16).copy()
    want[amax == 0] = 0x3C00
    want[want == 0] = 0x0001
    assert (s == want).all()
    sv = s.view(np.float16).astype(np.float32)
    y = (xb / sv[:, None]).astype(np.float32)
    ref = torch.from_numpy(np.clip(y, -FMAX[fmt], FMAX[fmt]).ravel()).to(TDT[fmt]
                                                                         ).view(torch.uint8).numpy()
    assert (q == ref).all()


def test_encode_block_nonfinite_gives_nan_block():
    x = np.zeros(256, np.float32)
    x[3] = np.inf
    x[200] = 1.0
    q, s = oracle.encode_block("e4m3", x)
    assert s[0] == 0x7E00 and (q[:128] == 0x7F).all()
    assert s[1] != 0x7E00 and (q[128:] != 0x7F).all()


@pytest.mark.parametrize("fmt", ["e4m3", "e5m2"])
def test_block_step_is_unscaled_step_then_block_encoding(fmt):
    rng = np.random.default_rng(1)
    nb = 48
    n = nb * 128
    q, s = oracle.encode_block(fmt, rng.normal(0, 0.02, n).astype(np.float32))
    m, v, ve = (np.zeros(n, np.float32) for _ in range(3))
    m2, v2, ve2 = (np.zeros(n, np.float32) for _ in range(3))
    for t in range(1, 6):
        g = (rng.normal(0, 1, n) * 10.0 ** rng.uniform(-5, -2, n)).astype(np.float32)
        w32 = dequant(fmt, q, s)
        codes32 = w32.view(np.uint32).copy()
        oracle.step("fp32", codes32, g, m2, v2, ve2, hp(step=t))
        q_want, s_want = oracle.encode_block(fmt, codes32.view(np.float32))
        oracle.step_block(fmt, q, s, g, m, v, ve, hp(step=t))
        assert (s == s_want).all()
        assert (oracle.decode_array(fmt, q) == oracle.decode_array(fmt, q_want)).all()
        assert m.tobytes() == m2.tobytes() and v.tobytes() == v2.tobytes()
        assert ve.tobytes() == ve2.tobytes()


def test_block_step_sr_lands_on_neighbours():
    fmt = "e4m3"
    rng = np.random.default_rng(2)
    n = 32 * 128
    q, s = oracle.encode_block(fmt, rng.normal(0, 0.02, n).astype(np.float32))
    g = rng.normal(0, 1e-3, n).astype(np.float32)
    w32 = dequant(fmt, q, s)
    codes32 = w32.view(np.uint32).copy()
    z = [np.zeros(n, np.float32) for _ in range(3)]
    oracle.step("fp32", codes32, g, *z, hp())
    wn = codes32.view(np.float32)
    z = [np.zeros(n, np.float32) for _ in range(3)]
    oracle.step_block(fmt, q, s, g, *z, hp(rounding="sr", seed=5))
    sv = oracle.decode_array("fp16", s)
    y = (wn.reshape(-1, 128) / sv[:, None].astype(np.float32)).astype(np.float32).ravel()
    lo = torch.from_numpy(y).to(TDT[fmt]).float().numpy()  # nearest grid point
    got = oracle.decode_array(fmt, q)
    # the nearest point or the neighbour on the other side of y
    grid = np.sort(np.unique(oracle.decode_array(fmt, np.arange(256, dtype=np.uint32))))
    grid = grid[np.isfinite(grid)]
    i = np.searchsorted(grid, y)
    below = grid[np.clip(i - 1, 0, grid.size - 1)]
    above = grid[np.clip(i, 0, grid.size - 1)]
    ok = (got == below) | (got == above) | (got == lo)
    assert ok.all()


# --------------------------------------------------------------------------
# bf16 compute copy
# --------------------------------------------------------------------------

def _torch_bf16(x: np.ndarray) -> np.ndarray:
    return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(torch.bfloat16).view(
        torch.int16).numpy().view(np.uint16)


@pytest.mark.parametrize("wfmt", ["bf16", "e4m3", "e5m2", "fp32"])
def test_compute_copy_is_bf16_of_the_stored_weight(wfmt):
    # The copy the GEMMs read is the new stored weight, dequantized and
    # rounded to bf16 by the library conversion.
    rng = np.random.default_rng(3)
    n = 4096
    codes = oracle.encode_array(wfmt, rng.normal(0, 0.3, n).astype(np.float32))
    copy = np.zeros(n, np.uint16)
    z = [np.zeros(n, np.float32) for _ in range(3)]
    g = rng.normal(0, 1e-2, n).astype(np.float32)
    oracle.step(wfmt, codes, g, *z, hp(rounding="sr", seed=1, lr_add=1e-2), copy=copy)
    assert (copy == _torch_bf16(oracle.decode_array(wfmt, codes))).all()


@pytest.mark.parametrize("fmt", ["e4m3", "e5m2"])
def test_block_compute_copy_is_bf16_of_payload_times_scale(fmt):
    rng = np.random.default_rng(4)
    n = 16 * 128
    q, s = oracle.encode_block(fmt, rng.normal(0, 0.05, n).astype(np.float32))
    copy = np.zeros(n, np.uint16)
    z = [np.zeros(n, np.float32) for _ in range(3)]
    g = rng.normal(0, 1e-3, n).astype(np.float32)
    oracle.step_block(fmt, q, s, g, *z, hp(rounding="sr", seed=2), copy=copy)
    assert (copy == _torch_bf16(dequant(fmt, q, s))).all()
