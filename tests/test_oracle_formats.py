"""Pins of the oracle's storage-format codecs (CPU).

The oracle decodes from each format's (sign, exponent, mantissa) definition
and encodes by searching its grid.  These tests pin both against independent
library conversions (torch's bfloat16 / float8 dtypes, numpy's float16), and
against exact rational arithmetic for round-to-nearest-even.
"""
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle


def _torch_decode(codes: np.ndarray, dtype) -> np.ndarray:
    if dtype == torch.bfloat16:
        t = torch.from_numpy(codes.astype(np.uint16).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(codes.astype(np.uint8)).view(dtype)
    with np.errstate(invalid="ignore"):
        return t.float().numpy().astype(np.float64)


def _same_values(a: np.ndarray, b: np.ndarray):
    nan = np.isnan(b)
    assert (np.isnan(a) == nan).all()
    assert (a[~nan] == b[~nan]).all()
    assert (np.signbit(a[~nan]) == np.signbit(b[~nan])).all()


@pytest.mark.parametrize("fmt,bits,dtype", [("bf16", 16, torch.bfloat16),
                                            ("e4m3", 8, torch.float8_e4m3fn),
                                            ("e5m2", 8, torch.float8_e5m2)])
def test_decode_every_code_matches_torch(fmt, bits, dtype):
    codes = np.arange(2 ** bits, dtype=np.uint32)
    _same_values(oracle.decode_array(fmt, codes), _torch_decode(codes, dtype))


def test_fp16_decode_every_code_matches_numpy():
    codes = np.arange(65536, dtype=np.uint16)
    _same_values(oracle.decode_array("fp16", codes), codes.view(np.float16).astype(np.float64))


@pytest.mark.parametrize("fmt,bits", [("bf16", 16), ("e4m3", 8), ("e5m2", 8), ("fp16", 16)])
def test_decode_is_monotone_in_code(fmt, bits):
    vals = oracle.decode_array(fmt, np.arange(2 ** (bits - 1), dtype=np.uint32))
    fin = vals[np.isfinite(vals)]
    assert (np.diff(fin) > 0).all()


def _probe_values(fmt: str, rng) -> np.ndarray:
    """fp32 values around every grid point of a format: the grid points, the
    midpoints between neighbours, one fp32 ulp either side of each midpoint,
    and random fp32 bit patterns."""
    bits = 16 if fmt in ("bf16", "fp16") else 8
    g = oracle.decode_array(fmt, np.arange(2 ** (bits - 1), dtype=np.uint32))
    g = np.sort(g[np.isfinite(g)])
    mids = ((g[1:] + g[:-1]) / 2).astype(np.float32)
    up = np.nextafter(mids, np.float32(np.inf))
    dn = np.nextafter(mids, np.float32(-np.inf))
    rnd = rng.integers(0, 2 ** 32, size=200_000, dtype=np.uint64).astype(np.uint32).view(np.float32)
    x = np.concatenate([g.astype(np.float32), mids, up, dn, rnd])
    x = np.concatenate([x, -x])
    return x[np.isfinite(x)]


def test_bf16_rne_matches_torch():
    x = _probe_values("bf16", np.random.default_rng(1))
    ours = oracle.encode_array("bf16", x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert (ours == ref).all()


@pytest.mark.parametrize("fmt,dtype,fmax", [("e4m3", torch.float8_e4m3fn, 448.0),
                                            ("e5m2", torch.float8_e5m2, 57344.0)])
def test_fp8_rne_matches_torch_in_range(fmt, dtype, fmax):
    x = _probe_values(fmt, np.random.default_rng(2))
    x = x[np.abs(x) <= fmax]
    ours = oracle.encode_array(fmt, x)
    ref = torch.from_numpy(x).to(dtype).view(torch.uint8).numpy()
    assert (ours == ref).all()


@pytest.mark.parametrize("fmt,maxcode", [("e4m3", 0x7E), ("e5m2", 0x7B)])
def test_fp8_saturates(fmt, maxcode):
    big = np.array([449.0, 1e4, 6e4, 1e30, np.inf], dtype=np.float32)
    big = big[big > (448.0 if fmt == "e4m3" else 57344.0)]
    assert (oracle.encode_array(fmt, big) == maxcode).all()
    assert (oracle.encode_array(fmt, -big) == (0x80 | maxcode)).all()


def test_fp16_rne_matches_numpy_including_overflow():
    x = _probe_values("fp16", np.random.default_rng(3))
    x = np.concatenate([x, np.array([65504, 65519.99, 65520, 70000, 1e10, np.inf, -np.inf],
                                    dtype=np.float32)])
    ours = oracle.encode_array("fp16", x)
    with np.errstate(over="ignore"):
        ref = x.astype(np.float16).view(np.uint16)
    assert (ours == ref).all()


def test_nan_codes():
    nan = np.array([np.nan, -np.nan], dtype=np.float32)
    assert (oracle.encode_array("bf16", nan) == 0x7FC0).all()
    assert (oracle.encode_array("fp16", nan) == 0x7E00).all()
    assert (oracle.encode_array("e4m3", nan) == 0x7F).all()
    assert (oracle.encode_array("e5m2", nan) == 0x7F).all()
    assert (oracle.encode_array("fp32", nan) == 0x7FC00000).all()


@pytest.mark.parametrize("fmt", ["bf16", "e4m3", "e5m2"])
def test_rne_is_nearest_by_exact_arithmetic(fmt):
    import bisect
    bits = 16 if fmt == "bf16" else 8
    g = oracle.decode_array(fmt, np.arange(2 ** (bits - 1), dtype=np.uint32))
    fin = np.isfinite(g)
    codes = np.arange(2 ** (bits - 1))[fin]
    order = np.argsort(g[fin])
    vals = [Fraction(float(v)) for v in g[fin][order]]
    cods = [int(c) for c in codes[order]]
    rng = np.random.default_rng(4)
    lim = float(g[fin].max())
    xs = np.concatenate([rng.uniform(0, lim, 300), np.exp(rng.uniform(-40, np.log(lim), 300))])
    for x in xs.astype(np.float32):
        c = oracle.encode(fmt, float(x))
        X = Fraction(float(x))
        i = bisect.bisect_left(vals, X)
        cands = [j for j in (i - 1, i) if 0 <= j < len(vals)]
        best = min(abs(vals[j] - X) for j in cands)
        near = [cods[j] for j in cands if abs(vals[j] - X) == best]
        want = near[0] if len(near) == 1 else [cc for cc in near if cc % 2 == 0][0]
        assert c == want, (fmt, float(x), hex(c), hex(want))
