"""Pins of the oracle's stochastic rounding and its counter-based generator.

The paper uses stochastic rounding (SR) so that small updates are preserved
in expectation, without defining it.  The reading used here rounds |x| up
with probability floor(frac * 2^16) / 2^16 from a 16-bit Philox4x32-10 draw.
Pins:
  * exact expectation: for BF16 the mean over all 2^16 draws equals x exactly
    (rational arithmetic); for FP8 it is within 2^-16 of a grid spacing;
  * the result is always one of the two neighbours, and representable values
    are returned unchanged;
  * unbiasedness through the keyed draws (seed, step, element index);
  * Philox4x32-10: Random123's published known-answer vectors, and rocRAND's
    implementation on random counters and keys (compiled here, host only);
  * uniformity and independence statistics of the 16-bit draws.
"""
import os
import shutil
import subprocess
from fractions import Fraction

import numpy as np
import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))


def _neighbours(fmt, x):
    """Grid neighbours lo <= |x| <= hi (by the oracle's RNE codes of the
    bracketing grid values), as (value, code) pairs."""
    bits = 16 if fmt == "bf16" else 8
    codes = np.arange(2 ** (bits - 1), dtype=np.uint32)
    vals = oracle.decode_array(fmt, codes)
    fin = np.isfinite(vals)
    vals, codes = vals[fin], codes[fin]
    a = abs(float(x))
    lo = vals[vals <= a].max()
    hi_c = vals[vals >= a]
    hi = hi_c.min() if hi_c.size else None
    return (lo, int(codes[vals == lo][0])), ((hi, int(codes[vals == hi][0])) if hi is not None
                                             else None)


SR_CASES = {
    "bf16": [1.0 + 2 ** -9, 0.0123, -3.3e-3, 1e-39, -2.5e-41, 3.0e38, 0.75 + 2 ** -12, 1.0],
    "e4m3": [0.3, -0.0123, 2 ** -10, 3 * 2 ** -11, 447.0, 100.1, -1.9e-3, 0.5],
    "e5m2": [0.3, -7.7e-5, 2 ** -17, 5 * 2 ** -18, 57000.0, 1.1e-6, -1234.5, 2.0],
}


@pytest.mark.parametrize("fmt", ["bf16", "e4m3", "e5m2"])
def test_sr_enumerated_over_all_draws(fmt):
    nb = 16 if fmt == "bf16" else 8
    sign_bit = 1 << (nb - 1)
    for x in SR_CASES[fmt]:
        x32 = float(np.float32(x))
        (lo, lo_c), hi = _neighbours(fmt, x32)
        codes = np.array([oracle.encode(fmt, x32, "sr", r) for r in range(65536)], dtype=np.int64)
        sgn = sign_bit if x32 < 0 else 0
        if lo == abs(x32):  # representable: never changes
            assert (codes == (sgn | lo_c)).all()
            continue
        hi_v, hi_c = hi
        assert set(np.unique(codes)) <= {sgn | lo_c, sgn | hi_c}
        ups = int((codes == (sgn | hi_c)).sum())
        frac = (Fraction(abs(x32)) - Fraction(lo)) / (Fraction(hi_v) - Fraction(lo))
        assert ups == int(frac * 65536)  # floor: frac >= 0
        mean = (Fraction(lo) * (65536 - ups) + Fraction(hi_v) * ups) / 65536
        err = abs(mean - Fraction(abs(x32)))
        if fmt == "bf16":
            assert err == 0  # exactly unbiased
        else:
            assert err <= (Fraction(hi_v) - Fraction(lo)) / 65536


@pytest.mark.parametrize("fmt", ["bf16", "e4m3"])
def test_sr_keyed_draws_are_unbiased(fmt):
    rng = np.random.default_rng(7)
    n = 1 << 15
    for x in rng.uniform(-0.05, 0.05, 4).astype(np.float32):
        (lo, _), (hi, _) = _neighbours(fmt, float(x))
        vals = np.array([oracle.decode(fmt, oracle.encode(fmt, float(x), "sr",
                                                          oracle.draw16(1234, 3, 0, i)))
                         for i in range(n)])
        p = (abs(float(x)) - lo) / (hi - lo)
        sigma = (hi - lo) * np.sqrt(p * (1 - p) / n) + 1e-30
        assert abs(vals.mean() - float(x)) < 5 * sigma + (hi - lo) / 65536


# Known-answer vectors for Philox4x32 with 10 rounds, as published with the
# Random123 library (Salmon et al., SC'11): (counter, key) -> output.
PHILOX_KAT = [
    ((0x00000000, 0x00000000, 0x00000000, 0x00000000), (0x00000000, 0x00000000),
     (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
    ((0xFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF), (0xFFFFFFFF, 0xFFFFFFFF),
     (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
    ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
     (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)),
]


@pytest.mark.parametrize("ctr,key,out", PHILOX_KAT)
def test_philox_known_answers(ctr, key, out):
    assert tuple(int(v) for v in oracle.philox(ctr, key)) == out


def test_philox_matches_rocrand(tmp_path):
    hipcc = "/opt/rocm/bin/hipcc" if os.path.exists("/opt/rocm/bin/hipcc") else shutil.which("hipcc")
    if hipcc is None or not os.path.exists("/opt/rocm/include/rocrand/rocrand_philox4x32_10.h"):
        pytest.skip("rocRAND headers or hipcc not available")
    exe = tmp_path / "probe"
    subprocess.run([hipcc, "-O1", "-o", str(exe), os.path.join(HERE, "philox_rocrand_probe.cpp")],
                   check=True, capture_output=True)
    rng = np.random.default_rng(11)
    rows = rng.integers(0, 2 ** 32, size=(300, 6), dtype=np.uint64)
    text = "\n".join(" ".join(f"{int(v):x}" for v in r) for r in rows) + "\n"
    res = subprocess.run([str(exe)], input=text, capture_output=True, text=True, check=True)
    lines = res.stdout.strip().splitlines()
    assert len(lines) == len(rows)
    for r, line in zip(rows, lines):
        want = [int(t, 16) for t in line.split()]
        got = oracle.philox(r[:4].astype(np.uint32), r[4:].astype(np.uint32))
        assert [int(v) for v in got] == want


def test_draw16_is_a_lane_of_philox():
    seed, t = 0x0123456789ABCDEF, 77
    for idx in [0, 1, 7, 8, 9, 2 ** 33 + 5, 6_738_415_615]:
        j = idx >> 3
        out = oracle.philox([j & 0xFFFFFFFF, j >> 32, t, 0], [seed & 0xFFFFFFFF, seed >> 32])
        word = int(out[(idx & 7) >> 1])
        want = (word >> 16) if idx & 1 else (word & 0xFFFF)
        assert oracle.draw16(seed, t, 0, idx) == want


def test_draw16_statistics():
    n = 1 << 15
    d = np.array([oracle.draw16(99, 5, 0, i) for i in range(n)], dtype=np.int64)
    # uniformity over 64 bins (chi-square, 63 dof: mean 63, sd ~ 11.2)
    h = np.bincount(d >> 10, minlength=64)
    chi2 = ((h - n / 64) ** 2 / (n / 64)).sum()
    assert chi2 < 63 + 6 * 11.2
    # bit balance
    for b in range(16):
        frac = ((d >> b) & 1).mean()
        assert abs(frac - 0.5) < 5 * 0.5 / np.sqrt(n)
    # neighbouring indices, and the same index at the next step, uncorrelated
    d2 = np.array([oracle.draw16(99, 6, 0, i) for i in range(n)], dtype=np.int64)
    for a, b in ((d[:-1], d[1:]), (d, d2)):
        r = np.corrcoef(a, b)[0, 1]
        assert abs(r) < 5 / np.sqrt(n)
