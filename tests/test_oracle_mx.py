"""Pins of the oracle's MXFP4 storage (CPU).

The paper's most aggressive regime stores master weights in a 4-bit
block-scaled format (Section 4.2, the NVFP4/FP8 setting) without defining
it.  The oracle uses the OCP Microscaling (MX) v1.0 block format MXFP4:
32-element blocks of E2M1 values sharing one E8M0 scale X = 2^s, with
s = floor(log2 max|w|) - 2 (2 = exponent of E2M1's largest value, 6).
Pins, none of which reuses the oracle's code path:
  * E2M1 decodes to the specification's value table; E8M0 decodes like
    torch's float8_e8m0fnu;
  * element rounding equals a brute-force nearest search over that table
    (ties to the even code, saturation at +-6); stochastic rounding has the
    exact expectation of the 16-bit rule;
  * the block scale satisfies 4 <= max|w| / X < 8 (the defining property of
    the floor rule), with the stated special cases;
  * a hand-computed block (packing order, scale, payloads);
  * the MXFP4 step equals the unscaled FP32 step on the dequantized weights
    followed by MXFP4 encoding; with stochastic rounding every payload is
    one of the two grid neighbours of w'/X.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2607_10611_amd.workloads import DEFAULT_HPARAMS

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "mxfp4_block.json")

# OCP MX v1.0, FP4 (E2M1) element values of codes 0..7 (code 8..15: negated)
E2M1_TABLE = [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]


def hp(**kw):
    h = dict(DEFAULT_HPARAMS)
    h["rounding"] = "rne"
    h.update(kw)
    return h


def nearest_e2m1(y: float) -> int:
    """Brute force: the E2M1 code nearest to y (ties: even code), saturating."""
    sign = 8 if np.signbit(y) else 0
    a = min(abs(y), 6.0)
    d = [abs(a - t) for t in E2M1_TABLE]
    best = min(d)
    cands = [c for c in range(8) if d[c] == best]
    even = [c for c in cands if c % 2 == 0]
    return sign | (even[0] if even else cands[0])


def test_e2m1_decodes_to_the_spec_table():
    for c in range(16):
        want = E2M1_TABLE[c & 7] * (-1.0 if c & 8 else 1.0)
        got = oracle.decode("e2m1", c)
        assert got == want and np.signbit(got) == bool(c & 8), c


def test_e8m0_decodes_like_torch():
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    ref = codes.view(torch.float8_e8m0fnu).double().numpy()
    got = oracle.decode_array("e8m0", np.arange(256, dtype=np.uint32))
    assert np.isnan(got[255]) and np.isnan(ref[255])
    assert (got[:255] == ref[:255]).all()


def test_e2m1_rne_is_brute_force_nearest():
    vals = set()
    for t in E2M1_TABLE + [6.5, 7.0, 8.0, 100.0]:
        for d in (0.0, 1e-3, 0.25, 0.5, 0.75, 1.0):
            vals.update({t + d, max(t - d, 0.0)})
    mids = [(a + b) / 2 for a, b in zip(E2M1_TABLE, E2M1_TABLE[1:])]
    for mpt in mids:  # ties, and one fp32 ulp to either side
        vals.update({mpt, float(np.nextafter(np.float32(mpt), np.float32(0))),
                     float(np.nextafter(np.float32(mpt), np.float32(10)))})
    vals.update({1e-30, 2.0 ** -149, float(np.inf)})
    for v in sorted(vals):
        for x in (v, -v):
            assert oracle.encode("e2m1", x) == nearest_e2m1(float(np.float32(x))), x


def test_e2m1_sr_has_the_exact_expectation_of_the_16_bit_rule():
    for y in (0.3, 1.1, 2.7, 4.9, 5.999):
        lo = max(t for t in E2M1_TABLE if t <= y)
        hi = min(t for t in E2M1_TABLE if t > y)
        k = np.floor((np.float32(y) - lo) / (hi - lo) * 65536.0)
        total = sum(abs(oracle.decode("e2m1", oracle.encode("e2m1", y, "sr", r)))
                    for r in range(0, 65536, 1))
        assert total / 65536.0 == pytest.approx(lo + k / 65536.0 * (hi - lo), abs=0, rel=1e-12)


def _blocks(rng, nb):
    mag = 2.0 ** rng.uniform(-20, 10, nb)
    x = rng.normal(0, 1, (nb, 32)) * mag[:, None]
    x[0] = 0.0                        # all-zero block
    x[1] = 0.0
    x[1, 7] = -2.0 ** -140            # tiny block: the scale exponent clamps at -127
    x[2] = 0.0
    x[2, 3] = 4.0                     # exact power of two
    x[3] = np.float32(np.nextafter(np.float32(8.0), np.float32(0))) * np.sign(x[3])
    return x.astype(np.float32).ravel()


def test_mx_encode_block_rule():
    rng = np.random.default_rng(10)
    x = _blocks(rng, 200)
    q, s = oracle.encode_mx(x)
    X = oracle.decode_array("e8m0", s)
    codes = oracle.unpack_e2m1(q)
    xb = x.reshape(-1, 32).astype(np.float64)
    amax = np.abs(xb).max(axis=1)
    for b in range(xb.shape[0]):
        if amax[b] == 0:
            assert s[b] == 127
        elif amax[b] < 2.0 ** -125:
            assert s[b] == 0
        else:
            assert 4.0 <= amax[b] / X[b] < 8.0, b
        for k in range(32):
            y = np.float32(xb[b, k] / X[b])  # exact: X is a power of two
            assert codes[32 * b + k] == nearest_e2m1(float(y)), (b, k)


def test_mx_nonfinite_block_gets_the_nan_scale_and_zero_payloads():
    x = np.ones(96, np.float32)
    x[40] = np.nan
    x[70] = -np.inf
    q, s = oracle.encode_mx(x)
    assert s.tolist() == [125, 255, 255]
    codes = oracle.unpack_e2m1(q)
    assert (codes[32:] == 0).all() and (codes[:32] == 6).all()  # 1.0 = 4 x 2^-2
    assert np.isnan(oracle.mx_values(q, s)[32:]).all()


def test_mx_hand_computed_block():
    # A block worked out by hand from the specification's rule (the JSON
    # fixture states the arithmetic).
    with open(GOLDEN) as f:
        ex = json.load(f)
    x = np.array(ex["x"], np.float32)
    q, s = oracle.encode_mx(x)
    assert s.tolist() == ex["scales"]
    assert q.tolist() == ex["packed"]


@pytest.mark.parametrize("sfmt", ["fp32", "bf16"])
def test_mx_step_is_unscaled_step_then_mx_encoding(sfmt):
    rng = np.random.default_rng(11)
    n = 64 * 32
    q, s = oracle.encode_mx(rng.normal(0, 0.02, n).astype(np.float32))
    zdt = np.float32 if sfmt == "fp32" else np.uint16
    st1 = [np.zeros(n, zdt) for _ in range(3)]
    st2 = [np.zeros(n, zdt) for _ in range(3)]
    for t in range(1, 6):
        g = (rng.normal(0, 1, n) * 10.0 ** rng.uniform(-5, -2, n)).astype(np.float32)
        w32 = oracle.mx_values(q, s).astype(np.float32)
        codes32 = w32.view(np.uint32).copy()
        oracle.step("fp32", codes32, g, *st2, hp(step=t, lr_add=1e-2), sfmt=sfmt)
        q_want, s_want = oracle.encode_mx(codes32.view(np.float32))
        oracle.step_mx(q, s, g, *st1, hp(step=t, lr_add=1e-2), sfmt=sfmt)
        assert (s == s_want).all() and (q == q_want).all(), t
        for a, b in zip(st1, st2):
            assert a.tobytes() == b.tobytes()


def test_mx_step_sr_lands_on_neighbours_and_moves_weights():
    rng = np.random.default_rng(12)
    n = 32 * 32
    q, s = oracle.encode_mx(rng.normal(0, 0.02, n).astype(np.float32))
    g = rng.normal(0, 1e-3, n).astype(np.float32)
    w32 = oracle.mx_values(q, s).astype(np.float32)
    codes32 = w32.view(np.uint32).copy()
    z = [np.zeros(n, np.float32) for _ in range(3)]
    oracle.step("fp32", codes32, g, *z, hp())
    wn = codes32.view(np.float32).astype(np.float64)
    z = [np.zeros(n, np.float32) for _ in range(3)]
    q0 = q.copy()
    oracle.step_mx(q, s, g, *z, hp(rounding="sr", seed=5))
    X = oracle.decode_array("e8m0", s)
    y = wn.reshape(-1, 32) / X[:, None]
    got = oracle.decode_array("e2m1", oracle.unpack_e2m1(q)).reshape(-1, 32)
    grid = np.array(sorted({-t for t in E2M1_TABLE} | set(E2M1_TABLE)))
    i = np.searchsorted(grid, y, side="right")
    below = grid[np.clip(i - 1, 0, grid.size - 1)]
    above = grid[np.clip(i, 0, grid.size - 1)]
    assert ((got == below) | (got == above) | (np.abs(y) >= 6) & (np.abs(got) == 6)).all()
    assert (q != q0).any()


def test_mx_sr_keys_by_global_index():
    rng = np.random.default_rng(13)
    n = 8 * 32
    x = rng.normal(0, 0.05, n).astype(np.float32)
    g = rng.normal(0, 1e-2, n).astype(np.float32)
    outs = []
    for kw in (dict(index_base=1000), dict(gidx=1000 + np.arange(n))):
        q, s = oracle.encode_mx(x)
        z = [np.zeros(n, np.float32) for _ in range(3)]
        oracle.step_mx(q, s, g, *z, hp(rounding="sr", seed=9, lr_add=1e-2), **kw)
        outs.append((q.copy(), s.copy()))
    assert (outs[0][0] == outs[1][0]).all() and (outs[0][1] == outs[1][1]).all()
    q, s = oracle.encode_mx(x)
    z = [np.zeros(n, np.float32) for _ in range(3)]
    oracle.step_mx(q, s, g, *z, hp(rounding="sr", seed=9, lr_add=1e-2), index_base=0)
    assert (q != outs[0][0]).any()


def test_mx_compute_copy_is_bf16_of_payload_times_scale():
    rng = np.random.default_rng(14)
    n = 16 * 32
    q, s = oracle.encode_mx(rng.normal(0, 0.05, n).astype(np.float32))
    copy = np.zeros(n, np.uint16)
    z = [np.zeros(n, np.float32) for _ in range(3)]
    g = rng.normal(0, 1e-3, n).astype(np.float32)
    oracle.step_mx(q, s, g, *z, hp(rounding="sr", seed=2), copy=copy)
    want = torch.from_numpy(oracle.mx_values(q, s).astype(np.float32)).to(torch.bfloat16)
    assert (copy == want.view(torch.int16).numpy().view(np.uint16)).all()


def test_mx_step_validation():
    z = [np.zeros(48, np.float32) for _ in range(4)]
    with pytest.raises(oracle.OracleError):
        oracle.step_mx(np.zeros(24, np.uint8), np.zeros(1, np.uint8), *z, hp())


@pytest.mark.parametrize("rounding", ["rne", "sr"])
def test_mx_zero_learning_rates_keep_every_stored_value(rounding):
    # eta_a = eta_m = 0 gives w' = the stored value q X.  A block whose largest
    # |q| is below 4 gets a smaller power-of-two scale X' = X 2^-k, and q 2^k
    # is again an E2M1 value (the grid doubles onto itself below 6), so the
    # scale code may change but no stored value does.
    rng = np.random.default_rng(15)
    nb = 200
    x = (rng.normal(0, 1, (nb, 32)) * 10.0 ** rng.uniform(-6, 2, nb)[:, None]).astype(np.float32)
    x[0] = 0.0
    x[1] = 0.0
    x[1, 5] = 3e-3
    x = x.ravel()
    q, s = oracle.encode_mx(x)
    before = oracle.mx_values(q, s).copy()
    z = [np.zeros(x.size, np.float32) for _ in range(3)]
    g = rng.normal(0, 1e-2, x.size).astype(np.float32)
    oracle.step_mx(q, s, g, *z, hp(lr_add=0.0, lr_mul=0.0, rounding=rounding, seed=4))
    assert (oracle.mx_values(q, s) == before).all()
