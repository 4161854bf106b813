"""The block-scale rules of the block-scaled encoders on every fp32 magnitude
(GPU).

MXFP4 (OCP MX): a block whose largest |x| is a has the shared exponent
s = floor(log2 a) - 2 (2 = the exponent of E2M1's largest value, 6), clamped
to [-127, 127], stored as the E8M0 code s + 127 (s = 0 for an all-zero
block); its elements are E2M1 codes of x / 2^s rounded to nearest-even,
saturating at 6.  Each test block holds one fp32 value a followed by 31
zeros, for every finite a > 0 and for a = 0, and the reference is written
here with torch integer and float ops on the device (2^-s built from its
bits; the products are exact).

NVFP4 with the tensor scale forced to 1 (one block holding 2688 = 6 x 448):
a block's E4M3 scale code is E4M3(a / 6) rounded to nearest-even, its factor
the code's value, and its elements E2M1 codes of x / factor (0 when the
factor is 0), for every fp32 a in [0, 2688].  torch's float8_e4m3fn cast and
fp32 division give the reference; the division is tensor by tensor, since
torch divides a device tensor by a Python scalar as a product with the
rounded reciprocal, one ulp off the quotient at times (which moves a ratio
onto an E4M3 midpoint).

Block-scaled FP8 (blocks of 128): the FP16 scale code of fp32(a / max)
rounded to nearest-even (1.0 for a zero block, never 0 or infinity) and the
payload of a / scale, saturating, for every finite fp32 a, in E4M3 and E5M2.
Each reference is also checked against the oracle on a seeded sample."""
import pytest
import torch

from paper_2607_10611_amd import binding as B

pytestmark = pytest.mark.gpu

MIDS = (0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0)   # between E2M1 magnitudes 0 .5 1 1.5 2 3 4 6


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    B.lib()
    yield
    torch.cuda.synchronize()


def e2m1_rne(v):
    """E2M1 code of v >= 0, nearest-even, saturating at 6 (code 7)."""
    s = torch.zeros_like(v, dtype=torch.int64)
    tie = torch.zeros_like(v, dtype=torch.bool)
    for m in MIDS:
        s += (v > m).to(torch.int64)
        tie |= v == m
    return s + (tie & (s % 2 == 1)).to(torch.int64)


def pow2(k):
    """2^k as fp32 for integer tensors k in [-126, 127], from its bits."""
    return ((k + 127).to(torch.int32) << 23).view(torch.float32)


def frexp_exponent(bits):
    """e with a = f 2^e, f in [0.5, 1), for the positive fp32 bit patterns
    `bits` (int64), from the fields: ef - 126 for normal numbers; for
    subnormal ones (mantissa m, a = m 2^-149) the same of m, exactly
    converted, minus 149."""
    ef = (bits >> 23) & 0xFF
    mf = (bits & 0x7FFFFF).to(torch.float32)      # exact: m < 2^23
    ef_m = (mf.view(torch.int32).to(torch.int64) >> 23) & 0xFF
    return torch.where(ef > 0, ef - 126, ef_m - 126 - 149)


def lead_codes(q, nb, per):
    """The code of each block's first element (the low nibble of its first byte)."""
    return (q.view(nb, per // 2)[:, 0] & 0xF).to(torch.int64)


def test_mxfp4_scale_and_payload_of_every_fp32_magnitude():
    per_call = 1 << 26
    top = 0x7F800000                                  # bit patterns 0 .. top-1: 0 and finite a > 0
    bad, examples = 0, []
    for start in range(0, top, per_call):
        nb = min(per_call, top - start)
        bits = torch.arange(start, start + nb, dtype=torch.int64, device="cuda")
        a = bits.to(torch.int32).view(torch.float32)
        x = torch.zeros(nb, 32, device="cuda")
        x[:, 0] = a
        q = torch.empty(nb * 16, dtype=torch.uint8, device="cuda")
        sc = torch.empty(nb, dtype=torch.uint8, device="cuda")
        B.madd_encode_weights(x.view(-1), q, "mxfp4", scales=sc)
        e = frexp_exponent(bits)                      # a = f 2^e, f in [0.5, 1)
        s = torch.clamp(e - 1 - 2, -127, 127)
        s = torch.where(a == 0, torch.zeros_like(s), s)
        want_sc = s + 127
        want_q = e2m1_rne(a * pow2(-s))
        got_sc = sc.to(torch.int64)
        got_q = lead_codes(q, nb, 32)
        rest_zero = bool((q.view(nb, 16)[:, 1:] == 0).all()) and bool(
            (q.view(nb, 16)[:, 0] >> 4 == 0).all())
        mism = (got_sc != want_sc) | (got_q != want_q)
        n = int(mism.sum()) + (0 if rest_zero else 1)
        if n and not examples:
            i = torch.nonzero(mism)[:5, 0]
            examples = [(hex(start + int(j)), int(got_sc[j]), int(want_sc[j]), int(got_q[j]),
                         int(want_q[j])) for j in i] or ["nonzero payload of a zero element"]
        bad += n
        del bits, a, x, q, sc, e, s, want_sc, want_q, got_sc, got_q, mism
    # non-finite blocks: the NaN scale code and zero payloads
    x = torch.zeros(3, 32, device="cuda")
    x[0, 5], x[1, 0], x[2, 31] = float("nan"), float("inf"), -float("inf")
    q = torch.empty(48, dtype=torch.uint8, device="cuda")
    sc = torch.empty(3, dtype=torch.uint8, device="cuda")
    B.madd_encode_weights(x.view(-1), q, "mxfp4", scales=sc)
    assert (sc == 0xFF).all() and (q == 0).all()
    assert bad == 0, f"{bad} magnitudes encode differently (bits, scale got/want, code got/want): " \
                     f"{examples}"


def test_nvfp4_block_scale_and_payload_of_every_fp32_magnitude_up_to_2688():
    per_call = 1 << 26
    top = 0x45280000 + 1                              # bit patterns of 0 .. 2688
    bad, examples = 0, []
    for start in range(0, top, per_call):
        nb = min(per_call, top - start)
        bits = torch.arange(start, start + nb, dtype=torch.int64, device="cuda")
        a = bits.to(torch.int32).view(torch.float32)
        x = torch.zeros(nb + 1, 16, device="cuda")
        x[:nb, 0] = a
        x[nb, 0] = 2688.0                             # tensor scale 2688 / 2688 = 1
        q = torch.empty((nb + 1) * 8, dtype=torch.uint8, device="cuda")
        sc = torch.empty(4 + nb + 1, dtype=torch.uint8, device="cuda")
        B.madd_encode_weights(x.view(-1), q, "nvfp4", scales=sc)
        assert float(sc[:4].view(torch.float32)[0]) == 1.0
        code = (a / torch.full_like(a, 6.0)).to(torch.float8_e4m3fn)
        want_sc = code.view(torch.uint8).to(torch.int64)
        den = code.to(torch.float32)
        want_q = torch.where(den == 0, torch.zeros_like(want_sc), e2m1_rne(a / den))
        got_sc = sc[4:4 + nb].to(torch.int64)
        got_q = lead_codes(q[:nb * 8], nb, 16)
        rest_zero = bool((q.view(nb + 1, 8)[:nb, 1:] == 0).all()) and bool(
            (q.view(nb + 1, 8)[:nb, 0] >> 4 == 0).all())
        mism = (got_sc != want_sc) | (got_q != want_q)
        n = int(mism.sum()) + (0 if rest_zero else 1)
        if n and not examples:
            i = torch.nonzero(mism)[:5, 0]
            examples = [(hex(start + int(j)), int(got_sc[j]), int(want_sc[j]), int(got_q[j]),
                         int(want_q[j])) for j in i] or ["nonzero payload of a zero element"]
        bad += n
        del bits, a, x, q, sc, code, want_sc, den, want_q, got_sc, got_q, mism
    assert bad == 0, f"{bad} magnitudes encode differently (bits, scale got/want, code got/want): " \
                     f"{examples}"


def test_references_agree_with_the_oracle_on_a_sample():
    """The two references above against the oracle's MXFP4 and NVFP4
    encoders on 20,000 seeded magnitudes (edges included, and the quotients
    a / 6 just below an E4M3 midpoint)."""
    import numpy as np

    import oracle
    rng = np.random.default_rng(17)
    bits = np.concatenate([[0, 1, 2, 0x7FFFFF, 0x800000, 0x40C00000, 0x45280000, 0x3DE3FFFF,
                            0x3E63FFFF, 0x3FE3FFFF],
                           rng.integers(1, 0x45280000, 20000)]).astype(np.int64)
    a = bits.astype(np.uint32).view(np.float32)
    # MXFP4
    x = np.zeros((a.size, 32), np.float32)
    x[:, 0] = a
    q, sc = oracle.encode_mx(x.reshape(-1))
    bt = torch.from_numpy(bits).cuda()
    at = torch.from_numpy(a.copy()).cuda()
    s = torch.clamp(frexp_exponent(bt) - 3, -127, 127)
    s = torch.where(at == 0, torch.zeros_like(s), s)
    assert np.array_equal((s + 127).cpu().numpy(), sc.astype(np.int64))
    assert np.array_equal(e2m1_rne(at * pow2(-s)).cpu().numpy(),
                          (q.reshape(a.size, 16)[:, 0] & 0xF).astype(np.int64))
    # NVFP4, tensor scale 1
    x = np.zeros((a.size + 1, 16), np.float32)
    x[:-1, 0] = a
    x[-1, 0] = 2688.0
    q, sc = oracle.encode_nv(x.reshape(-1))
    code = (at / torch.full_like(at, 6.0)).to(torch.float8_e4m3fn)
    den = code.to(torch.float32)
    want_q = torch.where(den == 0, torch.zeros_like(den, dtype=torch.int64), e2m1_rne(at / den))
    assert np.array_equal(code.view(torch.uint8).cpu().numpy(), sc[4:4 + a.size])
    assert np.array_equal(want_q.cpu().numpy(),
                          (q.reshape(a.size + 1, 8)[:-1, 0] & 0xF).astype(np.int64))


FP8 = {"e4m3": (torch.float8_e4m3fn, 448.0), "e5m2": (torch.float8_e5m2, 57344.0)}


def fp8_block_reference(a, fmt):
    """Block-scaled FP8 of a block led by a (the rest 0): the FP16 scale
    code of fp32(a / max) rounded to nearest-even (1.0 for a zero block, the
    smallest subnormal instead of 0, the largest finite instead of infinity)
    and the payload code of a / scale, saturating at the format's maximum."""
    ft, fmax = FP8[fmt]
    ratio = a / torch.full_like(a, fmax)
    sc = ratio.to(torch.float16).view(torch.int16).to(torch.int64) & 0xFFFF
    sc = torch.where(a == 0, torch.full_like(sc, 0x3C00), sc)
    sc = torch.where(sc == 0, torch.ones_like(sc), sc)
    sc = torch.where(sc == 0x7C00, torch.full_like(sc, 0x7BFF), sc)
    sf = sc.to(torch.int16).view(torch.float16).to(torch.float32)
    code = (a / sf).clamp(max=fmax).to(ft).view(torch.uint8).to(torch.int64)
    return sc, code


@pytest.mark.parametrize("fmt", ["e4m3", "e5m2"])
def test_block_fp8_scale_and_payload_of_every_fp32_magnitude(fmt):
    per_call = 1 << 24
    top = 0x7F800000
    bad, examples = 0, []
    for start in range(0, top, per_call):
        nb = min(per_call, top - start)
        bits = torch.arange(start, start + nb, dtype=torch.int64, device="cuda")
        a = bits.to(torch.int32).view(torch.float32)
        x = torch.zeros(nb, 128, device="cuda")
        x[:, 0] = a
        q = torch.empty(nb * 128, dtype=torch.uint8, device="cuda")
        sc = torch.empty(nb, dtype=torch.int16, device="cuda")
        B.madd_encode_weights(x.view(-1), q, fmt, scales=sc)
        want_sc, want_q = fp8_block_reference(a, fmt)
        got_sc = sc.to(torch.int64) & 0xFFFF
        qv = q.view(nb, 128)
        got_q = qv[:, 0].to(torch.int64)
        rest_zero = bool((qv[:, 1:] == 0).all())
        mism = (got_sc != want_sc) | (got_q != want_q)
        n = int(mism.sum()) + (0 if rest_zero else 1)
        if n and not examples:
            i = torch.nonzero(mism)[:5, 0]
            examples = [(hex(start + int(j)), hex(int(got_sc[j])), hex(int(want_sc[j])),
                         int(got_q[j]), int(want_q[j])) for j in i] or ["nonzero zero element"]
        bad += n
        del bits, a, x, q, sc, want_sc, want_q, got_sc, qv, got_q, mism
    assert bad == 0, f"{fmt}: {bad} magnitudes encode differently (bits, scale got/want, " \
                     f"code got/want): {examples}"


def test_fp8_block_reference_agrees_with_the_oracle_on_a_sample():
    import numpy as np

    import oracle
    rng = np.random.default_rng(23)
    bits = np.concatenate([[0, 1, 0x7FFFFF, 0x800000, 0x3F800000, 0x43E00000, 0x4B7FE000,
                            0x7F7FFFFF], rng.integers(1, 0x7F800000, 20000)]).astype(np.int64)
    a = bits.astype(np.uint32).view(np.float32)
    at = torch.from_numpy(a.copy()).cuda()
    for fmt in FP8:
        x = np.zeros((a.size, 128), np.float32)
        x[:, 0] = a
        q, sc = oracle.encode_block(fmt, x.reshape(-1))
        want_sc, want_q = fp8_block_reference(at, fmt)
        assert np.array_equal(want_sc.cpu().numpy(), sc.astype(np.int64)), fmt
        assert np.array_equal(want_q.cpu().numpy(), q.reshape(a.size, 128)[:, 0].astype(np.int64)), fmt
