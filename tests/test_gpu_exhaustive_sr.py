"""The step's stochastic rounding on every fp32 input (GPU).  With the weight
at 0, eta_a = 1 and eta_m = 0, Appendix B's additive rule (madd_plain_step)
makes w' = -g exactly for every finite nonzero g (+0 for a zero g, NaN for a
non-finite one), so feeding all 2^32 fp32 bit patterns as gradients, with
the index base chosen so that element i's global index is its own bit
pattern, rounds every fp32 value once with its keyed draw.  The reference is
written here on the device with torch integer and float ops: Philox4x32-10
from its definition (checked against the oracle's generator on a sample),
the 16-bit rule round-up iff floor(frac * 2^16) + r16 >= 2^16 (bf16 as the
integer form (u + r16) >> 16), FP8 saturating at its largest value, NaN as
the canonical code."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_10611_amd import binding as B
from paper_2607_10611_amd import workloads as W

pytestmark = pytest.mark.gpu

CHUNK = 1 << 27
MASK = 0xFFFFFFFF
SEED, STEP = 0x0123456789ABCDEF, 77
MINI = {"e4m3": (3, 7, -6, 448.0), "e5m2": (2, 15, -14, 57344.0)}   # M, bias, min exponent, max


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    B.lib()
    yield
    torch.cuda.synchronize()


def philox_words(j, t, seed):
    """Philox4x32-10 output words for counters (j lo, j hi, t, 0), key = seed."""
    c0, c1 = j & MASK, (j >> 32) & MASK
    c2 = torch.full_like(j, t & MASK)
    c3 = torch.zeros_like(j)
    k0, k1 = seed & MASK, (seed >> 32) & MASK
    for _ in range(10):
        p0 = c0 * 0xD2511F53
        p1 = c2 * 0xCD9E8D57
        c0, c1, c2, c3 = (((p1 >> 32) & MASK) ^ c1 ^ k0, p1 & MASK,
                          ((p0 >> 32) & MASK) ^ c3 ^ k1, p0 & MASK)
        k0, k1 = (k0 + 0x9E3779B9) & MASK, (k1 + 0xBB67AE85) & MASK
    return torch.stack([c0, c1, c2, c3], dim=1)


def draws16(idx, t, seed):
    """16-bit draw of each global index (lane idx & 7 of group idx >> 3)."""
    words = philox_words(idx >> 3, t, seed)
    lane = idx & 7
    w = torch.gather(words, 1, (lane >> 1).unsqueeze(1)).squeeze(1)
    return torch.where((lane & 1) == 1, w >> 16, w & 0xFFFF)


def test_reference_generator_matches_the_oracle():
    rng = np.random.default_rng(3)
    idx = np.concatenate([rng.integers(0, 2**33, 500), np.arange(16)])
    got = draws16(torch.from_numpy(idx).cuda(), STEP, SEED).cpu().numpy()
    want = np.array([oracle.draw16(SEED, STEP, 0, int(i)) for i in idx])
    assert (got == want).all()


def sr_fp8_reference(x, r16, fmt):
    M, bias, emin, fmax = MINI[fmt]
    sign = (x.view(torch.int32) < 0).to(torch.int64) << 7
    a = x.abs().clamp(max=fmax)
    e = ((a.view(torch.int32) >> 23) & 0xFF).to(torch.int64) - 127
    se = torch.clamp(e, min=emin) - M
    # a * 2^-se with the power of two built from its bits: exact (torch's
    # ldexp on the device goes through a rounded power)
    q = a * ((127 - se).to(torch.int32) << 23).view(torch.float32)
    k = torch.floor(q)
    f16 = torch.floor((q - k) * 65536.0).to(torch.int64)
    k = k.to(torch.int64) + ((f16 + r16) >= 65536).to(torch.int64)
    code = ((se + M + bias - 1) << M) + k
    code = code | sign
    return torch.where(torch.isnan(x), torch.full_like(code, 0x7F), code)


@pytest.mark.parametrize("fmt", ["bf16", "e4m3", "e5m2"])
def test_stochastic_rounding_of_every_fp32_value(fmt):
    code_t = torch.int16 if fmt == "bf16" else torch.uint8
    h = dict(W.DEFAULT_HPARAMS, lr_add=1.0, lr_mul=0.0, rounding="sr", seed=SEED, step=STEP)
    w = torch.zeros(CHUNK, dtype=code_t, device="cuda")
    bad, examples = 0, []
    for c in range((1 << 32) // CHUNK):
        idx = torch.arange(c * CHUNK, (c + 1) * CHUNK, dtype=torch.int64, device="cuda")
        g = idx.to(torch.int32).view(torch.float32)
        w.zero_()
        B.madd_plain_step(w, fmt, g, h, index_base=c * CHUNK)
        # w' of the additive rule from w = 0: -g, +0 for a zero g, NaN for a non-finite g
        wn = torch.where(g == 0, torch.zeros_like(g), -g)
        wn = torch.where(torch.isfinite(g), wn, torch.full_like(g, float("nan")))
        r16 = draws16(idx, STEP, SEED)
        if fmt == "bf16":
            u = wn.view(torch.int32).to(torch.int64) & MASK
            ref = ((u + r16) >> 16) & 0xFFFF
            ref = torch.where(torch.isnan(wn), torch.full_like(ref, 0x7FC0), ref)
            got = w.to(torch.int64) & 0xFFFF
        else:
            ref = sr_fp8_reference(wn, r16, fmt)
            got = w.to(torch.int64)
        mism = got != ref
        nb = int(mism.sum())
        if nb and not examples:
            i = torch.nonzero(mism)[:5, 0]
            examples = [(hex(int(idx[j])), int(got[j]), int(ref[j])) for j in i]
        bad += nb
        del idx, g, wn, r16, ref, got, mism
    assert bad == 0, f"{fmt}: {bad} of 2^32 values round differently, e.g. {examples}"
