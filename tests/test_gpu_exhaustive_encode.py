"""The library's round-to-nearest-even encoders (madd_encode_weights; the
same codecs the step uses with rounding = RNE) on every one of the 2^32 fp32
bit patterns, against torch's conversions on the device (GPU).  torch's
float8 casts do not saturate, so finite overflow and infinities are clamped
to the largest finite value first (the storage formats saturate); NaN
inputs must give the canonical NaN code (0x7FC0 bf16, 0x7F FP8)."""
import pytest
import torch

from paper_2607_10611_amd import binding as B

pytestmark = pytest.mark.gpu

CHUNK = 1 << 28
FMTS = {"bf16": (torch.int16, torch.bfloat16, None, 0x7FC0),
        "e4m3": (torch.uint8, torch.float8_e4m3fn, 448.0, 0x7F),
        "e5m2": (torch.uint8, torch.float8_e5m2, 57344.0, 0x7F)}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    B.lib()
    yield
    torch.cuda.synchronize()


@pytest.mark.parametrize("fmt", list(FMTS))
def test_rne_encode_on_every_fp32_input(fmt):
    code_t, ref_t, fmax, nan_code = FMTS[fmt]
    w = torch.empty(CHUNK, dtype=code_t, device="cuda")
    bad = 0
    examples = []
    for c in range((1 << 32) // CHUNK):
        bits = torch.arange(c * CHUNK, (c + 1) * CHUNK, dtype=torch.int64, device="cuda")
        x = bits.to(torch.int32).view(torch.float32)
        del bits
        B.madd_encode_weights(x, w, fmt)
        nan = torch.isnan(x)
        xr = x if fmax is None else x.clamp(-fmax, fmax)
        ref = xr.to(ref_t).view(code_t)
        got = w
        if fmt == "bf16":
            mism = (got != ref) & ~nan
            nan_bad = nan & (got != torch.tensor(nan_code, dtype=torch.int16, device="cuda"))
        else:
            mism = (got != ref) & ~nan
            nan_bad = nan & (got != nan_code)
        nb = int(mism.sum()) + int(nan_bad.sum())
        if nb and not examples:
            idx = torch.nonzero(mism | nan_bad)[:5, 0]
            examples = [(hex(c * CHUNK + int(i)), int(got[i]), int(ref[i])) for i in idx]
        bad += nb
        del x, nan, xr, ref
    assert bad == 0, f"{fmt}: {bad} of 2^32 inputs encode differently, e.g. {examples}"
