"""Every storage code through the step (GPU): each of the 65536 bf16 codes and
the 256 E4M3 and E5M2 codes, as weights of one tensor stepped with both
learning rates zero (so w' = w for every finite weight), the moments
updated from seeded gradients, and the bf16 compute copy of the result.

Each code's new code and compute copy are compared bit for bit with the
oracle, the moments to the parity bar; independently of it, a finite code must come back unchanged and
its compute copy must be the bf16 rounding of the value torch decodes the
code to (torch's bfloat16 / float8 types).  Infinite and NaN weights follow
the update's own arithmetic (inf x 0 is NaN), as the oracle computes it."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_10611_amd import binding as B
from paper_2607_10611_amd import workloads as W
from gpu_parity_util import assert_state_equal

pytestmark = pytest.mark.gpu

FMTS = {"bf16": (65536, torch.int16, np.uint16, torch.bfloat16),
        "e4m3": (256, torch.uint8, np.uint8, torch.float8_e4m3fn),
        "e5m2": (256, torch.uint8, np.uint8, torch.float8_e5m2)}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    B.lib()
    yield
    torch.cuda.synchronize()


@pytest.mark.parametrize("fmt", list(FMTS))
@pytest.mark.parametrize("rounding", ["rne", "sr"])
def test_every_code_steps_back_to_itself_with_zero_learning_rates(fmt, rounding):
    n, dt, npdt, tdt = FMTS[fmt]
    codes = np.arange(n, dtype=np.int64).astype(npdt)
    h = W.hparams("c2", step=3, lr_add=0.0, lr_mul=0.0, rounding=rounding, seed=99)
    rng = np.random.default_rng(4)
    g = (rng.normal(0, 1, n) * 1e-3).astype(np.float32)
    w = torch.from_numpy(codes.view(np.int16) if fmt == "bf16" else codes.copy()).cuda()
    m, v, ve = (torch.zeros(n, device="cuda") for _ in range(3))
    cp = torch.zeros(n, dtype=torch.int16, device="cuda")
    B.madd_step(w, fmt, torch.from_numpy(g).cuda(), m, v, ve, h, copy=cp)
    hw, hm, hv, hve = codes.copy(), *(np.zeros(n, np.float32) for _ in range(3))
    hcp = np.zeros(n, np.uint16)
    oracle.step(fmt, hw, g.copy(), hm, hv, hve, h, copy=hcp)
    torch.cuda.synchronize()
    gw = w.cpu().numpy().view(npdt)
    gcp = cp.cpu().numpy().view(np.uint16)
    assert np.array_equal(gw, hw), f"{fmt}: codes differ at {np.nonzero(gw != hw)[0][:5]}"
    assert np.array_equal(gcp, hcp), f"{fmt}: copies differ at {np.nonzero(gcp != hcp)[0][:5]}"
    # fp32 moments: the parity bar (within 2 ulp, NaN where NaN: NaN weights
    # make NaN exponent gradients, whose payloads are not compared)
    assert_state_equal(fmt, gw, hw, m.cpu().numpy(), hm, v.cpu().numpy(), hv,
                       ve.cpu().numpy(), hve)
    # independent of the oracle: finite weights keep their value (a zero may
    # change sign: w + w u_m + u_a adds signed zeros), and the copies are the
    # bf16 of torch's decoding
    def decoded(c):
        t = torch.from_numpy(c.view(np.int16) if fmt == "bf16" else c.copy())
        return t.view(tdt).to(torch.float32)
    val = decoded(codes)
    fin = torch.isfinite(val)
    assert bool((decoded(gw)[fin] == val[fin]).all())
    got_cp = torch.from_numpy(gcp.view(np.int16)).view(torch.bfloat16).to(torch.float32)
    assert bool((got_cp[fin] == val.to(torch.bfloat16).to(torch.float32)[fin]).all())
