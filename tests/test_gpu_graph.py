"""HIP graph capture of a multi-tensor step (GPU).  Once a list's descriptor
table is cached (first, eager call), a call only enqueues kernels, so it can
be captured; each replay repeats the captured step (same step counter and
seed) on the evolving state.  Checked replay by replay against the same
steps run eagerly on a copy, with eager work and synchronizations between
the replays; the NVFP4 current-scaling format's three kernels included."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_10611_amd import binding as B
from paper_2607_10611_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    B.lib()
    yield
    torch.cuda.synchronize()


def state(seed):
    rng = np.random.default_rng(seed)
    sizes, fmts = [8192 * 3 + 64, 2048 + 16, 4096], ["nvfp4_current", "nvfp4", "bf16"]
    st = dict(w=[], s=[], c=[], m=[], v=[], ve=[], g=[])
    for n, f in zip(sizes, fmts):
        x = rng.normal(0, 0.02, n).astype(np.float32)
        if f == "bf16":
            st["w"].append(torch.from_numpy(oracle.encode_array("bf16", x).view(np.int16)).cuda())
            st["s"].append(None)
            st["c"].append(None)
        else:
            q, s = oracle.encode_nv_current(x) if f == "nvfp4_current" else oracle.encode_nv(x)
            st["w"].append(torch.from_numpy(q).cuda())
            st["s"].append(torch.from_numpy(s).cuda())
            st["c"].append(torch.zeros(n, dtype=torch.int16, device="cuda"))
        for k in ("m", "v", "ve"):
            st[k].append(torch.zeros(n, device="cuda"))
        st["g"].append(torch.empty(n, device="cuda"))
    return st, fmts


def tl_of(st, fmts):
    return B.TensorList(st["w"], fmts, st["g"], st["m"], st["v"], st["ve"], scales=st["s"],
                        copies=st["c"])


def test_captured_step_replays_equal_eager_steps():
    a, fmts = state(3)
    b, _ = state(3)
    tla, tlb = tl_of(a, fmts), tl_of(b, fmts)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(99)
    for ga, gb in zip(a["g"], b["g"]):
        ga.normal_(0, 1e-3, generator=gen)
        gb.copy_(ga)
    torch.cuda.synchronize()
    h = W.hparams("c2", step=7)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        B.madd_multi_tensor_step(tla, h)          # eager call: caches the descriptor tables
    torch.cuda.current_stream().wait_stream(s)
    B.madd_multi_tensor_step(tlb, h)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        B.madd_multi_tensor_step(tla, h)
    for r in range(4):
        gen.manual_seed(r)
        for ga, gb in zip(a["g"], b["g"]):        # eager work between replays: fresh gradients
            ga.normal_(0, 1e-3, generator=gen)
            gb.copy_(ga)
        torch.cuda.synchronize()
        graph.replay()
        B.madd_multi_tensor_step(tlb, h)
        torch.cuda.synchronize()
        for k in ("w", "s", "c", "m", "v", "ve", "g"):
            for x, y in zip(a[k], b[k]):
                if x is not None:
                    assert torch.equal(x.view(torch.uint8), y.view(torch.uint8)), (r, k)
