"""HIP graph capture of a multi-tensor step (GPU).  Once a list's descriptor
table is cached (first, eager call), a call only enqueues kernels, so it can
be captured; each replay repeats the captured step (same step counter and
seed) on the evolving state.  Checked replay by replay against the same
steps run eagerly on a copy, with eager work and synchronizations between
the replays; the NVFP4 current-scaling format's three kernels included.
With madd_multi_tensor_step_dev the hyper-parameters come from device
memory, so one capture replays successive steps."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_10611_amd import binding as B
from paper_2607_10611_amd import workloads as W
from gpu_parity_util import encode_nv_current

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
            q, s = encode_nv_current(x) if f == "nvfp4_current" else oracle.encode_nv(x)
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


def dev_scalars(h):
    raw = np.frombuffer(B.prepare_scalars(h), dtype=np.uint8).copy()
    return torch.from_numpy(raw).cuda()


def assert_lists_equal(a, b, tag):
    for k in ("w", "s", "c", "m", "v", "ve", "g"):
        for x, y in zip(a[k], b[k]):
            if x is not None:
                assert torch.equal(x.view(torch.uint8), y.view(torch.uint8)), (tag, k)


def test_device_scalars_give_the_bits_of_host_scalars():
    """Eager madd_multi_tensor_step_dev steps equal madd_multi_tensor_step
    steps, step counter and learning rate changing from step to step."""
    a, fmts = state(5)
    b, _ = state(5)
    tla, tlb = tl_of(a, fmts), tl_of(b, fmts)
    gen = torch.Generator(device="cuda")
    for t in range(1, 4):
        gen.manual_seed(t)
        for ga, gb in zip(a["g"], b["g"]):
            ga.normal_(0, 1e-3, generator=gen)
            gb.copy_(ga)
        h = W.hparams("c2", step=t, lr_add=1e-3 * t, lr_mul=2e-3 / t)
        B.madd_multi_tensor_step_dev(tla, h, dev_scalars(h))
        B.madd_multi_tensor_step(tlb, h)
        torch.cuda.synchronize()
        assert_lists_equal(a, b, t)


def test_captured_step_with_device_scalars_replays_successive_steps():
    """One capture of madd_multi_tensor_step_dev; before each replay the
    device scalars are rewritten for the next step (counter, learning rates),
    and every replay equals an eager step with those hyper-parameters."""
    a, fmts = state(6)
    b, _ = state(6)
    tla, tlb = tl_of(a, fmts), tl_of(b, fmts)
    h0 = W.hparams("c2", step=1)
    sc = dev_scalars(h0)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(0)
    for ga, gb in zip(a["g"], b["g"]):
        ga.normal_(0, 1e-3, generator=gen)
        gb.copy_(ga)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        B.madd_multi_tensor_step_dev(tla, h0, sc)    # eager: caches the descriptor tables
    torch.cuda.current_stream().wait_stream(s)
    B.madd_multi_tensor_step(tlb, h0)
    torch.cuda.synchronize()
    assert_lists_equal(a, b, "eager")
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        B.madd_multi_tensor_step_dev(tla, h0, sc)
    for t in range(2, 7):
        h = W.hparams("c2", step=t, lr_add=1e-3 / t, seed=1000 + t)
        sc.copy_(dev_scalars(h))                     # the next step's scalars, written eagerly
        gen.manual_seed(t)
        for ga, gb in zip(a["g"], b["g"]):
            ga.normal_(0, 1e-3, generator=gen)
            gb.copy_(ga)
        torch.cuda.synchronize()
        graph.replay()
        B.madd_multi_tensor_step(tlb, h)
        torch.cuda.synchronize()
        assert_lists_equal(a, b, t)


def other_lists(k, n=2048 + 8):
    """k small lists of their own buffers (each a distinct descriptor table)."""
    out = []
    for i in range(k):
        w = torch.zeros(n, dtype=torch.int16, device="cuda")
        g, m, v, ve = (torch.full((n,), 1e-3 * (i + 1), device="cuda") for _ in range(4))
        out.append(B.TensorList([w], ["bf16"], [g], [m], [v], [ve]))
    return out


def test_captured_step_survives_forty_other_lists():
    """The descriptor table a captured step reads is pinned: after 40 other
    lists are stepped eagerly (more than the cache keeps unpinned, so tables
    are recycled meanwhile), replays still equal eager steps."""
    a, fmts = state(8)
    b, _ = state(8)
    tla, tlb = tl_of(a, fmts), tl_of(b, fmts)
    h = W.hparams("c2", step=3)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        B.madd_multi_tensor_step(tla, h)          # eager: caches the table
    torch.cuda.current_stream().wait_stream(s)
    B.madd_multi_tensor_step(tlb, h)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        B.madd_multi_tensor_step(tla, h)
    others = other_lists(40)
    gen = torch.Generator(device="cuda")
    for r in range(3):
        for tl in others:                         # 40 eager steps of other lists
            B.madd_multi_tensor_step(tl, W.hparams("c2", step=r + 1))
        gen.manual_seed(50 + r)
        for ga, gb in zip(a["g"], b["g"]):
            ga.normal_(0, 1e-3, generator=gen)
            gb.copy_(ga)
        torch.cuda.synchronize()
        graph.replay()
        B.madd_multi_tensor_step(tlb, h)
        torch.cuda.synchronize()
        assert_lists_equal(a, b, f"replay {r}")


def test_list_first_seen_during_capture_is_refused():
    """A list the library has not seen before cannot be captured (its table
    would have to be allocated and written inside the capture): the call
    returns MADD_ECAPTURE and touches nothing; stepped once outside the
    capture, the list captures.  (Tables are cached by content -- pointers,
    sizes, index bases -- and the allocator may hand this test the addresses
    of an earlier test's tensors, so an index base no other call uses makes
    the list new.)"""
    a, fmts = state(9)
    b, _ = state(9)
    tla, tlb = tl_of(a, fmts), tl_of(b, fmts)
    for ga, gb in zip(a["g"], b["g"]):
        ga.fill_(1e-3)
        gb.fill_(1e-3)
    torch.cuda.synchronize()
    h = W.hparams("c2", step=1)
    base = 3 * 2 ** 40 + 4096
    graph = torch.cuda.CUDAGraph()
    with pytest.raises(B.MaddError, match="ECAPTURE"):
        with torch.cuda.graph(graph):
            B.madd_multi_tensor_step(tla, h, index_base=base)
    torch.cuda.synchronize()
    assert_lists_equal(a, b, "refused capture")
    B.madd_multi_tensor_step(tla, h, index_base=base)
    B.madd_multi_tensor_step(tlb, h, index_base=base)
    torch.cuda.synchronize()
    assert_lists_equal(a, b, "eager after refusal")


def test_allocation_free_step_captures_a_list_never_stepped_before():
    """madd_multi_tensor_step_noalloc writes its tables on the stream, so a
    graph can capture a list the library has never seen; each replay rewrites
    the tables and equals an eager step, with other lists stepped through the
    same entry point (same fixed table array) between the replays."""
    a, fmts = state(10)
    b, _ = state(10)
    tla, tlb = tl_of(a, fmts), tl_of(b, fmts)
    h = W.hparams("c2", step=4)
    others = other_lists(3)
    B.madd_multi_tensor_step_noalloc(others[0], W.hparams("c2", step=1))  # first call on the GPU
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        B.madd_multi_tensor_step_noalloc(tla, h)
    gen = torch.Generator(device="cuda")
    for r in range(3):
        for tl in others:
            B.madd_multi_tensor_step_noalloc(tl, W.hparams("c2", step=r + 1))
        gen.manual_seed(70 + r)
        for ga, gb in zip(a["g"], b["g"]):
            ga.normal_(0, 1e-3, generator=gen)
            gb.copy_(ga)
        torch.cuda.synchronize()
        graph.replay()
        B.madd_multi_tensor_step(tlb, h)
        torch.cuda.synchronize()
        assert_lists_equal(a, b, f"replay {r}")
