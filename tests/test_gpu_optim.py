"""The torch.optim front end (paper_2607_10611_amd.optim.MAdam) against the
CPU oracle (GPU): every parameter's stored codes bit-exact and fp32 moments
within 2 ulp after each step, each parameter keyed by its own global index
base, with fp32 or bf16 gradients, fp32 / bf16 / stochastic bf16 moments,
bf16, fp32 and FP8 parameters, block-scaled master weights (FP8, MXFP4,
NVFP4) with bf16 compute copies, gaps (parameters without gradients),
state_dict round trips and a bf16 layer trained through autograd."""
import copy

import numpy as np
import pytest
import torch

import oracle
from paper_2607_10611_amd import binding as B
from paper_2607_10611_amd.optim import MAdam
from gpu_parity_util import HostState, assert_state_equal, encode_nv_current, oracle_step, to_host

pytestmark = pytest.mark.gpu

SHAPES = [(4096 + 40,), (1000,), (3, 2048 + 8), (33,), (64, 64)]
CODE = {torch.bfloat16: ("bf16", torch.int16, np.uint16), torch.float32: ("fp32", torch.int32, np.uint32),
        torch.float8_e4m3fn: ("e4m3", torch.uint8, np.uint8)}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    B.lib()
    yield
    torch.cuda.synchronize()


def make_params(seed, dtype=torch.bfloat16, grad_dtype=None):
    gen = torch.Generator().manual_seed(seed)
    ps = []
    for s in SHAPES:
        x = (torch.randn(s, generator=gen) * 0.02)
        if dtype == torch.float8_e4m3fn:
            x = x.clamp(-448, 448)
        p = torch.nn.Parameter(x.to(dtype).cuda())
        if grad_dtype is not None and grad_dtype != dtype:
            p.grad_dtype = None
        ps.append(p)
    return ps


def grads(seed, ps, dtype):
    gen = torch.Generator().manual_seed(seed)
    out = []
    for p in ps:
        g = torch.randn(p.shape, generator=gen) * 10.0 ** torch.empty(p.shape).uniform_(
            -6, -2, generator=gen)
        g[torch.rand(p.shape, generator=gen) < 0.05] = 0.0
        out.append(g.to(dtype))
    return out


def host_states(ps, sfmt):
    out = []
    for p in ps:
        fmt, it, nt = CODE[p.dtype]
        codes = to_host(p.detach().view(it).reshape(-1), nt)
        out.append(HostState(codes, p.numel(), sfmt=sfmt))
    return out


def group_hp(opt, p, step):
    g = next(gr for gr in opt.param_groups if any(q is p for q in gr["params"]))
    hp = {k: g[k] for k in ("lr_add", "lr_mul", "eps", "tau", "r_max", "eps0", "g_max",
                            "d_mult_max", "w_max", "rounding", "seed")}
    hp.update(beta1=g["betas"][0], beta2=g["betas"][1], bias_correction=int(g["bias_correction"]),
              step=step)
    return hp


def compare(tag, opt, ps, hs, sfmt):
    torch.cuda.synchronize()
    for i, (p, h) in enumerate(zip(ps, hs)):
        fmt, it, nt = CODE[p.dtype]
        st = opt.state[p]
        w = to_host(p.detach().view(it).reshape(-1), nt)
        sn = np.float32 if sfmt == "fp32" else np.uint16
        m, v, ve = (to_host(st[k], sn) for k in ("m", "v", "ve"))
        assert_state_equal(f"{tag} param {i}", w, h.w, m, h.m, v, h.v, ve, h.ve)


def oracle_steps(opt, ps, hs, gs, gfmt, have=None):
    for i, (p, h, g) in enumerate(zip(ps, hs, gs)):
        if have is not None and not have[i]:
            continue
        gh = g.reshape(-1).cpu()
        gh = gh.view(torch.int16).numpy().view(np.uint16) if gfmt == "bf16" else gh.numpy()
        oracle_step(CODE[p.dtype][0], h, gh.copy(), group_hp(opt, p, opt.state[p]["step"]),
                    gfmt=gfmt, index_base=opt._base[p])


@pytest.mark.parametrize("sfmt", ["fp32", "bf16", "bf16_sr"])
@pytest.mark.parametrize("gdt", [torch.float32, torch.bfloat16])
def test_madam_steps_match_the_oracle(sfmt, gdt):
    ps = make_params(1, grad_dtype=gdt)
    opt = MAdam([{"params": ps[:3]}, {"params": ps[3:], "lr_add": 3e-3, "lr_mul": 2e-3}],
                seed=0x5EED, state_format=sfmt)
    hs = host_states(ps, sfmt)
    gfmt = "fp32" if gdt == torch.float32 else "bf16"
    for t in range(1, 4):
        gs = grads(100 + t, ps, gdt)
        for p, g in zip(ps, gs):
            p.grad = g.cuda()
        opt.step()
        oracle_steps(opt, ps, hs, gs, gfmt)
        compare(f"{sfmt} {gfmt} t={t}", opt, ps, hs, sfmt)
    assert all(opt.state[p]["step"] == 3 for p in ps)


@pytest.mark.parametrize("dtype", [torch.float32, torch.float8_e4m3fn])
def test_fp32_and_fp8_parameters(dtype):
    ps = make_params(2, dtype=dtype, grad_dtype=torch.float32)
    opt = MAdam(ps, rounding="sr", seed=9)
    hs = host_states(ps, "fp32")
    for t in range(1, 3):
        gs = grads(200 + t, ps, torch.float32)
        for p, g in zip(ps, gs):
            p.grad = g.cuda()
        opt.step()
        oracle_steps(opt, ps, hs, gs, "fp32")
        compare(f"{dtype} t={t}", opt, ps, hs, "fp32")


def test_parameters_without_gradients_keep_the_others_keyed_by_their_own_bases():
    ps = make_params(3, grad_dtype=torch.float32)
    opt = MAdam(ps, seed=77)
    hs = host_states(ps, "fp32")
    pattern = [[1, 1, 1, 1, 1], [1, 0, 1, 0, 1], [0, 1, 1, 1, 1]]
    for t, have in enumerate(pattern, start=101):
        gs = grads(t, ps, torch.float32)
        for p, g, h in zip(ps, gs, have):
            p.grad = g.cuda() if h else None
        before = [p.detach().clone() for p in ps]
        opt.step()
        oracle_steps(opt, ps, hs, gs, "fp32", have=have)
        compare(f"gaps {have}", opt, ps, hs, "fp32")
        for p, b, h in zip(ps, before, have):
            if not h:
                assert torch.equal(p.detach().view(torch.int16), b.view(torch.int16))
    assert [opt.state[p]["step"] for p in ps] == [2, 2, 3, 2, 3]


def test_state_dict_round_trip_continues_bit_exact():
    for sfmt in ("fp32", "bf16"):
        ps = make_params(4, grad_dtype=torch.float32)
        opt = MAdam(ps, seed=3, state_format=sfmt)
        all_g = [grads(300 + t, ps, torch.float32) for t in range(4)]
        for t in range(2):
            for p, g in zip(ps, all_g[t]):
                p.grad = g.cuda()
            opt.step()
        sd = copy.deepcopy(opt.state_dict())
        qs = [torch.nn.Parameter(p.detach().clone()) for p in ps]
        for q in qs:
            q.grad_dtype = None
        opt2 = MAdam(qs, seed=3, state_format=sfmt)
        opt2.load_state_dict(sd)
        for p, q in zip(ps, qs):
            for k in ("m", "v", "ve"):
                assert opt2.state[q][k].dtype == opt.state[p][k].dtype
                assert torch.equal(opt2.state[q][k], opt.state[p][k])
        for t in range(2, 4):
            for p, q, g in zip(ps, qs, all_g[t]):
                p.grad = g.cuda()
                q.grad = g.cuda()
            opt.step()
            opt2.step()
        torch.cuda.synchronize()
        for p, q in zip(ps, qs):
            assert torch.equal(p.detach().view(torch.int16), q.detach().view(torch.int16))
            for k in ("m", "v", "ve"):
                assert torch.equal(opt.state[p][k], opt2.state[q][k])


def test_bf16_linear_layer_trained_through_autograd():
    torch.manual_seed(0)
    layer = torch.nn.Linear(64, 48, dtype=torch.bfloat16, device="cuda")
    ps = list(layer.parameters())
    opt = MAdam(ps, lr_add=1e-2, lr_mul=1e-2, seed=11)
    hs = host_states(ps, "fp32")
    x = torch.randn(128, 64, dtype=torch.bfloat16, device="cuda")
    y = torch.randn(128, 48, dtype=torch.bfloat16, device="cuda")
    losses = []
    for t in range(1, 6):
        opt.zero_grad(set_to_none=True)
        # fp32 products on the bf16 parameters: their gradients come back in bf16
        out = torch.nn.functional.linear(x.float(), layer.weight.float(), layer.bias.float())
        loss = ((out - y.float()) ** 2).mean()
        loss.backward()
        losses.append(float(loss.detach()))
        gs = [p.grad.detach().clone() for p in ps]
        opt.step()
        oracle_steps(opt, ps, hs, gs, "bf16")
        compare(f"linear t={t}", opt, ps, hs, "fp32")
    assert losses[-1] < losses[0]


def test_rejects_a_state_of_the_wrong_format():
    p = torch.nn.Parameter(torch.zeros(64, dtype=torch.bfloat16, device="cuda"))
    opt = MAdam([p], state_format="bf16")
    p.grad = torch.zeros_like(p)
    opt.step()
    opt.state[p]["m"] = torch.zeros(64, device="cuda")  # fp32 where bf16 moments live
    with pytest.raises(ValueError, match="bf16 moments"):
        opt.step()


def oracle_master(fmt, x):
    if fmt in ("e4m3", "e5m2"):
        return oracle.encode_block(fmt, x)
    return {"mxfp4": oracle.encode_mx, "nvfp4": oracle.encode_nv,
            "nvfp4_current": encode_nv_current}[fmt](x)


@pytest.mark.parametrize("master", ["e4m3", "e5m2", "mxfp4", "nvfp4", "nvfp4_current"])
def test_block_scaled_master_weights_with_bf16_compute_copies(master):
    """The paper's mixed list through the optimizer: block-scaled master
    weights for the 'linear' group (bf16 parameters hold the compute copy),
    bf16 storage for the rest; master codes, scales, compute copies and
    moments bit-exact against the oracle, which encodes its own starting
    codes from the same fp32 values."""
    gen = torch.Generator().manual_seed(5)
    lin = [torch.nn.Parameter((torch.randn(s, generator=gen) * 0.02).to(torch.bfloat16).cuda())
           for s in ((8, 128), (3, 512), (2048,))]
    rest = [torch.nn.Parameter((torch.randn(s, generator=gen) * 0.02).to(torch.bfloat16).cuda())
            for s in ((1000,), (33,))]
    for p in lin + rest:
        p.grad_dtype = None
    opt = MAdam([{"params": lin, "master_format": master}, {"params": rest}], seed=21,
                rounding="sr")
    hl = []
    for p in lin:
        q, sc = oracle_master(master, p.detach().float().cpu().numpy().reshape(-1))
        hl.append(HostState(q, p.numel(), scales=sc, copy=True))
    hr = host_states(rest, "fp32")
    for t in range(1, 4):
        gs = grads(400 + t, lin + rest, torch.float32)
        for p, g in zip(lin + rest, gs):
            p.grad = g.cuda()
        opt.step()
        for p, h, g in zip(lin, hl, gs[:len(lin)]):
            oracle_step(master, h, g.reshape(-1).numpy().copy(),
                        group_hp(opt, p, opt.state[p]["step"]), index_base=opt._base[p])
        oracle_steps(opt, rest, hr, gs[len(lin):], "fp32")
        torch.cuda.synchronize()
        for i, (p, h) in enumerate(zip(lin, hl)):
            st = opt.state[p]
            sc = to_host(st["scales"], np.uint8)
            if master in ("e4m3", "e5m2"):
                sc = sc.view(np.uint16)
            assert_state_equal(f"{master} t={t} param {i}", to_host(st["q"], np.uint8), h.w,
                               to_host(st["m"]), h.m, to_host(st["v"]), h.v, to_host(st["ve"]),
                               h.ve)
            assert np.array_equal(sc, h.scales), f"{master} t={t} param {i}: scales"
            cp = to_host(p.detach().view(torch.int16).reshape(-1), np.uint16)
            assert np.array_equal(cp, h.copy), f"{master} t={t} param {i}: compute copy"
        compare(f"{master} rest t={t}", opt, rest, hr, "fp32")


def test_state_dict_round_trip_keeps_master_codes_and_scales():
    gen = torch.Generator().manual_seed(6)
    ps = [torch.nn.Parameter((torch.randn(s, generator=gen) * 0.02).to(torch.bfloat16).cuda())
          for s in ((4, 128), (256,))]
    for p in ps:
        p.grad_dtype = None
    opt = MAdam(ps, master_format="nvfp4", seed=8)
    all_g = [grads(500 + t, ps, torch.float32) for t in range(3)]
    for p, g in zip(ps, all_g[0]):
        p.grad = g.cuda()
    opt.step()
    sd = copy.deepcopy(opt.state_dict())
    qs = [torch.nn.Parameter(p.detach().clone()) for p in ps]
    for q in qs:
        q.grad_dtype = None
    opt2 = MAdam(qs, master_format="nvfp4", seed=8)
    opt2.load_state_dict(sd)
    for p, q in zip(ps, qs):
        for k in ("q", "scales", "m", "v", "ve"):
            assert opt2.state[q][k].dtype == opt.state[p][k].dtype, k
            assert torch.equal(opt2.state[q][k], opt.state[p][k]), k
    for t in (1, 2):
        for p, q, g in zip(ps, qs, all_g[t]):
            p.grad = g.cuda()
            q.grad = g.cuda()
        opt.step()
        opt2.step()
    torch.cuda.synchronize()
    for p, q in zip(ps, qs):
        assert torch.equal(p.detach().view(torch.int16), q.detach().view(torch.int16))
        for k in ("q", "scales", "m", "v", "ve"):
            assert torch.equal(opt.state[p][k], opt2.state[q][k]), k


def test_capturable_step_replays_equal_eager_steps():
    """MAdam(capturable=True): one eager step, one captured step, then
    prepare_replay() + replay for the following steps; every replay equals
    an eager MAdam step on a copy (a bf16 group and an E4M3-master group)."""
    def build(seed):
        gen = torch.Generator().manual_seed(seed)
        lin = [torch.nn.Parameter((torch.randn(s, generator=gen) * 0.02).to(torch.bfloat16).cuda())
               for s in ((4, 128), (1024,))]
        rest = [torch.nn.Parameter((torch.randn(s, generator=gen) * 0.02).to(torch.bfloat16).cuda())
                for s in ((1000,), (33,))]
        for p in lin + rest:
            p.grad_dtype = None
            p.grad = torch.zeros(p.shape, device="cuda")
        return lin, rest
    la, ra = build(7)
    lb, rb = build(7)
    groups = lambda lin, rest: [{"params": lin, "master_format": "e4m3"},  # noqa: E731
                                {"params": rest, "lr_add": 2e-3}]
    opt_a = MAdam(groups(la, ra), seed=31, capturable=True)
    opt_b = MAdam(groups(lb, rb), seed=31)
    pa, pb = la + ra, lb + rb

    def new_grads(t):
        for p, q, g in zip(pa, pb, grads(600 + t, pa, torch.float32)):
            p.grad.copy_(g)   # in place: the captured step reads these tensors
            q.grad.copy_(g)

    def check(tag):
        torch.cuda.synchronize()
        for p, q in zip(pa, pb):
            assert torch.equal(p.detach().view(torch.int16), q.detach().view(torch.int16)), tag
            for k in ("m", "v", "ve", "q", "scales"):
                if k in opt_a.state[p]:
                    assert torch.equal(opt_a.state[p][k], opt_b.state[q][k]), (tag, k)
            assert opt_a.state[p]["step"] == opt_b.state[q]["step"], tag

    new_grads(1)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        opt_a.step()                    # eager: state, tables, scalars of step 1
    torch.cuda.current_stream().wait_stream(side)
    opt_b.step()
    check("eager")
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        opt_a.step()
    check("after capture")              # capturing ran nothing
    for t in range(2, 6):
        new_grads(t)
        opt_a.prepare_replay()
        graph.replay()
        opt_b.step()
        check(f"replay t={t}")
