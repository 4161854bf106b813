"""Seeded synthetic inputs for the M+Adam step: parameter lists, initial
weights and per-step gradients.

This module holds none of the update's arithmetic.  It produces fp32 values
(initial weights, gradients) and hyper-parameter settings; rounding the
initial weights into a storage format is left to whichever implementation
consumes them.  Both the HIP path and the CPU oracle take their inputs from
here, so they see identical bits.

The paper trains LLaMA-style models on C4; neither the dataset nor trained
weights are used here.  The lists below have the shapes of the benchmark
models and the value distributions stated for each configuration:

  c1  one 1024x1024 matrix, bf16, w ~ N(0, 0.02), g ~ N(0, 1e-3), RNE
  c2  GPT-2-small list (124,439,808 params, 148 tensors), bf16, SR;
      g ~ N(0, s_k) with s_k log-uniform in [1e-5, 1e-2] per tensor
  c3  Llama-1.1B list (1,100,048,384 params, 201 tensors), bf16, SR;
      gradients as c2, then 5% exact zeros and 0.1% outliers x100
  c4  c3 list in FP8 (E4M3; E5M2 variant), all weights N(0, 0.02)
  c5  Llama-7B list (6,738,415,616 params, 291 tensors), bf16, SR,
      gradients as c2

Initial weights by tensor kind: matrices and embeddings N(0, 0.02), norm
gains 1.0, biases 0.0 (c1 and c4: N(0, 0.02) for every tensor).
Seeds: numpy SeedSequence(20260701) with spawn key (config, purpose, tensor,
step) on the CPU; a torch generator seeded from the same key on the GPU.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

ROOT_SEED = 20260701
SR_SEED = 0x4D414444  # "MADD"

DEFAULT_HPARAMS = dict(lr_add=1e-3, lr_mul=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, tau=1e-8,
                       r_max=0.75, eps0=0.0, g_max=math.inf, d_mult_max=math.inf, w_max=math.inf,
                       bias_correction=1, rounding="sr", seed=SR_SEED, step=1)


@dataclass(frozen=True)
class TensorSpec:
    name: str
    shape: tuple
    kind: str  # "matrix" | "norm" | "bias"

    @property
    def numel(self) -> int:
        return int(np.prod(self.shape))


def _gpt2_small():
    d, ff, vocab, ctx, L = 768, 3072, 50257, 1024, 12
    out = [TensorSpec("wte", (vocab, d), "matrix"), TensorSpec("wpe", (ctx, d), "matrix")]
    for i in range(L):
        p = f"h{i}."
        out += [TensorSpec(p + "ln1.w", (d,), "norm"), TensorSpec(p + "ln1.b", (d,), "bias"),
                TensorSpec(p + "attn.qkv.w", (d, 3 * d), "matrix"),
                TensorSpec(p + "attn.qkv.b", (3 * d,), "bias"),
                TensorSpec(p + "attn.proj.w", (d, d), "matrix"),
                TensorSpec(p + "attn.proj.b", (d,), "bias"),
                TensorSpec(p + "ln2.w", (d,), "norm"), TensorSpec(p + "ln2.b", (d,), "bias"),
                TensorSpec(p + "mlp.fc.w", (d, ff), "matrix"),
                TensorSpec(p + "mlp.fc.b", (ff,), "bias"),
                TensorSpec(p + "mlp.proj.w", (ff, d), "matrix"),
                TensorSpec(p + "mlp.proj.b", (d,), "bias")]
    out += [TensorSpec("lnf.w", (d,), "norm"), TensorSpec("lnf.b", (d,), "bias")]
    return out


def _llama(d, ff, layers, vocab, kv_dim):
    out = [TensorSpec("embed", (vocab, d), "matrix")]
    for i in range(layers):
        p = f"l{i}."
        out += [TensorSpec(p + "q", (d, d), "matrix"), TensorSpec(p + "k", (kv_dim, d), "matrix"),
                TensorSpec(p + "v", (kv_dim, d), "matrix"), TensorSpec(p + "o", (d, d), "matrix"),
                TensorSpec(p + "gate", (ff, d), "matrix"), TensorSpec(p + "up", (ff, d), "matrix"),
                TensorSpec(p + "down", (d, ff), "matrix"),
                TensorSpec(p + "attn_norm", (d,), "norm"), TensorSpec(p + "mlp_norm", (d,), "norm")]
    out += [TensorSpec("norm", (d,), "norm"), TensorSpec("lm_head", (vocab, d), "matrix")]
    return out


# name -> description of the workload
CONFIGS = {
    "c1": dict(id=1, specs=lambda: [TensorSpec("w", (1024, 1024), "matrix")], wfmt="bf16",
               rounding="rne", steps=10, grad="fixed", init="normal_all"),
    "c2": dict(id=2, specs=_gpt2_small, wfmt="bf16", rounding="sr", steps=100, grad="loguniform",
               init="by_kind"),
    "c3": dict(id=3, specs=lambda: _llama(2048, 5632, 22, 32000, 256), wfmt="bf16", rounding="sr",
               steps=10, grad="loguniform_sparse", init="by_kind"),
    "c4": dict(id=4, specs=lambda: _llama(2048, 5632, 22, 32000, 256), wfmt="e4m3", rounding="sr",
               steps=10, grad="loguniform_sparse", init="normal_all"),
    "c5": dict(id=5, specs=lambda: _llama(4096, 11008, 32, 32000, 4096), wfmt="bf16",
               rounding="sr", steps=20, grad="loguniform", init="by_kind"),
}

PURPOSE_INIT, PURPOSE_GRAD, PURPOSE_SIGMA = 0, 1, 2


def specs(cfg: str):
    return CONFIGS[cfg]["specs"]()


def total_params(cfg: str) -> int:
    return sum(s.numel for s in specs(cfg))


def hparams(cfg: str, step: int = 1, **over) -> dict:
    hp = dict(DEFAULT_HPARAMS)
    hp["rounding"] = CONFIGS[cfg]["rounding"]
    hp["step"] = step
    hp.update(over)
    return hp


def _rng(cfg_id: int, purpose: int, tensor: int, step: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence(ROOT_SEED,
                                                        spawn_key=(cfg_id, purpose, tensor, step)))


def torch_seed(cfg_id: int, purpose: int, tensor: int, step: int = 0) -> int:
    ss = np.random.SeedSequence(ROOT_SEED, spawn_key=(cfg_id, purpose, tensor, step))
    return int(ss.generate_state(1, dtype=np.uint64)[0] & 0x7FFFFFFFFFFFFFFF)


def sigmas(cfg: str) -> np.ndarray:
    """Per-tensor gradient scale."""
    c = CONFIGS[cfg]
    n = len(specs(cfg))
    if c["grad"] == "fixed":
        return np.full(n, 1e-3)
    u = _rng(c["id"], PURPOSE_SIGMA, 0).uniform(math.log(1e-5), math.log(1e-2), size=n)
    return np.exp(u)


def _init_value(cfg: str, spec: TensorSpec):
    c = CONFIGS[cfg]
    if c["init"] == "normal_all" or spec.kind == "matrix":
        return None  # random
    return 1.0 if spec.kind == "norm" else 0.0


def init_fp32(cfg: str, i: int, n: int | None = None) -> np.ndarray:
    """Initial fp32 weights of tensor i (first n elements if n is given)."""
    spec = specs(cfg)[i]
    n = spec.numel if n is None else n
    const = _init_value(cfg, spec)
    if const is not None:
        return np.full(n, const, dtype=np.float32)
    x = _rng(CONFIGS[cfg]["id"], PURPOSE_INIT, i).standard_normal(n, dtype=np.float32) * np.float32(0.02)
    if CONFIGS[cfg]["wfmt"] in ("e4m3", "e5m2"):
        lim = np.float32(448.0 if CONFIGS[cfg]["wfmt"] == "e4m3" else 57344.0)
        x = np.clip(x, -lim, lim)
    return x.astype(np.float32)


def grad_fp32(cfg: str, i: int, step: int, n: int | None = None, sigma: float | None = None
              ) -> np.ndarray:
    """fp32 gradient of tensor i at step t (first n elements if n is given)."""
    c = CONFIGS[cfg]
    spec = specs(cfg)[i]
    n = spec.numel if n is None else n
    s = np.float32(sigmas(cfg)[i] if sigma is None else sigma)
    rng = _rng(c["id"], PURPOSE_GRAD, i, step)
    g = rng.standard_normal(n, dtype=np.float32) * s
    if c["grad"] == "loguniform_sparse":
        u = rng.random(n, dtype=np.float32)
        g = np.where(u < 0.05, np.float32(0.0), np.where(u > 0.999, g * np.float32(100.0), g))
    return g.astype(np.float32)


# ---------------------------------------------------------------------------
# Device-side generation for the large lists (torch on the GPU)
# ---------------------------------------------------------------------------

def init_fp32_device(cfg: str, i: int, device="cuda"):
    import torch
    spec = specs(cfg)[i]
    const = _init_value(cfg, spec)
    if const is not None:
        return torch.full((spec.numel,), const, dtype=torch.float32, device=device)
    gen = torch.Generator(device=device)
    gen.manual_seed(torch_seed(CONFIGS[cfg]["id"], PURPOSE_INIT, i))
    x = torch.randn(spec.numel, generator=gen, device=device, dtype=torch.float32) * 0.02
    if CONFIGS[cfg]["wfmt"] in ("e4m3", "e5m2"):
        lim = 448.0 if CONFIGS[cfg]["wfmt"] == "e4m3" else 57344.0
        x.clamp_(-lim, lim)
    return x


def grad_fp32_device_(cfg: str, i: int, step: int, out, sigma: float | None = None):
    """Fill the fp32 device tensor `out` with tensor i's gradient at step t."""
    import torch
    c = CONFIGS[cfg]
    s = float(sigmas(cfg)[i] if sigma is None else sigma)
    gen = torch.Generator(device=out.device)
    gen.manual_seed(torch_seed(c["id"], PURPOSE_GRAD, i, step))
    torch.randn(out.shape, generator=gen, device=out.device, dtype=torch.float32, out=out)
    out.mul_(s)
    if c["grad"] == "loguniform_sparse":
        u = torch.rand(out.shape, generator=gen, device=out.device, dtype=torch.float32)
        out.masked_fill_(u < 0.05, 0.0)
        out.mul_(torch.where(u > 0.999, 100.0, 1.0))
        del u
    return out


def low_precision_master_plan(cfg: str, linear_fmt: str = "e4m3"):
    """Per-tensor storage for the low-precision master settings of Section 4.2:
    attention and MLP linear weights block-scaled in ``linear_fmt`` -- "e4m3"
    (FP16 scale per 128 elements; the FP8/FP8 setting), "nvfp4" (E2M1 with an
    E4M3 scale per 16 elements and an fp32 scale per tensor; the 4-bit
    setting; "nvfp4_current" derives that scale anew every step) or "mxfp4"
    (E2M1 with an E8M0 scale per 32 elements) -- each
    with a bf16 compute copy; embeddings, norms and the LM head in bf16.  Returns (weight format, block-scaled, compute copy) per
    tensor."""
    plan = []
    for s in specs(cfg):
        linear = s.kind == "matrix" and s.name not in ("embed", "lm_head", "wte", "wpe")
        plan.append((linear_fmt, True, True) if linear else ("bf16", False, False))
    return plan


def fp8_master_plan(cfg: str):
    """The FP8-master setting: low_precision_master_plan with E4M3."""
    return low_precision_master_plan(cfg, "e4m3")


# ---------------------------------------------------------------------------
# Appendix B's BF16-stored matrix-fitting diagnostic: five regimes
# ---------------------------------------------------------------------------

TOY_N = 4096
TOY_REGIMES = ("sign_flip", "zero_revival", "small", "large", "mixed")


def toy_regime(name: str, seed: int = 0):
    """Targets w*, initial weights w0 and per-entry loss scales c of one regime
    (n = 4096 entries), as fp32 arrays.

    sign_flip: w* in {-1, +1}, w0 = -w*, c = 1; zero_revival: w* in {-1, +1},
    w0 = 0, c = 1; small: w* = 1e-4 z, w0 = 0, c = 1e8; large:
    w* = 900 max(|z|, 1/900), w0 = 100, c = 1e-7; mixed: first half small,
    second half large (z ~ N(0, 1))."""
    rng = np.random.default_rng(np.random.SeedSequence(ROOT_SEED, spawn_key=(6, 0, seed)))
    n = TOY_N
    z = rng.standard_normal(n)
    if name == "sign_flip":
        ws = rng.choice([-1.0, 1.0], n)
        w0, c = -ws, np.ones(n)
    elif name == "zero_revival":
        ws = rng.choice([-1.0, 1.0], n)
        w0, c = np.zeros(n), np.ones(n)
    elif name == "small":
        ws, w0, c = 1e-4 * z, np.zeros(n), np.full(n, 1e8)
    elif name == "large":
        ws, w0, c = 900.0 * np.maximum(np.abs(z), 1.0 / 900.0), np.full(n, 100.0), np.full(n, 1e-7)
    elif name == "mixed":
        h = n // 2
        ws = np.concatenate([1e-4 * z[:h], 900.0 * np.maximum(np.abs(z[h:]), 1.0 / 900.0)])
        w0 = np.concatenate([np.zeros(h), np.full(n - h, 100.0)])
        c = np.concatenate([np.full(h, 1e8), np.full(n - h, 1e-7)])
    else:
        raise KeyError(name)
    return ws.astype(np.float32), w0.astype(np.float32), c.astype(np.float32)
