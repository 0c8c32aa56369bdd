"""Seeded synthetic inputs shaped like the paper's workloads.

This module holds NO arithmetic of the method: it only draws golden tensors
and perturbed test tensors (Gaussian relative noise, bf16 rounding, planted NaN
and bit flips at positions it draws itself).  Bit flips that belong to the
method -- the random-bit-flip injector -- are applied by the caller with the
GPU library or with the oracle, never here.

The paper's own data (CIFAR-10/100, CoNLL-2003, ImageNet, trained weights,
recorded training tensors) is not available; these tensors stand in for them
with the shapes and value statistics of each workload:

  1. one f32 [1024, 1024] pair, G ~ N(0,1), T = G*(1+u), u ~ U(-2^-20, 2^-20),
     plus 16 single-bit flips at drawn positions/bits;
  2. 32 activation-shaped f32 [8, 512, 4096] pairs, G ~ N(0,1) with 0.1 %
     outliers x100, T = bf16-rounded G widened back;
  3. a GPT-style 1.3B checkpoint pair (292 tensors), G ~ N(0, 0.02),
     T = G*(1 + 1e-6 z), NaN planted at rate 1e-9;
  4. 1000 replayed calls of one f16 [4096, 4096] output, every 10th call with
     bit flips at rate 1e-7 (applied by the injector);
  5. a Llama-7B-shaped checkpoint with two Adam moments (873 f32 tensors),
     T = G*(1 + 1e-7 z), then exponent-bit flips at rate 1e-8 (applied by the
     injector).

Seeds: data seed 1000*c + k for tensor k of workload c; injector seed
0xC0FFEE00 + 1000*c + k.
"""
from __future__ import annotations

import numpy as np
import torch

BINS = (-40, 24, 64)           # 64 log2 bins over |err| in [2^-40, 2^24)
THRESHOLDS = (1e-6, 1e-3)      # absolute thresholds for mismatch counts

INJ_SEED_BASE = 0xC0FFEE00


def data_seed(config: int, k: int) -> int:
    return 1000 * config + k


def inject_seed(config: int, k: int) -> int:
    return INJ_SEED_BASE + 1000 * config + k


def _gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


# --------------------------------------------------------------------------
# Workload 1: single f32 pair with 16 planted single-bit flips.
# --------------------------------------------------------------------------
def config1(shape=(1024, 1024), seed: int | None = None, nflips: int = 16):
    """Host numpy arrays (G, T), float32."""
    rng = np.random.Generator(np.random.PCG64(data_seed(1, 0) if seed is None else seed))
    n = int(np.prod(shape))
    G = rng.standard_normal(n).astype(np.float32)
    u = rng.uniform(-2.0 ** -20, 2.0 ** -20, n)
    T = (G.astype(np.float64) * (1.0 + u)).astype(np.float32)
    k = min(nflips, n)
    pos = rng.choice(n, k, replace=False)
    bits = rng.integers(0, 32, k)
    Tb = T.view(np.uint32)
    Tb[pos] ^= (np.uint32(1) << bits.astype(np.uint32))
    return G.reshape(shape), T.reshape(shape)


# --------------------------------------------------------------------------
# Workload 2: activation-shaped batch, bf16 rounding error.
# --------------------------------------------------------------------------
CONFIG2_COUNT = 32
CONFIG2_SHAPE = (8, 512, 4096)


def config2_pair(k: int, device="cpu", shape=CONFIG2_SHAPE):
    g = _gen(device, data_seed(2, k))
    G = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    outlier = torch.rand(shape, generator=g, device=device) < 1e-3
    G = torch.where(outlier, G * 100.0, G)
    T = G.to(torch.bfloat16).to(torch.float32)   # round-to-nearest-even, widened back
    return G.contiguous(), T.contiguous()


# --------------------------------------------------------------------------
# Workload 3: GPT-style 1.3B checkpoint pair (24 layers, hidden 2048,
# FFN 8192, vocab 50304, context 2048).
# --------------------------------------------------------------------------
def gpt13b_shapes():
    h, f, v, ctx = 2048, 8192, 50304, 2048
    out = [("wte", (v, h)), ("wpe", (ctx, h))]
    for i in range(24):
        p = f"h{i}."
        out += [(p + "ln1.w", (h,)), (p + "ln1.b", (h,)),
                (p + "attn.qkv.w", (3 * h, h)), (p + "attn.qkv.b", (3 * h,)),
                (p + "attn.proj.w", (h, h)), (p + "attn.proj.b", (h,)),
                (p + "ln2.w", (h,)), (p + "ln2.b", (h,)),
                (p + "mlp.fc.w", (f, h)), (p + "mlp.fc.b", (f,)),
                (p + "mlp.proj.w", (h, f)), (p + "mlp.proj.b", (h,))]
    out += [("ln_f.w", (h,)), ("ln_f.b", (h,))]
    return out


def _relative_noise(G: torch.Generator, W: torch.Tensor, sigma: float, g) -> torch.Tensor:
    z = torch.randn(W.shape, generator=g, device=W.device, dtype=torch.float64)
    return (W.double() * (1.0 + sigma * z)).to(torch.float32)


def config3_pair(k: int, shape, device="cpu", nan_rate: float = 1e-9):
    g = _gen(device, data_seed(3, k))
    G = torch.randn(shape, generator=g, device=device, dtype=torch.float32) * 0.02
    T = _relative_noise(None, G, 1e-6, g)
    n = G.numel()
    rng = np.random.Generator(np.random.PCG64(data_seed(3, k)))
    nn = int(rng.binomial(n, nan_rate))
    if nn:
        pos = torch.from_numpy(rng.choice(n, nn, replace=False).astype(np.int64)).to(device)
        T.view(-1).view(torch.int32)[pos] = 0x7FC00000
    return G.contiguous(), T.contiguous()


# --------------------------------------------------------------------------
# Workload 4: 1000 replayed f16 [4096, 4096] calls, injected every 10th.
# --------------------------------------------------------------------------
CONFIG4_CALLS = 1000
CONFIG4_SHAPE = (4096, 4096)
CONFIG4_RATE = 1e-7
CONFIG4_MASK = 0xFFFF


def config4_golden(device="cpu", shape=CONFIG4_SHAPE):
    g = _gen(device, data_seed(4, 0))
    return torch.randn(shape, generator=g, device=device, dtype=torch.float32).half().contiguous()


def config4_injected(c: int) -> bool:
    """The 10th, 20th, ... call (0-based c = 9, 19, ...) carries injected flips."""
    return c % 10 == 9


# --------------------------------------------------------------------------
# Workload 5: Llama-7B-shaped checkpoint, weights + Adam m + Adam v.
# --------------------------------------------------------------------------
CONFIG5_RATE = 1e-8
CONFIG5_MASK = 0x7F800000      # the eight f32 exponent bits


def llama7b_shapes():
    h, f, v = 4096, 11008, 32000
    out = [("embed", (v, h))]
    for i in range(32):
        p = f"l{i}."
        out += [(p + "q", (h, h)), (p + "k", (h, h)), (p + "v", (h, h)), (p + "o", (h, h)),
                (p + "gate", (f, h)), (p + "up", (f, h)), (p + "down", (h, f)),
                (p + "in_norm", (h,)), (p + "post_norm", (h,))]
    out += [("norm", (h,)), ("lm_head", (v, h))]
    return out


def llama7b_states():
    """873 (name, shape, state) triples: state 0 weights, 1 Adam m, 2 Adam v."""
    return [(name, shape, s) for s in range(3) for name, shape in llama7b_shapes()]


def config5_pair(k: int, shape, state: int, device="cpu"):
    """(G, T) before injection.  Weights ~ N(0, 0.02); Adam m ~ N(0, 1e-3);
    Adam v = (N(0, 1e-3))^2; T = G*(1 + 1e-7 z)."""
    g = _gen(device, data_seed(5, k))
    G = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if state == 0:
        G.mul_(0.02)
    elif state == 1:
        G.mul_(1e-3)
    else:
        G.mul_(1e-3)
        G.mul_(G)
    T = _relative_noise(None, G, 1e-7, g)
    return G.contiguous(), T.contiguous()


def numel(shapes) -> int:
    return int(sum(int(np.prod(s)) for s in shapes))


def config2_all(device="cuda", shape=CONFIG2_SHAPE, count=CONFIG2_COUNT):
    return [config2_pair(k, device, shape) for k in range(count)]


def config3_all(device="cuda"):
    """All 292 (name, G, T) of the GPT-style checkpoint pair."""
    return [(name,) + config3_pair(k, shape, device) for k, (name, shape) in enumerate(gpt13b_shapes())]


def config5_all(device="cuda"):
    """All 873 (name, state, G, T_before_injection) of the Llama-7B-shaped pair."""
    out = []
    for k, (name, shape, state) in enumerate(llama7b_states()):
        G, T = config5_pair(k, shape, state, device)
        out.append((name, state, G, T))
    return out
