"""Seeded synthetic inputs for the LayUp layer-wise step.

The datasets the paper trains on (ImageNet-1k, CIFAR-100, MiniPile,
Wikitext-103; paper section 4, "Tasks") are not available, so every input is
drawn here from numpy's PCG64 generator with fixed seeds, at the shapes of the
paper's models (ResNet-50, GPT-2; section 4 "Setup", appendix B).

This module holds the model *shapes* (parameter names, shapes and order) and
the random draws only.  It contains none of the method's arithmetic: no
forward, no backward, no optimizer step and no mixing.  Both the CPU oracle and
the GPU path consume the arrays it returns.

Recipes (stds are standard deviations):

* tiny MLP 512-256-256-10, batch 32, 10 steps.  seed 0: inputs N(0,1) of shape
  (10, 32, 512) then labels uniform in [0, 10) of shape (10, 32); seed 1:
  weights He-uniform U(+-sqrt(6/fan_in)) in forward order, biases 0; seed 2:
  peer = own + 0.01 N(0,1), per tensor in forward order (weight, then bias).
* GPT decoder stacks.  seed 0: tokens uniform over the vocabulary, shape
  (batch, seq + 1) (targets are the inputs shifted by one); seed 1: every
  matrix and embedding N(0, 0.02) in the order of ``gpt_param_specs``, biases
  0, LayerNorm gain 1 and shift 0; seed 2: peer = own + 1e-3 N(0,1) per tensor
  in the same order.
* ResNet-50 parameter set (update+mix only).  seed 1: conv and fc weights
  He-uniform, BatchNorm gain 1 / shift 0, fc bias 0; seed 0: gradients
  1e-3 N(0,1) per tensor; seed 2: peer = own + 1e-3 N(0,1).
* peer slot per step: seed 3, uniform over the resident peer replicas.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List, Tuple

import numpy as np

# ---------------------------------------------------------------- configs


@dataclass(frozen=True)
class MLPConfig:
    dims: Tuple[int, ...] = (512, 256, 256, 10)
    batch: int = 32
    steps: int = 10
    lr: float = 0.05
    momentum: float = 0.9
    weight_decay: float = 0.0
    alpha: float = 0.5

    @property
    def n_classes(self) -> int:
        return self.dims[-1]


@dataclass(frozen=True)
class GPTConfig:
    n_layer: int
    d_model: int
    n_head: int
    d_ff: int
    seq: int
    batch: int
    vocab: int = 50257
    lr: float = 7.5249e-4
    beta1: float = 0.9
    beta2: float = 0.95
    eps: float = 1e-8
    weight_decay: float = 0.1
    alpha: float = 0.5
    n_peers: int = 1
    name: str = "gpt"

    @property
    def d_head(self) -> int:
        return self.d_model // self.n_head

    @property
    def n_tok(self) -> int:
        return self.batch * self.seq

    def n_params(self) -> int:
        return sum(int(np.prod(s)) for _, s, _ in gpt_param_specs(self))


# The five workloads: tiny MLP, GPT-2-small, ResNet-50 update+mix,
# GPT-2-medium, 1.3B decoder.
MLP_TINY = MLPConfig()
GPT2_SMALL = GPTConfig(n_layer=12, d_model=768, n_head=12, d_ff=3072, seq=1024,
                       batch=8, name="gpt2-small")
GPT2_MEDIUM = GPTConfig(n_layer=24, d_model=1024, n_head=16, d_ff=4096, seq=1024,
                        batch=8, name="gpt2-medium")
GPT_1P3B = GPTConfig(n_layer=24, d_model=2048, n_head=16, d_ff=8192, seq=2048,
                     batch=4, n_peers=3, name="gpt-1.3b")
# Small stacks used for element-by-element parity against the oracle.  They
# keep the GPT block structure and span several GEMM tiles with ragged tails.
GPT_TEST = GPTConfig(n_layer=2, d_model=128, n_head=2, d_ff=512, seq=128, batch=2,
                     vocab=1000, name="gpt-test")
GPT_TEST_RAGGED = GPTConfig(n_layer=2, d_model=96, n_head=3, d_ff=384, seq=80,
                            batch=3, vocab=517, name="gpt-test-ragged")
# Head width 128 (as in the 1.3B stack) with a ragged sequence, and head width
# 48, which the fused attention kernels do not cover (score GEMM + softmax).
GPT_TEST_DH128 = GPTConfig(n_layer=1, d_model=256, n_head=2, d_ff=512, seq=96, batch=2,
                           vocab=300, name="gpt-test-dh128")
# 2048 tokens: enough K for the split-K dW GEMMs (their float32 partial sums).
GPT_TEST_LONG = GPTConfig(n_layer=1, d_model=128, n_head=2, d_ff=256, seq=512, batch=4,
                          vocab=400, name="gpt-test-long")
GPT_TEST_DH48 = GPTConfig(n_layer=1, d_model=96, n_head=2, d_ff=256, seq=64, batch=2,
                          vocab=200, name="gpt-test-dh48")
# Wide rows: 832 and 1088 features (208 and 272 float4 groups, ragged over
# 64 lanes), the LayerNorm paths for rows wider than 768 features.
GPT_TEST_W832 = GPTConfig(n_layer=1, d_model=832, n_head=13, d_ff=256, seq=64, batch=2,
                          vocab=250, name="gpt-test-w832")
GPT_TEST_W1088 = GPTConfig(n_layer=1, d_model=1088, n_head=17, d_ff=256, seq=64, batch=2,
                           vocab=250, name="gpt-test-w1088")

# Four blocks: the backward's dY operands (double-buffered by block parity)
# are reused from the third block down, under both streams.
GPT_TEST4 = GPTConfig(n_layer=4, d_model=128, n_head=2, d_ff=512, seq=128, batch=2, vocab=1000,
                      name="gpt-test-4blocks")
# GPT-2-small's own widths (768 features, 12 heads of 64, MLP 3072, 1024
# tokens per sequence, the 50257-token vocabulary) with two blocks and two
# sequences: the LayerNorm, cross-entropy and attention kernels the full
# stack runs, at a size the oracle finishes in seconds.
GPT2_SMALL_2L = GPTConfig(n_layer=2, d_model=768, n_head=12, d_ff=3072, seq=1024, batch=2,
                          name="gpt2-small-width-2blocks")
# Head width 128 over 2048 tokens: the attention path of the 1.3B stack.
GPT_TEST_T2048 = GPTConfig(n_layer=1, d_model=256, n_head=2, d_ff=512, seq=2048, batch=1, vocab=300,
                           name="gpt-test-t2048-dh128")

# The GPT-2-medium and 1.3B stacks' widths (1024 features, 16 heads of 64,
# MLP 4096; 2048 features, 16 heads of 128, MLP 8192) with one block and a
# short sequence: their LayerNorm row widths, head widths and GEMM shapes.
GPT_TEST_W1024 = GPTConfig(n_layer=1, d_model=1024, n_head=16, d_ff=4096, seq=256, batch=2, vocab=2000,
                           name="gpt-test-medium-width")
GPT_TEST_W2048 = GPTConfig(n_layer=1, d_model=2048, n_head=16, d_ff=8192, seq=128, batch=2, vocab=500,
                           name="gpt-test-1.3b-width")

RESNET50_UPDATE = dict(lr=0.1, momentum=0.9, weight_decay=5e-5, alpha=0.5)

# ------------------------------------------------------------ param specs


def mlp_param_specs(cfg: MLPConfig) -> List[Tuple[str, Tuple[int, ...], bool]]:
    """(name, shape, decayed) in forward order: fc1.w, fc1.b, fc2.w, ..."""
    out = []
    for i in range(len(cfg.dims) - 1):
        out.append((f"fc{i+1}.w", (cfg.dims[i + 1], cfg.dims[i]), True))
        out.append((f"fc{i+1}.b", (cfg.dims[i + 1],), True))
    return out


def gpt_param_specs(cfg: GPTConfig) -> List[Tuple[str, Tuple[int, ...], bool]]:
    """(name, shape, decayed) in a fixed order.  Decay only on >=2-D tensors
    (matrices and embeddings), as in nanoGPT.  wte has the logical vocabulary
    rows only; it is tied with the output head."""
    d, f = cfg.d_model, cfg.d_ff
    out = [("wte", (cfg.vocab, d), True), ("wpe", (cfg.seq, d), True)]
    for l in range(cfg.n_layer):
        p = f"h{l}."
        out += [
            (p + "ln1.g", (d,), False), (p + "ln1.b", (d,), False),
            (p + "qkv.w", (3 * d, d), True), (p + "qkv.b", (3 * d,), False),
            (p + "proj.w", (d, d), True), (p + "proj.b", (d,), False),
            (p + "ln2.g", (d,), False), (p + "ln2.b", (d,), False),
            (p + "fc.w", (f, d), True), (p + "fc.b", (f,), False),
            (p + "mproj.w", (d, f), True), (p + "mproj.b", (d,), False),
        ]
    out += [("lnf.g", (d,), False), ("lnf.b", (d,), False)]
    return out


def resnet50_param_specs() -> List[Tuple[str, Tuple[int, ...], bool]]:
    """The 161 parameter tensors of ResNet-50 (53 conv, 106 BatchNorm, fc w/b)
    in forward order.  All are decayed (SGD weight decay on every tensor)."""
    out = [("conv1.w", (64, 3, 7, 7), True), ("bn1.g", (64,), True), ("bn1.b", (64,), True)]
    inp = 64
    for li, (width, blocks) in enumerate([(64, 3), (128, 4), (256, 6), (512, 3)]):
        for bi in range(blocks):
            p = f"layer{li+1}.{bi}."
            outc = width * 4
            out += [(p + "conv1.w", (width, inp, 1, 1), True), (p + "bn1.g", (width,), True),
                    (p + "bn1.b", (width,), True),
                    (p + "conv2.w", (width, width, 3, 3), True), (p + "bn2.g", (width,), True),
                    (p + "bn2.b", (width,), True),
                    (p + "conv3.w", (outc, width, 1, 1), True), (p + "bn3.g", (outc,), True),
                    (p + "bn3.b", (outc,), True)]
            if bi == 0:
                out += [(p + "down.w", (outc, inp, 1, 1), True), (p + "down.bn.g", (outc,), True),
                        (p + "down.bn.b", (outc,), True)]
            inp = outc
    out += [("fc.w", (1000, 2048), True), ("fc.b", (1000,), True)]
    return out


def resnet50_units() -> List[List[str]]:
    """Update units in forward order: one per conv with its BatchNorm, then fc.
    The layer-wise sweep visits them in reverse."""
    specs = resnet50_param_specs()
    units: List[List[str]] = []
    i = 0
    while i < len(specs):
        name = specs[i][0]
        if name == "fc.w":
            units.append([specs[i][0], specs[i + 1][0]])
            i += 2
        else:
            units.append([specs[i][0], specs[i + 1][0], specs[i + 2][0]])
            i += 3
    return units


# ------------------------------------------------------------- generators


def _he_uniform(rng, shape):
    fan_in = int(np.prod(shape[1:]))
    bound = np.sqrt(6.0 / fan_in)
    return rng.uniform(-bound, bound, size=shape).astype(np.float32)


def mlp_inputs(cfg: MLPConfig = MLP_TINY):
    """Returns (x [steps, batch, in] f32, labels [steps, batch] i32)."""
    rng = np.random.default_rng(0)
    x = rng.standard_normal((cfg.steps, cfg.batch, cfg.dims[0]), dtype=np.float32)
    y = rng.integers(0, cfg.n_classes, (cfg.steps, cfg.batch)).astype(np.int32)
    return x, y


def mlp_params(cfg: MLPConfig = MLP_TINY) -> Dict[str, np.ndarray]:
    rng = np.random.default_rng(1)
    out = {}
    for name, shape, _ in mlp_param_specs(cfg):
        out[name] = _he_uniform(rng, shape) if name.endswith(".w") else np.zeros(shape, np.float32)
    return out


def peer_of(params: Dict[str, np.ndarray], std: float, seed: int = 2,
            order: List[str] | None = None) -> Dict[str, np.ndarray]:
    """peer = own + std * N(0,1), drawn per tensor in ``order``."""
    rng = np.random.default_rng(seed)
    names = order if order is not None else list(params)
    out = {}
    for n in names:
        p = params[n]
        out[n] = (p + np.float32(std) * rng.standard_normal(p.shape, dtype=np.float32)).astype(np.float32)
    return out


def gpt_tokens(cfg: GPTConfig, seed: int = 0) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.integers(0, cfg.vocab, (cfg.batch, cfg.seq + 1)).astype(np.int32)


def gpt_params(cfg: GPTConfig, seed: int = 1) -> Dict[str, np.ndarray]:
    rng = np.random.default_rng(seed)
    out = {}
    for name, shape, _ in gpt_param_specs(cfg):
        if len(shape) >= 2:
            out[name] = (np.float32(0.02) * rng.standard_normal(shape, dtype=np.float32)).astype(np.float32)
        elif name.endswith(".g"):
            out[name] = np.ones(shape, np.float32)
        else:
            out[name] = np.zeros(shape, np.float32)
    return out


def gpt_peer(cfg: GPTConfig, params: Dict[str, np.ndarray], seed: int = 2, slot: int = 0):
    order = [n for n, _, _ in gpt_param_specs(cfg)]
    return peer_of(params, 1e-3, seed=seed + 100 * slot, order=order)


def peer_slots(n_steps: int, n_peers: int, seed: int = 3) -> np.ndarray:
    """Peer slot per step, uniform over the resident peer replicas."""
    rng = np.random.default_rng(seed)
    return rng.integers(0, n_peers, n_steps).astype(np.int32)


def gossip_pairs(n_steps: int, n_workers: int, seed: int = 4) -> List[Tuple[int, int]]:
    """(sender, receiver) per step for replicas that take their steps in turn:
    step s belongs to worker s mod M, whose receiver is drawn uniformly from
    the other M-1 workers."""
    rng = np.random.default_rng(seed)
    out = []
    for s in range(n_steps):
        i = s % n_workers
        r = int(rng.integers(0, n_workers - 1))
        out.append((i, r if r < i else r + 1))
    return out


def resnet50_tensors():
    """Returns (params, grads, peer) dicts for the ResNet-50 update+mix sweep."""
    specs = resnet50_param_specs()
    rng1 = np.random.default_rng(1)
    params = {}
    for name, shape, _ in specs:
        if name.endswith(".w"):
            params[name] = _he_uniform(rng1, shape)
        elif name.endswith(".g"):
            params[name] = np.ones(shape, np.float32)
        else:
            params[name] = np.zeros(shape, np.float32)
    rng0 = np.random.default_rng(0)
    grads = {n: (np.float32(1e-3) * rng0.standard_normal(s, dtype=np.float32)).astype(np.float32)
             for n, s, _ in specs}
    peer = peer_of(params, 1e-3, seed=2, order=[n for n, _, _ in specs])
    return params, grads, peer


def normal(shape, seed: int, std: float = 1.0, dtype=np.float32) -> np.ndarray:
    """Plain seeded normal draw, used for GEMM operands and update+mix inputs."""
    rng = np.random.default_rng(seed)
    return (np.float32(std) * rng.standard_normal(shape, dtype=np.float32)).astype(dtype)


def update_mix_inputs(n: int, seed: int, optim: str):
    """Seeded p, g, m, v, q for standalone update+mix parity: p ~ N(0, 0.02),
    g ~ N(0, 1e-3), m ~ N(0, 1e-4), v ~ |N(0, 1e-6)|, q = p + N(0, 1e-3)."""
    rng = np.random.default_rng(seed)
    p = (0.02 * rng.standard_normal(n)).astype(np.float32)
    g = (1e-3 * rng.standard_normal(n)).astype(np.float32)
    m = (1e-4 * rng.standard_normal(n)).astype(np.float32)
    v = np.abs(1e-6 * rng.standard_normal(n)).astype(np.float32) if optim == "adamw" else None
    q = (p + 1e-3 * rng.standard_normal(n)).astype(np.float32)
    return p, g, m, v, q
