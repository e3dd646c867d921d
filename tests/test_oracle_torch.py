"""Cross-check of the oracle against independent library routines on the CPU:
torch float64 autograd for the forward/backward, torch.optim for the
optimizer steps.  The GPU path never uses any of this.  CPU only."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle as O
from paper_2410_05985_amd import synthetic as S


def _torch_gpt_loss(tp, tokens, cfg):
    """GPT-2 in torch ops (nanoGPT structure): tied head, GELU tanh, causal
    attention, LayerNorm eps 1e-5."""
    tok = torch.as_tensor(tokens, dtype=torch.long)
    idx, tgt = tok[:, :-1], tok[:, 1:]
    B, T = idx.shape
    d, H = cfg.d_model, cfg.n_head
    x = tp["wte"][idx] + tp["wpe"][torch.arange(T)][None]
    mask = torch.ones(T, T, dtype=torch.bool).triu(1)
    for l in range(cfg.n_layer):
        p = f"h{l}."
        a = F.layer_norm(x, (d,), tp[p + "ln1.g"], tp[p + "ln1.b"], 1e-5)
        qkv = F.linear(a, tp[p + "qkv.w"], tp[p + "qkv.b"])
        q, k, v = qkv.split(d, dim=-1)
        q, k, v = (t.view(B, T, H, d // H).transpose(1, 2) for t in (q, k, v))
        s = (q @ k.transpose(-1, -2)) / math.sqrt(d // H)
        att = torch.softmax(s.masked_fill(mask, float("-inf")), dim=-1) @ v
        x = x + F.linear(att.transpose(1, 2).reshape(B, T, d), tp[p + "proj.w"], tp[p + "proj.b"])
        a2 = F.layer_norm(x, (d,), tp[p + "ln2.g"], tp[p + "ln2.b"], 1e-5)
        x = x + F.linear(F.gelu(F.linear(a2, tp[p + "fc.w"], tp[p + "fc.b"]), approximate="tanh"),
                         tp[p + "mproj.w"], tp[p + "mproj.b"])
    xf = F.layer_norm(x, (d,), tp["lnf.g"], tp["lnf.b"], 1e-5)
    logits = xf @ tp["wte"].T
    return F.cross_entropy(logits.reshape(-1, logits.shape[-1]), tgt.reshape(-1))


@pytest.mark.parametrize("cfg", [
    S.GPTConfig(n_layer=2, d_model=64, n_head=4, d_ff=256, seq=16, batch=2, vocab=97),
    S.GPTConfig(n_layer=1, d_model=48, n_head=3, d_ff=96, seq=9, batch=3, vocab=50),
])
def test_gpt_gradients_vs_torch_autograd(cfg):
    rng = np.random.default_rng(8)
    params = {n: rng.standard_normal(s) * (0.1 if len(s) >= 2 else 0.2) + (1.0 if n.endswith(".g") else 0.0)
              for n, s, _ in S.gpt_param_specs(cfg)}
    tokens = rng.integers(0, cfg.vocab, (cfg.batch, cfg.seq + 1))
    hp = dict(optim="adamw", lr=0.0, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.0)
    loss, grads, _, _ = O.gpt_step({k: v.copy() for k, v in params.items()}, None, None, None,
                                   tokens, cfg.n_head, hp, 0.0, rnd=O.ident, update=False,
                                   store=O.ident)
    tp = {k: torch.tensor(v, dtype=torch.float64, requires_grad=True) for k, v in params.items()}
    tl = _torch_gpt_loss(tp, tokens, cfg)
    tl.backward()
    assert abs(loss - tl.item()) < 1e-12
    for k in params:
        ref = tp[k].grad.numpy()
        err = np.max(np.abs(grads[k] - ref)) / max(np.max(np.abs(ref)), 1e-30)
        assert err < 1e-10, (k, err)


def test_gpt_bf16_storage_stays_close_to_exact():
    """The bfloat16 storage points perturb the gradient by about the bf16 unit
    roundoff, not more (a misplaced rounding of a high-precision stream or a
    dropped term would show up as a large deviation)."""
    cfg = S.GPT_TEST
    params = S.gpt_params(cfg)
    tokens = S.gpt_tokens(cfg)
    hp = dict(optim="adamw", lr=0.0, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.0)
    run = lambda rnd: O.gpt_step({k: v.astype(np.float64) for k, v in params.items()}, None, None,
                                 None, tokens, cfg.n_head, hp, 0.0, rnd=rnd, update=False,
                                 store=O.ident)
    l_lo, g_lo, _, _ = run(O.bf16)
    l_hi, g_hi, _, _ = run(O.ident)
    assert abs(l_lo - l_hi) < 1e-2 and abs(l_hi - math.log(cfg.vocab)) < 0.1
    for k in g_hi:
        num = np.linalg.norm(g_lo[k] - g_hi[k])
        den = np.linalg.norm(g_hi[k])
        if den > 0:
            assert num / den < 3e-2, (k, num / den)


@pytest.mark.parametrize("wd", [0.0, 5e-5, 0.1])
def test_sgd_momentum_vs_torch_optim(wd):
    rng = np.random.default_rng(9)
    p0 = rng.standard_normal(257)
    gs = [rng.standard_normal(257) for _ in range(4)]
    tp = torch.tensor(p0, requires_grad=True)
    opt = torch.optim.SGD([tp], lr=0.1, momentum=0.9, weight_decay=wd)
    p, m = p0.copy(), np.zeros_like(p0)
    for g in gs:
        tp.grad = torch.tensor(g)
        opt.step()
        p, m = O.sgd_momentum(p, g, m, 0.1, 0.9, wd, store=O.ident)
    np.testing.assert_allclose(p, tp.detach().numpy(), rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("wd", [0.0, 0.1])
def test_adamw_vs_torch_optim(wd):
    rng = np.random.default_rng(10)
    p0 = rng.standard_normal(257) * 0.02
    gs = [rng.standard_normal(257) * 1e-3 for _ in range(5)]
    tp = torch.tensor(p0, requires_grad=True)
    opt = torch.optim.AdamW([tp], lr=7.5249e-4, betas=(0.9, 0.95), eps=1e-8, weight_decay=wd)
    p, m, v = p0.copy(), np.zeros_like(p0), np.zeros_like(p0)
    for t, g in enumerate(gs, start=1):
        tp.grad = torch.tensor(g)
        opt.step()
        p, m, v = O.adamw(p, g, m, v, 7.5249e-4, 0.9, 0.95, 1e-8, wd, t, store=O.ident)
    np.testing.assert_allclose(p, tp.detach().numpy(), rtol=1e-12, atol=1e-16)


def test_mlp_ten_steps_vs_torch():
    """The tiny-MLP workload: 10 layer-wise steps of SGD-momentum + mix equal
    torch autograd + torch.optim.SGD + the same averaging, in float64.  For a
    single worker, updating each layer right after its own backward gives the
    same result as updating after the full backward."""
    cfg = S.MLP_TINY
    x, y = S.mlp_inputs(cfg)
    params = {k: v.astype(np.float64) for k, v in S.mlp_params(cfg).items()}
    peer = {k: v.astype(np.float64) for k, v in S.peer_of(S.mlp_params(cfg), 0.01).items()}
    hp = dict(optim="sgd", lr=cfg.lr, momentum=cfg.momentum, weight_decay=0.0)
    op = {k: v.copy() for k, v in params.items()}
    om = {k: np.zeros_like(v) for k, v in params.items()}
    tp = {k: torch.tensor(v, requires_grad=True) for k, v in params.items()}
    opt = torch.optim.SGD(list(tp.values()), lr=cfg.lr, momentum=cfg.momentum)
    for s in range(cfg.steps):
        loss, _, trace, _ = O.mlp_step(op, om, peer, x[s], y[s], hp, cfg.alpha, store=O.ident)
        assert trace == [2, 1, 0]
        h = torch.tensor(x[s], dtype=torch.float64)
        for i in range(3):
            h = F.linear(h, tp[f"fc{i+1}.w"], tp[f"fc{i+1}.b"])
            if i < 2:
                h = torch.relu(h)
        tl = F.cross_entropy(h, torch.tensor(y[s], dtype=torch.long))
        opt.zero_grad()
        tl.backward()
        opt.step()
        with torch.no_grad():
            for k in tp:
                tp[k].mul_(1 - cfg.alpha).add_(torch.tensor(peer[k]), alpha=cfg.alpha)
        assert abs(loss - tl.item()) < 1e-10
    for k in tp:
        np.testing.assert_allclose(op[k], tp[k].detach().numpy(), rtol=1e-10, atol=1e-13)
