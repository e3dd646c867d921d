"""Plain, slow, float64 reference of one LayUp worker's layer-wise step.

TEST INFRASTRUCTURE ONLY (see the package docstring): the product path never
imports this module.

What it computes, in the paper's order (Algorithm 1, "training loop on device
i" and "updater thread i"):

1. forward pass on the current parameters and the loss on the mini-batch;
2. for each layer (unit), from the output back to the input: the backward
   pass of that layer, then -- as soon as that layer's gradient exists
   (section 3.2, layer-wise updates) -- the local update of that layer
   (Algorithm 1, "Local Update") followed by the weighted average with the
   peer's copy of the same layer (Algorithm 1, "Peer Update"; section 3.1,
   push-sum weights).

The paper writes the local update as plain SGD; its experiments use SGD with
momentum and weight decay (ImageNet hyperparameter table) and AdamW (GPT-2
hyperparameter tables), implemented with LibTorch.  The optimizer steps below
are those optimizers as LibTorch defines them.  Optimizer state is local and is
never mixed (only the parameters are sent in Algorithm 1).

Precision: every sum is float64.  ``rnd`` marks each point where the GPU path
stores a bfloat16 tensor; ``bf16`` rounds there, ``ident`` turns the rounding
off (used by the finite-difference and autograd cross-checks).  Optimizer
outputs are rounded to float32, the precision of the master state.
"""
from __future__ import annotations

import math
from typing import Callable, Dict, List, Sequence, Tuple

import numpy as np

Array = np.ndarray

# ------------------------------------------------------------- roundings


def bf16(x) -> Array:
    """Round float64 values to the nearest bfloat16 value, ties to even,
    without going through float32 (no double rounding).  Returns float64.

    A bfloat16 keeps 8 significant bits.  For a float64 in the normal range
    of bfloat16 that means dropping the low 45 of its 52 stored mantissa bits
    with round-to-nearest-even, done on the integer bit pattern: add half an
    ulp minus one, plus the lowest kept bit (the tie goes to the even
    neighbour), then clear the dropped bits; a carry out of the mantissa
    moves the exponent up, which is the correct rounding across a binade.
    Below 2**-126 bfloat16 is subnormal with spacing 2**-133."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    out = np.empty_like(x)
    xf, of = x.reshape(-1), out.reshape(-1)
    step = 1 << 17                                        # slices small enough to stay in cache
    for s in range(0, xf.size, step):
        xs = xf[s: s + step]
        bits = xs.view(np.uint64)
        r = (bits >> np.uint64(45)) & np.uint64(1)        # lowest kept bit
        r += bits
        r += np.uint64((1 << 44) - 1)
        r &= ~np.uint64((1 << 45) - 1)
        of[s: s + step] = r.view(np.float64)
        ax = np.abs(xs)
        odd = ~(ax >= 2.0 ** -126) | (ax >= 2.0 ** 127)  # subnormal, zero, NaN, near or past overflow
        if np.any(odd):
            i = np.nonzero(odd)[0]
            xo = xs[i]
            ro = of[s + i]
            tiny = np.abs(xo) < 2.0 ** -126               # bfloat16 subnormals: spacing 2**-133
            ro = np.where(tiny, np.rint(np.where(tiny, xo, 0.0) * 2.0 ** 133) * 2.0 ** -133, ro)
            ro = np.where(np.abs(ro) >= 2.0 ** 128, np.copysign(np.inf, xo), ro)  # past the largest bfloat16
            ro = np.where(np.isnan(xo), xo, ro)
            of[s + i] = ro
    return out


def f32(x) -> Array:
    """Round to float32 (nearest, ties to even); returns float64."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def ident(x) -> Array:
    return np.asarray(x, dtype=np.float64)


# ------------------------------------------------------------ layer math
# Linear layers follow y = x W^T + b with W stored [out, in].


def linear_fwd(x: Array, w: Array, b: Array | None) -> Array:
    y = x @ w.T
    return y if b is None else y + b


def linear_bwd(dy: Array, x: Array, w: Array, need_dx: bool = True):
    """Chain rule of y = x W^T + b: dW = dy^T x, db = sum_rows dy, dx = dy W."""
    dw = dy.T @ x
    db = dy.sum(axis=0)
    dx = dy @ w if need_dx else None
    return dw, db, dx


def relu(x: Array) -> Array:
    return np.where(x > 0, x, 0.0)


def relu_bwd(dy: Array, y: Array) -> Array:
    """y = relu(x); the derivative is 1 where the output is positive."""
    return np.where(y > 0, dy, 0.0)


def layernorm_fwd(x: Array, g: Array, b: Array, eps: float = 1e-5) -> Array:
    """LayerNorm over the last axis, biased variance (Ba et al., 2016)."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * g + b


def layernorm_bwd(dy: Array, x: Array, g: Array, eps: float = 1e-5):
    """Backward of LayerNorm: with xh = (x - mu) * r, r = 1/sqrt(var + eps),
    dxh = dy * g and dx = r * (dxh - mean(dxh) - xh * mean(dxh * xh))."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    r = 1.0 / np.sqrt(var + eps)
    xh = (x - mu) * r
    dg = (dy * xh).sum(axis=0)
    db = dy.sum(axis=0)
    dxh = dy * g
    dx = r * (dxh - dxh.mean(axis=-1, keepdims=True) - xh * (dxh * xh).mean(axis=-1, keepdims=True))
    return dx, dg, db


_GELU_C = math.sqrt(2.0 / math.pi)


def gelu_tanh(x: Array) -> Array:
    """Tanh form of GELU (Hendrycks & Gimpel), as used by GPT-2."""
    return 0.5 * x * (1.0 + np.tanh(_GELU_C * (x + 0.044715 * x ** 3)))


def gelu_tanh_grad(x: Array) -> Array:
    """d/dx of gelu_tanh."""
    t = np.tanh(_GELU_C * (x + 0.044715 * x ** 3))
    return 0.5 * (1.0 + t) + 0.5 * x * (1.0 - t * t) * _GELU_C * (1.0 + 3.0 * 0.044715 * x * x)


def causal_softmax(s: Array) -> Array:
    """Row softmax of s [T, T] with entries above the diagonal masked out."""
    t = s.shape[-1]
    mask = np.triu(np.ones((t, t), dtype=bool), k=1)
    z = np.where(mask, -np.inf, s)
    z = z - z.max(axis=-1, keepdims=True)
    e = np.exp(z)
    return e / e.sum(axis=-1, keepdims=True)


def causal_logsumexp(s: Array) -> Array:
    """Natural log of the causal softmax normaliser of every row of s [.., T, T]:
    log sum_{j <= i} exp(s_ij).  exp(s_ij - lse_i) is causal_softmax(s)_ij."""
    t = s.shape[-1]
    mask = np.triu(np.ones((t, t), dtype=bool), k=1)
    z = np.where(mask, -np.inf, s)
    mx = z.max(axis=-1, keepdims=True)
    return (mx + np.log(np.exp(z - mx).sum(axis=-1, keepdims=True)))[..., 0]


def softmax_bwd(p: Array, dp: Array) -> Array:
    """Backward of a row softmax: ds = p * (dp - rowsum(dp * p))."""
    return p * (dp - (dp * p).sum(axis=-1, keepdims=True))


def cross_entropy(z: Array, y: Array):
    """Mean over rows of logsumexp(z) - z[y]; returns (loss, dz)."""
    n = z.shape[0]
    zm = z.max(axis=-1, keepdims=True)
    e = np.exp(z - zm)
    s = e.sum(axis=-1, keepdims=True)
    lse = np.log(s)[:, 0] + zm[:, 0]
    loss = float(np.mean(lse - z[np.arange(n), y]))
    dz = e / s
    dz[np.arange(n), y] -= 1.0
    return loss, dz / n


# ------------------------------------------------- optimizer and mixing
# Algorithm 1, "Local Update": x <- x - eta * grad, realised as the optimizer
# the experiments name (SGD with momentum for the ResNets, AdamW for GPT-2),
# with LibTorch semantics.  Inputs are float32 values; outputs are rounded to
# float32 (the master state).


def sgd_momentum(p, g, m, lr, momentum, weight_decay, wd_on=True, store=f32):
    """SGD with momentum, dampening 0, no Nesterov, coupled weight decay:
    g' = g + wd * p;  m = momentum * m + g';  p = p - lr * m."""
    p = np.asarray(p, np.float64)
    gg = np.asarray(g, np.float64)
    if wd_on and weight_decay != 0.0:
        gg = gg + weight_decay * p
    m_new = momentum * np.asarray(m, np.float64) + gg
    p_new = p - lr * m_new
    return p_new, store(m_new)


def adamw(p, g, m, v, lr, beta1, beta2, eps, weight_decay, t, wd_on=True, store=f32):
    """AdamW (decoupled weight decay, bias-corrected moments, no amsgrad):
    p *= 1 - lr*wd;  m = b1 m + (1-b1) g;  v = b2 v + (1-b2) g^2;
    p -= (lr / (1 - b1^t)) * m / (sqrt(v) / sqrt(1 - b2^t) + eps)."""
    p = np.asarray(p, np.float64)
    g = np.asarray(g, np.float64)
    if wd_on and weight_decay != 0.0:
        p = p * (1.0 - lr * weight_decay)
    m_new = beta1 * np.asarray(m, np.float64) + (1.0 - beta1) * g
    v_new = beta2 * np.asarray(v, np.float64) + (1.0 - beta2) * g * g
    bc1 = 1.0 - beta1 ** t
    bc2 = 1.0 - beta2 ** t
    p_new = p - (lr / bc1) * m_new / (np.sqrt(v_new) / math.sqrt(bc2) + eps)
    return p_new, store(m_new), store(v_new)


def mix(p, q, alpha):
    """Algorithm 1, "Peer Update": the receiving copy keeps weight
    w_self / (w_self + w_sender) and takes w_sender / (w_self + w_sender) of
    the incoming layer.  With alpha = w_sender / (w_self + w_sender):
    p <- (1 - alpha) * p + alpha * q, coefficients formed once on the host."""
    a = 1.0 - alpha
    b = alpha
    return a * np.asarray(p, np.float64) + b * np.asarray(q, np.float64)


def disagreement(p, q) -> float:
    """Model disagreement of one layer (appendix, disagreement measurement):
    the squared distance between the locally updated layer and the peer's."""
    d = np.asarray(p, np.float64) - np.asarray(q, np.float64)
    return float(np.sum(d * d))


def update_mix(p, g, m, v, q, hp: dict, alpha: float, t: int, wd_on=True, store=f32):
    """Local update then peer average of one tensor.  Returns float32-rounded
    (p, m, v) and the disagreement measured between the update and the mix."""
    if hp["optim"] == "sgd":
        p1, m1 = sgd_momentum(p, g, m, hp["lr"], hp["momentum"], hp["weight_decay"], wd_on, store)
        v1 = None
    else:
        p1, m1, v1 = adamw(p, g, m, v, hp["lr"], hp["beta1"], hp["beta2"], hp["eps"],
                           hp["weight_decay"], t, wd_on, store)
    dis = disagreement(p1, q)
    p2 = store(mix(p1, q, alpha))
    return p2, m1, v1, dis


def update_push(p, g, m, v, q, hp: dict, alpha: float, t: int, wd_on=True, store=f32):
    """Algorithm 1 as written, for one tensor: the sender's "Local Update" of
    its own copy, then the "Peer Update" of the receiver's copy q with the
    sent layer, q <- (1 - alpha) q + alpha p1, alpha = w_sender / (w_sender +
    w_receiver).  Returns float32-rounded (p1, m, v, q_new) and the
    disagreement between p1 and the receiver's copy before the mix."""
    if hp["optim"] == "sgd":
        p1, m1 = sgd_momentum(p, g, m, hp["lr"], hp["momentum"], hp["weight_decay"], wd_on, store)
        v1 = None
    else:
        p1, m1, v1 = adamw(p, g, m, v, hp["lr"], hp["beta1"], hp["beta2"], hp["eps"],
                           hp["weight_decay"], t, wd_on, store)
    dis = disagreement(p1, q)
    q2 = store(mix(q, p1, alpha))
    return p1, m1, v1, q2, dis


# --------------------------------------------------------- push-sum (host)


def push_sum_alpha(w_self: float, w_sender: float) -> float:
    """Section 3.1 / Algorithm 1: the sender has already halved its weight
    before sending; the receiver weighs the incoming layer by
    w_sender / (w_self + w_sender)."""
    return w_sender / (w_self + w_sender)


def push_sum_round(w: Sequence[float], sender: int, receiver: int) -> Tuple[List[float], float]:
    """One push-sum exchange: the sender halves its weight, the receiver mixes
    with alpha = w_sender' / (w_receiver + w_sender') and then adds the
    sender's weight.  Returns the new weights and alpha."""
    w = list(map(float, w))
    w[sender] = w[sender] / 2.0
    alpha = push_sum_alpha(w[receiver], w[sender])
    w[receiver] = w[receiver] + w[sender]
    return w, alpha


# ------------------------------------------------------------ units / order


def reverse_unit_order(n_units: int) -> List[int]:
    """Layer-wise order (Algorithm 1 loops over layers in backward order):
    the output-side unit first, the input-side unit last."""
    return list(range(n_units - 1, -1, -1))


def mlp_units(n_layers: int) -> List[List[str]]:
    return [[f"fc{i+1}.w", f"fc{i+1}.b"] for i in range(n_layers)]


def gpt_units(n_layer: int) -> List[List[str]]:
    """Unit 0: token and position embeddings (wte is tied with the output
    head, so its gradient is complete only after the embedding backward);
    units 1..L: the decoder blocks; unit L+1: the final LayerNorm."""
    units = [["wte", "wpe"]]
    for l in range(n_layer):
        p = f"h{l}."
        units.append([p + s for s in ("ln1.g", "ln1.b", "qkv.w", "qkv.b", "proj.w", "proj.b",
                                      "ln2.g", "ln2.b", "fc.w", "fc.b", "mproj.w", "mproj.b")])
    units.append(["lnf.g", "lnf.b"])
    return units


def _apply_unit(names, params, grads, m, v, peer, hp, alpha, t, decay_of, store=f32, push=False):
    """Update+mix of one unit's tensors.  push=False: the worker's copy
    absorbs the peer's (``peer`` read only); push=True: the worker keeps its
    update and the receiver's copy ``peer`` is mixed in place."""
    dis = 0.0
    for n in names:
        vn = None if v is None else v[n]
        if push:
            p2, m2, v2, q2, d = update_push(params[n], grads[n], m[n], vn, peer[n], hp, alpha, t,
                                            wd_on=decay_of(n), store=store)
            peer[n] = q2
        else:
            p2, m2, v2, d = update_mix(params[n], grads[n], m[n], vn, peer[n], hp, alpha, t,
                                       wd_on=decay_of(n), store=store)
        params[n], m[n] = p2, m2
        if v is not None:
            v[n] = v2
        dis += d
    return dis


# ------------------------------------------------------------ tiny MLP step


def mlp_step(params, m, peer, x, y, hp, alpha, t=1, store=f32, push=False):
    """One layer-wise step of the float32 MLP (ReLU between layers, softmax
    cross-entropy, mean over the batch).  Units are the linear layers.
    Returns (loss, grads, trace, disagreements); params and m are updated in
    place (dicts of float64 arrays holding float32 values)."""
    n_layers = len([k for k in params if k.endswith(".w")])
    x = np.asarray(x, np.float64)
    acts = [x]
    h = x
    for i in range(n_layers):
        z = linear_fwd(h, params[f"fc{i+1}.w"], params[f"fc{i+1}.b"])
        h = relu(z) if i < n_layers - 1 else z
        acts.append(h)
    loss, dz = cross_entropy(acts[-1], np.asarray(y))
    grads: Dict[str, Array] = {}
    trace, dis = [], {}
    units = mlp_units(n_layers)
    dy = dz
    for u in reverse_unit_order(n_layers):
        w = params[f"fc{u+1}.w"]
        dw, db, dx = linear_bwd(dy, acts[u], w, need_dx=u > 0)
        grads[f"fc{u+1}.w"], grads[f"fc{u+1}.b"] = store(dw), store(db)
        if u > 0:
            dy = relu_bwd(dx, acts[u])
        dis[u] = _apply_unit(units[u], params, grads, m, None, peer, hp, alpha, t,
                             lambda n: True, store, push)
        trace.append(u)
    return loss, grads, trace, dis


# ---------------------------------------------------------- GPT block step


def _heads(mat: Array, b: int, t: int, h: int, dh: int) -> Array:
    """[B*T, H*dh] -> [B, H, T, dh]"""
    return mat.reshape(b, t, h, dh).transpose(0, 2, 1, 3)


def _unheads(x: Array) -> Array:
    b, h, t, dh = x.shape
    return x.transpose(0, 2, 1, 3).reshape(b * t, h * dh)


def gpt_forward(params, tokens, n_head: int, rnd: Callable = bf16):
    """GPT-2 forward (nanoGPT structure, tied head, GELU-tanh, LN eps 1e-5).
    Returns (loss, dlogits, cache).  bf16 storage points (``rnd``): the
    weight copies used by the GEMMs, every LayerNorm output, qkv, the
    attention probabilities, the attention output, the MLP pre-activation and
    its GELU, the logits and the logit gradient.  The residual stream, scores
    and GEMM accumulations stay in high precision."""
    tok = np.asarray(tokens)
    bsz, t1 = tok.shape
    t = t1 - 1
    idx, tgt = tok[:, :t].reshape(-1), tok[:, 1:].reshape(-1)
    wte = np.asarray(params["wte"], np.float64)
    d = wte.shape[1]
    dh = d // n_head
    n_layer = len([k for k in params if k.endswith(".qkv.w")])
    scale = 1.0 / math.sqrt(dh)
    x = wte[idx] + np.asarray(params["wpe"], np.float64)[np.tile(np.arange(t), bsz)]
    cache = {"idx": idx, "tgt": tgt, "B": bsz, "T": t, "d": d, "H": n_head, "L": n_layer,
             "xs": [x]}
    for l in range(n_layer):
        p = f"h{l}."
        c = {}
        c["x"] = x
        c["a"] = a = rnd(layernorm_fwd(x, params[p + "ln1.g"], params[p + "ln1.b"]))
        c["qkv"] = qkv = rnd(linear_fwd(a, rnd(params[p + "qkv.w"]), params[p + "qkv.b"]))
        q = _heads(qkv[:, :d], bsz, t, n_head, dh)
        k = _heads(qkv[:, d:2 * d], bsz, t, n_head, dh)
        v = _heads(qkv[:, 2 * d:], bsz, t, n_head, dh)
        s = (q @ k.swapaxes(-1, -2)) * scale
        c["P"] = P = rnd(causal_softmax(s))
        c["lse"] = causal_logsumexp(s)
        c["o"] = o = rnd(_unheads(P @ v))
        h_res = x + linear_fwd(o, rnd(params[p + "proj.w"]), params[p + "proj.b"])
        c["h"] = h_res
        c["a2"] = a2 = rnd(layernorm_fwd(h_res, params[p + "ln2.g"], params[p + "ln2.b"]))
        f = linear_fwd(a2, rnd(params[p + "fc.w"]), params[p + "fc.b"])
        c["f"] = rnd(f)
        c["gl"] = gl = rnd(gelu_tanh(f))
        x = h_res + linear_fwd(gl, rnd(params[p + "mproj.w"]), params[p + "mproj.b"])
        cache[l] = c
        cache["xs"].append(x)
    cache["xL"] = x
    cache["xf"] = xf = rnd(layernorm_fwd(x, params["lnf.g"], params["lnf.b"]))
    logits = rnd(xf @ rnd(wte).T)
    loss, dlog = cross_entropy(logits, tgt)
    cache["dlogits"] = dlog = rnd(dlog)
    return loss, dlog, cache


def gpt_block_bwd(params, c, dx, l, bsz, t, n_head, rnd: Callable = bf16):
    """Backward of decoder block l given the gradient dx of its output
    (high precision).  Returns (grads of the block's tensors, dx of its
    input)."""
    p = f"h{l}."
    d = dx.shape[1]
    dh = d // n_head
    scale = 1.0 / math.sqrt(dh)
    g: Dict[str, Array] = {}
    # MLP output projection; the residual passes dx through unchanged.
    dy = rnd(dx)
    g[p + "mproj.w"], g[p + "mproj.b"], dgl = linear_bwd(dy, c["gl"], rnd(params[p + "mproj.w"]))
    df = rnd(dgl * gelu_tanh_grad(c["f"]))
    g[p + "fc.w"], g[p + "fc.b"], da2 = linear_bwd(df, c["a2"], rnd(params[p + "fc.w"]))
    dln2, g[p + "ln2.g"], g[p + "ln2.b"] = layernorm_bwd(da2, c["h"], params[p + "ln2.g"])
    dh_res = dx + dln2
    # attention output projection
    dy2 = rnd(dh_res)
    g[p + "proj.w"], g[p + "proj.b"], do = linear_bwd(dy2, c["o"], rnd(params[p + "proj.w"]))
    do = rnd(do)
    qkv, P = c["qkv"], c["P"]
    q = _heads(qkv[:, :d], bsz, t, n_head, dh)
    k = _heads(qkv[:, d:2 * d], bsz, t, n_head, dh)
    v = _heads(qkv[:, 2 * d:], bsz, t, n_head, dh)
    do_h = _heads(do, bsz, t, n_head, dh)
    dP = do_h @ v.swapaxes(-1, -2)
    dv = rnd(P.swapaxes(-1, -2) @ do_h)
    dS = rnd(scale * softmax_bwd(P, dP))
    dq = rnd(dS @ k)
    dk = rnd(dS.swapaxes(-1, -2) @ q)
    dqkv = np.concatenate([_unheads(dq), _unheads(dk), _unheads(dv)], axis=1)
    g[p + "qkv.w"], g[p + "qkv.b"], da = linear_bwd(dqkv, c["a"], rnd(params[p + "qkv.w"]))
    dln1, g[p + "ln1.g"], g[p + "ln1.b"] = layernorm_bwd(da, c["x"], params[p + "ln1.g"])
    return g, dh_res + dln1


def gpt_head_bwd(params, dlog, xf, xL, rnd: Callable = bf16):
    """Backward of the top unit: the tied output head (logits = xf wte^T)
    and the final LayerNorm, given the logit gradient.  Returns (grads of
    lnf.g and lnf.b, dx at the last block's output, the head's contribution
    to the wte gradient)."""
    dlog = np.asarray(dlog, np.float64)
    xf = np.asarray(xf, np.float64)
    dxf = dlog @ rnd(np.asarray(params["wte"], np.float64))
    wte_head = dlog.T @ xf
    dx, dg, db = layernorm_bwd(dxf, np.asarray(xL, np.float64), params["lnf.g"])
    return {"lnf.g": dg, "lnf.b": db}, dx, wte_head


def gpt_embed_bwd(dx, idx, wte_head, bsz, t):
    """Backward of the input embeddings x0 = wte[tok] + wpe[pos]: wte
    collects the head's gradient plus dx scattered over the input tokens;
    wpe sums dx over the batch per position."""
    dx = np.asarray(dx, np.float64)
    dwte = np.asarray(wte_head, np.float64).copy()
    np.add.at(dwte, np.asarray(idx), dx)
    return {"wte": dwte, "wpe": dx.reshape(bsz, t, -1).sum(axis=0)}


def gpt_step(params, m, v, peer, tokens, n_head, hp, alpha, t=1, rnd: Callable = bf16,
             update: bool = True, store: Callable = f32, push: bool = False):
    """One layer-wise LayUp step of a GPT stack.  ``params``, ``m``, ``v`` are
    dicts of arrays updated in place (float32 values).  Returns (loss, grads,
    trace, disagreements).  With ``update=False`` only the gradients are
    produced (all units use the pre-step weights either way: a unit's update
    happens after its own backward, and no earlier unit's backward reads it)."""
    params_f = {k_: np.asarray(a_, np.float64) for k_, a_ in params.items()}
    loss, dlog, cache = gpt_forward(params_f, tokens, n_head, rnd)
    bsz, t_len, n_layer = cache["B"], cache["T"], cache["L"]
    units = gpt_units(n_layer)
    decay = {n for n in params if params[n].ndim >= 2}
    grads: Dict[str, Array] = {}
    trace: List[int] = []
    dis: Dict[int, float] = {}

    def apply(u):
        trace.append(u)
        if update:
            dis[u] = _apply_unit(units[u], params, grads, m, v, peer, hp, alpha, t,
                                 lambda n: n in decay, store, push)

    # unit L+1: output head (tied wte) and final LayerNorm
    g, dx, wte_head = gpt_head_bwd(params_f, dlog, cache["xf"], cache["xL"], rnd)
    for k_, a_ in g.items():
        grads[k_] = store(a_)
    apply(n_layer + 1)
    for l in range(n_layer - 1, -1, -1):
        g, dx = gpt_block_bwd(params_f, cache[l], dx, l, bsz, t_len, n_head, rnd)
        for k_, a_ in g.items():
            grads[k_] = store(a_)
        apply(l + 1)
    # unit 0: embeddings
    g = gpt_embed_bwd(dx, cache["idx"], wte_head, bsz, t_len)
    for k_, a_ in g.items():
        grads[k_] = store(a_)
    apply(0)
    return loss, grads, trace, dis


def gpt_update_units(params, grads, m, v, peer, n_layer, hp, alpha, t=1, store: Callable = f32,
                     push: bool = False):
    """The update+mix part of a GPT step on given gradients, unit by unit in
    backward order (Algorithm 1's updater loop over the layers).  With the
    gradients of a run under test this checks that run's updates on their own
    inputs.  Returns the trace and the per-unit disagreements."""
    units = gpt_units(n_layer)
    decay = {n for n in params if np.ndim(params[n]) >= 2}
    trace, dis = [], {}
    for u in reverse_unit_order(len(units)):
        trace.append(u)
        dis[u] = _apply_unit(units[u], params, grads, m, v, peer, hp, alpha, t,
                             lambda n: n in decay, store, push)
    return trace, dis
