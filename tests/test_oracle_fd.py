"""Central finite differences in float64 pin every backward of the oracle
(bfloat16 rounding switched off).  CPU only."""
import numpy as np
import pytest

import oracle as O


def fd_grad(f, x, h_rel=1e-6):
    g = np.zeros_like(x)
    it = np.nditer(x, flags=["multi_index"])
    for _ in it:
        i = it.multi_index
        h = h_rel * max(1.0, abs(x[i]))
        old = x[i]
        x[i] = old + h
        fp = f()
        x[i] = old - h
        fm = f()
        x[i] = old
        g[i] = (fp - fm) / (2 * h)
    return g


def close(a, b, tol=1e-6):
    scale = max(np.max(np.abs(b)), 1e-12)
    assert np.max(np.abs(a - b)) <= tol * scale, (np.max(np.abs(a - b)), scale)


def test_fd_linear():
    rng = np.random.default_rng(0)
    x, w, b = rng.standard_normal((2, 4)), rng.standard_normal((3, 4)), rng.standard_normal(3)
    r = rng.standard_normal((2, 3))
    f = lambda: float(np.sum(r * O.linear_fwd(x, w, b)))
    dw, db, dx = O.linear_bwd(r, x, w)
    close(dw, fd_grad(f, w)); close(db, fd_grad(f, b)); close(dx, fd_grad(f, x))


def test_fd_layernorm():
    rng = np.random.default_rng(1)
    x, g, b = rng.standard_normal((3, 8)), rng.standard_normal(8), rng.standard_normal(8)
    r = rng.standard_normal((3, 8))
    f = lambda: float(np.sum(r * O.layernorm_fwd(x, g, b)))
    dx, dg, db = O.layernorm_bwd(r, x, g)
    close(dx, fd_grad(f, x)); close(dg, fd_grad(f, g)); close(db, fd_grad(f, b))


def test_fd_gelu_and_relu():
    rng = np.random.default_rng(2)
    x = rng.standard_normal(50) * 3
    for i in range(x.size):
        h = 1e-6
        fd = (O.gelu_tanh(x[i] + h) - O.gelu_tanh(x[i] - h)) / (2 * h)
        assert abs(fd - O.gelu_tanh_grad(x[i])) < 1e-8
    # GELU-tanh known values
    assert O.gelu_tanh(0.0) == 0.0
    assert abs(O.gelu_tanh(1.0) - 0.8411919906082768) < 1e-12
    y = O.relu(x)
    r = rng.standard_normal(50)
    f = lambda: float(np.sum(r * O.relu(x)))
    close(O.relu_bwd(r, y), fd_grad(f, x))


def test_fd_causal_attention_core():
    """softmax(q k^T * s, causal) v for one head, T=4, d_h=4."""
    rng = np.random.default_rng(3)
    q, k, v = (rng.standard_normal((4, 4)) for _ in range(3))
    r = rng.standard_normal((4, 4))
    s = 0.5

    def fwd():
        return O.causal_softmax(q @ k.T * s) @ v

    f = lambda: float(np.sum(r * fwd()))
    P = O.causal_softmax(q @ k.T * s)
    assert np.allclose(np.triu(P, 1), 0) and np.allclose(P.sum(1), 1)
    dP = r @ v.T
    dv = P.T @ r
    dS = s * O.softmax_bwd(P, dP)
    close(q * 0 + dS @ k, fd_grad(f, q)); close(dS.T @ q, fd_grad(f, k)); close(dv, fd_grad(f, v))


def test_fd_cross_entropy():
    rng = np.random.default_rng(4)
    z, y = rng.standard_normal((6, 5)), rng.integers(0, 5, 6)
    loss, dz = O.cross_entropy(z, y)
    close(dz, fd_grad(lambda: O.cross_entropy(z, y)[0], z))
    ref = np.mean([np.log(np.sum(np.exp(z[i]))) - z[i, y[i]] for i in range(6)])
    assert abs(loss - ref) < 1e-12


def test_fd_mlp_end_to_end():
    """Gradients the layer-wise MLP step feeds its updates equal the
    finite-difference gradient of the loss."""
    rng = np.random.default_rng(5)
    dims = (5, 4, 4, 3)
    params = {}
    for i in range(3):
        params[f"fc{i+1}.w"] = rng.standard_normal((dims[i + 1], dims[i]))
        params[f"fc{i+1}.b"] = rng.standard_normal(dims[i + 1]) * 0.1
    x, y = rng.standard_normal((2, 5)), rng.integers(0, 3, 2)

    def loss():
        h = x
        for i in range(3):
            h = O.linear_fwd(h, params[f"fc{i+1}.w"], params[f"fc{i+1}.b"])
            if i < 2:
                h = O.relu(h)
        return O.cross_entropy(h, y)[0]

    snap = {k: v.copy() for k, v in params.items()}
    hp = dict(optim="sgd", lr=0.0, momentum=0.9, weight_decay=0.0)
    m = {k: np.zeros_like(v) for k, v in params.items()}
    _, grads, trace, _ = O.mlp_step({k: v.copy() for k, v in snap.items()}, m,
                                    {k: v.copy() for k, v in snap.items()}, x, y, hp, 0.0,
                                    store=O.ident)
    assert trace == [2, 1, 0]
    for k in params:
        close(grads[k], fd_grad(loss, params[k]))


@pytest.mark.parametrize("n_layer", [1, 2])
def test_fd_gpt_end_to_end(n_layer):
    """Every gradient of the tiny GPT stack (tied head, two heads, causal
    attention, GELU MLP, LayerNorms, embeddings) against finite differences."""
    from paper_2410_05985_amd import synthetic as S
    cfg = S.GPTConfig(n_layer=n_layer, d_model=8, n_head=2, d_ff=16, seq=4, batch=2, vocab=11)
    rng = np.random.default_rng(6)
    params = {n: rng.standard_normal(s) * (0.3 if len(s) >= 2 else 0.1) + (1.0 if n.endswith(".g") else 0.0)
              for n, s, _ in S.gpt_param_specs(cfg)}
    tokens = rng.integers(0, cfg.vocab, (cfg.batch, cfg.seq + 1))
    hp = dict(optim="adamw", lr=0.0, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.0)
    _, grads, trace, _ = O.gpt_step({k: v.copy() for k, v in params.items()}, None, None, None,
                                    tokens, cfg.n_head, hp, 0.0, rnd=O.ident, update=False,
                                    store=O.ident)
    assert trace == list(range(n_layer + 1, -1, -1))
    loss = lambda: O.gpt_forward(params, tokens, cfg.n_head, rnd=O.ident)[0]
    for n in params:
        close(grads[n], fd_grad(loss, params[n]), tol=2e-6)
