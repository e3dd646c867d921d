"""Parity of the whole layer-wise step (layup_step / layup_forward /
layup_layer_backward / layup_unit_update_mix) with the oracle: unit order
(Algorithm 1 loops over layers in backward order; section 3.2 updates a layer
as soon as its gradient exists), gradients, optimizer state and mixed
parameters."""
import math

import numpy as np
import pytest

import oracle as O
from paper_2410_05985_amd import synthetic as S
from tests.gpt_cases import gpt_hp, gpt_setup
from tests.parity import compare, compare_chained

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
from paper_2410_05985_amd import layup as LU  # noqa: E402

DEV = "cuda"


# ------------------------------------------------------------------ MLP

def mlp_setup(two_streams=True):
    cfg = S.MLP_TINY
    x, y = S.mlp_inputs(cfg)
    params = S.mlp_params(cfg)
    peer = S.peer_of(params, 0.01)
    m = LU.Model(LU.mlp_config(cfg.dims, cfg.batch), "sgd", two_streams=two_streams)
    m.load("params", params)
    m.load("peers", peer)
    return cfg, x, y, params, peer, m


def test_mlp_ten_steps_parity():
    """Tiny MLP, float32, SGD momentum 0.9, lr 0.05, alpha 0.5, 10 layer-wise
    steps chained on both sides.  Tolerance 1e-4 (float32 GEMMs against a
    float64 reference, compounded over 10 steps; the float64 oracle and an
    independent float64 torch run agree to 1e-10)."""
    cfg, x, y, params, peer, m = mlp_setup()
    hp = LU.hparams("sgd", cfg.lr, cfg.momentum, 0.0)
    ohp = dict(optim="sgd", lr=cfg.lr, momentum=cfg.momentum, weight_decay=0.0)
    xd = torch.from_numpy(x).to(DEV)
    yd = torch.from_numpy(y).to(DEV)
    loss = torch.zeros(1, dtype=torch.float32, device=DEV)
    op = {k: v.astype(np.float64) for k, v in params.items()}
    om = {k: np.zeros_like(v) for k, v in op.items()}
    opeer = {k: v.astype(np.float64) for k, v in peer.items()}
    torch.cuda.synchronize()
    for s in range(cfg.steps):
        LU.layup_step(m.ctx, yd[s], xd[s], hp, cfg.alpha, 0, loss)
        oloss, ograds, otrace, _ = O.mlp_step(op, om, opeer, x[s], y[s], ohp, cfg.alpha)
        m.synchronize()
        assert abs(loss.item() - oloss) <= 1e-4 * abs(oloss), (s, loss.item(), oloss)
        g = m.read("grads")
        for k in ograds:
            compare(g[k], ograds[k].reshape(g[k].shape), 1e-4, f"step {s} grad {k}")
    got = m.read("params")
    mom = m.read("m")
    for k in op:
        compare(got[k], op[k].reshape(got[k].shape), 1e-4, f"param {k}")
        compare(mom[k], om[k].reshape(mom[k].shape), 1e-4, f"momentum {k}")
    # order trace: every step visits units 2, 1, 0
    assert m.read_trace() == [(s, u) for s in range(cfg.steps) for u in (2, 1, 0)]
    m.close()


def test_mlp_two_streams_equal_one_stream():
    """Overlapping update+mix with the next unit's backward changes timing
    only: results are bitwise identical to the serialized schedule."""
    outs = []
    for two in (True, False):
        cfg, x, y, params, peer, m = mlp_setup(two)
        hp = LU.hparams("sgd", cfg.lr, cfg.momentum, 0.0)
        xd, yd = torch.from_numpy(x).to(DEV), torch.from_numpy(y).to(DEV)
        torch.cuda.synchronize()
        for s in range(cfg.steps):
            LU.layup_step(m.ctx, yd[s], xd[s], hp, cfg.alpha, 0)
        m.synchronize()
        outs.append(m.params.cpu().numpy().copy())
        m.close()
    assert np.array_equal(outs[0], outs[1])


# ------------------------------------------------------------------ GPT

def check_adamw_params(got, ref, m_gpu, g_ref, cfg, name):
    """Chained check of the mixed parameters after the first AdamW step from
    zero moments.  The bias-corrected moments are then m = g and v = g^2, so
    the local update is u(g) = lr g / (|g| + eps), and two runs whose
    gradients differ move a parameter apart by (1 - alpha) |u(g_gpu) -
    u(g_ref)| (up to 2 lr (1 - alpha) where the two gradients differ in
    sign).  The GPU's gradient is read back from its first moment, m =
    (1 - beta1) g (for the fused schedule the only place it is kept).  Every
    element must lie within that distance plus 1e-5 (|ref| + rms(ref)); where
    the gradients agree, that is the 1e-5 bar of the update itself."""
    got, ref, m_gpu, g_ref = (np.asarray(a, np.float64) for a in (got, ref, m_gpu, g_ref))
    if ref.size == 0:
        return
    g_gpu = m_gpu / (1.0 - cfg.beta1)
    u = lambda g: cfg.lr * g / (np.abs(g) + cfg.eps)
    rms = np.sqrt(np.mean(ref * ref))
    allow = (1.0 - cfg.alpha) * np.abs(u(g_gpu) - u(g_ref)) + 1e-5 * (np.abs(ref) + rms)
    bad = np.abs(got - ref) > allow
    if bad.any():
        i = np.unravel_index(np.argmax(np.abs(got - ref) - allow), ref.shape)
        raise AssertionError(f"{name}: {int(bad.sum())}/{bad.size} parameters beyond the update's "
                             f"propagated bar; worst at {i}: gpu={got[i]!r} ref={ref[i]!r} "
                             f"g_gpu={g_gpu[i]!r} g_ref={g_ref[i]!r}")


@pytest.mark.parametrize("cfg", [S.GPT_TEST, S.GPT_TEST_RAGGED, S.GPT_TEST_DH128, S.GPT_TEST_DH48,
                                 S.GPT2_SMALL_2L, S.GPT_TEST_T2048],
                         ids=lambda c: c.name)
def test_gpt_forward_activations(cfg):
    """Saved forward activations against the oracle's forward (bf16 storage
    points on both sides; chained)."""
    params, tokens, peers, m = gpt_setup(cfg)
    td = torch.from_numpy(tokens).to(DEV)
    loss = torch.zeros(1, dtype=torch.float32, device=DEV)
    torch.cuda.synchronize()
    LU.layup_forward(m.ctx, td, None, loss)
    oloss, dlog, cache = O.gpt_forward({k: v.astype(np.float64) for k, v in params.items()}, tokens,
                                       cfg.n_head)
    m.synchronize()
    assert abs(loss.item() - oloss) <= 2e-3 * abs(oloss)
    N, d, F = cfg.batch * cfg.seq, cfg.d_model, cfg.d_ff
    for l in range(cfg.n_layer):
        c = cache[l]
        compare_chained(m.activation(0, l).reshape(N, d), c["x"], 2e-2, f"x[{l}]")
        compare_chained(m.activation(1, l).reshape(N, d), c["a"], 2e-2, f"ln1[{l}]")
        compare_chained(m.activation(2, l).reshape(N, 3 * d), c["qkv"], 2e-2, f"qkv[{l}]")
        if cfg.d_head in (32, 64, 128):
            # fused attention: P is not stored; its normaliser is (base 2)
            compare_chained(m.activation(12, l).reshape(c["lse"].shape) * np.log(2.0), c["lse"], 1e-2,
                            f"lse[{l}]")
            with pytest.raises(RuntimeError):
                m.activation(3, l)
        else:
            compare_chained(m.activation(3, l).reshape(c["P"].shape), c["P"], 2e-2, f"P[{l}]")
        compare_chained(m.activation(4, l).reshape(N, d), c["o"], 2e-2, f"o[{l}]")
        compare_chained(m.activation(5, l).reshape(N, d), c["h"], 2e-2, f"h[{l}]")
        compare_chained(m.activation(7, l).reshape(N, F), c["f"], 2e-2, f"f[{l}]")
        compare_chained(m.activation(8, l).reshape(N, F), c["gl"], 2e-2, f"gelu[{l}]")
    compare_chained(m.activation(9).reshape(N, d), cache["xf"], 2e-2, "xf")
    # run the backward so the context is left in a clean state
    for u in range(m.n_units - 1, -1, -1):
        LU.layup_layer_backward(m.ctx, u)
    m.close()


@pytest.mark.parametrize("cfg", [S.GPT_TEST, S.GPT_TEST_RAGGED, S.GPT_TEST_DH128, S.GPT_TEST_DH48,
                                 S.GPT_TEST_W832, S.GPT_TEST_W1088, S.GPT_TEST4, S.GPT2_SMALL_2L,
                                 S.GPT_TEST_W1024, S.GPT_TEST_W2048,
                                 S.GPT_TEST_T2048],
                         ids=lambda c: c.name)
def test_gpt_step_parity(cfg):
    """One layer-wise step, chained: every gradient at rel 2e-2 (bf16 GEMM
    operands, float32 accumulation), AdamW moments and the mixed parameters as
    described in check_adamw_params, order trace exact; then the update
    teacher-forced (the oracle's update of the GPU's gradients) at 1e-5."""
    _step_parity(cfg, LU.LAYUP_SCHEDULE_LAYERWISE)


@pytest.mark.parametrize("cfg", [S.GPT_TEST, S.GPT_TEST4], ids=lambda c: c.name)
def test_after_backward_schedule_matches_oracle(cfg):
    """The comparison schedule of section 3.2 (every update after the whole
    backward pass) against the oracle's step directly, with the same bars
    as the layer-wise step: on one worker the two schedules compute the same
    step, so the oracle's layer-wise step is the reference for both."""
    _step_parity(cfg, LU.LAYUP_SCHEDULE_AFTER_BACKWARD)


def _step_parity(cfg, schedule):
    params, tokens, peers, m = gpt_setup(cfg)
    hp, ohp = gpt_hp(cfg)
    td = torch.from_numpy(tokens).to(DEV)
    loss = torch.zeros(1, dtype=torch.float32, device=DEV)
    dis = torch.zeros(m.n_units, dtype=torch.float32, device=DEV)
    torch.cuda.synchronize()
    LU.layup_step_ex(m.ctx, td, None, hp, cfg.alpha, schedule=schedule, loss_out=loss, disagreement=dis)
    op = {k: v.astype(np.float64) for k, v in params.items()}
    om = {k: np.zeros_like(v) for k, v in op.items()}
    ov = {k: np.zeros_like(v) for k, v in op.items()}
    opeer = {k: v.astype(np.float64) for k, v in peers[0].items()}
    # the same step in exact arithmetic, on copies: the spread bf16 storage
    # alone causes in the gradients and moments
    xp, xm, xv = ({k: a.copy() for k, a in d.items()} for d in (op, om, ov))
    _, xgrads, _, _ = O.gpt_step(xp, xm, xv, opeer, tokens, cfg.n_head, ohp, cfg.alpha, rnd=O.ident)
    oloss, ograds, otrace, odis = O.gpt_step(op, om, ov, opeer, tokens, cfg.n_head, ohp, cfg.alpha)
    m.synchronize()
    assert abs(loss.item() - oloss) <= 2e-3 * abs(oloss)
    g = m.read("grads")
    for k, ref in ograds.items():
        compare_chained(g[k], ref.reshape(g[k].shape), 2e-2, f"grad {k}",
                        exact=xgrads[k].reshape(g[k].shape))
    got_p, got_m, got_v = m.read("params"), m.read("m"), m.read("v")
    for k in op:
        shp = got_p[k].shape
        check_adamw_params(got_p[k], op[k].reshape(shp), got_m[k], ograds[k].reshape(shp), cfg,
                           f"param {k}")
        compare_chained(got_m[k], om[k].reshape(shp), 2e-2, f"m {k}", exact=xm[k].reshape(shp))
        compare_chained(got_v[k], ov[k].reshape(shp), 4e-2, f"v {k}", exact=xv[k].reshape(shp))
    n_units = cfg.n_layer + 2
    assert otrace == list(range(n_units - 1, -1, -1))
    assert m.read_trace() == [(0, u) for u in otrace]
    dgpu = dis.cpu().numpy()
    for u in range(n_units):
        assert abs(dgpu[u] - odis[u]) <= 5e-2 * odis[u] + 1e-12, (u, dgpu[u], odis[u])
    # teacher-forced update: the oracle's update+mix of the GPU's own
    # gradients from the step's starting state gives the GPU's parameters
    # and moments to rel 1e-5, element by element
    tp = {k: v.astype(np.float64) for k, v in params.items()}
    tm = {k: np.zeros_like(v) for k, v in tp.items()}
    tv = {k: np.zeros_like(v) for k, v in tp.items()}
    gg = {k: a.astype(np.float64) for k, a in g.items()}
    O.gpt_update_units(tp, gg, tm, tv, opeer, cfg.n_layer, ohp, cfg.alpha, t=1)
    for k in tp:
        shp = got_p[k].shape
        compare(got_p[k], tp[k].reshape(shp), 1e-5, f"teacher-forced param {k}")
        compare(got_m[k], tm[k].reshape(shp), 1e-5, f"teacher-forced m {k}")
        compare(got_v[k], tv[k].reshape(shp), 1e-5, f"teacher-forced v {k}")
    m.close()


@pytest.mark.parametrize("cfg", [S.GPT_TEST, S.GPT_TEST4, S.GPT2_SMALL], ids=lambda c: c.name)
def test_gpt_two_streams_equal_one_stream_and_repeatable(cfg):
    """Two-stream overlap vs serialized schedule and two identical runs:
    bitwise identical parameters, moments, gradients and bf16 weight copies
    after two steps (race detector; no float atomics anywhere on the path).
    With four or more blocks the dY operands of the dW GEMMs, double-buffered
    by block parity, are overwritten two blocks later while the update
    stream may still read them: a missing or misplaced wait changes bits.
    GPT-2-small runs all twelve blocks at full size."""
    outs = []
    for two in (True, False, True):
        params, tokens, peers, m = gpt_setup(cfg, two)
        hp, _ = gpt_hp(cfg)
        td = torch.from_numpy(tokens).to(DEV)
        torch.cuda.synchronize()
        for s in range(2):
            hp.step = s + 1
            LU.layup_step(m.ctx, td, None, hp, cfg.alpha, 0)
        m.synchronize()
        outs.append([t.clone() for t in (m.params, m.m, m.v, m.grads, m.params_bf16)])
        m.close()
        del m
    for run in (1, 2):
        for name, a, b in zip(("params", "m", "v", "grads", "bf16 copy"), outs[0], outs[run]):
            assert torch.equal(a, b), (run, name)


def test_gpt_repeated_and_out_of_vocabulary_tokens_two_streams_equal_one_stream():
    """A batch of few distinct tokens, repeated, with some outside the
    vocabulary (which gather no embedding row and get no gradient): the
    two-stream step equals the one-stream step bit for bit over two steps,
    disagreements included."""
    cfg = S.GPT_TEST4
    rng = np.random.default_rng(77)
    tokens = rng.integers(0, 12, (cfg.batch, cfg.seq + 1)).astype(np.int32)
    tokens[0, ::7] = -1
    tokens[1, 3::11] = cfg.vocab + 5
    outs = []
    for two in (True, False):
        params, _, peers, m = gpt_setup(cfg, two)
        td = torch.from_numpy(tokens).to(DEV)
        dis = torch.zeros(m.n_units, dtype=torch.float32, device=DEV)
        torch.cuda.synchronize()
        for s in range(2):
            hp, _ = gpt_hp(cfg, s + 1)
            LU.layup_step(m.ctx, td, None, hp, cfg.alpha, 0, None, dis)
        m.synchronize()
        outs.append([t.clone() for t in (m.params, m.m, m.v, m.grads, m.params_bf16)] + [dis.clone()])
        assert m.read_trace() == [(s, u) for s in range(2) for u in range(m.n_units - 1, -1, -1)]
        m.close()
        del m
    for name, a, b in zip(("params", "m", "v", "grads", "bf16 copy", "disagreement"), outs[0], outs[1]):
        assert torch.equal(a, b), name


def test_gpt_manual_unit_calls_match_step():
    """Driving forward / backward(u) / update(u) by hand equals layup_step, and
    out-of-order calls are refused."""
    cfg = S.GPT_TEST
    params, tokens, peers, m = gpt_setup(cfg)
    hp, _ = gpt_hp(cfg)
    td = torch.from_numpy(tokens).to(DEV)
    torch.cuda.synchronize()
    with pytest.raises(LU.LayupError) as e:
        LU.layup_layer_backward(m.ctx, 0)
    assert e.value.status == LU.LAYUP_ERR_STATE
    LU.layup_forward(m.ctx, td, None, None)
    with pytest.raises(LU.LayupError) as e:
        LU.layup_layer_backward(m.ctx, 0)           # must start at the last unit
    assert e.value.status == LU.LAYUP_ERR_STATE
    for u in range(m.n_units - 1, -1, -1):
        LU.layup_layer_backward(m.ctx, u)
        LU.layup_unit_update_mix(m.ctx, u, hp, cfg.alpha, 0)
    m.synchronize()
    manual = m.params.cpu().numpy().copy()
    m.close()
    params, tokens, peers, m2 = gpt_setup(cfg)
    torch.cuda.synchronize()
    LU.layup_step(m2.ctx, td, None, hp, cfg.alpha, 0)
    m2.synchronize()
    assert np.array_equal(manual, m2.params.cpu().numpy())
    m2.close()


def test_gpt_peer_slots_select_replicas():
    """With three resident peer replicas, the step mixes with the slot it is
    given (1.3B workload reading: one peer slot drawn per step)."""
    cfg = S.GPT_TEST
    params, tokens, peers, m = gpt_setup(cfg, n_peers=3)
    hp, ohp = gpt_hp(cfg)
    td = torch.from_numpy(tokens).to(DEV)
    torch.cuda.synchronize()
    LU.layup_step(m.ctx, td, None, hp, cfg.alpha, 2)
    op = {k: v.astype(np.float64) for k, v in params.items()}
    om = {k: np.zeros_like(v) for k, v in op.items()}
    ov = {k: np.zeros_like(v) for k, v in op.items()}
    _, ograds, _, _ = O.gpt_step(op, om, ov, {k: v.astype(np.float64) for k, v in peers[2].items()},
                                 tokens, cfg.n_head, ohp, cfg.alpha)
    got, got_m = m.read("params"), m.read("m")
    for k in ["lnf.g", "h1.ln2.b", "h0.qkv.w"]:
        check_adamw_params(got[k], op[k].reshape(got[k].shape), got_m[k], ograds[k].reshape(got[k].shape),
                           cfg, k)
    m.close()


def test_gpt2_small_full_size_step_properties():
    """GPT-2-small at full size (12 x 768, 12 heads, T 1024, B 8, vocab 50257):
    the loss at initialisation matches its closed form, every gradient and
    parameter is finite, the order trace is exact, and the embedding padding
    rows stay zero.  Closed form: the final LayerNorm output has unit variance
    per feature and the tied head is N(0, 0.02^2), so the logits are close to
    Gaussian with variance s2 = d * 0.02^2 and E[logsumexp] = ln V + s2/2."""
    cfg = S.GPT2_SMALL
    params, tokens, peers, m = gpt_setup(cfg)
    hp, _ = gpt_hp(cfg)
    td = torch.from_numpy(tokens).to(DEV)
    loss = torch.zeros(1, dtype=torch.float32, device=DEV)
    torch.cuda.synchronize()
    LU.layup_step(m.ctx, td, None, hp, cfg.alpha, 0, loss)
    m.synchronize()
    expected = math.log(cfg.vocab) + 0.5 * cfg.d_model * 0.02 ** 2
    assert abs(loss.item() - expected) < 0.02, (loss.item(), expected)
    assert torch.isfinite(m.grads).all().item() and torch.isfinite(m.params).all().item()
    assert m.read_trace() == [(0, u) for u in range(13, -1, -1)]
    wte = m.by_name["wte"]
    pad = m.params[wte["offset"] + wte["numel"]: wte["offset"] + wte["padded_rows"] * wte["cols"]]
    assert pad.numel() == 47 * 768 and torch.count_nonzero(pad).item() == 0
    m.close()


def test_gemm_timing_counts_the_block_backward_gemms():
    """layup_gemm_timing brackets each block's eight linear-layer backward
    GEMMs (dX and dW of qkv, proj, fc, mproj): count and FLOPs are exact, the
    time positive; turning it off leaves later steps untimed."""
    cfg = S.GPT_TEST
    params, tokens, peers, m = gpt_setup(cfg)
    hp, _ = gpt_hp(cfg)
    td = torch.from_numpy(tokens).to(DEV)
    LU.layup_gemm_timing(m.ctx, True)
    LU.layup_step(m.ctx, td, None, hp, cfg.alpha, 0)
    ms, n, flops = LU.layup_gemm_timing_read(m.ctx)
    Ntok, d, F = cfg.batch * cfg.seq, cfg.d_model, cfg.d_ff
    per_block = 2 * Ntok * (3 * d * d + d * d + F * d + d * F) * 2   # dX and dW of each linear
    assert n == 8 * cfg.n_layer
    assert flops == per_block * cfg.n_layer
    assert ms > 0
    LU.layup_gemm_timing(m.ctx, False)
    hp.step = 2
    LU.layup_step(m.ctx, td, None, hp, cfg.alpha, 0)
    assert LU.layup_gemm_timing_read(m.ctx)[1] == 0
    m.close()


@pytest.mark.parametrize("cfg", [S.GPT_TEST, S.GPT_TEST_LONG], ids=lambda c: c.name)
def test_fused_dw_schedule_matches_oracle(cfg):
    """The fused schedule (each block's weight matrices updated and mixed by
    their dW GEMM, in its epilogue or, with 2048 tokens, in its split-K sum):
    parameters and AdamW moments against the oracle's layer-wise step as in
    test_gpt_step_parity, the order trace unchanged, and the bf16 copy equal
    to the nearest-even bf16 of the updated float32 weights."""
    params, tokens, peers, m = gpt_setup(cfg)
    hp, ohp = gpt_hp(cfg)
    td = torch.from_numpy(tokens).to(DEV)
    loss = torch.zeros(1, dtype=torch.float32, device=DEV)
    torch.cuda.synchronize()
    LU.layup_step_ex(m.ctx, td, None, hp, cfg.alpha, schedule=LU.LAYUP_SCHEDULE_FUSED_DW, loss_out=loss)
    op = {k: v.astype(np.float64) for k, v in params.items()}
    om = {k: np.zeros_like(v) for k, v in op.items()}
    ov = {k: np.zeros_like(v) for k, v in op.items()}
    opeer = {k: v.astype(np.float64) for k, v in peers[0].items()}
    xp, xm, xv = ({k: a.copy() for k, a in d.items()} for d in (op, om, ov))
    O.gpt_step(xp, xm, xv, opeer, tokens, cfg.n_head, ohp, cfg.alpha, rnd=O.ident)
    oloss, ograds, otrace, _ = O.gpt_step(op, om, ov, opeer, tokens, cfg.n_head, ohp, cfg.alpha)
    m.synchronize()
    assert abs(loss.item() - oloss) <= 2e-3 * abs(oloss)
    got_p, got_m, got_v = m.read("params"), m.read("m"), m.read("v")
    for k in op:
        shp = got_p[k].shape
        check_adamw_params(got_p[k], op[k].reshape(shp), got_m[k], ograds[k].reshape(shp), cfg,
                           f"param {k}")
        compare_chained(got_m[k], om[k].reshape(shp), 2e-2, f"m {k}", exact=xm[k].reshape(shp))
        compare_chained(got_v[k], ov[k].reshape(shp), 4e-2, f"v {k}", exact=xv[k].reshape(shp))
    assert m.read_trace() == [(0, u) for u in otrace]
    p16 = (m.params_bf16.to(torch.int32) << 16).view(torch.float32).cpu().numpy()
    assert np.array_equal(p16, O.bf16(m.params.cpu().numpy().astype(np.float64)))
    m.close()


def test_fused_dw_schedule_argument_checks():
    cfg = S.GPT_TEST
    params, tokens, peers, m = gpt_setup(cfg)
    hp, _ = gpt_hp(cfg)
    td = torch.from_numpy(tokens).to(DEV)
    dis = torch.zeros(m.n_units, dtype=torch.float32, device=DEV)
    with pytest.raises(LU.LayupError):
        LU.layup_step_ex(m.ctx, td, None, hp, 0.5, schedule=LU.LAYUP_SCHEDULE_FUSED_DW, disagreement=dis)
    other = torch.zeros_like(m.params)
    with pytest.raises(LU.LayupError):
        LU.layup_step_ex(m.ctx, td, None, hp, 0.5, schedule=LU.LAYUP_SCHEDULE_FUSED_DW,
                         mix_mode=LU.LAYUP_MIX_PUSH, push_params=other)
    m.close()
    mcfg = S.MLP_TINY
    mm = LU.Model(LU.mlp_config(mcfg.dims, mcfg.batch), "sgd")
    x, y = S.mlp_inputs(mcfg)
    with pytest.raises(LU.LayupError):
        LU.layup_step_ex(mm.ctx, torch.from_numpy(y[0]).to(DEV), torch.from_numpy(x[0]).to(DEV),
                         LU.hparams("sgd", mcfg.lr, mcfg.momentum, 0.0), 0.5,
                         schedule=LU.LAYUP_SCHEDULE_FUSED_DW)
    mm.close()
