"""Replicas resident on one GPU that exchange layers as Algorithm 1 writes
it (push mode: the sender keeps its local update and overwrites the
receiver's layer), with push-sum mixing weights (section 3.1), and the two
update schedules (section 3.2 layer-wise against updates after the whole
backward pass).  Every GPU result is compared with the oracle run on the same
seeded inputs; tolerances as for the single-worker step (rel 1e-5 for the
float32 update+mix alone, 1e-4 for the float32 MLP over several steps, the
chained bf16 rule for the GPT)."""
import numpy as np
import pytest

import oracle as O
from paper_2410_05985_amd import synthetic as S
from tests.parity import compare, compare_chained

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
from paper_2410_05985_amd import layup as LU  # noqa: E402

DEV = "cuda"
HP = dict(lr=7.5249e-4, momentum=0.9, weight_decay=0.1, beta1=0.9, beta2=0.95, eps=1e-8)


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _bf16_to_f32(t16):
    return (t16.to(torch.int32) << 16).view(torch.float32).cpu().numpy()


# ------------------------------------------------------------ push kernel

@pytest.mark.parametrize("optim", ["sgd", "adamw"])
@pytest.mark.parametrize("n", [5, 4096, 70001])
def test_push_update_parity(optim, n):
    """Push mode of the fused kernel: own layer locally updated, the
    receiver's layer mixed in place, both bf16 copies rewritten."""
    p, g, m, v, q = S.update_mix_inputs(n, 300 + n % 89, optim)
    alpha = float(np.float32(0.3))
    d = dict(p=_dev(p), g=_dev(g), m=_dev(m), v=_dev(v) if v is not None else None, q=_dev(q))
    p16 = torch.zeros(n, dtype=torch.int16, device=DEV)
    q16 = torch.zeros(n, dtype=torch.int16, device=DEV)
    desc = LU.layup_tensor(param=d["p"].data_ptr(), grad=d["g"].data_ptr(), state0=d["m"].data_ptr(),
                           state1=d["v"].data_ptr() if d["v"] is not None else None,
                           peer=d["q"].data_ptr(), param_bf16=p16.data_ptr(), peer_bf16=q16.data_ptr(),
                           numel=n, decay=1)
    hp = LU.hparams(optim, HP["lr"], HP["momentum"], HP["weight_decay"], HP["beta1"], HP["beta2"],
                    HP["eps"], 3)
    torch.cuda.synchronize()
    LU.layup_layer_update_mix(None, [desc], hp, alpha, stream=torch.cuda.current_stream(),
                              mix_mode=LU.LAYUP_MIX_PUSH)
    torch.cuda.synchronize()
    p1, m1, v1, q2, _ = O.update_push(p, g, m, v, q, dict(HP, optim=optim), alpha, 3, wd_on=True)
    compare(d["p"].cpu().numpy(), p1, 1e-5, "own p")
    compare(d["m"].cpu().numpy(), m1, 1e-5, "own m")
    if optim == "adamw":
        compare(d["v"].cpu().numpy(), v1, 1e-5, "own v")
    compare(d["q"].cpu().numpy(), q2, 1e-5, "receiver q")
    # the bf16 copies are the nearest-even bf16 of the stored float32 values
    assert np.array_equal(_bf16_to_f32(p16), O.bf16(d["p"].cpu().numpy().astype(np.float64)))
    assert np.array_equal(_bf16_to_f32(q16), O.bf16(d["q"].cpu().numpy().astype(np.float64)))


def test_push_sum_mass_conserved_on_device():
    """At lr 0 a push-sum exchange keeps sum_k w_k x_k: 40 exchanges among 3
    replicas, alpha from the library's push-sum functions, the mix in the
    kernel's push mode.  Float32 storage rounds each mix; the weighted sum
    stays within 1e-5 of the start and every replica matches the oracle."""
    M, n, steps = 3, 10007, 40
    rng = np.random.default_rng(5)
    xs = [rng.standard_normal(n).astype(np.float32) for _ in range(M)]
    dev = [_dev(x) for x in xs]
    zeros = torch.zeros(n, dtype=torch.float32, device=DEV)
    mom = [torch.zeros(n, dtype=torch.float32, device=DEV) for _ in range(M)]
    hp = LU.hparams("sgd", 0.0, 0.0, 0.0)
    w = np.full(M, 1.0 / M)
    mass0 = sum(w[k] * xs[k].astype(np.float64) for k in range(M))
    ox = [x.astype(np.float64) for x in xs]
    ow = [1.0 / M] * M
    pairs = S.gossip_pairs(steps, M, seed=6)
    torch.cuda.synchronize()
    for i, j in pairs:
        alpha = LU.layup_push_sum_send(w, i, j)
        desc = LU.layup_tensor(param=dev[i].data_ptr(), grad=zeros.data_ptr(), state0=mom[i].data_ptr(),
                               peer=dev[j].data_ptr(), numel=n, decay=0)
        LU.layup_layer_update_mix(None, [desc], hp, alpha, stream=torch.cuda.current_stream(),
                                  mix_mode=LU.LAYUP_MIX_PUSH)
        LU.layup_push_sum_receive(w, i, j)
        ow, oa = O.push_sum_round(ow, i, j)
        ox[j] = O.f32(O.mix(ox[j], ox[i], float(np.float32(oa))))
    torch.cuda.synchronize()
    got = [d.cpu().numpy() for d in dev]
    mass = sum(w[k] * got[k].astype(np.float64) for k in range(M))
    err = np.linalg.norm(mass - mass0) / np.linalg.norm(mass0)
    assert err < 1e-5, err
    assert abs(w.sum() - 1.0) < 1e-12
    for k in range(M):
        compare(got[k], ox[k], 1e-5, f"replica {k}")


# ------------------------------------------------------ resident replicas

def test_gossip_mlp_replicas_match_oracle():
    """Three float32 MLP replicas on one GPU take 6 steps in turn; each step
    is Algorithm 1 for its worker: forward and layer-wise backward on its own
    batch, local SGD-momentum update of each layer, the updated layer pushed
    into a random receiver with the push-sum alpha.  All replicas match the
    oracle run of the same schedule."""
    cfg = S.MLP_TINY
    M, steps = 3, 6
    x, y = S.mlp_inputs(cfg)
    base = S.mlp_params(cfg)
    init = [base] + [S.peer_of(base, 0.01, seed=2 + 100 * k) for k in range(1, M)]
    streams = (torch.cuda.Stream(), torch.cuda.Stream())
    models = []
    for k in range(M):
        mk = LU.Model(LU.mlp_config(cfg.dims, cfg.batch), "sgd", streams=streams)
        mk.load("params", init[k])
        models.append(mk)
    hp = LU.hparams("sgd", cfg.lr, cfg.momentum, 0.0)
    ohp = dict(optim="sgd", lr=cfg.lr, momentum=cfg.momentum, weight_decay=0.0)
    xd, yd = _dev(x), _dev(y)
    loss = torch.zeros(1, dtype=torch.float32, device=DEV)
    op = [{k_: v_.astype(np.float64) for k_, v_ in p.items()} for p in init]
    om = [{k_: np.zeros_like(v_) for k_, v_ in p.items()} for p in op]
    w = np.full(M, 1.0 / M)
    ow = [1.0 / M] * M
    torch.cuda.synchronize()
    for s, (i, j) in enumerate(S.gossip_pairs(steps, M)):
        b = s % cfg.steps
        alpha = LU.layup_push_sum_send(w, i, j)
        LU.layup_step_ex(models[i].ctx, yd[b], xd[b], hp, alpha, mix_mode=LU.LAYUP_MIX_PUSH,
                         push_params=models[j].params, loss_out=loss)
        LU.layup_push_sum_receive(w, i, j)
        ow, oa = O.push_sum_round(ow, i, j)
        assert alpha == float(np.float32(oa))
        oloss, _, _, _ = O.mlp_step(op[i], om[i], op[j], x[b], y[b], ohp, alpha, push=True)
        models[i].synchronize()
        assert abs(loss.item() - oloss) <= 1e-4 * abs(oloss), (s, loss.item(), oloss)
    for k in range(M):
        got = models[k].read("params")
        mom = models[k].read("m")
        for n_ in op[k]:
            compare(got[n_], op[k][n_].reshape(got[n_].shape), 1e-4, f"replica {k} {n_}")
            compare(mom[n_], om[k][n_].reshape(mom[n_].shape), 1e-4, f"replica {k} momentum {n_}")
        # trace of worker k: its own steps, units in reverse order
        own = [s for s, (i, _) in enumerate(S.gossip_pairs(steps, M)) if i == k]
        assert models[k].read_trace() == [(t, u) for t in range(len(own)) for u in (2, 1, 0)]
    for mk in models:
        mk.close()


def test_gossip_gpt_replicas_match_oracle():
    """Two bf16 GPT replicas (2 blocks x 128) alternate 4 steps with AdamW in
    push mode: the receiver's float32 layers and their bf16 copy (read by its
    next forward) come from the sender's kernel.  Teacher-forced per step:
    the step's gradients are compared with the oracle's on the same replica
    state (chained bf16 rule), then the oracle applies Algorithm 1's updates
    with the GPU's gradients, so the replicas' parameters are held to the
    float32 update bar (1e-5).  (Without teacher forcing, AdamW's sign-like
    early steps turn a bf16 sign flip of a near-zero gradient into a 2 lr
    move, which compounds over steps.)"""
    cfg = S.GPT_TEST
    M, steps = 2, 4
    base = S.gpt_params(cfg)
    init = [base, S.gpt_peer(cfg, base, slot=1)]
    lc = LU.gpt_config(cfg.n_layer, cfg.d_model, cfg.n_head, cfg.d_ff, cfg.seq, cfg.batch, cfg.vocab)
    streams = (torch.cuda.Stream(), torch.cuda.Stream())
    ws = None
    models = []
    for k in range(M):
        mk = LU.Model(lc, "adamw", streams=streams, workspace=ws)
        ws = mk.workspace      # one workspace: the replicas' steps never overlap
        mk.load("params", init[k])
        models.append(mk)
    ohp = dict(optim="adamw", lr=cfg.lr, weight_decay=cfg.weight_decay, beta1=cfg.beta1,
               beta2=cfg.beta2, eps=cfg.eps)
    op = [{k_: v_.astype(np.float64) for k_, v_ in p.items()} for p in init]
    om = [{k_: np.zeros_like(v_) for k_, v_ in p.items()} for p in op]
    ov = [{k_: np.zeros_like(v_) for k_, v_ in p.items()} for p in op]
    w = np.full(M, 1.0 / M)
    ow = [1.0 / M] * M
    t = [0] * M
    loss = torch.zeros(1, dtype=torch.float32, device=DEV)
    torch.cuda.synchronize()
    for s, (i, j) in enumerate(S.gossip_pairs(steps, M)):
        tokens = S.gpt_tokens(cfg, seed=10 + s)
        t[i] += 1
        hp = LU.hparams("adamw", cfg.lr, 0.0, cfg.weight_decay, cfg.beta1, cfg.beta2, cfg.eps, t[i])
        alpha = LU.layup_push_sum_send(w, i, j)
        td = _dev(tokens)     # read asynchronously by the step: kept until it is done
        LU.layup_step_ex(models[i].ctx, td, None, hp, alpha, mix_mode=LU.LAYUP_MIX_PUSH,
                         push_params=models[j].params, push_params_bf16=models[j].params_bf16,
                         loss_out=loss)
        LU.layup_push_sum_receive(w, i, j)
        ow, oa = O.push_sum_round(ow, i, j)
        assert alpha == float(np.float32(oa))
        oloss, ograds, _, _ = O.gpt_step(op[i], om[i], ov[i], op[j], tokens, cfg.n_head, ohp, alpha,
                                         t=t[i], update=False)
        # the same step in exact arithmetic: the spread bf16 storage alone causes
        _, xgrads, _, _ = O.gpt_step(op[i], om[i], ov[i], op[j], tokens, cfg.n_head, ohp, alpha,
                                     t=t[i], update=False, rnd=O.ident)
        models[i].synchronize()
        assert abs(loss.item() - oloss) <= 2e-3 * abs(oloss), (s, loss.item(), oloss)
        g = models[i].read("grads")
        for n_, ref in ograds.items():
            compare_chained(g[n_], ref.reshape(g[n_].shape), 2e-2, f"step {s} grad {n_}",
                            exact=xgrads[n_].reshape(g[n_].shape))
        gg = {n_: g[n_].astype(np.float64).reshape(op[i][n_].shape) for n_ in g}
        O.gpt_update_units(op[i], gg, om[i], ov[i], op[j], cfg.n_layer, ohp, alpha, t=t[i], push=True)
    for k in range(M):
        got = models[k].read("params")
        mom, vv = models[k].read("m"), models[k].read("v")
        for n_ in op[k]:
            compare(got[n_], op[k][n_].reshape(got[n_].shape), 1e-5, f"replica {k} {n_}")
            compare(mom[n_], om[k][n_].reshape(mom[n_].shape), 1e-5, f"replica {k} m {n_}")
            compare(vv[n_], ov[k][n_].reshape(vv[n_].shape), 1e-5, f"replica {k} v {n_}")
        # the bf16 copy is the nearest-even bf16 of the float32 parameters
        p16 = _bf16_to_f32(models[k].params_bf16)
        flat = models[k].params.cpu().numpy().astype(np.float64)
        assert np.array_equal(p16, O.bf16(flat))
    for mk in models:
        mk.close()


# ------------------------------------------------------------- schedules

def _gpt_model(cfg, params, peer, two_streams=True):
    lc = LU.gpt_config(cfg.n_layer, cfg.d_model, cfg.n_head, cfg.d_ff, cfg.seq, cfg.batch, cfg.vocab)
    m = LU.Model(lc, "adamw", two_streams=two_streams)
    m.load("params", params)
    m.load("peers", peer)
    return m


def test_after_backward_schedule_equals_layerwise_and_lands_later():
    """On one worker, updating every unit after the whole backward pass gives
    bit-identical results to the layer-wise schedule (no unit's backward reads
    a unit updated before it); the timeline shows the difference in when the
    updates land: after the whole backward, no update is applied before the
    last gradient is ready, while layer-wise updates land after their own
    gradient only."""
    cfg = S.GPT_TEST
    params = S.gpt_params(cfg)
    peer = S.gpt_peer(cfg, params)
    tokens = _dev(S.gpt_tokens(cfg))
    out = {}
    for sched in (LU.LAYUP_SCHEDULE_LAYERWISE, LU.LAYUP_SCHEDULE_AFTER_BACKWARD):
        m = _gpt_model(cfg, params, peer)
        dis = torch.zeros(m.n_units, dtype=torch.float32, device=DEV)
        for step in (1, 2):
            hp = LU.hparams("adamw", cfg.lr, 0.0, cfg.weight_decay, cfg.beta1, cfg.beta2, cfg.eps, step)
            LU.layup_step_ex(m.ctx, tokens, None, hp, cfg.alpha, schedule=sched, disagreement=dis)
        fwd, ready, applied = LU.layup_unit_timeline(m.ctx, m.n_units)
        assert 0 < fwd < min(ready)
        out[sched] = dict(p=m.params.cpu().numpy(), mo=m.m.cpu().numpy(), v=m.v.cpu().numpy(),
                          g=m.grads.cpu().numpy(), dis=dis.cpu().numpy(), trace=m.read_trace(),
                          ready=ready, applied=applied)
        m.close()
    a, b = out[LU.LAYUP_SCHEDULE_LAYERWISE], out[LU.LAYUP_SCHEDULE_AFTER_BACKWARD]
    for k in ("p", "mo", "v", "g", "dis"):
        assert np.array_equal(a[k], b[k]), k
    assert a["trace"] == b["trace"]
    U = len(a["ready"])
    for u in range(U):
        assert a["applied"][u] >= a["ready"][u], (u, a["ready"][u], a["applied"][u])
    assert min(b["applied"]) >= max(b["ready"]), (b["ready"], b["applied"])
    # the gradient of unit 0 is the last one produced in both schedules
    assert max(a["ready"]) == a["ready"][0] and max(b["ready"]) == b["ready"][0]


def test_drift_of_the_two_schedules_gpt2_small():
    """Section 3.2's drift at GPT-2-small's full size, from the HIP-event
    timeline of the third step of each schedule.  The drift of a unit is the
    delay from its gradient being ready to its update being applied.

    * After the whole backward pass, every update lands after the last
      gradient, and the delay grows with the unit's distance from the input
      over the blocks and the top unit (a unit's gradient is ready one
      unit-backward earlier than the one below it, and updates take a small
      fraction of a unit-backward).  The embeddings' unit is left out: its
      gradient comes last and its update is the largest.
    * The summed delay D lies within [0.5, 1.25] of the paper's model
      beta T (L + 1) / 2, with beta T the measured backward time and L the
      number of units: the model takes every unit's backward to last
      beta T / L, while here the top unit (the tied head) takes longer and the
      embeddings' unit much less.
    * The layer-wise schedule's summed delay is a small fraction of it."""
    cfg = S.GPT2_SMALL
    params = S.gpt_params(cfg)
    peer = S.gpt_peer(cfg, params)
    tokens = _dev(S.gpt_tokens(cfg))
    res = {}
    for sched in (LU.LAYUP_SCHEDULE_LAYERWISE, LU.LAYUP_SCHEDULE_AFTER_BACKWARD):
        m = _gpt_model(cfg, params, peer)
        for step in (1, 2, 3):
            hp = LU.hparams("adamw", cfg.lr, 0.0, cfg.weight_decay, cfg.beta1, cfg.beta2, cfg.eps, step)
            LU.layup_step_ex(m.ctx, tokens, None, hp, cfg.alpha, schedule=sched)
        res[sched] = LU.layup_unit_timeline(m.ctx, m.n_units)
        U = m.n_units
        m.close()
        del m
    fwd, ready, applied = res[LU.LAYUP_SCHEDULE_AFTER_BACKWARD]
    delay = [applied[u] - ready[u] for u in range(U)]
    assert min(applied) >= max(ready) == ready[0]
    for u in range(1, U - 1):
        assert delay[u + 1] > delay[u], (u, delay)
    d_after = sum(delay)
    beta_t = ready[0] - fwd
    model = beta_t * (U + 1) / 2
    assert 0.5 * model <= d_after <= 1.25 * model, (d_after, model)
    fwd_l, ready_l, applied_l = res[LU.LAYUP_SCHEDULE_LAYERWISE]
    d_layer = sum(applied_l[u] - ready_l[u] for u in range(U))
    assert 0 < d_layer < 0.2 * d_after, (d_layer, d_after)


def test_step_ex_argument_checks():
    cfg = S.GPT_TEST
    params = S.gpt_params(cfg)
    m = _gpt_model(cfg, params, S.gpt_peer(cfg, params))
    tokens = _dev(S.gpt_tokens(cfg))
    hp = LU.hparams("adamw", cfg.lr, 0.0, cfg.weight_decay, cfg.beta1, cfg.beta2, cfg.eps, 1)
    with pytest.raises(LU.LayupError):
        LU.layup_step_ex(m.ctx, tokens, None, hp, 0.5, schedule=7)
    with pytest.raises(LU.LayupError):
        LU.layup_step_ex(m.ctx, tokens, None, hp, 0.5, mix_mode=LU.LAYUP_MIX_PUSH)   # no receiver
    with pytest.raises(LU.LayupError):   # pushing into itself
        LU.layup_step_ex(m.ctx, tokens, None, hp, 0.5, mix_mode=LU.LAYUP_MIX_PUSH, push_params=m.params)
    with pytest.raises(LU.LayupError):
        LU.layup_unit_timeline(m.ctx, m.n_units)   # no step has run
    m.close()
