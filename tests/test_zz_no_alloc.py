"""The allocation-free update+mix entry point (layup_layer_update_mix_static,
for callers that cannot allocate device memory) against the entry point it
varies (layup_layer_update_mix with a context, whose workspace holds the
disagreement partial sums): the same kernels, so parameters, moments, bf16
copies and the disagreement must be bit-identical.  Two calls in a row, the
second with fewer elements (fewer partial sums than the first left in the
library's array), in both mixing forms and for both optimizers."""
import numpy as np
import pytest

from paper_2410_05985_amd import synthetic as S

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
from paper_2410_05985_amd import layup as LU  # noqa: E402

DEV = "cuda"


def _make(sizes, seed, optim):
    out = []
    for i, n in enumerate(sizes):
        p, g, m, v, q = S.update_mix_inputs(n, seed + i, optim)
        t = {k: torch.from_numpy(a).to(DEV) for k, a in (("p", p), ("g", g), ("m", m), ("q", q))}
        t["v"] = torch.from_numpy(v).to(DEV) if v is not None else None
        t["p16"] = torch.zeros(n, dtype=torch.int16, device=DEV)
        t["q16"] = torch.zeros(n, dtype=torch.int16, device=DEV)
        out.append(t)
    return out


def _clone(ts):
    return [{k: (a.clone() if a is not None else None) for k, a in t.items()} for t in ts]


def _descs(ts, push):
    ds = []
    for i, t in enumerate(ts):
        d = LU.layup_tensor()
        d.param, d.grad, d.state0 = t["p"].data_ptr(), t["g"].data_ptr(), t["m"].data_ptr()
        d.state1 = t["v"].data_ptr() if t["v"] is not None else None
        d.peer = t["q"].data_ptr()
        d.param_bf16 = t["p16"].data_ptr()
        d.peer_bf16 = t["q16"].data_ptr() if push else None
        d.numel = t["p"].numel()
        d.decay = i % 2
        ds.append(d)
    return ds


@pytest.mark.parametrize("push", [False, True], ids=["pull", "push"])
@pytest.mark.parametrize("optim", ["sgd", "adamw"])
def test_static_scratch_equals_context_entry_point(optim, push, layup_ctx):
    hp = (LU.hparams("adamw", 7.5249e-4, 0.0, 0.1, 0.9, 0.95, 1e-8, 3) if optim == "adamw"
          else LU.hparams("sgd", 0.1, 0.9, 5e-5))
    mode = LU.LAYUP_MIX_PUSH if push else LU.LAYUP_MIX_PULL
    stream = torch.cuda.current_stream()
    for call, sizes in enumerate([(2_000_003, 4097, 64, 5), (70_001, 3)]):
        a = _make(sizes, 100 + 10 * call, optim)
        b = _clone(a)
        dis_a = torch.full((1,), -1.0, dtype=torch.float32, device=DEV)
        dis_b = torch.full((1,), -2.0, dtype=torch.float32, device=DEV)
        torch.cuda.synchronize()
        LU.layup_layer_update_mix(layup_ctx, _descs(a, push), hp, 0.5, disagreement=dis_a, stream=stream,
                                  mix_mode=mode)
        LU.layup_layer_update_mix_static(_descs(b, push), hp, 0.5, disagreement=dis_b, stream=stream,
                                         mix_mode=mode)
        torch.cuda.synchronize()
        for ta, tb in zip(a, b):
            for k in ("p", "m", "v", "q", "p16", "q16"):
                if ta[k] is not None:
                    assert torch.equal(ta[k], tb[k]), (call, k)
        assert dis_a.item() > 0
        assert torch.equal(dis_a, dis_b), (call, dis_a.item(), dis_b.item())


def test_static_scratch_argument_checks():
    """More than 16 tensors with a disagreement output is refused before any
    work is enqueued; without the disagreement output they are accepted."""
    hp = LU.hparams("sgd", 0.1, 0.9, 0.0)
    ts = _make([8] * 17, 7, "sgd")
    dis = torch.zeros(1, dtype=torch.float32, device=DEV)
    with pytest.raises(LU.LayupError) as e:
        LU.layup_layer_update_mix_static(_descs(ts, False), hp, 0.5, disagreement=dis)
    assert e.value.status == LU.LAYUP_ERR_INVALID_ARG
    LU.layup_layer_update_mix_static(_descs(ts, False), hp, 0.5, stream=torch.cuda.current_stream())
    torch.cuda.synchronize()
