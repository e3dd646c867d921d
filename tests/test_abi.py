"""The C ABI library loads, exports every entry point include/layup.h
declares, and its host-side checks and layout logic behave -- no GPU needed
(no call here launches a kernel or touches a device)."""
import ctypes as C
import os
import re

import pytest

from paper_2410_05985_amd import layup as LU
from paper_2410_05985_amd import synthetic as S

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(LU.LIB_PATH):
        from paper_2410_05985_amd import build
        build.build()
    return LU.lib()


def header_functions():
    src = open(os.path.join(ROOT, "include", "layup.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w]+\**\s+\**(layup_\w+)\s*\(", src, flags=re.M)))


def test_every_declared_symbol_is_exported(L):
    names = header_functions()
    assert len(names) >= 17, names
    for n in names:
        assert hasattr(L, n), n
    assert sorted(LU.EXPORTS) == names


def test_gpt2_small_layout():
    cfg = LU.gpt_config(12, 768, 12, 3072, 1024, 8, 50257)
    nt, nu, total = LU.layup_param_layout(cfg)
    assert nu == 14 and nt == 2 + 12 * 12 + 2
    infos = [LU.layup_tensor_layout(cfg, i) for i in range(nt)]
    logical = sum(t["numel"] for t in infos)
    assert logical == 124_439_808 == S.GPT2_SMALL.n_params()
    for t in infos:
        assert t["offset"] % 64 == 0
    wte = [t for t in infos if t["name"] == "wte"][0]
    assert wte["padded_rows"] == 50304 and wte["rows"] == 50257 and wte["unit"] == 0
    # units are contiguous and in unit order; decayed tensors first in a unit
    units = [t["unit"] for t in infos]
    assert units == sorted(units)
    for u in range(nu):
        dec = [t["decay"] for t in infos if t["unit"] == u]
        assert dec == sorted(dec, reverse=True)
    # shapes agree with the model description used by the oracle
    spec = {n: s for n, s, _ in S.gpt_param_specs(S.GPT2_SMALL)}
    for t in infos:
        shape = (t["rows"], t["cols"]) if t["cols"] > 1 else (t["rows"],)
        assert spec[t["name"]] == shape, t["name"]


def test_mlp_layout_and_workspace():
    cfg = LU.mlp_config((512, 256, 256, 10), 32)
    nt, nu, total = LU.layup_param_layout(cfg)
    assert (nt, nu) == (6, 3)
    assert sum(LU.layup_tensor_layout(cfg, i)["numel"] for i in range(nt)) == 199_690
    assert LU.layup_workspace_size(cfg) > 0


def test_workspace_size_grows_with_model():
    small = LU.layup_workspace_size(LU.gpt_config(2, 128, 2, 512, 128, 2, 1000))
    big = LU.layup_workspace_size(LU.gpt_config(12, 768, 12, 3072, 1024, 8, 50257))
    assert 0 < small < big < 64 << 30


@pytest.mark.parametrize("bad", [
    dict(d_model=100),           # not a multiple of n_head * 8
    dict(seq=0),
    dict(n_head=0),
    dict(vocab=1 << 17),
    dict(batch=16, seq=1024),    # batch*seq above 8192
])
def test_bad_config_rejected(bad):
    base = dict(n_layer=2, d_model=128, n_head=2, d_ff=512, seq=128, batch=2, vocab=1000)
    base.update(bad)
    cfg = LU.gpt_config(**base)
    with pytest.raises(LU.LayupError) as e:
        LU.layup_param_layout(cfg)
    assert e.value.status == LU.LAYUP_ERR_SHAPE


def test_gemm_argument_checks_need_no_gpu(L):
    # misaligned operand: rejected on the host before any launch
    d = LU.gemm_desc(0x1002, 0x2000, 0x3000, 64, 64, 64, 64, 64, 64)
    with pytest.raises(LU.LayupError) as e:
        LU.layup_gemm_bf16(d)
    assert e.value.status == LU.LAYUP_ERR_ALIGN
    # contiguous dimension not a multiple of 8
    d = LU.gemm_desc(0x1000, 0x2000, 0x3000, 64, 64, 60, 60, 60, 64)
    with pytest.raises(LU.LayupError) as e:
        LU.layup_gemm_bf16(d)
    assert e.value.status == LU.LAYUP_ERR_ALIGN
    # null operand
    d = LU.gemm_desc(None, 0x2000, 0x3000, 64, 64, 64, 64, 64, 64)
    with pytest.raises(LU.LayupError) as e:
        LU.layup_gemm_bf16(d)
    assert e.value.status == LU.LAYUP_ERR_SHAPE
    assert L.layup_gemm_bf16(None, None) == LU.LAYUP_ERR_INVALID_ARG


def test_update_mix_argument_checks_need_no_gpu():
    hp = LU.hparams("adamw", 1e-3, step=1)
    t = LU.layup_tensor(param=0x1000, grad=0x2000, state0=0x3000, state1=None, peer=0x4000,
                        param_bf16=None, numel=16, decay=1)
    with pytest.raises(LU.LayupError) as e:      # AdamW without v
        LU.layup_layer_update_mix(None, [t], hp, 0.5)
    assert e.value.status == LU.LAYUP_ERR_INVALID_ARG
    t.state1 = 0x5008                             # misaligned v
    with pytest.raises(LU.LayupError) as e:
        LU.layup_layer_update_mix(None, [t], hp, 0.5)
    assert e.value.status == LU.LAYUP_ERR_ALIGN
    t.state1, t.peer = 0x5000, 0x1000             # param aliases peer
    with pytest.raises(LU.LayupError) as e:
        LU.layup_layer_update_mix(None, [t], hp, 0.5)
    assert e.value.status == LU.LAYUP_ERR_INVALID_ARG
    hp0 = LU.hparams("adamw", 1e-3, step=0)      # AdamW step 0
    t.peer = 0x4000
    with pytest.raises(LU.LayupError) as e:
        LU.layup_layer_update_mix(None, [t], hp0, 0.5)
    assert e.value.status == LU.LAYUP_ERR_INVALID_ARG
    with pytest.raises(LU.LayupError) as e:      # disagreement without a context
        LU.layup_layer_update_mix(None, [t], hp, 0.5, disagreement=0x6000)
    assert e.value.status == LU.LAYUP_ERR_INVALID_ARG


# ------------------------------------------------------------- push-sum (host)

def test_push_sum_host_functions_match_oracle(L):
    """layup_push_sum_send / _receive (host arithmetic in the library) follow
    the oracle's push-sum exchange exactly over a long random sequence: the
    same weights bit for bit, alpha equal to the oracle's rounded to float32,
    total weight 1."""
    import numpy as np
    import oracle as O
    rng = np.random.default_rng(11)
    M = 5
    w = np.full(M, 1.0 / M)
    wo = [1.0 / M] * M
    for _ in range(500):
        i = int(rng.integers(M))
        j = int((i + 1 + rng.integers(M - 1)) % M)
        alpha = LU.layup_push_sum_send(w, i, j)
        LU.layup_push_sum_receive(w, i, j)
        wo, ao = O.push_sum_round(wo, i, j)
        assert alpha == float(np.float32(ao))
        assert list(w) == wo
        assert abs(w.sum() - 1.0) < 1e-12


def test_push_sum_golden_exchange(L):
    """The worked two-worker exchange: weights 1/2 each, the sender halves to
    1/4, alpha = 1/3, the receiver ends at 3/4."""
    import json
    import numpy as np
    c = json.load(open(os.path.join(ROOT, "tests", "golden", "hand_2x2.json")))["push_sum_exchange"]
    w = np.array(c["w"], dtype=np.float64)
    alpha = LU.layup_push_sum_send(w, c["sender"], c["receiver"])
    assert alpha == float(np.float32(c["alpha"]))
    LU.layup_push_sum_receive(w, c["sender"], c["receiver"])
    assert list(w) == c["w_after"]


def test_push_sum_rejects_bad_arguments(L):
    import numpy as np
    w = np.full(3, 1.0 / 3)
    for args in ((0, 0), (-1, 1), (0, 3)):
        with pytest.raises(LU.LayupError):
            LU.layup_push_sum_send(w, *args)
        with pytest.raises(LU.LayupError):
            LU.layup_push_sum_receive(w, *args)
    with pytest.raises(LU.LayupError):
        LU.layup_push_sum_send(np.full(1, 1.0), 0, 0)
    bad = np.array([0.5, 0.0, 0.5])
    with pytest.raises(LU.LayupError):
        LU.layup_push_sum_send(bad, 0, 1)
    assert list(w) == [1.0 / 3] * 3   # nothing changed by the rejected calls
