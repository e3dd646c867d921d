"""Benchmark of the LayUp layer-wise step on one MI355X.

A step is one pass of the whole path on one batch of synthetic data: forward
pass and loss, then for every unit from the output back to the input its
backward GEMMs and glue kernels on the compute stream and, overlapped on the
update stream, its fused AdamW update + gossip mix with the peer replica
(LayUp Algorithm 1 with the layer-wise updates of section 3.2).  Workload:
GPT-2-small-shaped decoder, 12 blocks x 768, 12 heads, MLP 3072, T 1024,
batch 8, vocab 50257 (tokens uniform, weights N(0, 0.02), peer = weights +
N(0, 1e-3)), AdamW (0.9, 0.95), wd 0.1 on matrices, alpha 0.5.

Prints ONE JSON line.  ``value`` is ms per layer-wise step (lower is better);
the per-kernel figures (update+mix HBM GB/s, backward-GEMM TFLOP/s) are
measured with HIP events on the stream the kernels run on.

Other workloads (one JSON line each, not the default bench line):
  --workload gpt2-medium   24 x 1024, 16 heads, MLP 4096, T 1024, batch 8
  --workload gpt-1.3b      24 x 2048, 16 heads, MLP 8192, T 2048, batch 4, 3
                           resident peer replicas, peer slot drawn per step
  --workload resnet50-update  update+mix sweep over the 161 ResNet-50
                           tensors (54 units in reverse order), SGD momentum
  --workload mlp           tiny float32 MLP, 10 layer-wise steps
  --workload gossip        4 GPT-2-small replicas resident on the GPU taking
                           steps in turn, push mode with push-sum weights
  --workload gemm-yardstick  the backward GEMM shapes of a GPT-2-small block,
                           its tied head and a 1.3B block, each timed with
                           this library's GEMM and with torch.matmul
                           (hipBLASLt) on the same operands, cold operands
  --workload kernels       one launch each of: a 1 GiB copy (counter
                           calibration), one GPT-2-small block's 8 backward
                           GEMMs, one block's update+mix -- for rocprofv3 --pmc

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
                       [--workload NAME]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import hashlib

PEAK_HBM_GBS = 8000.0       # MI355X HBM3E, GB/s
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA, TFLOP/s


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--kernel-reps", type=int, default=20)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--serialize", action="store_true", help="update on the compute stream")
    ap.add_argument("--only-step", action="store_true",
                    help="time the layer-wise steps only (for kernel traces of the step)")
    ap.add_argument("--pmc-summary", nargs=2, default=None, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="no GPU run: turn the FETCH_SIZE and WRITE_SIZE counter collections of "
                         "`rocprofv3 --pmc ... -- python3 bench.py --workload kernels` into "
                         "profiles/pmc_traffic.json (copy-calibrated bytes per dispatch group)")
    ap.add_argument("--trace-overlap", default=None, metavar="CSV",
                    help="no GPU run: read a rocprofv3 kernel trace of --only-step and report how much of "
                         "the update stream's kernel time ran concurrently with compute-stream kernels")
    ap.add_argument("--workload", default="gpt2-small",
                    choices=["gpt2-small", "gpt2-medium", "gpt-1.3b", "resnet50-update", "mlp",
                             "gossip", "kernels", "gemm-yardstick"])
    return ap.parse_args()


def measured_traffic(key, source):
    """HBM bytes per launch sequence from the committed counter summary
    (profiles/pmc_traffic.json: FETCH_SIZE + WRITE_SIZE, copy-calibrated),
    or None when the kernel source has changed since the counters were
    taken."""
    try:
        rec = json.load(open(os.path.join(ROOT, "profiles", "pmc_traffic.json")))[key]
        sha = hashlib.sha256(open(os.path.join(ROOT, "paper_2410_05985_amd", "csrc", source), "rb").read())
        if sha.hexdigest()[:16] != rec["source_sha256_16"]:
            return None
        return rec["hbm_bytes"]
    except (OSError, KeyError, ValueError):
        return None


def backward_gemm_shapes(cfg):
    """(name, M, N, K, a_kmajor, b_kmajor) of one block's dX/dW GEMMs and the
    tied head's, at the workload's shape (N_tok = batch * seq)."""
    n, d, f, vp = cfg.batch * cfg.seq, cfg.d_model, cfg.d_ff, (cfg.vocab + 63) // 64 * 64
    out = []
    for name, o, i in (("qkv", 3 * d, d), ("proj", d, d), ("fc", f, d), ("mproj", d, f)):
        out.append((name + ".dX", n, i, o, True, False))
        out.append((name + ".dW", o, i, n, False, False))
    head = [("head.dX", n, d, vp, True, False), ("head.dW", vp, d, n, False, False)]
    return out, head


def time_gemms(torch, LU, shapes, reps, stream, cold_bytes=512 << 20):
    """Average duration of each GEMM launch with HIP events on its stream:
    reps launches back to back between two events.  The launches rotate over
    enough copies of the operands and output (up to 16) to exceed the 256 MB
    MALL, so, as inside the step, every launch reads its operands from HBM."""
    res = []
    ws = torch.empty(64 << 20, dtype=torch.uint8, device="cuda")
    for name, M, N, K, ak, bk in shapes:
        per = 2 * M * K + 2 * N * K + 4 * M * N
        R = max(1, min(16, -(-cold_bytes // per)))
        bufs, descs = [], []
        for _ in range(R):
            A = torch.randn((M, K) if ak else (K, M), device="cuda").to(torch.bfloat16)
            B = torch.randn((N, K) if bk else (K, N), device="cuda").to(torch.bfloat16)
            C = torch.empty((M, N), dtype=torch.float32, device="cuda")
            bufs.append((A, B, C))
            descs.append(LU.gemm_desc(A, B, C, M, N, K, K if ak else M, K if bk else N, N, ak, bk, True,
                                      workspace=ws, workspace_bytes=64 << 20))
        with torch.cuda.stream(stream):
            for d in descs:
                LU.layup_gemm_bf16(d, stream)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for r in range(reps):
                LU.layup_gemm_bf16(descs[r % R], stream)
            e1.record(stream)
        e1.synchronize()
        ms = e0.elapsed_time(e1) / reps
        res.append(dict(name=name, M=M, N=N, K=K, ms=ms, copies=R,
                        tflops=2.0 * M * N * K / (ms * 1e-3) / 1e12))
        del bufs, descs
    return res


def time_update_mix(torch, LU, m, units, hp, alpha, reps, stream):
    """Update+mix launches (AdamW + bf16 copy) of the given units, back to
    back, one launch per unit as in the step, timed with HIP events on the
    update stream.  Returns the time of one round over the units and, for
    units of equal size, of one launch.  A round over the 12 GPT-2-small
    block units moves 12 x 241 MB, far more than the 256 MB MALL, so no
    launch finds its operands in the cache."""
    descs = []
    numels = []
    for unit in units:
        t = [x for x in m.infos if x["unit"] == unit]
        numels.append(sum(x["numel"] for x in t))
        d = []
        for x in t:
            o = x["offset"]
            d.append(LU.layup_tensor(param=m.params.data_ptr() + 4 * o, grad=m.grads.data_ptr() + 4 * o,
                                     state0=m.m.data_ptr() + 4 * o, state1=m.v.data_ptr() + 4 * o,
                                     peer=m.peers.data_ptr() + 4 * o,
                                     param_bf16=m.params_bf16.data_ptr() + 2 * o,
                                     numel=x["numel"], decay=x["decay"]))
        descs.append(d)
    hp.step = 1
    with torch.cuda.stream(stream):
        for d in descs:
            LU.layup_layer_update_mix(None, d, hp, alpha, stream=stream)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            for d in descs:
                LU.layup_layer_update_mix(None, d, hp, alpha, stream=stream)
        e1.record(stream)
    e1.synchronize()
    round_ms = e0.elapsed_time(e1) / reps
    nbytes = 34 * sum(numels)   # AdamW 32 B/param + 2 B bf16 copy
    out = dict(units=len(descs), round_ms=round_ms, round_bytes=nbytes,
               gbs=nbytes / (round_ms * 1e-3) / 1e9)
    if len(set(numels)) == 1:
        out.update(numel=numels[0], ms=round_ms / len(descs), bytes=34 * numels[0])
    return out


def percentiles(xs):
    xs = sorted(xs)
    pick = lambda q: xs[min(len(xs) - 1, int(round(q * (len(xs) - 1))))]
    return dict(p10=round(pick(0.1), 4), median=round(pick(0.5), 4), p90=round(pick(0.9), 4))


def host_cpu():
    """Cores this process may run on and the CPU model (from /proc/cpuinfo)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return n, model


def cpu_baseline(cfg_full):
    """The oracle on the host cores: one whole layer-wise step of a stack with
    the full width, sequence length and vocabulary but 1 block and 2 of the 8
    sequences, scaled to the full step by the ratio of the two steps' GEMM
    FLOPs (the oracle's time is dominated by its float64 matrix products).
    Timed twice on the same sample: with every thread the BLAS library uses
    (the reported value) and with one thread."""
    import threadpoolctl
    import oracle as O
    from paper_2410_05985_amd import synthetic as S
    cfg1 = S.GPTConfig(n_layer=1, d_model=cfg_full.d_model, n_head=cfg_full.n_head,
                       d_ff=cfg_full.d_ff, seq=cfg_full.seq, batch=2,
                       vocab=cfg_full.vocab)
    params0 = {k: v.astype(np.float64) for k, v in S.gpt_params(cfg1).items()}
    peer = {k: v.astype(np.float64) for k, v in S.gpt_peer(cfg1, S.gpt_params(cfg1)).items()}
    tokens = S.gpt_tokens(cfg1)
    hp = dict(optim="adamw", lr=cfg1.lr, weight_decay=cfg1.weight_decay, beta1=cfg1.beta1,
              beta2=cfg1.beta2, eps=cfg1.eps)

    def one_step():
        params = {k: a.copy() for k, a in params0.items()}
        m = {k: np.zeros_like(a) for k, a in params.items()}
        v = {k: np.zeros_like(a) for k, a in params.items()}
        t0 = time.perf_counter()
        O.gpt_step(params, m, v, peer, tokens, cfg1.n_head, hp, cfg1.alpha)
        return time.perf_counter() - t0

    threads = max((p.get("num_threads", 1) for p in threadpoolctl.threadpool_info()), default=1)
    dt = one_step()
    with threadpoolctl.threadpool_limits(limits=1):
        dt1 = one_step()

    def flops(c):
        n, d, f, V = c.batch * c.seq, c.d_model, c.d_ff, c.vocab
        blk = 2 * n * (3 * d * d + d * d + 2 * d * f) * 3 + 4 * c.batch * c.seq * c.seq * d * 3
        return c.n_layer * blk + 2 * n * d * V * 3
    scale = flops(cfg_full) / flops(cfg1)
    nproc, model = host_cpu()
    return dict(value=dt * scale * 1e3, unit="ms/step", cores=int(threads), kind="oracle",
                sample=f"one oracle step of a 1-block, batch-2 stack at full width/seq/vocab "
                       f"({dt:.1f} s with {threads} threads, {dt1:.1f} s with 1), scaled by GEMM FLOPs "
                       f"x{scale:.2f} to 12 blocks x batch 8",
                one_thread_ms_per_step=round(dt1 * scale * 1e3, 1),
                sample_s={"all_threads": round(dt, 3), "one_thread": round(dt1, 3)},
                host={"nproc": nproc, "cpu_model": model})


def gpt_model_on_device(torch, LU, S, cfg, n_peers):
    """Model buffers filled on the device from seeded torch generators (the
    1.3B stack would take minutes to draw on the host): matrices and
    embeddings N(0, 0.02), biases 0, LayerNorm gain 1; peer replica k = own +
    N(0, 1e-3) from seed 2 + 100 k.  Embedding padding rows stay zero."""
    lc = LU.gpt_config(cfg.n_layer, cfg.d_model, cfg.n_head, cfg.d_ff, cfg.seq, cfg.batch, cfg.vocab,
                       n_peers)
    model = LU.Model(lc, "adamw")
    gen = torch.Generator(device="cuda")
    gen.manual_seed(1)
    for t in model.infos:
        view = model.params[t["offset"]: t["offset"] + t["numel"]]
        if t["cols"] > 1:
            view.normal_(0.0, 0.02, generator=gen)
        elif t["name"].endswith(".g"):
            view.fill_(1.0)
    for k in range(n_peers):
        gen.manual_seed(2 + 100 * k)
        peer = model.peers[k * model.total: (k + 1) * model.total]
        peer.copy_(model.params)
        noise = torch.empty_like(peer).normal_(0.0, 1e-3, generator=gen)
        for t in model.infos:   # logical elements only
            o = t["offset"]
            peer[o: o + t["numel"]] += noise[o: o + t["numel"]]
        del noise
    torch.cuda.synchronize()
    LU.layup_refresh_shadow(model.ctx)
    model.synchronize()
    return model


def bench_gpt_other(args, torch, LU, S, name):
    cfg = S.GPT2_MEDIUM if name == "gpt2-medium" else S.GPT_1P3B
    model = gpt_model_on_device(torch, LU, S, cfg, cfg.n_peers)
    tokens = torch.from_numpy(S.gpt_tokens(cfg)).to("cuda")
    slots = S.peer_slots(args.warmup + args.steps, cfg.n_peers)
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    hp = LU.hparams("adamw", cfg.lr, 0.0, cfg.weight_decay, cfg.beta1, cfg.beta2, cfg.eps, 1)
    step = 0
    for _ in range(args.warmup):
        hp.step = step + 1
        LU.layup_step(model.ctx, tokens, None, hp, cfg.alpha, int(slots[step]), loss)
        step += 1
    model.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        hp.step = step + 1
        LU.layup_step(model.ctx, tokens, None, hp, cfg.alpha, int(slots[step]), loss)
        step += 1
    model.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    ks = torch.cuda.Stream()
    blk, _ = backward_gemm_shapes(cfg)
    g = time_gemms(torch, LU, blk, args.kernel_reps, ks)
    blk_ms = sum(x["ms"] for x in g)
    blk_flops = sum(2.0 * x["M"] * x["N"] * x["K"] for x in g)
    um = time_update_mix(torch, LU, model, range(1, cfg.n_layer + 1), hp, cfg.alpha, args.kernel_reps, ks)
    out = {"metric": "ms per layer-wise step", "value": round(ms, 3), "unit": "ms/step",
           "workload": name, "n_params": cfg.n_params(), "steps": args.steps, "warmup": args.warmup,
           "tokens_per_s": round(cfg.batch * cfg.seq / (ms * 1e-3), 1), "loss": round(float(loss.item()), 5),
           "backward_gemm_TFLOPs": round(blk_flops / (blk_ms * 1e-3) / 1e12, 2),
           "backward_gemm_frac": round(blk_flops / (blk_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
           "update_mix_GBps": round(um["gbs"], 1), "update_mix_frac_hbm": round(um["gbs"] / PEAK_HBM_GBS, 4),
           "update_mix_unit_bytes": um["bytes"], "data": "synthetic (device-seeded)",
           "peer_slots": "seed 3, uniform over %d resident replicas" % cfg.n_peers}
    model.close()
    print(json.dumps(out), flush=True)


def bench_resnet(args, torch, LU, S):
    """Update+mix sweep over the 161 ResNet-50 tensors, 54 units in reverse
    order, SGD momentum 0.9, wd 5e-5 on every tensor, lr 0.1, alpha 0.5;
    24 B/param (read p, g, m, q; write p, m).  Reported four ways: the
    kernel-time-weighted rate of the per-unit launches, the wall-clock rate of
    the sweep (launch gaps included), one launch sequence covering all 161
    tensors (16 per launch), and the 54 units -- all ready -- in reverse order
    in one pass of layup_units_update_mix (the headline value)."""
    params, grads, peer = S.resnet50_tensors()
    specs = S.resnet50_param_specs()
    units = S.resnet50_units()
    off, o = {}, 0
    for n, shp, _ in specs:
        off[n] = o
        o += (int(np.prod(shp)) + 63) // 64 * 64
    total = o
    bufs = {k: torch.zeros(total, dtype=torch.float32, device="cuda") for k in ("p", "g", "m", "q")}
    for name, arr in (("p", params), ("g", grads), ("q", peer)):
        host = torch.zeros(total, dtype=torch.float32)
        for n, a in arr.items():
            host[off[n]: off[n] + a.size] = torch.from_numpy(a.reshape(-1))
        bufs[name].copy_(host.cuda())
    def desc(n):
        k = off[n]
        return LU.layup_tensor(param=bufs["p"].data_ptr() + 4 * k, grad=bufs["g"].data_ptr() + 4 * k,
                               state0=bufs["m"].data_ptr() + 4 * k, state1=None,
                               peer=bufs["q"].data_ptr() + 4 * k, param_bf16=None,
                               numel=int(params[n].size), decay=1)
    unit_descs = [[desc(n) for n in u] for u in units]
    all_descs = [desc(n) for n, _, _ in specs]
    # every unit's gradient is ready: the units in reverse order, one pass
    rev_descs = [d for u in reversed(range(len(units))) for d in unit_descs[u]]
    rev_units = [u for u in reversed(range(len(units))) for _ in unit_descs[u]]
    trace = torch.zeros(2 * len(units), dtype=torch.int32, device="cuda")
    counter = torch.zeros(1, dtype=torch.int32, device="cuda")
    n_params = sum(a.size for a in params.values())
    hp = LU.hparams("sgd", 0.1, 0.9, 5e-5)
    st = torch.cuda.Stream()
    flush = torch.empty(128 << 20, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    # per-unit kernel times
    kern_ms, wall_ms, single_ms = 0.0, 0.0, 0.0
    reps = max(1, args.kernel_reps // 4)
    with torch.cuda.stream(st):
        for r in range(reps + 1):
            flush.add_(1.0)
            evs = [torch.cuda.Event(enable_timing=True) for _ in range(2 * len(units))]
            w0, w1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            w0.record(st)
            for i, u in enumerate(reversed(range(len(units)))):
                evs[2 * i].record(st)
                LU.layup_layer_update_mix(None, unit_descs[u], hp, 0.5, stream=st)
                evs[2 * i + 1].record(st)
            w1.record(st)
            w1.synchronize()
            if r > 0:
                kern_ms += sum(evs[2 * i].elapsed_time(evs[2 * i + 1]) for i in range(len(units)))
                wall_ms += w0.elapsed_time(w1)
        for r in range(reps + 1):
            flush.add_(1.0)
            w0, w1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            w0.record(st)
            LU.layup_layer_update_mix(None, all_descs, hp, 0.5, stream=st)
            w1.record(st)
            w1.synchronize()
            if r > 0:
                single_ms += w0.elapsed_time(w1)
        pass_ms = 0.0
        for r in range(reps + 1):
            flush.add_(1.0)
            counter.zero_()
            w0, w1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            w0.record(st)
            LU.layup_units_update_mix(rev_descs, rev_units, hp, 0.5, trace=trace, trace_counter=counter,
                                      trace_capacity=len(units), trace_step=r, stream=st)
            w1.record(st)
            w1.synchronize()
            if r > 0:
                pass_ms += w0.elapsed_time(w1)
        tr = trace.cpu().numpy().reshape(-1, 2)
        assert [int(u) for u in tr[:, 1]] == list(range(len(units) - 1, -1, -1)), "unit order"
    nbytes = 24 * n_params
    kern_ms, wall_ms, single_ms, pass_ms = kern_ms / reps, wall_ms / reps, single_ms / reps, pass_ms / reps
    gbs = lambda ms: round(nbytes / (ms * 1e-3) / 1e9, 1)
    out = {"metric": "update+mix HBM GB/s (ResNet-50 parameter set, layer-wise sweep)",
           "workload": "resnet50-update", "value": gbs(pass_ms), "unit": "GB/s",
           "n_tensors": len(specs), "n_units": len(units), "n_params": int(n_params), "bytes": nbytes,
           "units_one_pass_GBps": gbs(pass_ms), "units_one_pass_ms": round(pass_ms, 4),
           "frac_hbm": round(nbytes / (pass_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
           "per_unit_launches_kernel_weighted_GBps": gbs(kern_ms),
           "per_unit_launches_wall_GBps": gbs(wall_ms),
           "sixteen_tensor_launches_GBps": gbs(single_ms),
           "per_unit_launches_kernel_ms": round(kern_ms, 4), "per_unit_launches_wall_ms": round(wall_ms, 4),
           "note": "value: the 54 units, all ready, in reverse order in one pass (layup_units_update_mix), "
                   "one trace entry per unit checked; per-unit launches as a layer-wise step issues them "
                   "one gradient at a time are reported beside it",
           "data": "synthetic"}
    print(json.dumps(out), flush=True)


def bench_mlp(args, torch, LU, S):
    cfg = S.MLP_TINY
    x, y = S.mlp_inputs(cfg)
    m = LU.Model(LU.mlp_config(cfg.dims, cfg.batch), "sgd")
    m.load("params", S.mlp_params(cfg))
    m.load("peers", S.peer_of(S.mlp_params(cfg), 0.01))
    xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    hp = LU.hparams("sgd", cfg.lr, cfg.momentum, 0.0)
    torch.cuda.synchronize()
    for s_ in range(cfg.steps):
        LU.layup_step(m.ctx, yd[s_], xd[s_], hp, cfg.alpha, 0)
    m.synchronize()
    reps = 20
    t0 = time.perf_counter()
    for r in range(reps):
        for s_ in range(cfg.steps):
            LU.layup_step(m.ctx, yd[s_], xd[s_], hp, cfg.alpha, 0)
    m.synchronize()
    us = (time.perf_counter() - t0) * 1e6 / (reps * cfg.steps)
    print(json.dumps({"metric": "us per layer-wise step (tiny MLP, float32)", "workload": "mlp",
                      "value": round(us, 2), "unit": "us/step", "steps": reps * cfg.steps,
                      "note": "launch-latency bound: 3 units, 4.8 MB of update+mix and ~30 MFLOP per step"}),
          flush=True)
    m.close()


def bench_gossip(args, torch, LU, S):
    """M = 4 GPT-2-small replicas resident on one GPU take layer-wise steps in
    turn (worker s mod 4 at step s), each on its own token batch; every unit's
    locally updated layer is pushed into a receiver drawn per step (seed 4)
    with the push-sum alpha (Algorithm 1 as written; section 3.1 weights).
    The replicas share one pair of streams and one workspace.  Reports ms per
    step and the model disagreement sum((p_updated - q)^2) over all units."""
    cfg = S.GPT2_SMALL
    M = 4
    lc = LU.gpt_config(cfg.n_layer, cfg.d_model, cfg.n_head, cfg.d_ff, cfg.seq, cfg.batch, cfg.vocab)
    streams = (torch.cuda.Stream(), torch.cuda.Stream())
    models, ws = [], None
    gen = torch.Generator(device="cuda")
    for k in range(M):
        mk = LU.Model(lc, "adamw", streams=streams, workspace=ws, trace_capacity=16)
        ws = mk.workspace
        models.append(mk)
    gen.manual_seed(1)
    for t in models[0].infos:
        view = models[0].params[t["offset"]: t["offset"] + t["numel"]]
        if t["cols"] > 1:
            view.normal_(0.0, 0.02, generator=gen)
        elif t["name"].endswith(".g"):
            view.fill_(1.0)
    for k in range(1, M):
        gen.manual_seed(2 + 100 * k)
        models[k].params.copy_(models[0].params)
        noise = torch.empty_like(models[k].params).normal_(0.0, 1e-3, generator=gen)
        for t in models[k].infos:
            o = t["offset"]
            models[k].params[o: o + t["numel"]] += noise[o: o + t["numel"]]
        del noise
    torch.cuda.synchronize()
    for mk in models:
        LU.layup_refresh_shadow(mk.ctx)
        mk.synchronize()
    tokens = [torch.from_numpy(S.gpt_tokens(cfg, seed=10 + k)).cuda() for k in range(M)]
    pairs = S.gossip_pairs(args.warmup + args.steps, M)
    w = np.full(M, 1.0 / M)
    t_own = [0] * M
    U = models[0].n_units
    dis = torch.zeros((len(pairs), U), dtype=torch.float32, device="cuda")

    def step(s):
        i, j = pairs[s]
        t_own[i] += 1
        hp = LU.hparams("adamw", cfg.lr, 0.0, cfg.weight_decay, cfg.beta1, cfg.beta2, cfg.eps, t_own[i])
        alpha = LU.layup_push_sum_send(w, i, j)
        LU.layup_step_ex(models[i].ctx, tokens[i], None, hp, alpha, mix_mode=LU.LAYUP_MIX_PUSH,
                         push_params=models[j].params, push_params_bf16=models[j].params_bf16,
                         disagreement=dis[s])
        LU.layup_push_sum_receive(w, i, j)

    for s_ in range(args.warmup):
        step(s_)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(streams[0])
    for s_ in range(args.warmup, args.warmup + args.steps):
        step(s_)
    e1.record(streams[0])
    e1.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    d = dis.sum(dim=1).cpu().numpy()
    print(json.dumps({"metric": "ms per layer-wise step, 4 resident replicas in push mode",
                      "workload": "gossip-gpt2-small-x4", "value": round(ms, 3), "unit": "ms/step",
                      "steps": args.steps, "warmup": args.warmup,
                      "tokens_per_s": round(cfg.batch * cfg.seq / (ms * 1e-3), 1),
                      "disagreement_first_last": [float(d[0]), float(d[-1])],
                      "push_sum_weights": [round(float(x), 6) for x in w], "weight_sum": float(w.sum()),
                      "data": "synthetic (device-seeded replicas, per-worker token batches)"}), flush=True)
    for mk in models:
        mk.close()


def time_torch_mm(torch, shapes, reps, stream, cold_bytes=512 << 20):
    """torch.matmul (hipBLASLt) on the layouts of time_gemms: C = A B with A
    [M, K] (a_kmajor) or the transpose of a [K, M] array, B [K, N] (b not
    k-major) or the transpose of [N, K].  bf16 in, bf16 out (torch has no
    float32-output bf16 matmul), operands rotated as in time_gemms."""
    res = []
    for name, M, N, K, ak, bk in shapes:
        per = 2 * M * K + 2 * N * K + 2 * M * N
        R = max(1, min(16, -(-cold_bytes // per)))
        ops = []
        for _ in range(R):
            A = torch.randn((M, K) if ak else (K, M), device="cuda").to(torch.bfloat16)
            B = torch.randn((N, K) if bk else (K, N), device="cuda").to(torch.bfloat16)
            ops.append((A if ak else A.t(), B.t() if bk else B))
        with torch.cuda.stream(stream):
            for a, b in ops:
                torch.matmul(a, b)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for r in range(reps):
                a, b = ops[r % R]
                torch.matmul(a, b)
            e1.record(stream)
        e1.synchronize()
        ms = e0.elapsed_time(e1) / reps
        res.append(dict(name=name, ms=ms, tflops=2.0 * M * N * K / (ms * 1e-3) / 1e12))
        del ops
    return res


def bench_gemm_yardstick(args, torch, LU, S):
    """This library's GEMM next to hipBLASLt on the backward shapes: one
    GPT-2-small block and its tied head, and one 1.3B block."""
    stream = torch.cuda.Stream()
    rows = []
    for tag, cfg in (("gpt2-small", S.GPT2_SMALL), ("gpt-1.3b", S.GPT_1P3B)):
        blk, head = backward_gemm_shapes(cfg)
        shapes = blk + (head if tag == "gpt2-small" else [])
        ours = time_gemms(torch, LU, shapes, args.kernel_reps, stream)
        ref = time_torch_mm(torch, shapes, args.kernel_reps, stream)
        for (name, M, N, K, ak, bk), o, r in zip(shapes, ours, ref):
            rows.append(dict(config=tag, gemm=name, M=M, N=N, K=K, ours_us=round(o["ms"] * 1e3, 1),
                             ours_tflops=round(o["tflops"], 1), hipblaslt_us=round(r["ms"] * 1e3, 1),
                             hipblaslt_tflops=round(r["tflops"], 1)))
    print(json.dumps({"workload": "gemm-yardstick", "peak_tflops": PEAK_BF16_TFLOPS, "gemms": rows,
                      "note": "ours: float32 output (dW, dX as in the step); hipBLASLt: bf16 output"}),
          flush=True)


def bench_kernels(args, torch, LU, S):
    """Single launches for hardware-counter runs, in this order: a 1 GiB
    device copy (known traffic: 1 GiB read + 1 GiB written), the 8 backward
    GEMMs of one GPT-2-small block (qkv, proj, fc, mproj; dX then dW), the
    update+mix of one GPT-2-small block (AdamW + bf16 copy).  The device is
    synchronised between launches so each dispatch stands alone."""
    cfg = S.GPT2_SMALL
    src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    blk, _ = backward_gemm_shapes(cfg)
    ops = []
    ws = torch.empty(64 << 20, dtype=torch.uint8, device="cuda")
    for name, M, N, K, ak, bk in blk:
        A = torch.randn((M, K) if ak else (K, M), device="cuda").to(torch.bfloat16)
        B = torch.randn((N, K) if bk else (K, N), device="cuda").to(torch.bfloat16)
        C = torch.empty((M, N), dtype=torch.float32, device="cuda")
        ops.append((name, LU.gemm_desc(A, B, C, M, N, K, K if ak else M, K if bk else N, N, ak, bk, True,
                                       workspace=ws, workspace_bytes=64 << 20), (A, B, C)))
    n = 7_087_872
    bufs = [torch.randn(n, device="cuda") * 1e-3 for _ in range(5)]
    p16 = torch.zeros(n, dtype=torch.int16, device="cuda")
    bufs[3].abs_()
    t = LU.layup_tensor(param=bufs[0].data_ptr(), grad=bufs[1].data_ptr(), state0=bufs[2].data_ptr(),
                        state1=bufs[3].data_ptr(), peer=bufs[4].data_ptr(), param_bf16=p16.data_ptr(),
                        numel=n, decay=1)
    hp = LU.hparams("adamw", cfg.lr, 0.0, cfg.weight_decay, cfg.beta1, cfg.beta2, cfg.eps, 1)
    flush = torch.empty(128 << 20, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    for name, d, _ in ops:
        LU.layup_gemm_bf16(d, torch.cuda.current_stream())
        torch.cuda.synchronize()
    flush.add_(1.0)
    torch.cuda.synchronize()
    LU.layup_layer_update_mix(None, [t], hp, cfg.alpha, stream=torch.cuda.current_stream())
    torch.cuda.synchronize()
    print(json.dumps({"workload": "kernels", "copy_bytes": 2 * src.numel() * 4,
                      "gemms": [o[0] for o in ops], "update_mix_numel": n,
                      "update_mix_algorithmic_bytes": 34 * n}), flush=True)


def pmc_summary(fetch_csv, write_csv):
    """HBM bytes of the kernels of `bench.py --workload kernels` from two
    counter passes.  The 1 GiB device copy calibrates the counters (it reads
    and writes 1 GiB): fetch and write counts are scaled so that the copy
    reads and writes exactly that.  The dispatches after the copy are the 8
    backward GEMMs of a GPT-2-small block (each with its split-K reduction,
    if any), then the block's update+mix."""
    import csv

    def load(path, counter):
        rows = {}
        with open(path, newline="") as f:
            for r in csv.DictReader(f):
                if r["Counter_Name"] != counter:
                    continue
                d = int(r["Dispatch_Id"])
                rows.setdefault(d, [r["Kernel_Name"], 0.0])[1] += float(r["Counter_Value"])
        return [rows[k] for k in sorted(rows)]

    f, w = load(fetch_csv, "FETCH_SIZE"), load(write_csv, "WRITE_SIZE")
    assert [a[0] for a in f] == [a[0] for a in w], "the two passes ran different dispatches"
    names = [a[0] for a in f]
    ci = next(i for i, n in enumerate(names) if "copyBuffer" in n)
    gib = float(1 << 30)
    ff, wf = gib / (f[ci][1] * 1024), gib / (w[ci][1] * 1024)
    gemm_names = ["qkv.dX", "qkv.dW", "proj.dX", "proj.dW", "fc.dX", "fc.dW", "mproj.dX", "mproj.dW"]
    groups, um = [], None
    for i in range(ci + 1, len(names)):
        if "gemm_bf16_kernel" in names[i]:
            groups.append([i])
        elif "splitk_reduce" in names[i]:
            groups[-1].append(i)
        elif "update_mix_kernel" in names[i]:
            um = i
            break
    assert len(groups) == 8 and um is not None, [names[g[0]][:40] for g in groups]
    sha = lambda src: hashlib.sha256(open(os.path.join(ROOT, "paper_2410_05985_amd", "csrc", src), "rb")
                                     .read()).hexdigest()[:16]
    per, tot = [], 0.0
    for nm, g in zip(gemm_names, groups):
        fb = sum(f[i][1] for i in g) * 1024 * ff
        wb = sum(w[i][1] for i in g) * 1024 * wf
        tot += fb + wb
        per.append(dict(gemm=nm, dispatches=len(g), fetch_bytes=fb, write_bytes=wb))
    ufb, uwb = f[um][1] * 1024 * ff, w[um][1] * 1024 * wf
    out = dict(fetch_factor=ff, write_factor=wf,
               gemm_block_backward=dict(source_sha256_16=sha("gemm_bf16.hip"), hbm_bytes=tot, per_gemm=per),
               update_mix_block=dict(source_sha256_16=sha("update_mix.hip"), hbm_bytes=ufb + uwb,
                                     fetch_bytes=ufb, write_bytes=uwb, algorithmic_bytes=34 * 7_087_872))
    with open(os.path.join(ROOT, "profiles", "pmc_traffic.json"), "w") as fo:
        json.dump(out, fo, indent=1)
    print(json.dumps({"fetch_factor": ff, "write_factor": wf, "gemm_block_backward_bytes": tot,
                      "per_gemm": per, "update_mix_block_bytes": ufb + uwb}), flush=True)


def trace_overlap(path):
    """Concurrency of the two streams in a rocprofv3 kernel trace (CSV) of
    `bench.py --only-step`: the compute stream is the one that runs the
    attention backward, the update stream the one that runs the update+mix.
    For the update+mix kernels, and for every kernel of the update stream
    (dW GEMMs, the head's dW, the forward's second half, the token sort),
    the fraction of their summed duration during which at least one
    compute-stream kernel was running, over every step in the trace
    (warm-up and timed steps are the same step)."""
    import csv
    rows = []
    with open(path, newline="") as f:
        for r in csv.DictReader(f):
            rows.append((r["Kernel_Name"], r["Stream_Id"], int(r["Start_Timestamp"]), int(r["End_Timestamp"])))
    from collections import Counter
    um_streams = Counter(sid for n, sid, _, _ in rows if "update_mix_kernel" in n)
    at_streams = Counter(sid for n, sid, _, _ in rows if "attn_bwd_dq_kernel" in n)
    comp_c = [k for k in at_streams if k not in um_streams]
    upd_c = [k for k in um_streams if k not in at_streams]
    if len(comp_c) != 1 or len(upd_c) != 1:
        raise SystemExit(f"expected the trace of one two-stream model (bench.py --only-step): compute-stream "
                         f"candidates {comp_c}, update-stream candidates {upd_c}")
    comp, upd = comp_c[0], upd_c[0]
    cint = sorted((a, b) for n, sid, a, b in rows if sid == comp)
    merged = []
    for a, b in cint:
        if merged and a <= merged[-1][1]:
            merged[-1][1] = max(merged[-1][1], b)
        else:
            merged.append([a, b])
    import bisect
    starts = [m[0] for m in merged]

    def covered(a, b):
        i = max(0, bisect.bisect_right(starts, a) - 1)
        tot = 0
        while i < len(merged) and merged[i][0] < b:
            tot += max(0, min(b, merged[i][1]) - max(a, merged[i][0]))
            i += 1
        return tot

    def stats(ks):
        dur = sum(b - a for a, b in ks)
        conc = sum(covered(a, b) for a, b in ks)
        return dict(kernels=len(ks), ms_per_step=round(dur * 1e-6 / n_steps, 4),
                    concurrent_ms_per_step=round(conc * 1e-6 / n_steps, 4),
                    concurrent_frac=round(conc / max(dur, 1), 4))

    # each step launches the 14 units' update+mix in reverse order: the
    # 14th of a step is the embeddings' unit, whose gradient is the step's
    # last (nothing is left on the compute stream to overlap it with)
    um = sorted((a, b) for n, sid, a, b in rows if sid == upd and "update_mix_kernel" in n)
    n_steps = max(1, len(um) // 14)
    out = {"trace": os.path.basename(path), "steps": n_steps,
           "update_mix": stats(um),
           "update_mix_blocks_and_final_ln": stats([k for i, k in enumerate(um) if i % 14 != 13]),
           "update_mix_embeddings": stats([k for i, k in enumerate(um) if i % 14 == 13]),
           "update_stream_all": stats([(a, b) for n, sid, a, b in rows if sid == upd]),
           "compute_stream_busy_ms_per_step": round(sum(b - a for a, b in merged) * 1e-6 / n_steps, 4)}
    print(json.dumps(out), flush=True)


def main():
    args = parse()
    if args.trace_overlap:
        trace_overlap(args.trace_overlap)
        return
    if args.pmc_summary:
        pmc_summary(*args.pmc_summary)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "the benchmark runs on one GPU: the layer-wise step of one worker; "
                                   "multi-GPU runs are not part of it", "n_gpus": args.gpus}))
        sys.exit(2)
    import torch
    if args.workload != "gpt2-small":
        from paper_2410_05985_amd import layup as LU
        from paper_2410_05985_amd import synthetic as S
        if args.workload == "resnet50-update":
            bench_resnet(args, torch, LU, S)
        elif args.workload == "kernels":
            bench_kernels(args, torch, LU, S)
        elif args.workload == "mlp":
            bench_mlp(args, torch, LU, S)
        elif args.workload == "gossip":
            bench_gossip(args, torch, LU, S)
        elif args.workload == "gemm-yardstick":
            bench_gemm_yardstick(args, torch, LU, S)
        else:
            bench_gpt_other(args, torch, LU, S, args.workload)
        return
    from paper_2410_05985_amd import layup as LU
    from paper_2410_05985_amd import synthetic as S

    cfg = S.GPT2_SMALL
    params = S.gpt_params(cfg)
    tokens = S.gpt_tokens(cfg)
    peer = S.gpt_peer(cfg, params)
    lc = LU.gpt_config(cfg.n_layer, cfg.d_model, cfg.n_head, cfg.d_ff, cfg.seq, cfg.batch, cfg.vocab)
    model = LU.Model(lc, "adamw", two_streams=not args.serialize)
    model.load("params", params)
    model.load("peers", peer)
    del params, peer
    td = torch.from_numpy(tokens).to("cuda")
    loss = torch.zeros(1, dtype=torch.float32, device="cuda")
    hp = LU.hparams("adamw", cfg.lr, 0.0, cfg.weight_decay, cfg.beta1, cfg.beta2, cfg.eps, 1)
    torch.cuda.synchronize()
    step = 0
    for _ in range(args.warmup):
        step += 1
        hp.step = step
        LU.layup_step(model.ctx, td, None, hp, cfg.alpha, 0, loss)
    model.synchronize()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    t0 = time.perf_counter()
    ev[0].record(model.compute_stream)
    for i in range(args.steps):
        step += 1
        hp.step = step
        LU.layup_step(model.ctx, td, None, hp, cfg.alpha, 0, loss)
        ev[i + 1].record(model.compute_stream)   # after the step's join
    model.synchronize()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps
    step_ms = [ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps)]
    loss_v = float(loss.item())
    if args.only_step:
        print(json.dumps({"metric": "ms per layer-wise step (GPT-2-small), steps only", "value": round(ms_step, 4),
                          "unit": "ms/step", "steps": args.steps, "warmup": args.warmup,
                          "step_ms_events": percentiles(step_ms), "loss": round(loss_v, 5),
                          "streams": 1 if args.serialize else 2}), flush=True)
        return

    # drift (section 3.2): delay from each unit's gradient to its applied
    # update, layer-wise (the last timed step) against one step with every
    # update after the whole backward pass; model D = beta T (U + 1) / 2
    drift = {}
    for name, sched in (("layerwise", LU.LAYUP_SCHEDULE_LAYERWISE),
                        ("after_backward", LU.LAYUP_SCHEDULE_AFTER_BACKWARD)):
        if sched == LU.LAYUP_SCHEDULE_AFTER_BACKWARD:
            step += 1
            hp.step = step
            LU.layup_step_ex(model.ctx, td, None, hp, cfg.alpha, schedule=sched, loss_out=loss)
        f_ms, ready, applied = LU.layup_unit_timeline(model.ctx, model.n_units)
        delays = [a - r for a, r in zip(applied, ready)]
        drift[name] = dict(D_ms=round(sum(delays), 4), max_unit_delay_ms=round(max(delays), 4),
                           step_ms=round(max(applied), 4))
        if name == "layerwise":
            bwd = max(ready) - f_ms
    U = model.n_units
    drift["backward_ms"] = round(bwd, 4)
    drift["model_after_backward_D_ms"] = round(bwd * (U + 1) / 2, 4)



    # forward pass alone (saved activations + loss gradient), compute stream
    f0, f1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    LU.layup_forward(model.ctx, td, None, loss)
    f0.record(model.compute_stream)
    for _ in range(args.steps):
        LU.layup_forward(model.ctx, td, None, loss)
    f1.record(model.compute_stream)
    f1.synchronize()
    fwd_ms = f0.elapsed_time(f1) / args.steps

    # the same step with the update on the compute stream (no overlap)
    ser = LU.Model(lc, "adamw", two_streams=False)
    for a, b in ((ser.params, model.params), (ser.m, model.m), (ser.v, model.v), (ser.peers, model.peers)):
        a.copy_(b)
    torch.cuda.synchronize()
    LU.layup_refresh_shadow(ser.ctx)
    for _ in range(2):
        LU.layup_step(ser.ctx, td, None, hp, cfg.alpha, 0, loss)
    s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s0.record(ser.compute_stream)
    for _ in range(args.steps):
        LU.layup_step(ser.ctx, td, None, hp, cfg.alpha, 0, loss)
    s1.record(ser.compute_stream)
    s1.synchronize()
    serial_ms = s0.elapsed_time(s1) / args.steps
    ser.close()
    del ser

    # the fused schedule: each block's weight matrices updated by their dW GEMM
    for _ in range(2):
        step += 1
        hp.step = step
        LU.layup_step_ex(model.ctx, td, None, hp, cfg.alpha, schedule=LU.LAYUP_SCHEDULE_FUSED_DW, loss_out=loss)
    fz0, fz1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    fz0.record(model.compute_stream)
    for _ in range(args.steps):
        step += 1
        hp.step = step
        LU.layup_step_ex(model.ctx, td, None, hp, cfg.alpha, schedule=LU.LAYUP_SCHEDULE_FUSED_DW, loss_out=loss)
    fz1.record(model.compute_stream)
    fz1.synchronize()
    fused_ms = fz0.elapsed_time(fz1) / args.steps
    print(f"[bench] {args.steps} steps, {ms_step:.3f} ms/step, loss {loss_v:.4f}", file=sys.stderr,
          flush=True)

    # per-kernel timing with HIP events on the stream the kernels run on
    ks = torch.cuda.Stream()
    blk, head = backward_gemm_shapes(cfg)
    g = time_gemms(torch, LU, blk + head, args.kernel_reps, ks)
    blk_ms = sum(x["ms"] for x in g[:len(blk)])
    blk_flops = sum(2.0 * x["M"] * x["N"] * x["K"] for x in g[:len(blk)])
    gemm_tflops = blk_flops / (blk_ms * 1e-3) / 1e12
    um = time_update_mix(torch, LU, model, range(1, cfg.n_layer + 1), hp, cfg.alpha, args.kernel_reps, ks)
    um_all = time_update_mix(torch, LU, model, range(model.n_units), hp, cfg.alpha, args.kernel_reps, ks)
    moved = serial_ms - ms_step
    print(f"[bench] step events p10/median/p90 {percentiles(step_ms)}; forward {fwd_ms:.3f} ms; "
          f"serialized {serial_ms:.3f} ms; fused dW {fused_ms:.3f} ms; update+mix of all {model.n_units} units {um_all['round_ms']:.3f} ms; "
          f"critical path moved {moved:.3f} ms", file=sys.stderr, flush=True)
    for x in g:
        print(f"[bench] gemm {x['name']:9s} {x['M']}x{x['N']}x{x['K']}: {x['ms']*1e3:8.1f} us "
              f"{x['tflops']:7.1f} TFLOP/s", file=sys.stderr, flush=True)
    print(f"[bench] update+mix block unit: {um['ms']*1e3:.1f} us {um['gbs']:.0f} GB/s",
          file=sys.stderr, flush=True)

    # dominant kernel of the step: the backward GEMMs of a block (MFMA bound)
    traffic = measured_traffic("gemm_block_backward", "gemm_bf16.hip")
    roofline = dict(bound="mfma", achieved=round(gemm_tflops, 2), peak=PEAK_BF16_TFLOPS,
                    unit="TFLOP/s", frac=round(gemm_tflops / PEAK_BF16_TFLOPS, 4),
                    traffic=traffic,
                    kernel="gemm_bf16_kernel (a block's 8 backward dX/dW GEMMs + split-K sums, operands from HBM)",
                    algorithmic_flops_per_block=blk_flops,
                    launch_ms_per_block=round(blk_ms, 5))
    out = {
        "metric": "update+mix HBM GB/s; backward GEMM TFLOPS; ms per layer-wise step (GPT-2-small)",
        "value": round(ms_step, 4),
        "unit": "ms/step",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 GEMM operands / f32 accumulate, f32 master + AdamW + mix",
        "data": "synthetic",
        "config": {"workload": "gpt2-small layer-wise step: 12x768, 12 heads, MLP 3072, seq 1024, "
                               "batch 8, vocab 50257, AdamW, alpha 0.5",
                   "global_batch": cfg.batch, "seq_len": cfg.seq, "parallelism": "single worker",
                   "streams": 1 if args.serialize else 2},
        "tokens_per_s": round(cfg.batch * cfg.seq / (ms_step * 1e-3), 1),
        "update_mix_GBps": round(um["gbs"], 1),
        "update_mix_frac_hbm": round(um["gbs"] / PEAK_HBM_GBS, 4),
        "update_mix_roofline": {"bound": "hbm", "achieved": round(um["gbs"], 1), "peak": PEAK_HBM_GBS,
                                "unit": "GB/s", "frac": round(um["gbs"] / PEAK_HBM_GBS, 4),
                                "traffic": measured_traffic("update_mix_block", "update_mix.hip"),
                                "algorithmic_bytes": um["bytes"]},
        "backward_gemm_TFLOPs": round(gemm_tflops, 2),
        "head_gemm_TFLOPs": [round(x["tflops"], 1) for x in g[len(blk):]],
        "loss": round(loss_v, 5),
        "step_ms_events": percentiles(step_ms),
        "forward_ms": round(fwd_ms, 4),
        "serialized_ms_per_step": round(serial_ms, 4),
        "fused_dw_ms_per_step": round(fused_ms, 4),
        "update_mix_all_units_ms": round(um_all["round_ms"], 4),
        "critical_path_moved_ms": round(moved, 4),
        "moved_off_compute_stream": "serialized minus two-stream step time; the update stream takes the "
                                    "update+mix of every unit, every dW GEMM with its bias sum, the head's dW, "
                                    "the forward's second batch half and the token sort (the concurrency of "
                                    "the update+mix itself comes from a kernel trace: bench.py --trace-overlap)",
        "drift": drift,
        "roofline": roofline,
    }
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle sample ...", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(cfg)
    model.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
