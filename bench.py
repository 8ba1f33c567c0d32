#!/usr/bin/env python3
"""Benchmark of the GRPO loss hot path on one MI355X.

A step is one pass of the whole logits path over one batch resident in HBM:
group advantages (grpo_advantages), then grpo_loss_fwd_bwd (segment pass,
row pass with dlogits, loss reduction).  Workload: 16 task groups x G = 8
trajectories, T = 120,000 action tokens, V = 151,936, bf16 logits (the
realistic-vocabulary rollout batch), synthetic and seeded.

The same batch with the per-trajectory normaliser 1/|tau_i| is reported under
"normaliser_traj_steps", one device's share of the vocabulary-parallel loss (the
batch's vocabulary split 8 ways, 18,992 columns) under "vocab_shard", and the
forward-only log-prob + entropy pass under "token_logp".  The other logits
workloads run the same step: "long" (32 groups, T = 250,000, V = 151,936, 76 GB
of logits and 76 GB of dlogits resident), "v32k" (8 groups, T of about 32,000,
V = 32,000, bf16) and "tiny" (one group of 4, fp32 [192, 1024]), each with its
own roofline line.

The fused LM-head path is measured in the same run on its own workload
(hidden bf16 [65,536, 3,584], W bf16 [3,584, 151,936]) and reported under
"fused_lmhead" against the bf16 dense MFMA peak with the algorithmic work of
three products (6 T H V flop): token blocks of 8192 rows with each block's D
pass on a second stream (the line's value), the same on one stream, and
vocabulary chunks of 8192 (four products executed) beside it.  Under
"library_gemm", the three products of one token block done by torch.matmul
(hipBLASLt, no epilogue) in the same process: context for the MFMA kernels, as
the copy ceiling is for the row pass.

Prints one JSON line.  ``value`` is tokens/s of the whole step.  ``roofline``
reports the dominant kernel (the row pass): algorithmic bytes per launch,
T * (4V + 16), over its average duration from HIP events recorded around it
on its stream, with the copy ceiling of the same two buffers beside it (the
fastest hand-written streaming copy of the logits into the dlogits buffer, timed
in the same process); ``traffic`` is the HBM traffic measured with rocprofv3 counters
(FETCH_SIZE, WRITE_SIZE) scaled by a plain copy's reading, when the committed
measurement matches the current kernel source, else null.  ``cpu_baseline``
times the fp64 oracle on the host on a bounded sample of the same batch.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "GRPO loss fwd+bwd tokens/s at V=151,936 bf16; % of HBM (or MFMA) roofline"
HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_rows_pipe_v152k_traffic.md")
KERNEL_SOURCES = ["paper_2606_05597_amd/csrc/loss.hip", "paper_2606_05597_amd/csrc/device.h"]
FUSED_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "lmhead_fused_65536x3584x151936_traffic.md")
FUSED_SOURCES = ["paper_2606_05597_amd/csrc/lmhead.hip", "paper_2606_05597_amd/csrc/gemm.h",
                 "paper_2606_05597_amd/csrc/device.h"]


def _code_hash(paths) -> str:
    """A hash of the sources' code: comments and whitespace removed, so that a measurement stays current across
    edits of the comments alone."""
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p)) as f:
            src = f.read()
        src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
        src = re.sub(r"//[^\n]*", " ", src)
        h.update(" ".join(src.split()).encode())
    return h.hexdigest()[:16]


def kernel_source_hash() -> str:
    return _code_hash(KERNEL_SOURCES)


def fused_source_hash() -> str:
    return _code_hash(FUSED_SOURCES)


def measured_fused_traffic(schedule: str):
    """HBM bytes per fused call of one schedule ("chunked" or "blocked") from the committed counter summary, if it
    is current."""
    if not os.path.exists(FUSED_TRAFFIC_FILE):
        return None
    kv = dict(re.findall(r"^- (\w+): (\S+)", open(FUSED_TRAFFIC_FILE).read(), re.M))
    key = f"traffic_bytes_per_call_{schedule}"
    if kv.get("kernel_source_sha256") != fused_source_hash() or key not in kv:
        return None
    return float(kv[key])


def measured_traffic(T: int):
    """HBM bytes per launch of the row kernel from the committed counter summary, if it is current."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    kv = dict(re.findall(r"^- (\w+): (\S+)", open(TRAFFIC_FILE).read(), re.M))
    if kv.get("kernel_source_sha256") != kernel_source_hash() or int(kv.get("T", -1)) != T:
        return None
    return float(kv["traffic_bytes_per_launch"])


def fused_schedules(args):
    return FUSED_SCHEDULES if args.fused_schedule == "all" else (args.fused_schedule,)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="oracle timing budget (0 = skip)")
    ap.add_argument("--fused-steps", type=int, default=3, help="timed steps of the fused path (0 = skip)")
    ap.add_argument("--logp-steps", type=int, default=10,
                    help="timed steps of the forward-only log-prob + entropy path (0 = skip)")
    ap.add_argument("--shard-steps", type=int, default=10,
                    help="timed steps of one device's share of the vocabulary-parallel loss (0 = skip)")
    ap.add_argument("--config-steps", type=int, default=10,
                    help="timed steps of each other logits-path workload: long, v32k, tiny (0 = skip)")
    ap.add_argument("--skip-logits", action="store_true", help="measure only the fused path")
    ap.add_argument("--token-block", type=int, default=8192, help="token block of the blocked fused schedule")
    ap.add_argument("--fused-schedule", choices=("all",) + FUSED_SCHEDULES, default="all",
                    help="fused schedules to time (all: the three, two-stream token blocks first)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a plain device copy of known size (for counter calibration)")
    return ap.parse_args()


def copy_calibration():
    import torch
    n = 8 << 30  # 8 GiB
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(2):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": n, "copies": 2}))


def cpu_baseline(b: dict, adv64, budget_s: float) -> dict:
    """The fp64 oracle on host cores, on the first rows of the same batch, cycled for ~budget_s."""
    import numpy as np
    import torch

    import oracle
    st = b["structure"]
    R = min(st.T, 16384)
    zl = b["logits"][:R].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    seg = oracle.segments(st.T, st.step_tok_off, st.traj_step_off)
    actions = b["actions"].cpu().numpy()
    behave = b["behave"].cpu().numpy()
    cfg = b["cfg"]
    chunk = 256
    rows = 0
    t0 = time.perf_counter()
    r0 = 0
    while True:
        r1 = min(R, r0 + chunk)
        oracle.loss_rows(zl[r0:r1], actions, behave, None, adv64, seg, cfg.G, norm=oracle.NORM_CONST_K, k=cfg.k,
                         dual_clip_c=3.0, row_begin=r0, row_end=r1, row_offset=r0)
        rows += r1 - r0
        r0 = 0 if r1 == R else r1
        if time.perf_counter() - t0 >= budget_s:
            break
    el = time.perf_counter() - t0
    cores = oracle.threads()
    # the same oracle on one thread, over fewer rows
    oracle.set_threads(1)
    r1 = 1024
    t1 = time.perf_counter()
    oracle.loss_rows(zl[:r1], actions, behave, None, adv64, seg, cfg.G, norm=oracle.NORM_CONST_K, k=cfg.k,
                     dual_clip_c=3.0, row_begin=0, row_end=r1, row_offset=0)
    el1 = time.perf_counter() - t1
    oracle.set_threads(cores)
    return {"value": rows / el, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": f"first {R} token rows of the same batch (loss + fp64 dlogits), cycled in blocks of "
                      f"{chunk}; {rows} rows in {el:.1f} s",
            "single_thread": {"value": r1 / el1, "unit": "tokens/s", "cores": 1,
                              "sample": f"first {r1} token rows, {el1:.1f} s"}}


def copy_ceiling(src, dst, reps: int = 3) -> dict:
    """The memory-only ceiling of the row pass: src copied into dst -- the same logits and dlogits buffers the row
    kernel reads and writes, so the same physical placement -- by each hand-written streaming-copy variant
    (libgrpo_bench.so) and by torch's copy_, best of ``reps`` each, read + write bytes per second.  The ceiling is
    the fastest hand-written variant."""
    import ctypes

    import torch

    from paper_2606_05597_amd.build import BENCH_SO
    lib = ctypes.CDLL(BENCH_SO)
    lib.stream_copy.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
    lib.stream_copy.restype = ctypes.c_int
    lib.stream_copy_name.argtypes = [ctypes.c_int]
    lib.stream_copy_name.restype = ctypes.c_char_p
    nbytes = src.numel() * src.element_size()
    assert dst.numel() * dst.element_size() == nbytes and src.is_contiguous() and dst.is_contiguous()
    assert nbytes % 16 == 0
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def best(run):
        ms = []
        for _ in range(reps):
            e0.record(stream)
            run()
            e1.record(stream)
            torch.cuda.synchronize()
            ms.append(e0.elapsed_time(e1))
        return min(ms)

    variants = []
    for v in range(lib.stream_copy_variants()):
        def run(v=v):
            rc = lib.stream_copy(v, src.data_ptr(), dst.data_ptr(), nbytes // 16, ctypes.c_void_p(stream.cuda_stream))
            assert rc == 0, rc
        ms = best(run)
        variants.append({"kernel": lib.stream_copy_name(v).decode(), "ms": ms, "GBps": 2.0 * nbytes / (ms * 1e-3) / 1e9})
    tms = best(lambda: dst.copy_(src))
    top = max(variants, key=lambda x: x["GBps"])
    return {"GBps": top["GBps"], "ms": top["ms"], "bytes": 2.0 * nbytes, "kernel": top["kernel"],
            "what": "hand-written streaming copy of the logits buffer into the dlogits buffer (16-byte non-temporal "
                    "loads and stores), the fastest of the variants",
            "variants": variants, "torch_copy_GBps": 2.0 * nbytes / (tms * 1e-3) / 1e9}


def device_info() -> dict:
    import torch
    p = torch.cuda.get_device_properties(0)
    out = {"name": p.name, "compute_units": p.multi_processor_count, "hbm_GiB": round(p.total_memory / 2**30, 1)}
    clk = getattr(p, "clock_rate", None)
    if clk:
        out["max_clock_MHz"] = clk / 1000.0
    return out


def time_logits(b: dict, norm: int, steps: int, warmup: int, dlogits=None) -> dict:
    """Times one logits-path step on batch b (group advantages, then grpo_loss_fwd_bwd with dlogits) under the
    normaliser ``norm``: the whole step by the host clock, the row pass by the HIP events the library records
    around it on its stream.  Returns the step's figures and the row pass's roofline."""
    import torch

    import paper_2606_05597_amd as grpo
    cfg, st = b["cfg"], b["structure"]
    T, V = b["logits"].shape
    N = len(st.rewards)
    dev = b["logits"].device
    sto = torch.from_numpy(st.step_tok_off).to(dev)
    tso = torch.from_numpy(st.traj_step_off).to(dev)
    adv = torch.empty(N, dtype=torch.float32, device=dev)
    dl = torch.empty_like(b["logits"]) if dlogits is None else dlogits
    ws = torch.empty(grpo.grpo_loss_workspace_bytes(T, N), dtype=torch.uint8, device=dev)
    loss = torch.empty(1, dtype=torch.float64, device=dev)
    stream = torch.cuda.current_stream()
    ev0 = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    ev1 = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    for e in ev0 + ev1:
        e.record(stream)  # creates the underlying hipEvent_t
    torch.cuda.synchronize()

    def step(i=None):
        grpo.grpo_advantages(b["rewards"], cfg.G, out=adv)
        aux = None if i is None else grpo.LossAux(hot_events=(ev0[i].cuda_event, ev1[i].cuda_event))
        grpo.grpo_loss_fwd_bwd(b["logits"], b["actions"], b["behave"], adv, sto, tso, cfg.G, V=b["V"], norm=norm,
                               k=cfg.k, eps_low=0.2, eps_high=0.2, dual_clip_c=3.0, dlogits=dl, aux=aux,
                               workspace=ws, loss_out=loss)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        step(i)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    hot_ms = sum(ev0[i].elapsed_time(ev1[i]) for i in range(steps)) / steps
    esz = b["logits"].element_size()
    alg = T * (2.0 * esz * V + 16.0)  # the row read once, dlogits written once, action + behave + weight + advantage
    achieved = alg / (hot_ms * 1e-3) / 1e9
    out = {"value": T / (ms * 1e-3), "unit": "tokens/s", "ms_per_step": ms, "steps": steps,
           "loss": float(loss.item()),
           "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                        "frac": achieved / HBM_PEAK_GBS, "traffic": None, "kernel_ms": hot_ms,
                        "algorithmic_bytes_per_launch": alg}}
    if dlogits is None:
        del dl
    del ws
    return out


def time_logits_graph(b: dict, norm: int, steps: int) -> dict:
    """The same logits-path step (group advantages, then grpo_loss_fwd_bwd with dlogits) captured once into a HIP
    graph and replayed: for launch-bound batches the launches, not the kernels, set the step time.  Every buffer is
    allocated before the capture; the replays' loss is checked against an eager call's, bit for bit."""
    import torch

    import paper_2606_05597_amd as grpo
    cfg, st = b["cfg"], b["structure"]
    T, V = b["logits"].shape
    N = len(st.rewards)
    dev = b["logits"].device
    sto = torch.from_numpy(st.step_tok_off).to(dev)
    tso = torch.from_numpy(st.traj_step_off).to(dev)
    adv = torch.empty(N, dtype=torch.float32, device=dev)
    dl = torch.empty_like(b["logits"])
    ws = torch.empty(grpo.grpo_loss_workspace_bytes(T, N), dtype=torch.uint8, device=dev)
    loss = torch.empty(1, dtype=torch.float64, device=dev)

    def step():
        grpo.grpo_advantages(b["rewards"], cfg.G, out=adv)
        grpo.grpo_loss_fwd_bwd(b["logits"], b["actions"], b["behave"], adv, sto, tso, cfg.G, V=b["V"], norm=norm,
                               k=cfg.k, eps_low=0.2, eps_high=0.2, dual_clip_c=3.0, dlogits=dl, workspace=ws,
                               loss_out=loss)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    eager = float(loss.item())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    loss.fill_(float("nan"))
    for _ in range(3):
        graph.replay()
    torch.cuda.synchronize()
    first = float(loss.item())
    t0 = time.perf_counter()
    for _ in range(steps):
        graph.replay()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    if not (first == eager and float(loss.item()) == eager):
        raise RuntimeError(f"graph replay loss {first!r} / {float(loss.item())!r} differs from the eager {eager!r}")
    del graph, dl, ws
    return {"value": T / (ms * 1e-3), "unit": "tokens/s", "ms_per_step": ms, "steps": steps, "loss": eager,
            "note": "the same step captured once into a HIP graph and replayed (host clock around the replays)"}


def bench_logits_config(name: str, steps: int, warmup: int = 2, kernel: str = "", norms=None,
                        graph: bool = False) -> dict:
    """One of the other logits-path workloads, generated, timed under each normaliser (and, with ``graph``, as a
    captured HIP graph under the first), and freed."""
    import torch

    import paper_2606_05597_amd as grpo
    from synth import make_batch
    b = make_batch(name, torch.device("cuda:0"))
    T, V = b["logits"].shape
    cfg = b["cfg"]
    dt = "bf16" if b["logits"].dtype == torch.bfloat16 else "fp32"
    norms = norms or [("1/k", grpo.GRPO_NORM_CONST_K)]
    res = {}
    for label, norm in norms:
        r = time_logits(b, norm, steps, warmup)
        r["roofline"]["kernel"] = kernel
        res[label] = r
    head = dict(res[norms[0][0]])
    head["workload"] = (f"{name}: {cfg.n_groups} groups x G={cfg.G}, T={T} action tokens, V={V}, {dt} logits; "
                        f"normaliser {norms[0][0]} (k={cfg.k:g})")
    for label, _ in norms[1:]:
        head[f"normaliser {label}"] = res[label]
    if graph:
        head["graph_replay"] = time_logits_graph(b, norms[0][1], max(steps, 100))
    del b
    torch.cuda.empty_cache()
    return head


def bench_logp(b: dict, steps: int, warmup: int = 2) -> dict:
    """Times grpo_token_logp (action log-prob + entropy, forward only) on the resident logits batch."""
    import torch

    import paper_2606_05597_amd as grpo
    T, V = b["logits"].shape
    stream = torch.cuda.current_stream()
    ev0 = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    ev1 = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    for _ in range(warmup):
        grpo.grpo_token_logp(b["logits"], b["actions"])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        ev0[i].record(stream)
        grpo.grpo_token_logp(b["logits"], b["actions"])
        ev1[i].record(stream)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    hot_ms = sum(ev0[i].elapsed_time(ev1[i]) for i in range(steps)) / steps
    alg = T * (2.0 * V + 12.0)  # logits row read once, action id read, log-prob and entropy written
    achieved = alg / (hot_ms * 1e-3) / 1e9
    return {"value": T / (ms * 1e-3), "unit": "tokens/s", "ms_per_step": ms, "steps": steps,
            "workload": f"forward only: action log-prob and entropy of the same {T} x {V} bf16 logits",
            "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                         "kernel": "k_logp_vec<bf16, 256, 4> (one workgroup per row)", "kernel_ms": hot_ms,
                         "algorithmic_bytes_per_launch": alg}}


def bench_vocab_shard(b: dict, steps: int, n_shards: int = 8, warmup: int = 2) -> dict:
    """Times one device's share of the vocabulary-parallel loss: the vocabulary of the resident batch split
    n_shards ways, the first shard held contiguous [T, V / n_shards].  A step is that shard's statistics pass and
    its loss/dlogits pass, with every shard's records already gathered (they are computed once, untimed, from
    the other column ranges of the same logits)."""
    import torch

    import paper_2606_05597_amd as grpo
    cfg, st = b["cfg"], b["structure"]
    T, V = b["logits"].shape
    Vs = V // n_shards
    dev = b["logits"].device
    N = len(st.rewards)
    stats = torch.empty((n_shards, T, grpo.VOCAB_STATS_BYTES), dtype=torch.uint8, device=dev)
    for g in range(n_shards):
        grpo.grpo_vocab_shard_stats(b["logits"][:, g * Vs:(g + 1) * Vs], b["actions"], g * Vs, stats=stats[g])
    shard = b["logits"][:, :Vs].contiguous()
    dshard = torch.empty_like(shard)
    sto = torch.from_numpy(st.step_tok_off).to(dev)
    tso = torch.from_numpy(st.traj_step_off).to(dev)
    adv = grpo.grpo_advantages(b["rewards"], cfg.G)
    ws = torch.empty(grpo.grpo_loss_workspace_bytes(T, N), dtype=torch.uint8, device=dev)
    loss = torch.empty(1, dtype=torch.float64, device=dev)
    stream = torch.cuda.current_stream()
    es = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    el = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for e in [x for pair in es + el for x in pair]:
        e.record(stream)  # creates the underlying hipEvent_t
    torch.cuda.synchronize()

    def step(i=None):
        if i is not None:
            es[i][0].record(stream)
        grpo.grpo_vocab_shard_stats(shard, b["actions"], 0, stats=stats[0])
        if i is not None:
            es[i][1].record(stream)
        aux = grpo.LossAux(hot_events=(el[i][0].cuda_event, el[i][1].cuda_event)) if i is not None else None
        grpo.grpo_loss_fwd_bwd_vocab_shard(shard, stats, 0, V, b["actions"], b["behave"], adv, sto, tso, cfg.G,
                                           norm=grpo.GRPO_NORM_CONST_K, k=cfg.k, dual_clip_c=3.0, dlogits=dshard,
                                           aux=aux, workspace=ws, loss_out=loss)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        step(i)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    stats_ms = sum(a.elapsed_time(c) for a, c in es) / steps
    rows_ms = sum(a.elapsed_time(c) for a, c in el) / steps
    rec = grpo.VOCAB_STATS_BYTES
    alg_stats = T * (2.0 * Vs + 4 + rec)  # the shard's row read once, the action id, one record written
    alg_rows = T * (4.0 * Vs + 16 + rec * n_shards)  # read + dlogits written, token inputs, every shard's record

    def roof(alg, kms, kernel):
        a = alg / (kms * 1e-3) / 1e9
        return {"bound": "hbm", "achieved": a, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": a / HBM_PEAK_GBS,
                "traffic": None, "kernel": kernel, "kernel_ms": kms, "algorithmic_bytes_per_launch": alg}

    return {"value": T / (ms * 1e-3), "unit": "tokens/s", "ms_per_step": ms, "steps": steps,
            "workload": f"one device's share of the {V}-column vocabulary split {n_shards} ways: bf16 [{T}, {Vs}], "
                        f"statistics pass + loss/dlogits pass",
            "loss": float(loss.item()),
            "roofline_stats": roof(alg_stats, stats_ms, "k_logp_vec<bf16, 256, 4> in record mode"),
            "roofline_rows": roof(alg_rows, rows_ms, "k_shard_rows_vec<bf16, 512, 5>")}


def fused_cpu_baseline(b: dict, rows: int = 64) -> dict:
    """The fp64 fused oracle (z = h W, the loss rows, dhidden = D W^T, dW += h^T D) on the first rows of the fused
    batch, timed on the host cores and scaled to tokens/s."""
    import numpy as np
    import torch

    import oracle
    from oracle import fused
    st, cfg = b["structure"], b["cfg"]
    hb = b["hidden"][:rows].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    W64 = fused.as_f64(b["W"].contiguous().view(torch.int16).cpu().numpy().view(np.uint16))
    seg = oracle.segments(st.T, st.step_tok_off, st.traj_step_off)
    A = oracle.advantages(st.rewards, cfg.G).astype(np.float32).astype(np.float64)
    actions, behave = b["actions"].cpu().numpy(), b["behave"].cpu().numpy()
    t0 = time.perf_counter()
    h64 = fused.as_f64(hb)
    z = h64 @ W64
    res = oracle.loss_rows(z, actions, behave, None, A, seg, cfg.G, norm=oracle.NORM_CONST_K, k=cfg.k,
                           dual_clip_c=3.0, row_begin=0, row_end=rows, row_offset=0)
    D = res.dlogits
    dh = D @ W64.T
    dW = h64.T @ D
    el = time.perf_counter() - t0
    del z, D, dh, dW, W64
    return {"value": rows / el, "unit": "tokens/s", "cores": oracle.threads(), "kind": "oracle",
            "sample": f"first {rows} token rows of the fused batch: the three fp64 products and the loss rows, "
                      f"{el:.1f} s (numpy float64 matmul on the host's cores; the per-token rate extrapolates "
                      f"to the whole batch)"}


def time_fused(b: dict, adv, sto, tso, steps: int, warmup: int, token_block: int = 0,
               two_streams: bool = False) -> dict:
    """Times one schedule of the fused LM head on batch b: the vocabulary-chunked fused_lmhead_grpo (token_block 0)
    or the token-blocked fused_lmhead_grpo_blocked.  The hot region, timed with events the library records on its
    stream, is the first forward product through the last backward product."""
    import torch

    import paper_2606_05597_amd as grpo
    cfg, st = b["cfg"], b["structure"]
    T, H, V = st.T, b["H"], b["V"]
    N = len(st.rewards)
    dev = b["hidden"].device
    dh = torch.empty_like(b["hidden"])
    dw = torch.empty((H, V), dtype=torch.float32, device=dev)
    if token_block:
        need = grpo.fused_lmhead_blocked_workspace_bytes(T, H, V, token_block, N)
        entry, kw = grpo.fused_lmhead_grpo_blocked, dict(token_block=token_block)
        if two_streams:
            kw["aux_stream"] = torch.cuda.Stream(device=dev)
    else:
        need = grpo.fused_lmhead_workspace_bytes(T, H, V, cfg.vocab_chunk, N)
        entry, kw = grpo.fused_lmhead_grpo, dict(vocab_chunk=cfg.vocab_chunk)
    ws = torch.empty(need, dtype=torch.uint8, device=dev)
    loss = torch.empty(1, dtype=torch.float64, device=dev)
    stream = torch.cuda.current_stream()
    ev0 = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    ev1 = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    for e in ev0 + ev1:
        e.record(stream)
    torch.cuda.synchronize()

    def step(i=None):
        grpo.grpo_advantages(b["rewards"], cfg.G, out=adv)
        aux = None if i is None else grpo.LossAux(hot_events=(ev0[i].cuda_event, ev1[i].cuda_event))
        entry(b["hidden"], b["W"], b["actions"], b["behave"], adv, sto, tso, cfg.G, norm=grpo.GRPO_NORM_CONST_K,
              k=cfg.k, dual_clip_c=3.0, dhidden=dh, dw_lm=dw, aux=aux, workspace=ws, loss_out=loss, **kw)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        step(i)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    hot_ms = sum(ev0[i].elapsed_time(ev1[i]) for i in range(steps)) / steps
    products = 3 if token_block else 4
    alg = 6.0 * T * H * V
    achieved = alg / (hot_ms * 1e-3) / 1e12
    out = {"value": T / (ms * 1e-3), "unit": "tokens/s", "ms_per_step": ms, "steps": steps, "hot_ms": hot_ms,
           "loss": float(loss.item()), "workspace_bytes": need,
           "schedule": (f"token blocks of {token_block} (their logits kept between the products as fp16 terms exp(z - m); "
                        f"3 products)"
                        if token_block else
                        f"vocabulary chunks of {cfg.vocab_chunk} (logits recomputed for the backward; 4 products)"),
           "roofline": {"bound": "mfma", "achieved": achieved, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                        "frac": achieved / MFMA_BF16_PEAK_TFLOPS, "hot_ms": hot_ms,
                        "algorithmic_flop_per_launch": alg,
                        "executed_frac": (2.0 * products * T * H * V) / (hot_ms * 1e-3) / 1e12
                        / MFMA_BF16_PEAK_TFLOPS}}
    del dh, dw, ws
    torch.cuda.empty_cache()
    return out


def bench_fused_logp(b: dict, steps: int, warmup: int = 1) -> dict:
    """Forward only from hidden states (fused_lmhead_token_logp): the action log-probs and entropies of the fused
    workload, z = h W formed once on the matrix cores and never stored; the whole call timed with HIP events."""
    import torch

    import paper_2606_05597_amd as grpo
    st = b["structure"]
    T, H, V = st.T, b["H"], b["V"]
    dev = b["hidden"].device
    ws = torch.empty(grpo._lib.load().fused_lmhead_token_logp_workspace_bytes(T, H, V), dtype=torch.uint8,
                     device=dev)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for _ in range(warmup):
        grpo.fused_lmhead_token_logp(b["hidden"], b["W"], b["actions"], workspace=ws)
    torch.cuda.synchronize()
    for i in range(steps):
        ev[i][0].record()
        grpo.fused_lmhead_token_logp(b["hidden"], b["W"], b["actions"], workspace=ws)
        ev[i][1].record()
    torch.cuda.synchronize()
    ms = sum(a.elapsed_time(c) for a, c in ev) / steps
    alg = 2.0 * T * H * V
    achieved = alg / (ms * 1e-3) / 1e12
    del ws
    torch.cuda.empty_cache()
    return {"value": T / (ms * 1e-3), "unit": "tokens/s", "ms_per_step": ms, "steps": steps,
            "workload": f"forward only from hidden states: log-prob and entropy per token, hidden bf16 [{T}, {H}], "
                        f"W bf16 [{H}, {V}]",
            "roofline": {"bound": "mfma", "achieved": achieved, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                         "frac": achieved / MFMA_BF16_PEAK_TFLOPS, "traffic": None,
                         "algorithmic_flop_per_launch": alg}}


def library_gemm(b: dict, token_block: int, reps: int = 3) -> dict:
    """Context for the fused line, as the copy ceiling is for the row pass: the three products of one token block
    done by torch.matmul (hipBLASLt), bf16 in and out, no epilogue, operands laid out as the library's kernels read
    them (both K-contiguous), and what the whole call's products would take at those rates."""
    import torch

    st = b["structure"]
    T, H, V = st.T, b["H"], b["V"]
    tb = min(token_block, T)
    dev = b["hidden"].device
    gen = torch.Generator(device=dev).manual_seed(7)
    h = b["hidden"][:tb]
    wt = b["W"].t().contiguous()                          # [V, H]
    d = (torch.randn((tb, V), device=dev, generator=gen) * 1e-3).to(torch.bfloat16)
    ht = h.t().contiguous()                               # [H, tb]
    dt = d.t().contiguous()                               # [V, tb]
    prods = {"forward z = h W": (lambda: torch.matmul(h, wt.t()), (tb, V, H)),
             "dhidden = D W^T": (lambda: torch.matmul(d, b["W"].t()), (tb, H, V)),
             "dW = h^T D": (lambda: torch.matmul(ht, dt.t()), (H, V, tb))}
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    res, block_ms = {}, 0.0
    for name, (fn, (m, n, k)) in prods.items():
        fn()
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        block_ms += ms
        res[name] = {"shape_mnk": [m, n, k], "ms": ms, "TFLOPs": 2.0 * m * n * k / (ms * 1e-3) / 1e12}
    del wt, d, ht, dt
    torch.cuda.empty_cache()
    call_ms = block_ms * T / tb
    return {"kernel": "torch.matmul (hipBLASLt), bf16 in and out, no epilogue", "token_block": tb,
            "products": res, "block_ms": block_ms, "call_ms": call_ms,
            "call_TFLOPs": 6.0 * T * H * V / (call_ms * 1e-3) / 1e12}


FUSED_SCHEDULES = ("blocked", "blocked1", "chunked")


def bench_fused(steps: int, warmup: int = 1, shard_steps: int = 0, cpu: bool = False, token_block: int = 8192,
                schedules=FUSED_SCHEDULES) -> dict:
    """The fused workload in the chosen schedules: "blocked" (token blocks, each block's D pass on a second stream
    beside the next block's forward product), "blocked1" (token blocks on one stream), "chunked" (vocabulary
    chunks, logits recomputed).  The first one chosen is the line's value; the others are reported beside it."""
    import torch

    from synth import make_fused_batch

    dev = torch.device("cuda:0")
    b = make_fused_batch("fused", dev)
    cfg, st = b["cfg"], b["structure"]
    T, H, V = st.T, b["H"], b["V"]
    N = len(st.rewards)
    sto = torch.from_numpy(st.step_tok_off).to(dev)
    tso = torch.from_numpy(st.traj_step_off).to(dev)
    adv = torch.empty(N, dtype=torch.float32, device=dev)
    res = {}
    for sch in schedules:
        if sch == "chunked":
            r = time_fused(b, adv, sto, tso, steps, warmup, 0)
            r["roofline"]["traffic"] = measured_fused_traffic("chunked")
        else:
            r = time_fused(b, adv, sto, tso, steps, warmup, token_block, two_streams=(sch == "blocked"))
            r["roofline"]["traffic"] = measured_fused_traffic("blocked")
            if sch == "blocked":
                r["schedule"] += "; each block's D pass on a second stream beside the next block's forward product"
        res[sch] = r
    head = schedules[0]
    out = dict(res[head])
    out["workload"] = (f"fused: hidden bf16 [{T}, {H}], W bf16 [{H}, {V}], {cfg.n_groups} groups x G={cfg.G}; "
                       f"{out['schedule']}")
    names = {"blocked": "token_blocked_two_streams", "blocked1": "token_blocked_one_stream",
             "chunked": "vocab_chunked"}
    for sch in schedules[1:]:
        out[names[sch]] = res[sch]
    lib = library_gemm(b, token_block or 8192)
    lib["frac_of_library_products"] = lib["call_ms"] / out["hot_ms"]
    out["library_gemm"] = lib
    out["forward_only"] = bench_fused_logp(b, max(1, steps))
    if shard_steps > 0:
        out["vocab_shard"] = bench_fused_shard(b, adv, sto, tso, shard_steps, keep=True)
        out["vocab_shard"]["recompute"] = bench_fused_shard(b, adv, sto, tso, shard_steps, keep=False)
    if cpu:
        out["cpu_baseline"] = fused_cpu_baseline(b)
    return out


def bench_fused_shard(b: dict, adv, sto, tso, steps: int, n_shards: int = 8, warmup: int = 1,
                      keep: bool = True) -> dict:
    """One device's share of the vocabulary-parallel fused LM head on the fused workload: W's columns split n_shards
    ways, the first shard's statistics call and backward call timed, every shard's records gathered beforehand.
    keep: the statistics call keeps the shard's logits and the backward call uses them (three products in the two
    calls); otherwise the backward call forms them again (four)."""
    import torch

    import paper_2606_05597_amd as grpo
    cfg, st = b["cfg"], b["structure"]
    T, H, V = st.T, b["H"], b["V"]
    N = len(st.rewards)
    Vs = V // n_shards
    chunk = (Vs + 511) // 512 * 256  # the shard's columns in one pair of chunks
    dev = b["hidden"].device
    stats = torch.empty((n_shards, T, grpo.VOCAB_STATS_BYTES), dtype=torch.uint8, device=dev)
    for g in range(n_shards):
        grpo.fused_lmhead_vocab_shard_stats(b["hidden"], b["W"][:, g * Vs:(g + 1) * Vs].contiguous(), b["actions"],
                                            g * Vs, stats=stats[g])
    w = b["W"][:, :Vs].contiguous()
    dhp = torch.empty((T, H), dtype=torch.float32, device=dev)
    dws = torch.empty((H, Vs), dtype=torch.float32, device=dev)
    ws1 = torch.empty(grpo._lib.load().fused_lmhead_vocab_shard_stats_workspace_bytes(T, H, Vs), dtype=torch.uint8,
                      device=dev)
    kept = grpo.vocab_shard_logits_buffer(T, Vs, dev) if keep else None
    if keep:
        chunk = (Vs + 255) // 256 * 256  # the whole shard as one chunk
    ws2 = torch.empty(grpo.fused_lmhead_workspace_bytes(T, H, Vs, chunk, N), dtype=torch.uint8, device=dev)
    loss = torch.empty(1, dtype=torch.float64, device=dev)
    stream = torch.cuda.current_stream()
    es = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    eb = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for e in [x for pair in es + eb for x in pair]:
        e.record(stream)
    torch.cuda.synchronize()

    def step(i=None):
        if i is not None:
            es[i][0].record(stream)
        grpo.fused_lmhead_vocab_shard_stats(b["hidden"], w, b["actions"], 0, stats=stats[0], workspace=ws1,
                                            logits_out=kept)
        if i is not None:
            es[i][1].record(stream)
            eb[i][0].record(stream)
        grpo.fused_lmhead_grpo_vocab_shard(b["hidden"], w, stats, 0, V, b["actions"], b["behave"], adv, sto, tso,
                                           cfg.G, vocab_chunk=chunk, norm=grpo.GRPO_NORM_CONST_K, k=cfg.k,
                                           dual_clip_c=3.0, dhidden_partial=dhp, dw_shard=dws, workspace=ws2,
                                           loss_out=loss, logits_in=kept)
        if i is not None:
            eb[i][1].record(stream)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        step(i)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    stats_ms = sum(a.elapsed_time(c) for a, c in es) / steps
    bwd_ms = sum(a.elapsed_time(c) for a, c in eb) / steps
    alg = 6.0 * T * H * Vs
    achieved = alg / ((stats_ms + bwd_ms) * 1e-3) / 1e12
    how = ("the statistics call keeps the shard's fp32 logits, the backward call forms D from them"
           if keep else f"the backward call forms the logits again in chunks of {chunk}")
    products = 3 if keep else 4
    return {"value": T / (ms * 1e-3), "unit": "tokens/s", "ms_per_step": ms, "steps": steps,
            "workload": f"one device's share of the fused LM head with W's {V} columns split {n_shards} ways: "
                        f"hidden bf16 [{T}, {H}], W shard bf16 [{H}, {Vs}]; statistics call + backward call "
                        f"(records of all {n_shards} shards gathered beforehand); {how}",
            "loss": float(loss.item()), "stats_ms": stats_ms, "backward_ms": bwd_ms,
            "roofline": {"bound": "mfma", "achieved": achieved, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                         "frac": achieved / MFMA_BF16_PEAK_TFLOPS, "traffic": None,
                         "algorithmic_flop_per_launch": alg,
                         "executed_frac": (2.0 * products * T * H * Vs) / ((stats_ms + bwd_ms) * 1e-3) / 1e12
                         / MFMA_BF16_PEAK_TFLOPS}}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: the benchmark runs on one GPU only (asked for --gpus {args.gpus}); "
              "the loss shards by whole task groups, one process per GPU, with one fp64 all-reduce of the loss", file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return
    if args.skip_logits:
        print(json.dumps({"fused_lmhead": bench_fused(max(1, args.fused_steps), shard_steps=args.shard_steps and 3,
                                                          token_block=args.token_block,
                                                          schedules=fused_schedules(args))}),
              flush=True)
        return
    import numpy as np
    import torch

    import paper_2606_05597_amd as grpo
    from synth import make_batch

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    b = make_batch("v152k", dev)
    cfg, st = b["cfg"], b["structure"]
    T, V = b["logits"].shape
    N = len(st.rewards)
    dlogits = torch.empty_like(b["logits"])
    head = time_logits(b, grpo.GRPO_NORM_CONST_K, args.steps, args.warmup, dlogits=dlogits)
    roof = head["roofline"]
    roof["traffic"] = measured_traffic(T)
    roof["kernel"] = "k_rows_pipe<19, 6> (bf16, 1024 threads, one workgroup per CU)"
    out = {
        "metric": METRIC,
        "value": head["value"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "v152k: 16 groups x G=8 rollouts, T=120,000 action tokens, V=151,936, bf16 logits",
                   "T": T, "V": V, "n_traj": N, "n_steps": int(st.step_tok_off.shape[0] - 1),
                   "normalizer": "1/k (k=10)", "eps": 0.2, "dual_clip_c": 3.0, "loss": head["loss"]},
        "roofline": roof,
    }
    # the memory-only ceiling on the same two buffers, then the row pass again, so that a placement that changes
    # between the two would show
    cc = copy_ceiling(b["logits"], dlogits)
    again = time_logits(b, grpo.GRPO_NORM_CONST_K, max(3, args.steps // 2), 1, dlogits=dlogits)
    roof["copy_ceiling_GBps"] = cc["GBps"]
    roof["copy_ceiling_kernel"] = cc["kernel"]
    roof["copy_variants"] = cc["variants"]
    roof["torch_copy_GBps"] = cc["torch_copy_GBps"]
    roof["frac_of_copy_ceiling"] = roof["achieved"] / cc["GBps"]
    roof["kernel_ms_after_copy"] = again["roofline"]["kernel_ms"]
    # the paper's baseline normaliser 1/|tau_i| on the same batch (Sec. 3.2; the workload names both)
    trs = time_logits(b, grpo.GRPO_NORM_TRAJ_STEPS, max(3, args.steps // 2), 1, dlogits=dlogits)
    trs["roofline"]["kernel"] = roof["kernel"]
    out["normaliser_traj_steps"] = trs
    del dlogits
    torch.cuda.empty_cache()
    out["device"] = device_info()
    if args.cpu_seconds > 0:
        import oracle
        A = oracle.advantages(st.rewards, cfg.G).astype(np.float32).astype(np.float64)
        out["cpu_baseline"] = cpu_baseline(b, A, args.cpu_seconds)
    if args.logp_steps > 0:
        out["token_logp"] = bench_logp(b, args.logp_steps)
    if args.shard_steps > 0:
        out["vocab_shard"] = bench_vocab_shard(b, args.shard_steps)
    del b
    torch.cuda.empty_cache()
    if args.config_steps > 0:
        out["long"] = bench_logits_config("long", args.config_steps, kernel=roof["kernel"])
        out["v32k"] = bench_logits_config(
            "v32k", args.config_steps, kernel="k_rows_resident<bf16, 1024, 4> (one workgroup per row)",
            norms=[("1/k", grpo.GRPO_NORM_CONST_K), ("1/|tau_i|", grpo.GRPO_NORM_TRAJ_STEPS)])
        tiny = bench_logits_config(
            "tiny", max(20, args.config_steps), kernel="k_rows_resident<fp32, 64, 4> (one workgroup per row)",
            norms=[("1/k", grpo.GRPO_NORM_CONST_K), ("1/|tau_i|", grpo.GRPO_NORM_TRAJ_STEPS)], graph=True)
        tiny["note"] = ("launch-bound: four small launches per step (advantages, segments, row pass, reduction); "
                        "graph_replay: the same step as one captured HIP graph")
        out["tiny"] = tiny
    if args.fused_steps > 0:
        out["fused_lmhead"] = bench_fused(args.fused_steps, shard_steps=args.shard_steps and 3,
                                          cpu=args.cpu_seconds > 0, token_block=args.token_block,
                                          schedules=fused_schedules(args))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
