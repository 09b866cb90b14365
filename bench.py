#!/usr/bin/env python3
"""Decode-step throughput of the language-decode hot path on one MI355X.

A step is one decode step (hs_decode_step): embedding gather, every decoder layer
(RMSNorm + q/k/v + RoPE + KV append, split-K attention and combine, output
projection, RMSNorm + gate/up + SwiGLU, down projection) and the final norm,
LM head and greedy selection, for every request of the batch.  Inputs are
seeded synthetic tensors generated directly in HBM; the KV cache is filled by
prefill from the vision rows and text tokens (or, for the one-layer workload,
with synthetic rows) before timing.  The timed steps are replayed from HIP
graphs (one captured step per graph, the greedy tokens chaining on the device);
the same number of direct calls is timed beside them.

The default run measures the headline workload (LLaVA-7B-shaped fp16,
batch 1) and then, in the same process, the batched LLaVA-shaped, the
Qwen2.5-VL-shaped and the one-layer batch-256 workloads.  For each it reports
tokens/s, algorithmic HBM GB/s, the dominant kernel against the HBM roofline,
the CPU oracle's rate on a bounded sample, and the parity of the GPU with that
oracle on the same teacher-forced steps.

Prints one JSON line on stdout; progress goes to stderr.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-workloads]
    python bench.py --summarise-stats TRACE_DIR BENCH_LOG WORKLOAD "COMMAND"
    python bench.py --summarise-counters FETCH_DIR WRITE_DIR WORKLOAD KIND "KERNEL" "COMMAND"
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import re
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0  # MI355X HBM3E
WEIGHT_COPIES = 4  # one-layer workloads: weight sets rotated over the steps (4 x 0.47 GB > 256 MB Infinity Cache)
METRIC = "decode tokens/s at batch B + achieved HBM GB/s vs peak, 7B-shaped fp16"
HEADLINE = "llava7b_b1"
WORKLOADS = ("llava7b_b32", "qwen7b_b16", "qwen_layer_b256")
LOGIT_TOL = 2e-2
# oracle steps per workload (bounded CPU sample, a few seconds per step at 7B size)
ORACLE_STEPS = {"llava7b_b1": 5, "llava7b_b32": 2, "qwen7b_b16": 2, "qwen_layer_b256": 3}


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def weight_bytes(cfg: dict) -> dict:
    """Algorithmic bytes of each weight set streamed once per step."""
    b = 2 if cfg["dtype"] != "f32" else 4
    d, nh, nkv, hd, F, V = (cfg[k] for k in ("d_model", "n_heads", "n_kv_heads", "head_dim", "ffn_dim", "vocab"))
    qkv = (nh + 2 * nkv) * hd * d + (nh + 2 * nkv) * hd * cfg["qkv_bias"] + d  # + attn_norm gain
    out = {
        "qkv": qkv * b,
        "oproj": d * nh * hd * b,
        "gateup": (2 * F * d + d) * b,  # + mlp_norm gain
        "down": d * F * b,
    }
    out["head"] = (V * d + d) * b if cfg.get("lm_head", True) else 0
    return out


def step_bytes(cfg: dict, lens: list) -> int:
    """Algorithmic HBM bytes of one step: every weight once, the embedding
    rows, every request's K/V rows 0..len_b (read) and the appended row
    (written)."""
    b = 2 if cfg["dtype"] != "f32" else 4
    wb = weight_bytes(cfg)
    L, nkv, hd, d = cfg["n_layers"], cfg["n_kv_heads"], cfg["head_dim"], cfg["d_model"]
    per_layer = wb["qkv"] + wb["oproj"] + wb["gateup"] + wb["down"]
    kv_row = 2 * L * nkv * hd * b
    B = len(lens)
    return L * per_layer + wb["head"] + B * d * b + sum(kv_row * (n + 1) for n in lens) + B * kv_row


def attn_bytes(cfg: dict, lens: list) -> int:
    """Algorithmic bytes of one attention launch (one layer): K and V rows
    0..len_b of every request, its q rows read and its output rows written."""
    b = 2 if cfg["dtype"] != "f32" else 4
    nkv, nh, hd = cfg["n_kv_heads"], cfg["n_heads"], cfg["head_dim"]
    return sum(2 * nkv * hd * (n + 1) * b for n in lens) + len(lens) * 2 * nh * hd * b


# what each replayable kind launches, for the roofline line
KIND_NAMES = {
    "qkv": "q/k/v projection (RMSNorm + GEMM + RoPE + KV append)",
    "attn": "split-K attention over the KV cache",
    "oproj": "O projection + residual",
    "gateup": "gate/up projection (RMSNorm + GEMM + SwiGLU)",
    "down": "down projection + residual",
    "head": "final RMSNorm + LM head",
}


def kernel_source_hash(kind: str = "gateup") -> str:
    """Hash of the sources that build the kernels of one replayable kind."""
    h = hashlib.sha256()
    main = "hs_attn.hip" if kind in ("attn", "combine") else "hs_gemm.hip"
    for rel in ("paper_2603_12707_amd/csrc/" + main, "paper_2603_12707_amd/csrc/hs_device.h",
                "paper_2603_12707_amd/csrc/hs_internal.h"):
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def stored_traffic(workload: str, kernel: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or
    None if there is none for this kernel source."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_counters.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    src = re.search(r"kernel_source_sha256:\s*([0-9a-f]+)", text)
    val = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not src or not val or src.group(1) != kernel_source_hash(kernel):
        return None
    return float(val.group(1))


DEFAULT_WARMUP, DEFAULT_STEPS = 8, 120
PREFILL_ROWS = 16384  # packed prefill rows per pass at batch > 1
STREAM_READ_BYTES, STREAM_READ_BLOCKS = 4 << 30, (1024, 2048, 4096)


def steps_after_context(warmup: int, steps: int) -> int:
    """Positions a bench run needs after the context: warm-up, the timed region,
    and one spare position that kernel replays rewrite."""
    return warmup + steps + 1


def make_weights(cfg: dict):
    """Weight sets generated and packed in HBM (several copies for a one-layer
    workload, so that the 256 MB Infinity Cache cannot carry one step's weights
    into the next)."""
    import torch

    import paper_2603_12707_amd as hs
    from workload import synth
    t = time.time()
    copies = WEIGHT_COPIES if "kv_len" in cfg else 1
    ws = []
    for k in range(copies):
        w = {}
        for name in synth.weight_names(cfg):  # generate and pack one matrix at a time
            t_row = synth.make_weight(cfg, name, device="cuda", seed=None if k == 0 else cfg["seed"] + 7919 * k)
            w[name] = hs.pack_weight(cfg, name, t_row)
            del t_row
        ws.append(w)
    torch.cuda.synchronize()
    log(f"{cfg['name']}: weights generated and packed in HBM: {copies} x "
        f"{sum(v.numel() * v.element_size() for v in ws[0].values()) / 1e9:.2f} GB in {time.time() - t:.1f} s")
    return ws


def context_lengths(cfg: dict) -> tuple:
    from workload import synth
    if "kv_len" in cfg:  # layer stack fed from a synthetic cache
        return [0] * cfg["batch"], synth.kv_lengths(cfg)
    n_v, s_text = synth.request_lengths(cfg)
    return n_v, [a + b for a, b in zip(n_v, s_text)]


def fill_synthetic(cfg: dict, kv, lens: list) -> None:
    """Every request's cache rows [0, len) from the seeded generator (the rows
    the oracle leg reads too); RoPE position = length."""
    from workload import synth
    for r, n in enumerate(lens):
        kv.set_length(r, n, n)  # a pool takes the blocks here
        for layer in range(cfg["n_layers"]):
            for sel in (0, 1):
                for h in range(cfg["n_kv_heads"]):
                    kv.write(r, layer, sel, h, 0, synth.kv_block(cfg, r, layer, sel, h, n, device="cuda"))


def setup(cfg: dict, ws: list, n_steps_total: int, pool_block: int = 0):
    import torch

    import paper_2603_12707_amd as hs
    from workload import synth
    B = cfg["batch"]
    n_v, lens = context_lengths(cfg)
    caps = [n + n_steps_total for n in lens]
    models = [hs.Model(cfg, w, max_batch=B, max_ctx=max(caps), packed=True) for w in ws]
    model = models[0]
    if pool_block:  # block-granular cache: one slot per request, admitted up front
        n_blocks = sum((c + pool_block - 1) // pool_block for c in caps)
        kv = hs.KVPool(model, B, pool_block, n_blocks)
        for r in range(B):
            kv.admit(r, n_v[r], caps[r])
    else:
        kv = hs.KVCache(model, n_v, caps)
    first = torch.empty(B, dtype=torch.int32, device="cuda")
    t = time.time()
    prefill_ms = None
    if "kv_len" in cfg:
        fill_synthetic(cfg, kv, lens)
        first.copy_(synth.decode_tokens(cfg, 0, B, device="cuda"))
    else:
        _, s_text = synth.request_lengths(cfg)
        # inputs first, packed request by request; then the timed prefill
        embs = [synth.vision_rows(cfg, r, n_v[r], device="cuda") for r in range(B) if n_v[r]]
        idss = [synth.text_ids(cfg, r, s_text[r], device="cuda") for r in range(B) if s_text[r]]
        emb = torch.cat(embs) if embs else None
        ids = torch.cat(idss) if idss else None
        pos = (torch.cat([synth.mrope_positions(n_v[r], s_text[r]) for r in range(B)], dim=1).contiguous().cuda()
               if cfg["rope_kind"] == 1 else None)
        if B > 1:  # room for several requests per packed pass
            model.reserve_rows(min(sum(lens), PREFILL_ROWS))
        torch.cuda.synchronize()
        t = time.time()
        if B == 1:
            kv.prefill(0, emb, ids, pos, first_token=first)
        else:
            kv.prefill_batch(list(range(B)), emb, ids, s_text, pos, first_tokens=first)
    torch.cuda.synchronize()
    ready_s = time.time() - t
    log(f"{cfg['name']}: context ready for {B} request(s) in {ready_s * 1e3:.1f} ms (lengths {min(lens)}..{max(lens)})")
    if "kv_len" not in cfg:
        prefill_ms = ready_s * 1e3 / B
    return models, kv, first, lens, prefill_ms


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def stream_read_rate() -> float:
    """The plain streaming-read rate of this GPU (the same 16-byte
    non-temporal loads as the weight stream), best of three grids."""
    import torch

    import paper_2603_12707_amd as hs
    buf = torch.empty(STREAM_READ_BYTES, dtype=torch.uint8, device="cuda")
    sink = torch.empty(max(STREAM_READ_BLOCKS), dtype=torch.int32, device="cuda")
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    best = 0.0
    for blocks in STREAM_READ_BLOCKS:
        hs.stream_read(buf, sink, blocks)  # warm
        ev0.record()
        for _ in range(5):
            hs.stream_read(buf, sink, blocks)
        ev1.record()
        torch.cuda.synchronize()
        best = max(best, 5 * STREAM_READ_BYTES / (ev0.elapsed_time(ev1) / 1e3) / 1e9)
    del buf, sink
    return best


def prewarm(seconds: float = 0.5) -> None:
    """Streaming reads for about `seconds` before a timed region, so that the
    GPU's clocks have left any idle state (an oracle leg or a weight upload
    leaves the GPU idle for seconds; a short timed region after that measured
    up to 6 % slow)."""
    import torch

    import paper_2603_12707_amd as hs
    buf = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    sink = torch.empty(2048, dtype=torch.int32, device="cuda")
    t = time.time()
    while time.time() - t < seconds:
        for _ in range(50):
            hs.stream_read(buf, sink, 2048)
        torch.cuda.synchronize()
    del buf, sink


def measure(cfg: dict, ws: list, steps: int, warmup: int, eager: bool = False, pool_block: int = 0,
            stream_gbs: float = 0.0) -> dict:
    """Times `steps` decode steps after `warmup`, then the per-kernel breakdown
    and the dominant kernel replayed back to back.

    The timed steps are replayed from HIP graphs, one captured decode step
    each (the paper's engine runs its decode iteration from CUDA graphs,
    §5.4): graph i decodes from token buffer i % 2 into the other (greedy
    tokens chain from step to step on the device) with weight copy
    i % copies.  The same number of steps called directly is timed after
    them and reported beside (`eager`: the other way round)."""
    import torch
    B = cfg["batch"]
    copies = len(ws)
    has_head = cfg.get("lm_head", True)
    P = copies if copies % 2 == 0 or not has_head else 2 * copies  # graphs: token ping-pong x weight rotation
    models, kv, first, lens0, prefill_ms = setup(cfg, ws, steps_after_context(warmup, 2 * steps), pool_block)
    tb = [first.clone(), torch.empty_like(first)]
    graphs = []
    for i in range(P):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            kv.decode(tb[i % 2] if has_head else tb[0], tb[(i + 1) % 2] if has_head else None,
                      model=models[i % copies])
        graphs.append(g)
    kv.sync()  # capture launched nothing: the lengths are those after prefill
    assert kv.lengths() == lens0

    def replayed(n):
        graphs[n % P].replay()

    def called(n):
        kv.decode(tb[n % 2] if has_head else tb[0], tb[(n + 1) % 2] if has_head else None,
                  model=models[n % copies])

    first_run, second_run = (called, replayed) if eager else (replayed, called)
    prewarm()
    for n in range(warmup):
        first_run(n)
    torch.cuda.synchronize()
    # timed region: K steps bracketed by device synchronisation
    t0 = time.perf_counter()
    for n in range(warmup, warmup + steps):
        first_run(n)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    kv.sync()
    lens_after = kv.lengths()
    t0 = time.perf_counter()
    for n in range(warmup + steps, warmup + 2 * steps):
        second_run(n)
    torch.cuda.synchronize()
    other_ms = (time.perf_counter() - t0) / steps * 1e3
    kv.sync()
    del graphs

    # per-kernel breakdown, the same way for every replayable kind: each
    # layer's launch replayed once per weight copy, HIP events around the
    # batch on the stream the library launches on (torch's current stream)
    def replay_all(kind, passes):
        for _ in range(passes):
            for m in models:
                kv.replay(kind, cfg["n_layers"], model=m)
    launches = cfg["n_layers"] * len(models)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    breakdown = {}
    for kind in ("qkv", "attn", "combine", "oproj", "gateup", "down", "head"):
        try:
            kv.replay(kind, 1)
        except Exception:  # combine: single split; head: no LM head
            continue
        ev0.record()
        replay_all(kind, 1)
        ev1.record()
        torch.cuda.synchronize()
        breakdown[kind] = ev0.elapsed_time(ev1) / launches * 1e3  # us per launch
    # dominant kernel: the kind with the most time per step, replayed back
    # to back over every layer's weights (4 passes over each copy)
    per_step = {k: v * (1 if k == "head" else cfg["n_layers"]) for k, v in breakdown.items() if k in KIND_NAMES}
    dominant = max(per_step, key=per_step.get)
    lens_replay = kv.lengths()
    reps = 4 * launches
    replay_all(dominant, 1)  # warm
    ev0.record()
    replay_all(dominant, 4)
    ev1.record()
    torch.cuda.synchronize()
    dom_avg_s = ev0.elapsed_time(ev1) / 1e3 / reps

    ms_per_step = elapsed / steps * 1e3
    lens_start = [n + warmup for n in lens0]
    total_bytes = sum(step_bytes(cfg, [n + k for n in lens_start]) for k in range(steps))
    gbs = total_bytes / elapsed / 1e9
    assert lens_after == [n + steps for n in lens_start], (lens_after[:4], lens_start[:4])
    assert kv.lengths() == [n + 2 * steps for n in lens_start]
    dom_bytes = attn_bytes(cfg, lens_replay) if dominant == "attn" else weight_bytes(cfg)[dominant]
    achieved = dom_bytes / dom_avg_s / 1e9
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": stored_traffic(cfg["name"], dominant),
                "kernel": KIND_NAMES[dominant], "kind": dominant,
                "bytes_per_launch": dom_bytes, "avg_launch_us": round(dom_avg_s * 1e6, 2), "launches": reps}
    if stream_gbs:
        roofline["stream_read_gbps"] = round(stream_gbs, 1)
        roofline["frac_of_stream_read"] = round(achieved / stream_gbs, 4)
    out = {
        "value": round(B * steps / elapsed, 2),
        "unit": "tokens/s",
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(ms_per_step, 4),
        "dtype": cfg["dtype"],
        "config": {"workload": cfg["name"], "batch": B,
                   "context_at_start": lens_start[0] if B == 1 else [min(lens_start), max(lens_start)],
                   "n_layers": cfg["n_layers"], "d_model": cfg["d_model"], "n_heads": cfg["n_heads"],
                   "n_kv_heads": cfg["n_kv_heads"], "ffn_dim": cfg["ffn_dim"],
                   "vocab": cfg["vocab"] if has_head else None, "qkv_bias": cfg["qkv_bias"],
                   "rope": "3-section M-RoPE" if cfg["rope_kind"] == 1 else "1-D RoPE",
                   "parallelism": "none (one GPU)",
                   "kv_cache": f"pool of {pool_block}-position blocks" if pool_block else "contiguous",
                   "weight_copies": copies},
        "hbm_gbps": round(gbs, 1),
        "hbm_frac": round(gbs / PEAK_HBM_GBS, 4),
        "bytes_per_step": total_bytes // steps,
        "roofline": roofline,
        "kernel_us": {k: round(v, 2) for k, v in breakdown.items()},
    }
    if prefill_ms is not None:
        out["prefill_ms_per_request"] = round(prefill_ms, 2)
    out["timed_as"] = "direct hs_decode_step calls" if eager else "decode steps replayed from HIP graphs"
    out["eager" if not eager else "graph"] = {
        "ms_per_step": round(other_ms, 4), "tokens_per_s": round(B / other_ms * 1e3, 2),
        "note": ("the same number of steps right after, called directly (hs_decode_step per step)" if not eager
                 else "the same number of steps right after, replayed from HIP graphs")}
    kv.close()
    for m in models:
        m.close()
    return out


def oracle_leg(cfg: dict, w: dict, n_steps: int) -> tuple:
    """The CPU oracle against the GPU on the same teacher-forced steps.

    Every request of the workload gets a synthetic cache of its context
    length (rows from the seeded generator) on the GPU; request 0 gets the
    same rows in the oracle.  Step k feeds every request a fixed seeded token.
    The GPU runs the workload's batch (its launch configuration); the oracle
    runs request 0 alone (decode rows are independent), single-threaded and
    pinned to one host core, and is timed: its per-step time, scaled by the
    batch, is the CPU baseline.  Parity: the largest relative error of
    request 0's logits (of its residual stream without an LM head) over the
    steps, and the near ties among its greedy choices."""
    import numpy as np
    import torch

    import paper_2603_12707_amd as hs
    from oracle import oracle as O
    from workload import synth
    B = cfg["batch"]
    has_head = cfg.get("lm_head", True)
    _, lens = context_lengths(cfg)
    caps = [n + n_steps + 1 for n in lens]
    model = hs.Model(cfg, w, max_batch=B, max_ctx=max(caps), packed=True)
    kv = hs.KVCache(model, [0] * B, caps)
    t = time.time()
    fill_synthetic(cfg, kv, lens)
    toks = [synth.decode_tokens(cfg, 1000 + k, B) for k in range(n_steps)]
    g_out = []
    tout = torch.empty(B, dtype=torch.int32, device="cuda")
    logits = torch.empty(B, cfg["vocab"], dtype=torch.float32, device="cuda") if has_head else None
    hidden = torch.empty(B, cfg["d_model"], dtype=torch.float32, device="cuda")
    for k in range(n_steps):
        kv.decode(toks[k].cuda(), tout if has_head else None, logits, hidden)
        torch.cuda.synchronize()
        g_out.append((logits[0].cpu().numpy() if has_head else hidden[0].cpu().numpy(), int(tout[0].item())))
    kv.close()
    model.close()
    # the oracle's row-major weights from the same generator (run on the GPU)
    w_cpu = {n: synth.make_weight(cfg, n, device="cuda").cpu() for n in synth.weight_names(cfg)}
    seq = O.Model(cfg, w_cpu).new_seq(caps[0])
    for layer in range(cfg["n_layers"]):
        for sel in (0, 1):
            for h in range(cfg["n_kv_heads"]):
                seq.write_kv(layer, sel, h, 0, synth.kv_block(cfg, 0, layer, sel, h, lens[0], device="cuda").float().cpu())
    seq.set_len(lens[0], lens[0])
    log(f"{cfg['name']}: GPU parity steps and oracle inputs ready in {time.time() - t:.1f} s")
    allowed = os.sched_getaffinity(0)
    core = min(allowed)
    os.sched_setaffinity(0, {core})  # timed on one host core
    try:
        outs = []
        t0 = time.perf_counter()
        for k in range(n_steps):
            outs.append(seq.decode(int(toks[k][0])))
        el = time.perf_counter() - t0
    finally:
        os.sched_setaffinity(0, allowed)
    del w_cpu
    worst, ties, mismatches = 0.0, 0, 0
    for (g, g_tok), (r_log, r_hid, r_tok) in zip(g_out, outs):
        ref = np.asarray(r_log if has_head else r_hid, np.float64)
        g = np.asarray(g, np.float64)
        delta = float(np.max(np.abs(g - ref)))
        worst = max(worst, delta / max(float(np.max(np.abs(ref))), 1e-30))
        if has_head and g_tok != r_tok:
            if float(ref[r_tok] - ref[g_tok]) <= 2 * delta:
                ties += 1
            else:
                mismatches += 1
    per_step = el / n_steps
    log(f"{cfg['name']}: oracle {n_steps} steps in {el:.1f} s; parity max rel err {worst:.3g}")
    sample = (f"{n_steps} teacher-forced decode steps of request 0 from a synthetic {lens[0]}-position cache, "
              f"single-threaded plain C oracle (fp64 dot products), pinned to one host core"
              + (f"; rate scaled by the batch of {B} (decode rows are independent)" if B > 1 else ""))
    base = {"value": B / per_step, "unit": "tokens/s", "cores": 1, "kind": "oracle", "sample": sample,
            "cpu_model": cpu_model(), "host_cpus_available": len(allowed), "pinned_core": core}
    parity = {"steps": n_steps, "request": 0, "batch": B, "bound": LOGIT_TOL,
              ("max_logit_rel_err" if has_head else "max_hidden_rel_err"): round(worst, 6),
              "near_ties": ties, "token_mismatches": mismatches,
              "ok": worst <= LOGIT_TOL and mismatches == 0}
    return base, parity


def run_workload(name: str, args, ws_cache: dict, stream_gbs: float, headline: bool) -> dict:
    import torch

    from workload import configs
    cfg = configs.get(name)
    model_key = json.dumps({k: v for k, v in cfg.items() if k not in ("name", "batch", "n_v", "s_text", "n_dec")},
                           sort_keys=True, default=str)
    if model_key not in ws_cache:
        ws_cache.clear()
        torch.cuda.empty_cache()
        ws_cache[model_key] = make_weights(cfg)
    ws = ws_cache[model_key]
    out = measure(cfg, ws, args.steps, args.warmup, eager=args.eager,
                  pool_block=args.kv_pool_block if headline else 0, stream_gbs=stream_gbs)
    other = out.get("eager") or out.get("graph")
    log(f"{name}: {out['ms_per_step']:.4f} ms/step ({out['timed_as']}; the other way {other['ms_per_step']:.4f}), "
        f"{out['value']:.1f} tokens/s, {out['hbm_frac']:.4f} of HBM peak")
    if not args.no_cpu_baseline:
        out["cpu_baseline"], out["parity"] = oracle_leg(cfg, ws[0], ORACLE_STEPS.get(name, 2))
    return out


# ---------------------------------------------------------------------------
# rocprofv3 summaries (the files under profiles/)
# ---------------------------------------------------------------------------

KERNEL_LEGEND = """Template arguments. `k_gemm<dtype, row tiles, column tiles, waves, k-blocks per group, prologue, LDS
staging, epilogue, packed SwiGLU output, packed activations>` (columns <= 32); `k_gemm_lds<dtype, epilogue, row tiles,
column tiles>` (LDS-staged, many columns); `k_gemm_ws<dtype, epilogue>` (weight-stationary: gate/up and the LM head at
129..256 columns); `k_gemm_tile<dtype, row tiles/wave, column tiles/wave, wave rows, wave columns, epilogue>`;
`k_attn<dtype, head_dim, group, waves, paged cache>` (scalar split attention), `k_attn_mma<...>` (GQA on the matrix
cores), `k_attn_prefill<...>` (causal prefill); `k_combine<dtype, head_dim, splits unrolled>`. dtype 1 = f16,
2 = bf16; prologue 0 = plain activations, 1 = RMSNorm, 2 = attention split combine; epilogue 0 = logits,
1 = residual, 2 = SwiGLU, 3 = q/k/v + RoPE + KV append, 5 = residual as two fp64 K-split partials. `k_splitk_sum`
adds the K-split partials of a residual GEMM; `k_rmsnorm<dtype, pending splits>` normalises rows into a workspace
when a GEMM has more columns than its prologue stages, after adding a deferred residual sum's partials."""


def _short(name: str) -> str:
    m = re.search(r"(k_\w+)(<[^>]*>)?", name)
    return (m.group(1) + (m.group(2) or "")) if m else name[:60]


def _csv_rows(d: str, suffix: str) -> list:
    path = d if d.endswith(".csv") else next(
        os.path.join(r, f) for r, _, fs in os.walk(d) for f in fs if f.endswith(suffix))
    with open(path) as f:
        return list(csv.DictReader(f))


def _steps_summary(trace: list) -> str:
    """Per-kernel durations inside the decode steps of a kernel trace (a step
    runs from one k_embed to the next and ends in k_argmax / k_advance)."""
    rows = sorted((r for r in trace if "hs::" in r["Kernel_Name"]), key=lambda r: int(r["Start_Timestamp"]))
    steps, cur = [], None
    for r in rows:
        k = _short(r["Kernel_Name"]).replace(" ", "")
        if k.startswith("k_embed"):
            if cur:
                steps.append(cur)
            cur = []
        if cur is not None:
            cur.append((k, int(r["Start_Timestamp"]), int(r["End_Timestamp"])))
    if cur:
        steps.append(cur)
    full = [s for s in steps if any(k.startswith(("k_argmax", "k_advance")) for k, _, _ in s)]
    inner = full[2:-2] if len(full) > 6 else full
    if not inner:
        return "no complete decode step in the trace"
    dur, gaps, spans = {}, [], []
    for s in inner:
        spans.append(s[-1][2] - s[0][1])
        for i, (k, a, b) in enumerate(s):
            dur.setdefault(k, []).append(b - a)
            if i:
                gaps.append(a - s[i - 1][2])
    lines = [f"steps {len(inner)} (of {len(full)})  step span median {statistics.median(spans) / 1e3:.1f} us"]
    tot = 0.0
    for k, v in sorted(dur.items(), key=lambda kv: -sum(kv[1])):
        per = sum(v) / len(inner)
        tot += per
        lines.append(f"{k:48s} n/step {len(v) / len(inner):5.1f}  avg {statistics.mean(v) / 1e3:8.2f} us  "
                     f"per step {per / 1e3:8.1f} us")
    lines.append(f"kernel time per step {tot / 1e3:.1f} us; gaps between launches: median "
                 f"{statistics.median(gaps) / 1e3 if gaps else 0:.2f} us")
    return "\n".join(lines)


def summarise_stats(trace_dir: str, bench_log: str, workload: str, command: str) -> str:
    """profiles/decode_<workload>_kernel_stats.md from a `rocprofv3 --kernel-trace
    --stats --output-format csv` run of bench.py and that run's output."""
    stats = [r for r in _csv_rows(trace_dir, "kernel_stats.csv") if "hs::" in r["Name"]]
    trace = _csv_rows(trace_dir, "kernel_trace.csv")
    line = [ln for ln in open(bench_log) if ln.startswith("{")][-1]
    j = json.loads(line)
    res = j if j.get("config", {}).get("workload") == workload else j.get("workloads", {}).get(workload, j)
    tab = "\n".join(f"| `{_short(r['Name'])}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                    f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} |" for r in stats)
    rl = res["roofline"]
    md = f"""# Decode, `{workload}` — rocprofv3 kernel statistics

Command (GPU box, repository root), then `python bench.py --summarise-stats` on its output:

```
{command}
```

From the run's kernel statistics, libhs kernels only (torch's input-generation kernels omitted). Calls include the
prefill (or the synthetic KV fill), the warm-up and timed decode steps, bench.py's kernel replays and (without
--no-cpu-baseline) its parity steps.

{KERNEL_LEGEND}

| Kernel | Calls | Avg µs | Min µs | Max µs |
|---|---|---|---|---|
{tab}

Inside the decode steps (from the kernel trace's start/end stamps):

```
{_steps_summary(trace)}
```

bench.py measured the dominant kernel ({rl.get('kernel')}) with HIP events at {rl['avg_launch_us']} µs per launch.
This workload's result from the same run (under the profiler):

```
{json.dumps({k: res.get(k) for k in ("value", "unit", "ms_per_step", "hbm_gbps", "hbm_frac", "roofline", "kernel_us")})}
```
"""
    path = os.path.join(ROOT, "profiles", f"decode_{workload}_kernel_stats.md")
    with open(path, "w") as f:
        f.write(md)
    return path


def summarise_counters(fetch_dir: str, write_dir: str, workload: str, kind: str, kernel: str, command: str) -> str:
    """profiles/<kind>_<workload>_counters.md from two `rocprofv3 --pmc` runs of
    bench.py (FETCH_SIZE, then WRITE_SIZE) that also copy 1 GiB device to
    device: each counter is scaled by what it reads for that copy."""
    from workload import configs
    cfg = configs.get(workload)

    def per(d, counter):
        rs = [r for r in _csv_rows(d, "counter_collection.csv") if r["Counter_Name"] == counter]
        copy = [float(r["Counter_Value"]) for r in rs if "copyBuffer" in r["Kernel_Name"]]
        ours = [float(r["Counter_Value"]) for r in rs if kernel.replace(" ", "") in r["Kernel_Name"].replace(" ", "")]
        return max(copy), ours
    if kind == "attn":
        _, lens = context_lengths(cfg)
        alg = attn_bytes(cfg, [n + DEFAULT_WARMUP for n in lens])
        alg_note = "K/V rows 0..len of every request at the context of the first replay, q and output rows"
    else:
        alg = weight_bytes(cfg)[kind]
        alg_note = "every weight byte (and gain / bias) once"
    cf, fk = per(fetch_dir, "FETCH_SIZE")
    cw, wk = per(write_dir, "WRITE_SIZE")
    ff, fw = 1048576.0 / cf, 1048576.0 / cw
    # a kernel that serves two projections (the residual GEMM: O and down) is
    # told apart by what it fetches: the dispatches within 0.5x..3x of this
    # kind's algorithmic bytes, and the same dispatches of the WRITE_SIZE run
    # (the two runs launch the same sequence)
    pick = [i for i, v in enumerate(fk) if 0.5 <= v * 1024 * ff / alg <= 3.0] or list(range(len(fk)))
    fk = [fk[i] for i in pick]
    wk = [wk[i] for i in pick if i < len(wk)]
    mf, mw = statistics.median(fk), statistics.median(wk)
    traffic = mf * 1024 * ff + mw * 1024 * fw
    md = f"""# {KIND_NAMES[kind]}, `{workload}` — HBM traffic counters

kernel: `{kernel}`
kernel_source_sha256: {kernel_source_hash(kind)}

Commands (GPU box, repository root), one counter per run, then `python bench.py --summarise-counters` on their
output:

```
{command}
```

Calibration: the same runs copy 1 GiB device to device (`--copy-calibration-mib 1024`: one copy dispatch reading
1,048,576 KiB and writing 1,048,576 KiB); each counter is scaled by known / counted for that copy.

| Counter | 1 GiB copy (KiB) | factor = known / counted | kernel per dispatch (KiB, median of {len(fk)}) | scaled bytes |
|---|---|---|---|---|
| FETCH_SIZE | {cf:.2f} | {ff:.5f} | {mf:.1f} | {mf * 1024 * ff:.0f} |
| WRITE_SIZE | {cw:.1f} | {fw:.5f} | {mw:.1f} | {mw * 1024 * fw:.0f} |

traffic_bytes_per_launch: {traffic:.0f}
algorithmic_bytes_per_launch: {alg} ({alg_note})
ratio traffic / algorithmic: {traffic / alg:.4f}
"""
    path = os.path.join(ROOT, "profiles", f"{kind}_{workload}_counters.md")
    with open(path, "w") as f:
        f.write(md)
    return path


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=DEFAULT_STEPS)
    ap.add_argument("--warmup", type=int, default=DEFAULT_WARMUP)
    ap.add_argument("--workload", default=HEADLINE, help="the workload of the headline line")
    ap.add_argument("--no-workloads", action="store_true",
                    help="measure the headline workload only (default: also " + ", ".join(WORKLOADS) + ")")
    ap.add_argument("--no-cpu-baseline", action="store_true", help="skip the oracle leg (CPU baseline and parity)")
    ap.add_argument("--eager", action="store_true",
                    help="time direct hs_decode_step calls (default: the steps replayed from HIP graphs; the other "
                         "way is timed beside)")
    ap.add_argument("--kv-pool-block", type=int, default=0,
                    help="headline decode from a block-granular KV pool with blocks of this many positions")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="also run a plain device copy of this many MiB (counter calibration)")
    ap.add_argument("--summarise-stats", nargs=4, metavar=("TRACE_DIR", "BENCH_LOG", "WORKLOAD", "COMMAND"))
    ap.add_argument("--summarise-counters", nargs=6,
                    metavar=("FETCH_DIR", "WRITE_DIR", "WORKLOAD", "KIND", "KERNEL", "COMMAND"))
    args = ap.parse_args()
    if args.summarise_stats:
        print(summarise_stats(*args.summarise_stats))
        return 0
    if args.summarise_counters:
        print(summarise_counters(*args.summarise_counters))
        return 0
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one MI355X: the library has no multi-GPU path (the decode step would be "
              "sharded by request across GPUs with no exchange). Run with --gpus 1.",
              file=sys.stderr)
        return 2

    import torch
    torch.cuda.set_device(0)
    stream_gbs = stream_read_rate()
    log(f"streaming read: {stream_gbs:.0f} GB/s")
    ws_cache: dict = {}
    head = run_workload(args.workload, args, ws_cache, stream_gbs, headline=True)
    extra = {}
    if not args.no_workloads:
        for name in WORKLOADS:
            if name != args.workload:
                extra[name] = run_workload(name, args, ws_cache, stream_gbs, headline=False)
    ws_cache.clear()
    if args.copy_calibration_mib:
        src = torch.empty(args.copy_calibration_mib << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copy calibration: {args.copy_calibration_mib} MiB")

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
        "dtype": head["dtype"],
        "data": "synthetic (seeded: N(0,0.02) weights, N(0,1) vision rows, uniform text ids; generated in HBM)",
    }
    out.update({k: v for k, v in head.items() if k not in out and k not in ("steps", "warmup")})
    if extra:
        out["workloads"] = extra
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
