#!/usr/bin/env python3
"""Decode-step throughput of the language-decode hot path on one MI355X.

A step is one hs_decode_step call: embedding gather, every decoder layer
(RMSNorm + q/k/v + RoPE + KV append, split-K attention and combine, output
projection, RMSNorm + gate/up + SwiGLU, down projection) and the final norm,
LM head and greedy selection, for every request of the batch.  Inputs are
seeded synthetic tensors generated directly in HBM; the KV cache is filled by
hs_prefill_embeddings from the vision rows and text tokens before timing.

Prints one JSON line on stdout; progress goes to stderr.
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

PEAK_HBM_GBS = 8000.0  # MI355X HBM3E
WEIGHT_COPIES = 4  # one-layer workloads: weight sets rotated over the steps (4 x 0.47 GB > 256 MB Infinity Cache)
METRIC = "decode tokens/s at batch B + achieved HBM GB/s vs peak, 7B-shaped fp16"


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


def setup(cfg: dict, n_steps_total: int, pool_block: int = 0):
    import torch

    import paper_2603_12707_amd as hs
    from workload import synth
    B = cfg["batch"]
    t = time.time()
    # a one-layer workload rotates copies of its weights, so that the 256 MB
    # Infinity Cache cannot serve one step's weights to the next
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
    log(f"weights generated and packed in HBM: {copies} x "
        f"{sum(v.numel() * v.element_size() for v in ws[0].values()) / 1e9:.2f} GB in {time.time() - t:.1f} s")
    if "kv_len" in cfg:  # layer stack fed from a synthetic cache
        lens = synth.kv_lengths(cfg)
        n_v = [0] * B
    else:
        n_v, s_text = synth.request_lengths(cfg)
        lens = [a + b for a, b in zip(n_v, s_text)]
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
    if "kv_len" in cfg:
        for r in range(B):
            kv.set_length(r, lens[r], lens[r])  # a pool takes the blocks here
            for layer in range(cfg["n_layers"]):
                for sel in (0, 1):
                    for h in range(cfg["n_kv_heads"]):
                        kv.write(r, layer, sel, h, 0, synth.kv_block(cfg, r, layer, sel, h, lens[r], device="cuda"))
        first.copy_(synth.decode_tokens(cfg, 0, B, device="cuda"))
    else:
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
    log(f"context ready for {B} request(s) in {ready_s * 1e3:.1f} ms (lengths {min(lens)}..{max(lens)})")
    setup.prefill_ms = None if "kv_len" in cfg else ready_s * 1e3 / B
    return ws, models, kv, first, lens


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg: dict, ctx: int, n_tokens: int = 2) -> dict:
    """The oracle, single-threaded on one host core, decoding n_tokens for one
    request of the workload from a synthetic cache of ctx positions.  Its
    row-major weights come from the same seeded generator (run on the GPU for
    speed; the generator is bit-identical on CPU and GPU)."""
    from oracle import oracle as O
    from workload import synth
    t = time.time()
    w_cpu = {n: synth.make_weight(cfg, n, device="cuda").cpu() for n in synth.weight_names(cfg)}
    model = O.Model(cfg, w_cpu)
    seq = model.new_seq(ctx + n_tokens)
    for layer in range(cfg["n_layers"]):
        for sel in (0, 1):
            for h in range(cfg["n_kv_heads"]):
                seq.write_kv(layer, sel, h, 0, synth.kv_block(cfg, 0, layer, sel, h, ctx, device="cuda").float().cpu())
    seq.set_len(ctx, ctx)
    log(f"oracle inputs ready in {time.time() - t:.1f} s")
    tok = int(synth.decode_tokens(cfg, 0, 1)[0])
    # timed on one host core (the process is pinned to it meanwhile)
    allowed = os.sched_getaffinity(0)
    core = min(allowed)
    os.sched_setaffinity(0, {core})
    try:
        t = time.perf_counter()
        for _ in range(n_tokens):
            _, _, nxt = seq.decode(tok)
            tok = nxt if cfg.get("lm_head", True) else tok
        el = time.perf_counter() - t
    finally:
        os.sched_setaffinity(0, allowed)
    log(f"oracle: {n_tokens} tokens in {el:.1f} s")
    del w_cpu
    return {"value": n_tokens / el, "unit": "tokens/s", "cores": 1, "kind": "oracle",
            "sample": f"{n_tokens} greedy decode steps of one request of the workload from a synthetic "
                      f"{ctx}-position KV cache, single-threaded plain C oracle (fp64 accumulation), pinned to one "
                      f"host core",
            "cpu_model": cpu_model(), "host_cpus_available": len(allowed), "pinned_core": core}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=DEFAULT_STEPS)
    ap.add_argument("--warmup", type=int, default=DEFAULT_WARMUP)
    ap.add_argument("--workload", default="llava7b_b1")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--graph", action="store_true",
                    help="also time the decode step replayed from a HIP graph (stream capture)")
    ap.add_argument("--kv-pool-block", type=int, default=0,
                    help="decode from a block-granular KV pool with blocks of this many positions (0: contiguous)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="also run a plain device copy of this many MiB (counter calibration)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one MI355X: the library has no multi-GPU path (the decode step would be "
              "sharded by request across GPUs with no exchange). Run with --gpus 1.",
              file=sys.stderr)
        return 2

    import torch

    import paper_2603_12707_amd as hs
    from workload import configs
    cfg = configs.get(args.workload)
    B = cfg["batch"]
    torch.cuda.set_device(0)
    copies = WEIGHT_COPIES if "kv_len" in cfg else 1
    per_graph = max(2, copies)  # decode steps captured in one graph: the token ping-pong and the weight rotation
    graph_steps = per_graph * (max(1, args.steps // 4) + 1) if args.graph else 0
    ws, models, kv, first, lens0 = setup(cfg, steps_after_context(args.warmup, args.steps) + graph_steps,
                                       args.kv_pool_block)

    tin = first.clone()
    tout = torch.empty_like(tin)
    has_head = cfg.get("lm_head", True)

    n_step = 0

    def step():
        nonlocal tin, tout, n_step
        kv.decode(tin, tout if has_head else None, model=models[n_step % len(models)])
        n_step += 1
        if has_head:
            tin, tout = tout, tin

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # timed region: K steps bracketed by device synchronisation
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    lens_after = kv.lengths()

    graph_ms = None
    if args.graph:
        # per_graph steps per graph (token buffers ping-pong, weight sets
        # rotate), graphs replayed back to back
        ga, gb = tin.clone(), torch.empty_like(tin)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for k in range(per_graph):
                a, b = (ga, gb) if k % 2 == 0 else (gb, ga)
                kv.decode(a, b if has_head else None, model=models[k % len(models)])
        kv.sync()
        reps_g = max(1, args.steps // 4)
        graph.replay()  # warm
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(reps_g):
            graph.replay()
        torch.cuda.synchronize()
        graph_ms = (time.perf_counter() - t0) / (per_graph * reps_g) * 1e3
        kv.sync()
        lens_after = [n - per_graph * (reps_g + 1) for n in kv.lengths()]

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

    # the plain streaming-read rate of this GPU (the same loads as the weight
    # stream), for reading roofline.frac against what HBM delivers
    sr_buf = torch.empty(STREAM_READ_BYTES, dtype=torch.uint8, device="cuda")
    sr_sink = torch.empty(max(STREAM_READ_BLOCKS), dtype=torch.int32, device="cuda")
    stream_read_gbs = 0.0
    for blocks in STREAM_READ_BLOCKS:  # the best grid
        hs.stream_read(sr_buf, sr_sink, blocks)  # warm
        ev0.record()
        for _ in range(5):
            hs.stream_read(sr_buf, sr_sink, blocks)
        ev1.record()
        torch.cuda.synchronize()
        stream_read_gbs = max(stream_read_gbs, 5 * STREAM_READ_BYTES / (ev0.elapsed_time(ev1) / 1e3) / 1e9)
    del sr_buf, sr_sink

    if args.copy_calibration_mib:
        src = torch.empty(args.copy_calibration_mib << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copy calibration: {args.copy_calibration_mib} MiB")

    ms_per_step = elapsed / args.steps * 1e3
    tok_s = B * args.steps / elapsed
    lens_start = [n + args.warmup for n in lens0]
    total_bytes = sum(step_bytes(cfg, [n + k for n in lens_start]) for k in range(args.steps))
    gbs = total_bytes / elapsed / 1e9
    assert lens_after == [n + args.steps for n in lens_start], (lens_after[:4], lens_start[:4])

    dom_bytes = attn_bytes(cfg, lens_replay) if dominant == "attn" else weight_bytes(cfg)[dominant]
    achieved = dom_bytes / dom_avg_s / 1e9
    traffic = stored_traffic(args.workload, dominant)
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": traffic,
                "kernel": KIND_NAMES[dominant], "kind": dominant,
                "bytes_per_launch": dom_bytes, "avg_launch_us": round(dom_avg_s * 1e6, 2), "launches": reps,
                "stream_read_gbps": round(stream_read_gbs, 1), "frac_of_stream_read": round(achieved / stream_read_gbs, 4)}
    kernels = {k: round(v, 2) for k, v in breakdown.items()}

    out = {
        "metric": METRIC,
        "value": round(tok_s, 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg["dtype"],
        "data": "synthetic (seeded: N(0,0.02) weights, N(0,1) vision rows, uniform text ids; generated in HBM)",
        "config": {"workload": args.workload, "batch": B, "context_at_start": lens_start[0] if B == 1 else
                   [min(lens_start), max(lens_start)], "n_layers": cfg["n_layers"], "d_model": cfg["d_model"],
                   "n_heads": cfg["n_heads"], "n_kv_heads": cfg["n_kv_heads"], "ffn_dim": cfg["ffn_dim"],
                   "vocab": cfg["vocab"] if has_head else None, "parallelism": "none (one GPU)",
                   "kv_cache": f"pool of {args.kv_pool_block}-position blocks" if args.kv_pool_block else "contiguous",
                   "weight_copies": copies},
        "hbm_gbps": round(gbs, 1),
        "hbm_frac": round(gbs / PEAK_HBM_GBS, 4),
        "bytes_per_step": total_bytes // args.steps,
        "roofline": roofline,
        "kernel_us": kernels,
    }
    if getattr(setup, "prefill_ms", None) is not None:
        out["prefill_ms_per_request"] = round(setup.prefill_ms, 2)
    if graph_ms is not None:
        out["graph"] = {"ms_per_step": round(graph_ms, 4), "tokens_per_s": round(B / graph_ms * 1e3, 2),
                        "note": "the same step replayed from a HIP graph (stream capture)"}
    if not args.no_cpu_baseline:
        del ws, models
        out["cpu_baseline"] = cpu_baseline(cfg, lens_start[0])
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
