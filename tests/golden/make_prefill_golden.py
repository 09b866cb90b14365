"""Writes the oracle's prefill outputs for the wide-prefill parity test to
tests/golden/prefill_wide.json.

Two 2-layer models (d = 1024, d_h = 128, F = 2048, V = 512): an fp16 MHA model
with 1-D RoPE and a bf16 GQA-7 model (14 query / 2 KV heads) with 3-section
M-RoPE and q/k/v bias.  Each gets one request of 576 vision rows + 64 text
tokens (640 rows, prefilled alone) and four requests of 960 vision rows + 64
text tokens (1024 rows each, prefilled packed: two of them in 2048 rows, all
four in 4096).  For every request the fixture holds the first greedy token,
the prefill's last-row logits, and layer-1 K and V rows of the first and the
last KV head at sampled positions.  Layer-1 rows are computed from the whole
of layer 0 (its attention over all earlier rows, its O, gate/up and down
projections), so they check every layer-0 kernel the prefill ran.

It calls only the oracle and the seeded input generator.  Single-threaded;
a few minutes.

    python tests/golden/make_prefill_golden.py
"""
from __future__ import annotations

import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from oracle import oracle as O  # noqa: E402
from workload import synth  # noqa: E402

MODELS = {
    "mha_f16": dict(name="wide_mha_f16", n_layers=2, d_model=1024, n_heads=8, n_kv_heads=8, head_dim=128,
                    ffn_dim=2048, vocab=512, rope_theta=1e4, rms_eps=1e-5, rope_kind=0, mrope_section=(0, 0, 0),
                    qkv_bias=0, dtype="f16", lm_head=True, seed=5),
    "gqa7_bf16": dict(name="wide_gqa7_bf16", n_layers=2, d_model=1024, n_heads=14, n_kv_heads=2, head_dim=128,
                      ffn_dim=2048, vocab=512, rope_theta=1e6, rms_eps=1e-6, rope_kind=1, mrope_section=(16, 24, 24),
                      qkv_bias=1, dtype="bf16", lm_head=True, seed=6),
}
# request 0: 640 rows alone; requests 1..4: 1024 rows each, packed
REQUESTS = [(576, 64), (960, 64), (960, 64), (960, 64), (960, 64)]


def sample_positions(n_v: int, s_text: int) -> list:
    T = n_v + s_text
    return sorted({1, T // 3, n_v, T - 1})


def f32s(a) -> list:
    """Values to 6 significant digits (the parity bound is 2e-2)."""
    return [float(f"{v:.6g}") for v in np.asarray(a, np.float32).ravel()]


def main() -> str:
    out = {"what": "oracle prefill of each request: first token, last-row logits, layer-1 K/V rows of KV heads "
                   "0 and n_kv-1 at sampled positions",
           "requests": [{"n_v": n, "s_text": s} for n, s in REQUESTS], "models": {}}
    for key, cfg in MODELS.items():
        W = synth.make_weights(cfg)
        om = O.Model(cfg, W)
        reqs = []
        for r, (n_v, s_text) in enumerate(REQUESTS):
            t0 = time.time()
            emb = synth.vision_rows(cfg, r, n_v)
            ids = synth.text_ids(cfg, r, s_text)
            pos = synth.mrope_positions(n_v, s_text) if cfg["rope_kind"] == 1 else None
            seq = om.new_seq(n_v + s_text)
            logits, tok = seq.prefill(emb, ids, pos)
            lg = np.asarray(logits, np.float64)
            order = np.argsort(-lg, kind="stable")
            rows = {}
            for p in sample_positions(n_v, s_text):
                for h in sorted({0, cfg["n_kv_heads"] - 1}):
                    for sel in (0, 1):
                        rows[f"{p}.{h}.{sel}"] = f32s(seq.read_kv(1, sel, h, p, 1))
            reqs.append({"first_token": int(tok), "margin": float(lg[order[0]] - lg[order[1]]),
                         "last_logits": f32s(logits), "layer1_rows": rows})
            print(f"[golden] {key} request {r}: {n_v + s_text} rows in {time.time() - t0:.0f} s, token {tok}",
                  flush=True)
        out["models"][key] = {"config": {k: (list(v) if isinstance(v, tuple) else v) for k, v in cfg.items()},
                              "requests": reqs}
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "prefill_wide.json")
    with open(path + ".tmp", "w") as f:
        json.dump(out, f, separators=(",", ":"))
    os.replace(path + ".tmp", path)
    print(f"[golden] wrote {path}", flush=True)
    return path


if __name__ == "__main__":
    main()
