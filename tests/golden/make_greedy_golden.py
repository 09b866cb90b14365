"""Writes the oracle's free-running greedy decode of one workload request to a
JSON fixture under tests/golden/.

The fixture holds, for the first request of the workload: the context
lengths, the first token (from the prefill's last row), and for every decode
step the greedy token, the oracle's top-1 / top-2 logits (the margin a GPU
logit error must stay under for the choice to be unambiguous), the largest
|logit| (the denominator of the relative logit error), the 8 largest logits
with their indices, and the logits at a fixed seeded sample of vocabulary
indices.  The GPU parity test replays the same request free-running and
compares token for token.

It calls only the oracle and the seeded input generator: no value comes from
the HIP library.  Single-threaded and slow (the oracle runs every context
row through every layer): at the LLaVA-shaped batch-1 size about an hour.

    python tests/golden/make_greedy_golden.py llava7b_b1 [n_dec]
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
from workload import configs, synth  # noqa: E402

N_SAMPLE = 48
N_TOP = 8


def sample_indices(cfg: dict) -> list:
    """Fixed vocabulary indices at which every step's logits are stored."""
    return sorted(set(synth.uniform_int(cfg["seed"], "golden.logit_sample", N_SAMPLE, 0, cfg["vocab"] - 1).tolist()))


def step_record(logits: np.ndarray, token: int, sample: list) -> dict:
    lg = np.asarray(logits, np.float64)
    order = np.argsort(-lg, kind="stable")[:N_TOP]
    return {
        "token": int(token),
        "top1": float(lg[order[0]]),
        "top2": float(lg[order[1]]),
        "max_abs": float(np.max(np.abs(lg))),
        "top": [[int(i), float(lg[i])] for i in order],
        "sample": [float(lg[i]) for i in sample],
    }


def main(name: str, n_dec: int | None = None) -> str:
    cfg = configs.get(name)
    n_dec = cfg["n_dec"] if n_dec is None else n_dec
    n_v, s_text = synth.request_lengths(cfg)
    n_v, s_text = n_v[0], s_text[0]
    t0 = time.time()
    weights = synth.make_weights(cfg)
    print(f"[golden] {name}: weights generated in {time.time() - t0:.0f} s", flush=True)
    emb = synth.vision_rows(cfg, 0, n_v)
    ids = synth.text_ids(cfg, 0, s_text)
    pos = synth.mrope_positions(n_v, s_text) if cfg["rope_kind"] == 1 else None
    seq = O.Model(cfg, weights).new_seq(n_v + s_text + n_dec)
    sample = sample_indices(cfg)
    t0 = time.time()
    logits, tok = seq.prefill(emb, ids, pos)
    print(f"[golden] prefill of {n_v + s_text} rows in {time.time() - t0:.0f} s, first token {tok}", flush=True)
    steps = [step_record(logits, tok, sample)]
    for k in range(n_dec):
        t1 = time.time()
        logits, _, tok = seq.decode(tok)
        steps.append(step_record(logits, tok, sample))
        print(f"[golden] step {k + 1}/{n_dec}: token {tok} margin {steps[-1]['top1'] - steps[-1]['top2']:.4g} "
              f"({time.time() - t1:.1f} s)", flush=True)
    margins = [s["top1"] - s["top2"] for s in steps]
    out = {
        "what": "oracle free-running greedy decode of request 0 (prefill from its vision rows and text ids, "
                "then n_dec steps each fed the previous greedy token); step 0 is the prefill's last row",
        "workload": name,
        "seed": cfg["seed"],
        "n_v": n_v,
        "s_text": s_text,
        "n_dec": n_dec,
        "sample_indices": sample,
        "min_margin": float(min(margins)),
        "steps": steps,
    }
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), f"greedy_{name}.json")
    tmp = path + ".tmp"
    with open(tmp, "w") as f:
        json.dump(out, f, separators=(",", ":"))
    os.replace(tmp, path)
    print(f"[golden] wrote {path}; min top-1 margin {min(margins):.4g}", flush=True)
    return path


if __name__ == "__main__":
    main(sys.argv[1], int(sys.argv[2]) if len(sys.argv) > 2 else None)
