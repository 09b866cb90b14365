"""Shared test helpers: build the GPU model and the oracle from the same seeded
CPU inputs, and compare their outputs under the parity rules.

Parity rules (tolerance 2e-2 max-abs relative on logits, greedy ids exact):
  * logits: max_j |gpu_j - ref_j| / max_j |ref_j| <= 2e-2 per (step, request);
  * tokens: equal to the oracle's argmax, except that when the oracle's top-1
    margin over the GPU's token is within 2 * max_j |gpu_j - ref_j| the step
    is a near tie (several results are correct) and is counted, not failed.
"""
from __future__ import annotations

import numpy as np
import torch

from oracle import oracle as O
from workload import synth

LOGIT_TOL = 2e-2
# Appended K/V rows (not logits).  At layer 0 a row depends on its input row
# alone and the two sides round it identically up to one storage rounding:
# each row against its own maximum.  A deeper layer's rows are rounded
# projections of the residual stream, which carries the depth-accumulated
# error that LOGIT_TOL bounds on the logits: the K (or V) rows of all KV heads
# of the position are compared as one vector, with the logits' statistic and
# bound (max-abs error against the vector's maximum).
KV_ROW0_TOL = 2.0 ** -8
KV_ROWS_DEEP_TOL = LOGIT_TOL


def small_cfg(**kw) -> dict:
    base = dict(name="small", n_layers=2, d_model=384, n_heads=6, n_kv_heads=6, head_dim=64, ffn_dim=1000,
                vocab=997, rope_theta=1e4, rms_eps=1e-5, rope_kind=0, mrope_section=(0, 0, 0), qkv_bias=0,
                dtype="f16", lm_head=True, seed=3)
    base.update(kw)
    return base


def to_device(w: dict) -> dict:
    return {k: v.to("cuda") for k, v in w.items()}


def rel_err(gpu, ref) -> float:
    gpu, ref = np.asarray(gpu, np.float64), np.asarray(ref, np.float64)
    return float(np.max(np.abs(gpu - ref)) / max(np.max(np.abs(ref)), 1e-30))


def token_ok(gpu_tok: int, gpu_logits, ref_logits) -> tuple:
    """(ok, near_tie) for one greedy choice."""
    ref = np.asarray(ref_logits, np.float64)
    want = int(np.argmax(ref))
    if gpu_tok == want:
        return True, False
    delta = float(np.max(np.abs(np.asarray(gpu_logits, np.float64) - ref)))
    margin = float(ref[want] - ref[gpu_tok])
    return margin <= 2 * delta, True


class Pair:
    """The same seeded model on the GPU (libhs) and in the oracle."""

    def __init__(self, cfg: dict, max_batch: int, max_ctx: int, weights_cpu: dict | None = None):
        import paper_2603_12707_amd as hs
        self.cfg = cfg
        self.w_cpu = weights_cpu if weights_cpu is not None else synth.make_weights(cfg)
        self.w_gpu = to_device(self.w_cpu)
        self.gpu = hs.Model(cfg, self.w_gpu, max_batch, max_ctx)
        self.ora = O.Model(cfg, self.w_cpu)

    def request_inputs(self, req: int, n_v: int, s_text: int):
        emb = synth.vision_rows(self.cfg, req, n_v)
        ids = synth.text_ids(self.cfg, req, s_text)
        pos = synth.mrope_positions(n_v, s_text) if self.cfg["rope_kind"] == 1 else None
        return emb, ids, pos
