"""Parity of the wide prefill paths with the oracle, through outputs that
depend on the whole of layer 0.

Two 2-layer models (d = 1024, d_h = 128, F = 2048; fp16 MHA with 1-D RoPE, and
bf16 GQA-7 with 3-section M-RoPE and q/k/v bias) are prefilled
  * one request of 640 rows alone: causal matrix-core prefill attention at 640
    rows, the 8 x 8-tile LDS GEMM for gate/up, K splits for q/k/v, O and down;
  * two requests of 1024 rows packed into one 2048-row pass: the 16 x 8-tile
    LDS GEMM for q/k/v and gate/up, the unsplit 8 x 8-tile one for O and down;
  * four such requests packed into one 4096-row pass: the 16 x 16-tile LDS GEMM
    for q/k/v and gate/up, the 16 x 8-tile one for O and down.
(The tile choice follows the work-group counts of the GEMM launcher's rule at
these shapes.)  Each request's first token and last-row logits, and its
layer-1 K/V rows at sampled positions, are compared with the oracle's values
in tests/golden/prefill_wide.json, written by make_prefill_golden.py from the
oracle alone.  Layer-1 rows are projections of the residual stream after
layer 0, which holds every layer-0 kernel's output.
"""
from __future__ import annotations

import json
import os

import numpy as np
import pytest
import torch

from helpers import LOGIT_TOL, rel_err, to_device, token_ok
from workload import synth

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "prefill_wide.json")
TDT = {"f16": torch.float16, "bf16": torch.bfloat16}
PHASES = {"single_640": [0], "packed_2048": [1, 2], "packed_4096": [1, 2, 3, 4]}


def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


@pytest.mark.parametrize("phase", list(PHASES))
@pytest.mark.parametrize("model", ["mha_f16", "gqa7_bf16"])
def test_wide_prefill_matches_oracle(model, phase):
    import paper_2603_12707_amd as hs
    gold = _golden()
    spec = gold["models"][model]
    cfg = dict(spec["config"])
    cfg["mrope_section"] = tuple(cfg["mrope_section"])
    reqs = PHASES[phase]
    shapes = [(r["n_v"], r["s_text"]) for r in gold["requests"]]
    caps = [n + s for n, s in shapes]
    gpu = hs.Model(cfg, to_device(synth.make_weights(cfg)), max_batch=len(shapes), max_ctx=max(caps))
    kv = hs.KVCache(gpu, [n for n, _ in shapes], caps)
    V = cfg["vocab"]
    inputs = []
    for r in reqs:
        n_v, s_text = shapes[r]
        inputs.append((synth.vision_rows(cfg, r, n_v), synth.text_ids(cfg, r, s_text),
                       synth.mrope_positions(n_v, s_text) if cfg["rope_kind"] == 1 else None))
    logits = torch.empty(len(reqs), V, dtype=torch.float32, device="cuda")
    if len(reqs) == 1:
        emb, ids, pos = inputs[0]
        toks = kv.prefill(reqs[0], emb.cuda(), ids.cuda(), None if pos is None else pos.cuda(), last_logits=logits[0])
    else:
        rows = sum(caps[r] for r in reqs)
        gpu.reserve_rows(rows)
        emb = torch.cat([e for e, _, _ in inputs]).cuda()
        ids = torch.cat([i for _, i, _ in inputs]).cuda()
        pos = torch.cat([p for _, _, p in inputs], dim=1).contiguous().cuda() if cfg["rope_kind"] == 1 else None
        toks = kv.prefill_batch(reqs, emb, ids, [shapes[r][1] for r in reqs], pos, last_logits=logits)
    torch.cuda.synchronize()
    toks = toks.cpu().tolist()
    logits = logits.cpu().numpy()
    lens = kv.lengths()
    near = 0
    for k, r in enumerate(reqs):
        ref = spec["requests"][r]
        assert lens[r] == caps[r]
        ref_logits = np.asarray(ref["last_logits"], np.float64)
        err = rel_err(logits[k], ref_logits)
        assert err <= LOGIT_TOL, (r, err)
        ok, tie = token_ok(toks[k], logits[k], ref_logits)
        assert ok, (r, toks[k], ref["first_token"])
        near += tie
        for key, want in ref["layer1_rows"].items():
            p, h, sel = (int(v) for v in key.split("."))
            g = torch.empty(1, cfg["head_dim"], dtype=TDT[cfg["dtype"]], device="cuda")
            kv.read(r, 1, sel, h, p, 1, g)
            err = rel_err(g.float().cpu().numpy(), want)
            assert err <= LOGIT_TOL, (r, key, err)
    assert near == 0
    assert gpu.status() == 0
    kv.close()
    gpu.close()
