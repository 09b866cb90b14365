"""Greedy decode against the oracle's free-running run, token for token.

The oracle's run of request 0 of a workload (prefill from its vision rows and
text ids, then n_dec greedy steps each fed the previous token) is stored in
tests/golden/greedy_<workload>.json by make_greedy_golden.py, which calls
only the oracle and the input generator.  Here the GPU prefills the same
request for real and decodes it in the launch configuration bench.py uses
(the same capacity, so the same attention splits), each step fed the
oracle's previous token -- which is the GPU's own wherever the two agree, so
the run is free-running up to the first disagreement.  At every step the
logits are compared at the oracle's 8 largest and at a fixed sample of
vocabulary indices, relative to the oracle's largest |logit|, against the
2e-2 bound; and the GPU's token must be the oracle's, or else a near tie:
among the oracle's 8 largest, with an oracle margin no more than twice the
GPU's largest logit error on that step (several results correct).  Near ties
are counted and reported with the smallest margin-to-error ratio.  The
batched workloads' stored runs (request 0 alone in the oracle) are replayed
with request 0 decoding among the whole batch, every request prefilled from
its real inputs in packed passes, as bench.py runs them.
"""
from __future__ import annotations

import json
import os

import pytest
import torch

import bench
from helpers import LOGIT_TOL
from workload import configs, synth

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _gpu_model(cfg, cap):
    import paper_2603_12707_amd as hs
    w = {}
    for name in synth.weight_names(cfg):  # generated on the GPU, bit-identical to the CPU generator
        t = synth.make_weight(cfg, name, device="cuda")
        w[name] = hs.pack_weight(cfg, name, t)
        del t
    return hs.Model(cfg, w, max_batch=1, max_ctx=cap, packed=True)


def _step_check(gold_step, sample, logits):
    """(relative, absolute) largest logit error at the stored indices."""
    pairs = list(gold_step["top"]) + list(zip(sample, gold_step["sample"]))
    err = max(abs(float(logits[i]) - v) for i, v in pairs)
    return err / gold_step["max_abs"], err


def _free_running(name):
    import paper_2603_12707_amd as hs
    with open(os.path.join(GOLDEN, f"greedy_{name}.json")) as f:
        gold = json.load(f)
    cfg = configs.get(name)
    n_v, s_text, n_dec = gold["n_v"], gold["s_text"], gold["n_dec"]
    assert gold["seed"] == cfg["seed"] and (n_v, s_text) == tuple(x[0] for x in synth.request_lengths(cfg))
    cap = n_v + s_text + max(n_dec, bench.steps_after_context(bench.DEFAULT_WARMUP, bench.DEFAULT_STEPS))
    model = _gpu_model(cfg, cap)
    kv = hs.KVCache(model, [n_v], [cap])
    emb = synth.vision_rows(cfg, 0, n_v, device="cuda")
    ids = synth.text_ids(cfg, 0, s_text, device="cuda")
    pos = synth.mrope_positions(n_v, s_text).cuda() if cfg["rope_kind"] == 1 else None
    V = cfg["vocab"]
    logits = torch.empty(1, V, dtype=torch.float32, device="cuda")
    tin = torch.empty(1, dtype=torch.int32, device="cuda")
    tout = torch.empty(1, dtype=torch.int32, device="cuda")
    kv.prefill(0, emb, ids, pos, last_logits=logits[0], first_token=tin)
    worst_rel, worst_ratio, ties, equal = 0.0, float("inf"), [], 0
    for k, gs in enumerate(gold["steps"]):
        if k > 0:
            tin.fill_(gold["steps"][k - 1]["token"])
            kv.decode(tin, tout, logits)
        torch.cuda.synchronize()
        tok = int((tin if k == 0 else tout).item())
        lg = logits[0].cpu().numpy()
        rel, err = _step_check(gs, gold["sample_indices"], lg)
        assert rel <= LOGIT_TOL, (k, rel)
        worst_rel = max(worst_rel, rel)
        worst_ratio = min(worst_ratio, (gs["top1"] - gs["top2"]) / max(err, 1e-30))
        if tok == gs["token"]:
            equal += 1
            continue
        ref = dict((i, v) for i, v in gs["top"])
        assert tok in ref and gs["top1"] - ref[tok] <= 2 * err, (k, tok, gs["token"], gs["top1"] - gs["top2"], err)
        ties.append(k)
    assert kv.lengths() == [n_v + s_text + n_dec]
    assert model.status() == 0
    kv.close()
    model.close()
    print(f"\n[greedy {name}] {equal} of {n_dec + 1} tokens equal, near ties at steps {ties}; max logit rel err "
          f"{worst_rel:.3g}; smallest oracle margin / GPU logit error {worst_ratio:.3g}", flush=True)
    return ties


def test_tiny_free_running_matches_stored_oracle_run():
    assert _free_running("tiny") == []


@pytest.mark.slow
@pytest.mark.timeout(900)
def test_llava7b_b1_free_running_128_steps_token_for_token():
    """The LLaVA-shaped fp16 batch-1 workload: the real 576 + 64-row prefill,
    then all 128 greedy steps."""
    assert len(_free_running("llava7b_b1")) <= 1


def _free_running_batch(name):
    """Request 0 of a batched workload against the oracle's stored run, in
    bench.py's launch configuration: every request prefilled from its real
    inputs in packed passes, then the whole batch decodes n_dec steps; request
    0 is fed the oracle's previous token (its own wherever the two agree), the
    other requests their own tokens."""
    with open(os.path.join(GOLDEN, f"greedy_{name}.json")) as f:
        gold = json.load(f)
    cfg = configs.get(name)
    n_v, s_text = synth.request_lengths(cfg)
    assert gold["seed"] == cfg["seed"] and (gold["n_v"], gold["s_text"]) == (n_v[0], s_text[0])
    n_dec, B, V = gold["n_dec"], cfg["batch"], cfg["vocab"]
    tail = max(n_dec, bench.steps_after_context(bench.DEFAULT_WARMUP, bench.DEFAULT_STEPS))
    models, kv, first, lens, _ = bench.setup(cfg, bench.make_weights(cfg), tail)
    model = models[0]
    torch.cuda.synchronize()
    s0 = gold["steps"][0]
    tok0 = int(first[0].item())
    assert tok0 == s0["token"] or (tok0 in dict((i, v) for i, v in s0["top"]) and
                                   s0["top1"] - dict((i, v) for i, v in s0["top"])[tok0] <= 2 * LOGIT_TOL * s0["max_abs"])
    idx = torch.tensor(sorted(set(gold["sample_indices"]) | {i for s in gold["steps"] for i, _ in s["top"]}),
                       dtype=torch.long, device="cuda")
    pos_of = {int(i): k for k, i in enumerate(idx.tolist())}
    logits = torch.empty(B, V, dtype=torch.float32, device="cuda")
    tin, tout = first.clone(), torch.empty_like(first)
    worst_rel, ties, equal = 0.0, [], int(tok0 == s0["token"])
    for k in range(1, n_dec + 1):
        gs = gold["steps"][k]
        tin[0] = gold["steps"][k - 1]["token"]
        kv.decode(tin, tout, logits)
        row = logits[0].index_select(0, idx).cpu().numpy()
        tok = int(tout[0].item())
        lg = {i: float(row[pos_of[i]]) for i in pos_of}
        pairs = list(gs["top"]) + list(zip(gold["sample_indices"], gs["sample"]))
        err = max(abs(lg[int(i)] - v) for i, v in pairs)
        rel = err / gs["max_abs"]
        assert rel <= LOGIT_TOL, (k, rel)
        worst_rel = max(worst_rel, rel)
        if tok == gs["token"]:
            equal += 1
        else:
            ref = dict((i, v) for i, v in gs["top"])
            assert tok in ref and gs["top1"] - ref[tok] <= 2 * err, (k, tok, gs["token"], gs["top1"] - gs["top2"], err)
            ties.append(k)
        tin, tout = tout, tin
    assert kv.lengths()[0] == lens[0] + n_dec
    assert model.status() == 0
    kv.close()
    for m in models:
        m.close()
    print(f"\n[greedy {name} request 0 at batch {B}] {equal} of {n_dec + 1} tokens equal, near ties at steps "
          f"{ties}; max logit rel err {worst_rel:.3g}", flush=True)
    return ties


@pytest.mark.slow
@pytest.mark.timeout(900)
def test_qwen7b_b16_request0_free_running_256_steps_at_batch_16():
    """The Qwen-shaped bf16 batch-16 workload (GQA 28/4, 3-section M-RoPE,
    q/k/v bias): the real 515 + 128-row prefill of request 0 among 16 packed
    requests, then all 256 greedy steps of the batch.  Every differing token
    is a near tie by the per-step rule; in bf16 the oracle's top-2 margin is
    within twice the 2e-2 bound on 141 of the 257 steps, and at most 5 % of
    the steps may differ (measured: 10, steps 5 ... 253)."""
    ties = _free_running_batch("qwen7b_b16")
    assert len(ties) <= 0.05 * 257


@pytest.mark.slow
@pytest.mark.timeout(900)
def test_llava7b_b32_request0_free_running_128_steps_at_batch_32():
    """The LLaVA-shaped fp16 batch-32 workload: the real 576 + 223-row
    prefill of request 0 among 32 packed requests, then all 128 greedy steps
    of the batch."""
    ties = _free_running_batch("llava7b_b32")
    assert len(ties) <= 0.05 * 129
