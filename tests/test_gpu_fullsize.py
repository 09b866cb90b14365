"""Parity at the full workload sizes, in the launch configuration bench.py
uses, on outputs the oracle can compute one by one.

The oracle cannot prefill 640+ rows of a 7B-shaped model in reasonable time
(single-threaded, ~9 s per row), so at these sizes:
  * decode is checked from a synthetic cache written identically to both
    sides (hs_kv_write / the oracle's own cache), for sampled requests,
    teacher-forced: logits, greedy tokens (near-tie rule), the residual
    stream after the last layer and the appended K/V rows;
  * prefill is checked through the layer-0 K/V rows at sampled positions,
    which depend on that row alone.
Weights come from the seeded generator run on the GPU; its CPU/GPU bit
identity is checked in test_gpu_abi.py.
"""
from __future__ import annotations

import gc

import numpy as np
import pytest
import torch

import bench
from helpers import KV_ROW0_TOL, KV_ROWS_DEEP_TOL, LOGIT_TOL, rel_err, token_ok
from oracle import oracle as O
from workload import configs, synth

pytestmark = [pytest.mark.gpu, pytest.mark.slow, pytest.mark.timeout(900)]
# positions bench.py allocates after each request's context (its default run)
BENCH_TAIL = bench.steps_after_context(bench.DEFAULT_WARMUP, bench.DEFAULT_STEPS)
TDT = {"f16": torch.float16, "bf16": torch.bfloat16, "f32": torch.float32}


def _weights(cfg):
    """(row-major CPU copies for the oracle, packed GPU weights)."""
    import paper_2603_12707_amd as hs
    cpu, gpu = {}, {}
    for name in synth.weight_names(cfg):
        t = synth.make_weight(cfg, name, device="cuda")
        cpu[name] = t.cpu()
        gpu[name] = hs.pack_weight(cfg, name, t)
        del t
    torch.cuda.synchronize()
    return cpu, gpu


def _fill_both(cfg, kv, req, seq, length, rope_pos):
    """Writes the same synthetic cache rows [0, length) of request req into
    the GPU cache and into the oracle sequence."""
    kv.set_length(req, length, rope_pos)  # a pooled cache takes the blocks here
    for layer in range(cfg["n_layers"]):
        for sel in (0, 1):
            for h in range(cfg["n_kv_heads"]):
                rows = synth.kv_block(cfg, req, layer, sel, h, length, device="cuda")
                kv.write(req, layer, sel, h, 0, rows)
                if seq is not None:
                    seq.write_kv(layer, sel, h, 0, rows.float().cpu())
    if seq is not None:
        seq.set_len(length, rope_pos)


def _decode_compare(cfg, kv, seqs, sample, tokens, lens):
    """One teacher-forced decode step for the whole batch; compares the
    sampled requests with the oracle."""
    B = kv.batch
    has_head = cfg.get("lm_head", True)
    tin = torch.tensor(tokens, dtype=torch.int32, device="cuda")
    tout = torch.empty(B, dtype=torch.int32, device="cuda")
    logits = torch.empty(B, cfg["vocab"], dtype=torch.float32, device="cuda") if has_head else None
    hidden = torch.empty(B, cfg["d_model"], dtype=torch.float32, device="cuda")
    kv.decode(tin, tout if has_head else None, logits, hidden)
    torch.cuda.synchronize()
    ties = 0
    for r in sample:
        r_log, r_hid, r_tok = seqs[r].decode(tokens[r])
        assert rel_err(hidden[r].cpu().numpy(), r_hid) <= LOGIT_TOL, r
        if has_head:
            g_log = logits[r].cpu().numpy()
            assert rel_err(g_log, r_log) <= LOGIT_TOL, (r, rel_err(g_log, r_log))
            ok, tie = token_ok(int(tout[r].item()), g_log, r_log)
            assert ok, r
            ties += tie
        # the appended K/V rows of every head at the first and the last layer:
        # layer 0 row by row (one storage rounding from the oracle); the last
        # layer's K (and V) rows of all heads as one vector, like the logits
        for layer in sorted({0, cfg["n_layers"] - 1}):
            for sel in (0, 1):
                gs, refs = [], []
                for h in range(cfg["n_kv_heads"]):
                    g = torch.empty(1, cfg["head_dim"], dtype=TDT[cfg["dtype"]], device="cuda")
                    kv.read(r, layer, sel, h, lens[r], 1, g)
                    ref = seqs[r].read_kv(layer, sel, h, lens[r], 1)
                    if layer == 0:
                        err = rel_err(g.float().cpu().numpy(), ref)
                        assert err <= KV_ROW0_TOL, (r, layer, h, sel, err)
                    gs.append(g.float().cpu().numpy().ravel())
                    refs.append(np.asarray(ref).ravel())
                if layer > 0:
                    err = rel_err(np.concatenate(gs), np.concatenate(refs))
                    assert err <= KV_ROWS_DEEP_TOL, (r, layer, sel, err)
    return ties


def _prefill_layer0_compare(cfg, w_cpu, kv, req, emb, ids, pos_thw, positions):
    """Layer-0 K/V rows written by hs_prefill_embeddings at sampled positions
    against the oracle's first layer on those rows alone."""
    one = dict(cfg, n_layers=1, lm_head=False)
    keep = {k: v for k, v in w_cpu.items() if k == "embed" or k.startswith("layers.0.")}
    om = O.Model(one, keep)
    n_v = emb.shape[0]
    for p in positions:
        x = emb[p].float() if p < n_v else w_cpu["embed"][int(ids[p - n_v])].float()
        pos3 = (p, p, p) if pos_thw is None else tuple(int(pos_thw[c, p]) for c in range(3))
        seq = om.new_seq(p + 1)
        seq.set_len(p, 0)
        seq.forward_row(x.numpy(), pos3, want_logits=False)
        for h in sorted({0, cfg["n_kv_heads"] // 2, cfg["n_kv_heads"] - 1}):
            for sel in (0, 1):
                g = torch.empty(1, cfg["head_dim"], dtype=TDT[cfg["dtype"]], device="cuda")
                kv.read(req, 0, sel, h, p, 1, g)
                ref = seq.read_kv(0, sel, h, p, 1)
                assert rel_err(g.float().cpu().numpy(), ref) <= KV_ROW0_TOL, (p, h, sel)


@pytest.fixture(scope="module")
def llava():
    cfg = configs.get("llava7b_b1")
    cpu, gpu = _weights(cfg)
    yield cfg, cpu, gpu
    del cpu, gpu
    gc.collect()
    torch.cuda.empty_cache()


def test_llava7b_b1_bench_configuration(llava):
    """Batch 1, the capacity bench.py allocates: sampled prefill rows, then
    two teacher-forced decode steps from a synthetic 640-position cache."""
    import paper_2603_12707_amd as hs
    cfg, w_cpu, w_gpu = llava
    n_v, s_text = synth.request_lengths(cfg)
    ctx = n_v[0] + s_text[0]
    cap = ctx + BENCH_TAIL
    model = hs.Model(cfg, w_gpu, max_batch=1, max_ctx=cap, packed=True)
    # prefill from the real inputs
    kv = hs.KVCache(model, n_v, [cap])
    emb = synth.vision_rows(cfg, 0, n_v[0])
    ids = synth.text_ids(cfg, 0, s_text[0])
    kv.prefill(0, emb.cuda(), ids.cuda())
    torch.cuda.synchronize()
    assert kv.lengths() == [ctx]
    _prefill_layer0_compare(cfg, w_cpu, kv, 0, emb, ids, None, [0, 1, 301, n_v[0] - 1, n_v[0], ctx - 1])
    kv.close()
    # decode from a synthetic cache
    kv = hs.KVCache(model, n_v, [cap])
    seq = O.Model(cfg, w_cpu).new_seq(cap)
    _fill_both(cfg, kv, 0, seq, ctx, ctx)
    toks = synth.decode_tokens(cfg, 0, 2).tolist()
    ties = 0
    for k in range(2):
        ties += _decode_compare(cfg, kv, [seq], [0], [toks[k]], [ctx + k])
    assert ties == 0
    kv.close()
    model.close()


def test_llava7b_b32_sampled_requests(llava):
    import paper_2603_12707_amd as hs
    cfg, w_cpu, w_gpu = llava
    cfg = configs.get("llava7b_b32")
    n_v, s_text = synth.request_lengths(cfg)
    lens = [a + b for a, b in zip(n_v, s_text)]
    caps = [n + BENCH_TAIL for n in lens]
    model = hs.Model(cfg, w_gpu, max_batch=32, max_ctx=max(caps), packed=True)
    kv = hs.KVCache(model, n_v, caps)
    sample = [0, 17, 31]
    om = O.Model(cfg, w_cpu)
    seqs = {}
    for r in range(32):
        seqs[r] = om.new_seq(caps[r]) if r in sample else None
        _fill_both(cfg, kv, r, seqs[r], lens[r], lens[r])
    toks = synth.decode_tokens(cfg, 1, 32).tolist()
    assert _decode_compare(cfg, kv, seqs, sample, toks, lens) <= 1
    kv.close()
    model.close()


@pytest.fixture(scope="module")
def qwen():
    cfg = configs.get("qwen7b_b16")
    cpu, gpu = _weights(cfg)
    yield cfg, cpu, gpu
    del cpu, gpu
    gc.collect()
    torch.cuda.empty_cache()


def test_qwen7b_b16_sampled_requests_mrope(qwen):
    """GQA 28/4, bf16, 3-section M-RoPE: prefill rows of one request with its
    (t, h, w) ids, then one teacher-forced step for two sampled requests."""
    import paper_2603_12707_amd as hs
    cfg, w_cpu, w_gpu = qwen
    n_v, s_text = synth.request_lengths(cfg)
    lens = [a + b for a, b in zip(n_v, s_text)]
    caps = [n + BENCH_TAIL for n in lens]
    model = hs.Model(cfg, w_gpu, max_batch=16, max_ctx=max(caps), packed=True)
    kv = hs.KVCache(model, n_v, caps)
    r0 = 3
    emb = synth.vision_rows(cfg, r0, n_v[r0])
    ids = synth.text_ids(cfg, r0, s_text[r0])
    pos = synth.mrope_positions(n_v[r0], s_text[r0])
    kv.prefill(r0, emb.cuda(), ids.cuda(), pos.cuda())
    torch.cuda.synchronize()
    _prefill_layer0_compare(cfg, w_cpu, kv, r0, emb, ids, pos, [0, 37, n_v[r0] - 1, n_v[r0], lens[r0] - 1])
    kv.close()
    kv = hs.KVCache(model, n_v, caps)
    sample = [0, 15]
    om = O.Model(cfg, w_cpu)
    seqs = {}
    for r in range(16):
        rope = int(synth.mrope_positions(n_v[r], s_text[r]).max()) + 1
        seqs[r] = om.new_seq(caps[r]) if r in sample else None
        _fill_both(cfg, kv, r, seqs[r], lens[r], rope)
    toks = synth.decode_tokens(cfg, 2, 16).tolist()
    assert _decode_compare(cfg, kv, seqs, sample, toks, lens) <= 1
    kv.close()
    model.close()


@pytest.mark.parametrize("pool_block", [0, 256])
def test_qwen_layer_b256_sampled_requests(pool_block):
    """One Qwen-shaped layer, batch 256, KV lengths U[1024, 8192]: the
    residual stream after the layer and the appended rows, for sampled
    requests, over two appending steps; in a contiguous cache and in a pool
    of 256-position blocks (decode splits of several thousand positions
    read dozens of blocks)."""
    import paper_2603_12707_amd as hs
    cfg = configs.get("qwen_layer_b256")
    w_cpu, w_gpu = _weights(cfg)
    lens = synth.kv_lengths(cfg)
    caps = [n + BENCH_TAIL for n in lens]
    model = hs.Model(cfg, w_gpu, max_batch=256, max_ctx=max(caps), packed=True)
    if pool_block:
        kv = hs.KVPool(model, 256, pool_block, sum((c + pool_block - 1) // pool_block for c in caps))
        for r in range(256):
            kv.admit(r, 0, caps[r])
    else:
        kv = hs.KVCache(model, [0] * 256, caps)
    sample = [0, 100, int(np.argmax(lens)), 255]
    om = O.Model(cfg, w_cpu)
    seqs = {}
    for r in range(256):
        seqs[r] = om.new_seq(caps[r]) if r in sample else None
        _fill_both(cfg, kv, r, seqs[r], lens[r], lens[r])
    toks = synth.decode_tokens(cfg, 0, 256).tolist()
    for k in range(2):
        _decode_compare(cfg, kv, seqs, sample, toks, [n + k for n in lens])
    kv.close()
    model.close()
