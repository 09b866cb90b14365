"""Parity of the HIP path (through the C ABI) with the CPU oracle on the same
seeded inputs, at sizes the oracle finishes in seconds that still span several
tiles, splits and ragged tails."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from helpers import LOGIT_TOL, Pair, rel_err, small_cfg, token_ok
from workload import configs, synth

pytestmark = pytest.mark.gpu


def _packed_inputs(inputs, order):
    """The inputs of the requests in `order`, packed request by request as
    hs_prefill_batch takes them (device tensors or None)."""
    embs = [inputs[b][0] for b in order if inputs[b][0].shape[0]]
    ids = [inputs[b][1] for b in order if inputs[b][1].shape[0]]
    pos = [inputs[b][2] for b in order] if inputs[order[0]][2] is not None else None
    return (torch.cat(embs).cuda() if embs else None, torch.cat(ids).cuda() if ids else None,
            torch.cat(pos, dim=1).contiguous().cuda() if pos else None)


def _run_pair(cfg, n_v_list, s_text_list, n_dec, extra_cap=0, free_running=False, packed=None, weights=None):
    """Prefills every request on both sides, then runs n_dec decode steps for
    the whole batch (teacher-forced on the oracle's tokens unless
    free_running).  With packed = {"order": [...], "rows": R}, the GPU side
    prefills all requests in one hs_prefill_batch call, in that order, with
    the row workspaces grown to R rows (0: as created).  Returns the number
    of near ties.  `weights` (CPU tensors) replaces the seeded weights."""
    import paper_2603_12707_amd as hs
    B = len(n_v_list)
    caps = [n + s + n_dec + extra_cap for n, s in zip(n_v_list, s_text_list)]
    pair = Pair(cfg, max_batch=B, max_ctx=max(caps), weights_cpu=weights)
    kv = hs.KVCache(pair.gpu, n_v_list, caps)
    seqs, cur_ref, cur_gpu = [], [], []
    near = 0
    V = cfg["vocab"]
    inputs = [pair.request_inputs(b, n_v_list[b], s_text_list[b]) for b in range(B)]
    refs = []
    for b in range(B):
        emb, ids, pos = inputs[b]
        s = pair.ora.new_seq(caps[b])
        refs.append(s.prefill(emb if n_v_list[b] else None, ids, pos))
        seqs.append(s)
    g_first = [None] * B
    if packed is None:
        for b in range(B):
            emb, ids, pos = inputs[b]
            lg = torch.empty(V, dtype=torch.float32, device="cuda")
            tok = kv.prefill(b, emb.cuda() if n_v_list[b] else None, ids.cuda() if s_text_list[b] else None,
                             None if pos is None else pos.cuda(), last_logits=lg)
            torch.cuda.synchronize()
            g_first[b] = (int(tok.item()), lg.cpu().numpy())
    else:
        order = packed["order"]
        if packed.get("rows"):
            pair.gpu.reserve_rows(packed["rows"])
        emb, ids, pos = _packed_inputs(inputs, order)
        lg = torch.empty(len(order), V, dtype=torch.float32, device="cuda")
        toks = kv.prefill_batch(order, emb, ids, [s_text_list[b] for b in order], pos, last_logits=lg)
        torch.cuda.synchronize()
        for k, b in enumerate(order):
            g_first[b] = (int(toks[k].item()), lg[k].cpu().numpy())
    for b in range(B):
        ref_logits, ref_tok = refs[b]
        tok, g = g_first[b]
        assert rel_err(g, ref_logits) <= LOGIT_TOL, (b, rel_err(g, ref_logits))
        ok, tie = token_ok(tok, g, ref_logits)
        assert ok, (b, tok, ref_tok)
        near += tie
        cur_ref.append(ref_tok)
        cur_gpu.append(tok)
    assert kv.lengths() == [n + s for n, s in zip(n_v_list, s_text_list)]
    tin = torch.empty(B, dtype=torch.int32, device="cuda")
    tout = torch.empty(B, dtype=torch.int32, device="cuda")
    logits = torch.empty(B, V, dtype=torch.float32, device="cuda")
    hidden = torch.empty(B, cfg["d_model"], dtype=torch.float32, device="cuda")
    for step in range(n_dec):
        feed = cur_gpu if free_running else cur_ref
        tin.copy_(torch.tensor(feed, dtype=torch.int32))
        kv.decode(tin, tout, logits, hidden)
        torch.cuda.synchronize()
        g_tok = tout.cpu().tolist()
        g_log = logits.cpu().numpy()
        g_hid = hidden.cpu().numpy()
        nxt_ref = []
        for b in range(B):
            r_log, r_hid, r_tok = seqs[b].decode(feed[b])
            assert rel_err(g_log[b], r_log) <= LOGIT_TOL, (step, b, rel_err(g_log[b], r_log))
            assert rel_err(g_hid[b], r_hid) <= LOGIT_TOL, (step, b)
            ok, tie = token_ok(g_tok[b], g_log[b], r_log)
            assert ok, (step, b, g_tok[b], r_tok)
            near += tie
            nxt_ref.append(r_tok)
        if free_running:
            assert g_tok == nxt_ref, (step, g_tok, nxt_ref)
        cur_ref, cur_gpu = nxt_ref, g_tok
    assert kv.lengths() == [n + s + n_dec for n, s in zip(n_v_list, s_text_list)]
    assert pair.gpu.status() == 0
    kv.close()
    pair.gpu.close()
    return near


def test_tiny_config_free_running_token_for_token():
    """The tiny fp32 decoder: 576 vision rows + 32 text tokens, 16 greedy
    steps, tokens identical to the oracle's without teacher forcing."""
    cfg = configs.get("tiny")
    n_v, s_text = synth.request_lengths(cfg)
    near = _run_pair(cfg, n_v, s_text, cfg["n_dec"], free_running=True)
    assert near == 0


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
def test_mha_batch_ragged(dtype):
    # three requests with different vision/text lengths; d = 384 leaves one
    # wave without K blocks, F = 1000 and V = 997 leave ragged tails
    near = _run_pair(small_cfg(dtype=dtype), [40, 0, 129], [7, 33, 1], 5)
    assert near <= 1


@pytest.mark.parametrize("group,n_heads,head_dim", [(2, 4, 128), (4, 8, 64), (7, 14, 64), (8, 8, 64)])
def test_gqa_groups(group, n_heads, head_dim):
    cfg = small_cfg(n_heads=n_heads, n_kv_heads=n_heads // group, head_dim=head_dim, dtype="bf16")
    near = _run_pair(cfg, [33, 5], [20, 260], 4)
    assert near <= 1


def test_mrope_qkv_bias_gqa7():
    cfg = small_cfg(n_heads=14, n_kv_heads=2, head_dim=64, dtype="bf16", rope_kind=1, mrope_section=(8, 12, 12),
                    qkv_bias=1, rope_theta=1e6, rms_eps=1e-6)
    near = _run_pair(cfg, [70, 16, 121], [12, 12, 3], 5)
    assert near <= 1


@pytest.mark.parametrize("B", [17, 33])
def test_column_tiles(B):
    """Batches spanning two and three 16-column tiles."""
    cfg = small_cfg(n_layers=1, dtype="f16")
    n_v = [(7 * b) % 23 for b in range(B)]
    s_text = [1 + (5 * b) % 11 for b in range(B)]
    near = _run_pair(cfg, n_v, s_text, 3)
    assert near <= 2


def test_packed_activation_layout():
    """24 requests at d = 1024 (GQA-4 with bias, F = 1000): the q/k/v, gate/up,
    down and LM head GEMMs read their activations from memory in the packed
    MFMA-operand layout, written by the RMSNorm and by the SwiGLU epilogue
    (F pads to 1024 there).  The prefills, 2..31 rows each, mix the producer
    and consumer paths: a small prefill stages q/k/v and gate/up activations
    in LDS while its down projection reads the packed layout."""
    cfg = small_cfg(n_layers=1, d_model=1024, n_heads=8, n_kv_heads=2, head_dim=128, ffn_dim=1000, dtype="bf16",
                    qkv_bias=1)
    n_v = [(9 * b) % 27 for b in range(24)]
    s_text = [2 + (5 * b) % 3 for b in range(24)]
    near = _run_pair(cfg, n_v, s_text, 3)
    assert near <= 2


@pytest.mark.parametrize("dtype,B,d", [("bf16", 12, 2056), ("f16", 16, 1032), ("f16", 5, 4360)])
def test_one_column_tile_read_from_memory(dtype, B, d):
    """5..16 requests whose activations do not fit the LDS copy: every GEMM of
    the decode step reads one column tile from memory in the packed layout
    (2-wave q/k/v, SwiGLU and LM head work groups, 4-wave residual ones), after
    the separate RMSNorm.  d = 2056 and 1032 end in a half row tile and a
    partial k-block; two layers, GQA-4 with q/k/v bias."""
    cfg = small_cfg(n_layers=2, d_model=d, n_heads=8, n_kv_heads=2, head_dim=128, ffn_dim=1000, dtype=dtype,
                    qkv_bias=1)
    n_v = [(11 * b) % 29 for b in range(B)]
    s_text = [1 + (3 * b) % 7 for b in range(B)]
    near = _run_pair(cfg, n_v, s_text, 3)
    assert near <= 2


@pytest.mark.parametrize("dtype", ["f16", "f32"])
def test_packed_prefill_mha(dtype):
    """Six requests of mixed shapes (no vision rows, no text, one row)
    prefilled by one hs_prefill_batch call in a shuffled order; the row
    workspaces hold 86 rows (the largest capacity), so the 225 rows go in
    three packed passes."""
    cfg = small_cfg(n_layers=2, dtype=dtype)
    n_v = [0, 37, 70, 1, 16, 45]
    s_text = [9, 0, 13, 0, 30, 4]
    near = _run_pair(cfg, n_v, s_text, 3, packed={"order": [4, 1, 5, 0, 3, 2], "rows": 0})
    assert near <= 1


def test_packed_prefill_gqa7_mrope_bias():
    """Packed prefill with 7 query heads per KV head (2 query rows per matrix
    tile), M-RoPE ids taken section-major over all packed rows, q/k/v bias;
    one pass holds every request."""
    cfg = small_cfg(n_heads=14, n_kv_heads=2, head_dim=64, dtype="bf16", rope_kind=1, mrope_section=(8, 12, 12),
                    qkv_bias=1, rope_theta=1e6, rms_eps=1e-6)
    n_v = [70, 16, 121, 9]
    s_text = [12, 12, 3, 31]
    near = _run_pair(cfg, n_v, s_text, 3, packed={"order": [2, 0, 3, 1], "rows": 512})
    assert near <= 1


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("packed", [False, True])
def test_prefill_wide_score_range(dtype, packed):
    """The q and k projections scaled by 8, so that attention scores spread
    over tens of units (std ~10): the prefill attention's running maximum,
    raised only when a score passes it by more than its slack, is raised
    past the first key tiles too, with o and l already accumulated."""
    cfg = small_cfg(n_layers=1, dtype=dtype)
    w = synth.make_weights(cfg)
    for name in ("layers.0.wq", "layers.0.wk"):
        w[name] = w[name] * 8
    n_v = [300, 0, 61]
    s_text = [20, 150, 9]
    near = _run_pair(cfg, n_v, s_text, 2, weights=w,
                     packed={"order": [1, 2, 0], "rows": 512} if packed else None)
    assert near <= 1


def test_packed_prefill_more_requests_than_a_pass():
    """37 short requests: a pass takes at most 32 of them."""
    cfg = small_cfg(n_layers=1, dtype="bf16")
    B = 37
    n_v = [(5 * b) % 11 for b in range(B)]
    s_text = [1 + (3 * b) % 6 for b in range(B)]
    order = list(range(B))[::-1]
    near = _run_pair(cfg, n_v, s_text, 2, packed={"order": order, "rows": 4096})
    assert near <= 2


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_many_columns_split_k(dtype):
    """40 requests (three column tiles) and a long, ragged down projection
    (K = 2040), two layers: the residual GEMM splits K four ways into fp32
    partials and sums them into the residual stream that the second layer
    and the LM head read."""
    cfg = small_cfg(n_layers=2, ffn_dim=2040, dtype=dtype)
    n_v = [(11 * b) % 29 for b in range(40)]
    s_text = [1 + (3 * b) % 7 for b in range(40)]
    near = _run_pair(cfg, n_v, s_text, 2)
    assert near <= 2


def test_many_columns_split_k_qkv():
    """40 requests and K = 1024: the q/k/v GEMM (GQA-2, with bias) splits K
    and a second kernel sums the partials before the bias, RoPE and the K/V
    append."""
    cfg = small_cfg(n_layers=1, d_model=1024, n_heads=8, n_kv_heads=4, head_dim=128, ffn_dim=1024, dtype="bf16",
                    qkv_bias=1)
    n_v = [(7 * b) % 19 for b in range(40)]
    s_text = [1 + (5 * b) % 9 for b in range(40)]
    near = _run_pair(cfg, n_v, s_text, 2)
    assert near <= 2


@pytest.mark.parametrize("d_model,n_heads,n_kv_heads,qkv_bias,dtype", [(1024, 8, 2, 1, "bf16"), (512, 4, 4, 0, "f16")])
def test_weight_stationary_columns(d_model, n_heads, n_kv_heads, qkv_bias, dtype):
    """150 requests (129..256 columns): gate/up and the LM head take the
    weight-stationary GEMM (two column groups, the second ragged; F = 1000
    leaves a ragged last gate/up task and V = 997 a ragged LM head), while
    q/k/v, O and down stay on the LDS-staged kernel (at d = 1024 with K
    split two ways)."""
    cfg = small_cfg(n_layers=1, d_model=d_model, n_heads=n_heads, n_kv_heads=n_kv_heads, head_dim=128, ffn_dim=1000,
                    dtype=dtype, qkv_bias=qkv_bias)
    n_v = [(13 * b) % 11 for b in range(150)]
    s_text = [1 + (5 * b) % 4 for b in range(150)]
    near = _run_pair(cfg, n_v, s_text, 2)
    assert near <= 3


@pytest.mark.parametrize("B", [2, 6])
def test_rows_longer_than_one_pass(B):
    """d = 4608: the RMSNorm holds a row's first 4096 elements in registers
    and reads the remaining 512 in a second pass -- in the GEMM prologue at 2
    columns, in the separate normalisation kernel at 6 columns and in
    prefill."""
    cfg = small_cfg(n_layers=1, d_model=4608, n_heads=4, n_kv_heads=4, head_dim=128, ffn_dim=512, vocab=512,
                    dtype="bf16")
    n_v = [(7 * b) % 13 for b in range(B)]
    s_text = [2 + b % 3 for b in range(B)]
    near = _run_pair(cfg, n_v, s_text, 3)
    assert near <= 1


def test_deferred_residual_sum_rows_longer_than_one_pass():
    """6 requests at d = 4608 whose O and down projections (3072 inputs each)
    read their activations from memory: each leaves two fp64 K-split partials
    that the next RMSNorm adds, in both of its passes (a row's first 4096
    elements held in registers, the remaining 512 read again); two layers,
    so the second layer's q/k/v norm takes the first layer's down partials,
    and the LM head's norm the last ones."""
    cfg = small_cfg(n_layers=2, d_model=4608, n_heads=24, n_kv_heads=6, head_dim=128, ffn_dim=3072, vocab=512,
                    dtype="bf16")
    n_v = [(7 * b) % 13 for b in range(6)]
    s_text = [2 + b % 3 for b in range(6)]
    near = _run_pair(cfg, n_v, s_text, 3)
    assert near <= 1


@pytest.mark.parametrize("n_heads,ffn_dim", [(18, 2560), (16, 2560), (18, 1536)])
def test_deferred_residual_sum_without_lm_head(n_heads, ffn_dim):
    """8 requests of a two-layer model without an LM head, whose output is the
    residual stream after the last layer, at d = 2304.  A residual projection
    leaves its sum pending when its activations do not fit the LDS copy
    (8 x K x 2 bytes > 32 KB): O over 2304 inputs and down over 2560 both do;
    O over 2048 inputs (16 heads) adds its sum itself while down defers; down
    over 1536 adds its own while O defers.  Each pending sum goes to the next
    norm, and the last down projection's, when pending, to the step's own
    kernel.  Caches of 5..54 positions written alike to both sides, three
    teacher-forced steps, every request's residual stream against the
    oracle's."""
    import paper_2603_12707_amd as hs
    cfg = small_cfg(n_layers=2, d_model=2304, n_heads=n_heads, n_kv_heads=n_heads // 2, head_dim=128,
                    ffn_dim=ffn_dim, dtype="bf16", qkv_bias=1, lm_head=False)
    B = 8
    lens = [5 + 7 * b for b in range(B)]
    caps = [n + 3 for n in lens]
    pair = Pair(cfg, max_batch=B, max_ctx=max(caps))
    kv = hs.KVCache(pair.gpu, [0] * B, caps)
    seqs = []
    for r in range(B):
        kv.set_length(r, lens[r], lens[r])
        s = pair.ora.new_seq(caps[r])
        for layer in range(cfg["n_layers"]):
            for sel in (0, 1):
                for h in range(cfg["n_kv_heads"]):
                    rows = synth.kv_block(cfg, r, layer, sel, h, lens[r], device="cuda")
                    kv.write(r, layer, sel, h, 0, rows)
                    s.write_kv(layer, sel, h, 0, rows.float().cpu())
        s.set_len(lens[r], lens[r])
        seqs.append(s)
    hidden = torch.empty(B, cfg["d_model"], dtype=torch.float32, device="cuda")
    for step in range(3):
        toks = synth.decode_tokens(cfg, step, B).tolist()
        kv.decode(torch.tensor(toks, dtype=torch.int32, device="cuda"), None, None, hidden)
        torch.cuda.synchronize()
        g_hid = hidden.cpu().numpy()
        for b in range(B):
            _, r_hid, _ = seqs[b].decode(toks[b])
            assert rel_err(g_hid[b], r_hid) <= LOGIT_TOL, (step, b, rel_err(g_hid[b], r_hid))
    assert kv.lengths() == [n + 3 for n in lens]
    assert pair.gpu.status() == 0
    kv.close()
    pair.gpu.close()


@pytest.mark.parametrize("n_v,dtype", [(1100, "f16"), (2400, "f16"), (2400, "f32")])
def test_long_context_many_splits(n_v, dtype):
    """Contexts long enough for many attention splits in decode: at most 8
    (combined in the O projection's prologue), up to 16 (partials requested
    at once by the combine kernel) and more (the combine's general loop)."""
    cfg = small_cfg(n_layers=1, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64, ffn_dim=512, vocab=512,
                    dtype=dtype)
    near = _run_pair(cfg, [n_v], [37], 3, extra_cap=400)
    assert near == 0


def test_batch_invariance():
    """A request's logits do not depend on the other requests of its batch
    (the property that lets decode shard by request across GPUs)."""
    import paper_2603_12707_amd as hs
    cfg = small_cfg(dtype="bf16", n_heads=8, n_kv_heads=2, head_dim=64)
    n_v, s_text = [30, 3, 70, 0, 12], [5, 40, 2, 9, 200]
    caps = [n + s + 3 for n, s in zip(n_v, s_text)]
    pair = Pair(cfg, max_batch=5, max_ctx=max(caps))
    out = {}
    for batch in ([2], [0, 1, 2, 3, 4]):
        kv = hs.KVCache(pair.gpu, [n_v[r] for r in batch], [caps[r] for r in batch])
        for i, r in enumerate(batch):
            emb, ids, _ = pair.request_inputs(r, n_v[r], s_text[r])
            kv.prefill(i, emb.cuda() if n_v[r] else None, ids.cuda())
        logits = torch.empty(len(batch), cfg["vocab"], device="cuda")
        tout = torch.empty(len(batch), dtype=torch.int32, device="cuda")
        kv.decode(torch.full((len(batch),), 11, dtype=torch.int32, device="cuda"), tout, logits)
        out[len(batch)] = logits[batch.index(2)].cpu().numpy()
        kv.close()
    assert rel_err(out[5], out[1]) <= 1e-3


@pytest.mark.parametrize("rope_kind", [0, 1])
def test_prefill_then_decode_matches_longer_prefill(rope_kind):
    """prefill(s + 1) last-row logits agree with prefill(s) followed by one
    decode step of token s (a property that holds at any size)."""
    import paper_2603_12707_amd as hs
    extra = dict(rope_kind=1, mrope_section=(8, 12, 12), rope_theta=1e6) if rope_kind else {}
    cfg = small_cfg(dtype="f16", n_heads=6, n_kv_heads=3, head_dim=64, **extra)
    n_v, s_text = 50, 9
    pair = Pair(cfg, max_batch=1, max_ctx=80)
    emb, ids, pos = pair.request_inputs(0, n_v, s_text)
    a = hs.KVCache(pair.gpu, [n_v], [80])
    pos_short = None if pos is None else pos[:, :-1].contiguous()
    a.prefill(0, emb.cuda(), ids[:-1].cuda(), None if pos is None else pos_short.cuda())
    la = torch.empty(1, cfg["vocab"], device="cuda")
    tout = torch.empty(1, dtype=torch.int32, device="cuda")
    if rope_kind:  # the decode position must be the one the longer prefill gives the last token
        assert int(pos[0, -1]) == int(pos_short.max()) + 1
    a.decode(ids[-1:].cuda(), tout, la)
    b = hs.KVCache(pair.gpu, [n_v], [80])
    lb = torch.empty(cfg["vocab"], device="cuda")
    b.prefill(0, emb.cuda(), ids.cuda(), None if pos is None else pos.cuda(), last_logits=lb)
    torch.cuda.synchronize()
    assert rel_err(la[0].cpu().numpy(), lb.cpu().numpy()) <= 2e-3


@pytest.mark.parametrize("case", ["three", "packed", "wide"])
def test_decode_step_replays_from_a_hip_graph(case):
    """hs_decode_step recorded by stream capture (two steps, ping-ponging the
    token buffers) and replayed gives, replay after replay, the tokens and
    logits of eager calls on an identical cache, and the replayed logits of
    sampled requests agree with the oracle fed the same tokens; eager work and
    synchronisation run between the replays.  Cases: 3 requests (activations
    staged in LDS), 20 requests at d = 1024 (packed activations read from
    memory), 150 requests (the weight-stationary gate/up and LM head)."""
    import paper_2603_12707_amd as hs
    if case == "three":
        cfg = small_cfg(dtype="bf16", n_heads=8, n_kv_heads=2, head_dim=64)
        n_v, s_text = [30, 9, 50], [5, 40, 2]
    elif case == "packed":
        cfg = small_cfg(n_layers=1, d_model=1024, n_heads=8, n_kv_heads=2, head_dim=128, ffn_dim=1000, dtype="bf16")
        n_v, s_text = [(9 * b) % 27 for b in range(20)], [2 + b % 3 for b in range(20)]
    else:
        cfg = small_cfg(n_layers=1, dtype="bf16", n_heads=8, n_kv_heads=2, head_dim=64)
        n_v, s_text = [(13 * b) % 11 for b in range(150)], [1 + (5 * b) % 4 for b in range(150)]
    B = len(n_v)
    caps = [n + s + 12 for n, s in zip(n_v, s_text)]
    pair = Pair(cfg, max_batch=B, max_ctx=max(caps))
    handles = []
    for _ in range(2):
        kv = hs.KVCache(pair.gpu, n_v, caps)
        first = torch.empty(B, dtype=torch.int32, device="cuda")
        for r in range(B):
            emb, ids, _ = pair.request_inputs(r, n_v[r], s_text[r])
            kv.prefill(r, emb.cuda() if n_v[r] else None, ids.cuda(), first_token=first[r:r + 1])
        handles.append((kv, first))
    torch.cuda.synchronize()
    V = cfg["vocab"]
    # eager reference: 8 steps
    kv_e, t_e = handles[0]
    a, b = t_e.clone(), torch.empty_like(t_e)
    ref_tok, ref_log = [], []
    lg = torch.empty(B, V, device="cuda")
    for _ in range(8):
        kv_e.decode(a, b, lg)
        ref_tok.append(b.cpu().clone())
        ref_log.append(lg.cpu().clone())
        a, b = b, a
    # the oracle on sampled requests, fed the tokens every step was fed
    sample = sorted({0, B // 2, B - 1})
    seqs = {}
    for r in sample:
        emb, ids, _ = pair.request_inputs(r, n_v[r], s_text[r])
        seqs[r] = pair.ora.new_seq(caps[r])
        seqs[r].prefill(emb if n_v[r] else None, ids)
    feeds = [t_e.cpu().clone()] + ref_tok[:-1]
    near = 0

    def check_oracle(step, g_log, g_tok):
        nonlocal near
        for r in sample:
            r_log, _, _ = seqs[r].decode(int(feeds[step][r]))
            assert rel_err(g_log[r].numpy(), r_log) <= LOGIT_TOL, (step, r, rel_err(g_log[r].numpy(), r_log))
            ok, tie = token_ok(int(g_tok[r]), g_log[r].numpy(), r_log)
            assert ok, (step, r)
            near += tie
    # captured: two steps per graph, replayed four times
    kv_g, t_g = handles[1]
    ga, gb = t_g.clone(), torch.empty_like(t_g)
    lg1, lg2 = torch.empty(B, V, device="cuda"), torch.empty(B, V, device="cuda")
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        kv_g.decode(ga, gb, lg1)
        kv_g.decode(gb, ga, lg2)
    kv_g.sync()  # capture ran no kernel: the device lengths are those after prefill
    assert kv_g.lengths() == [n + s for n, s in zip(n_v, s_text)]
    for k in range(4):
        graph.replay()
        torch.cuda.synchronize()
        scratch = torch.randn(1 << 16, device="cuda").sum()  # eager work between replays
        torch.cuda.synchronize()
        assert torch.isfinite(scratch)
        assert torch.equal(gb.cpu(), ref_tok[2 * k]), k
        assert torch.equal(ga.cpu(), ref_tok[2 * k + 1]), k
        assert torch.equal(lg1.cpu(), ref_log[2 * k]), k
        assert torch.equal(lg2.cpu(), ref_log[2 * k + 1]), k
        check_oracle(2 * k, lg1.cpu(), gb.cpu())
        check_oracle(2 * k + 1, lg2.cpu(), ga.cpu())
    assert near <= 1
    kv_g.sync()
    assert kv_g.lengths() == kv_e.lengths() == [n + s + 8 for n, s in zip(n_v, s_text)]
    for kv, _ in handles:
        kv.close()
    pair.gpu.close()


@pytest.mark.parametrize("case", ["b1_splits", "b40"])
def test_repeat_runs_are_bit_identical(case):
    """Determinism: the same prefills and decode steps on two fresh caches give
    bit-identical tokens, logits and K/V rows (no floating-point atomics; every
    reduction in a fixed order): one request long enough for split attention
    merged in the O projection's prologue, and 40 requests (K-split LDS GEMMs,
    split attention and the combine kernel)."""
    import paper_2603_12707_amd as hs
    if case == "b1_splits":
        cfg = small_cfg(dtype="f16")
        n_v, s_text = [900], [20]
    else:
        cfg = small_cfg(dtype="bf16", n_heads=8, n_kv_heads=2, head_dim=64)
        n_v, s_text = [(37 * b) % 300 for b in range(40)], [1 + (5 * b) % 9 for b in range(40)]
    B, steps = len(n_v), 3
    caps = [n + s + steps for n, s in zip(n_v, s_text)]
    pair = Pair(cfg, max_batch=B, max_ctx=max(caps))
    runs = []
    for _ in range(2):
        kv = hs.KVCache(pair.gpu, n_v, caps)
        first = torch.empty(B, dtype=torch.int32, device="cuda")
        for r in range(B):
            emb, ids, _ = pair.request_inputs(r, n_v[r], s_text[r])
            kv.prefill(r, emb.cuda() if n_v[r] else None, ids.cuda(), first_token=first[r:r + 1])
        tin, tout = first.clone(), torch.empty_like(first)
        lg = torch.empty(B, cfg["vocab"], device="cuda")
        out = [first.cpu()]
        for _ in range(steps):
            kv.decode(tin, tout, lg)
            out += [tout.cpu().clone(), lg.cpu().clone()]
            tin, tout = tout, tin
        n = kv.lengths()[B - 1]
        rows = torch.empty(n, cfg["head_dim"], dtype=torch.float16 if cfg["dtype"] == "f16" else torch.bfloat16)
        kv.read(B - 1, cfg["n_layers"] - 1, 1, cfg["n_kv_heads"] - 1, 0, n, rows)
        out.append(rows)
        runs.append(out)
        kv.close()
    for a, b in zip(*runs):
        assert torch.equal(a, b)
    pair.gpu.close()
