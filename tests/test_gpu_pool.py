"""Block-granular KV pool (hs_kv_pool_create / hs_kv_admit / hs_kv_release):
parity with the oracle across block boundaries, continuous batching (a slot
released and refilled between decode steps), bit-identical layer-0 cache rows
against a contiguous cache, graph replays that take blocks on the device, and
the capacity checks."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from helpers import LOGIT_TOL, Pair, rel_err, small_cfg, token_ok

pytestmark = pytest.mark.gpu

BT = 256  # positions per block


class PoolRun:
    """A pooled cache on the GPU and one oracle sequence per live slot."""

    def __init__(self, cfg, slots, n_blocks, max_ctx=512):
        import paper_2603_12707_amd as hs
        self.cfg = cfg
        self.pair = Pair(cfg, max_batch=slots, max_ctx=max_ctx)
        self.pool = hs.KVPool(self.pair.gpu, slots, BT, n_blocks)
        self.slots = slots
        self.seqs = {}   # slot -> oracle sequence
        self.next = {}   # slot -> token to feed next (the oracle's)
        self.near = 0

    def admit_and_prefill(self, entries, key):
        """entries: [(slot, n_v, s_text, cap)] prefilled in one batch call;
        `key` salts the request inputs."""
        V = self.cfg["vocab"]
        inputs = []
        for slot, n_v, s_text, cap in entries:
            self.pool.admit(slot, n_v, cap)
            emb, ids, pos = self.pair.request_inputs(key + slot, n_v, s_text)
            s = self.pair.ora.new_seq(cap)
            ref = s.prefill(emb if n_v else None, ids, pos)
            self.seqs[slot] = s
            inputs.append((emb, ids, pos, ref))
        embs = [e for e, _, _, _ in inputs if e.shape[0]]
        idss = [i for _, i, _, _ in inputs if i.shape[0]]
        lg = torch.empty(len(entries), V, dtype=torch.float32, device="cuda")
        toks = self.pool.prefill_batch([e[0] for e in entries], torch.cat(embs).cuda() if embs else None,
                                       torch.cat(idss).cuda() if idss else None, [e[2] for e in entries],
                                       last_logits=lg)
        torch.cuda.synchronize()
        for k, (slot, *_rest) in enumerate(entries):
            ref_logits, ref_tok = inputs[k][3]
            g = lg[k].cpu().numpy()
            assert rel_err(g, ref_logits) <= LOGIT_TOL, (slot, rel_err(g, ref_logits))
            ok, tie = token_ok(int(toks[k].item()), g, ref_logits)
            assert ok, (slot, int(toks[k].item()), ref_tok)
            self.near += tie
            self.next[slot] = ref_tok

    def release(self, slot):
        self.pool.release(slot)
        del self.seqs[slot]
        del self.next[slot]

    def decode(self, n_steps):
        V = self.cfg["vocab"]
        live = sorted(self.seqs)
        tin = torch.zeros(self.slots, dtype=torch.int32, device="cuda")
        tout = torch.full((self.slots,), -7, dtype=torch.int32, device="cuda")
        logits = torch.empty(len(live), V, dtype=torch.float32, device="cuda")
        for step in range(n_steps):
            tin.copy_(torch.tensor([self.next.get(s, 0) for s in range(self.slots)], dtype=torch.int32))
            self.pool.decode(tin, tout, logits)
            torch.cuda.synchronize()
            g_tok, g_log = tout.cpu().tolist(), logits.cpu().numpy()
            for k, slot in enumerate(live):  # logits rows follow slot order
                r_log, _, r_tok = self.seqs[slot].decode(self.next[slot])
                assert rel_err(g_log[k], r_log) <= LOGIT_TOL, (step, slot, rel_err(g_log[k], r_log))
                ok, tie = token_ok(g_tok[slot], g_log[k], r_log)
                assert ok, (step, slot, g_tok[slot], r_tok)
                self.near += tie
                self.next[slot] = r_tok
            assert all(g_tok[s] == -7 for s in range(self.slots) if s not in self.seqs), g_tok


def _used(lengths):
    return sum((n + BT - 1) // BT for n in lengths)


def test_pool_parity_across_blocks_and_continuous_batching():
    """Three requests in slots 0, 2, 3 of five, contexts 254, 256 and 299
    positions (256-position blocks): the decode steps cross block
    boundaries.  Then slot 2 is released, a new request is admitted into it
    (reusing the freed blocks) and prefilled while the others wait, and all
    decode on."""
    cfg = small_cfg(n_layers=2, dtype="bf16")
    run = PoolRun(cfg, slots=5, n_blocks=16)
    assert run.pool.blocks() == (16, 16)
    run.admit_and_prefill([(3, 200, 99, 340), (0, 40, 214, 300), (2, 0, 256, 300)], key=0)
    assert run.pool.lengths() == [254, 0, 256, 299, 0]
    assert run.pool.blocks() == (16 - _used([254, 256, 299]), 16)
    run.decode(4)
    assert run.pool.lengths() == [258, 0, 260, 303, 0]
    assert run.pool.blocks() == (16 - _used([258, 260, 303]), 16)
    run.release(2)
    assert run.pool.blocks() == (16 - _used([258, 303]), 16)
    run.admit_and_prefill([(2, 17, 240, 300)], key=50)
    assert run.pool.lengths() == [258, 0, 257, 303, 0]
    run.decode(3)
    assert run.pool.lengths() == [261, 0, 260, 306, 0]
    assert run.pool.blocks() == (16 - _used([261, 260, 306]), 16)
    assert run.pair.gpu.status() == 0
    assert run.near <= 2


def test_pool_packed_activations_and_wide_prefill():
    """20 requests in 22 slots at d = 1024 (GQA-4 with bias, F = 1000): one
    prefill call packs their ~150 rows (gate/up and the LM head on the
    weight-stationary kernel), and the 20-column decode steps read packed
    activations while the q/k/v epilogue appends into the blocks."""
    cfg = small_cfg(n_layers=1, d_model=1024, n_heads=8, n_kv_heads=2, head_dim=128, ffn_dim=1000, dtype="bf16",
                    qkv_bias=1)
    run = PoolRun(cfg, slots=22, n_blocks=24, max_ctx=64)
    entries = [(s, (5 * s) % 11, 2 + s % 3, 24) for s in range(1, 21)]
    run.admit_and_prefill(entries, key=7)
    run.decode(3)
    assert run.pool.lengths() == [0] + [n + t + 3 for _, n, t, _ in entries] + [0]
    assert run.pair.gpu.status() == 0
    assert run.near <= 2


def test_pool_gqa7_mrope():
    """Pooled cache with 7 query heads per KV head (matrix-core decode
    attention reading the blocks batch by batch) and M-RoPE."""
    cfg = small_cfg(n_heads=14, n_kv_heads=2, head_dim=64, dtype="bf16", rope_kind=1, mrope_section=(8, 12, 12),
                    qkv_bias=1, rope_theta=1e6, rms_eps=1e-6)
    import paper_2603_12707_amd as hs
    pair = Pair(cfg, max_batch=3, max_ctx=400)
    pool = hs.KVPool(pair.gpu, 3, BT, 6)
    V = cfg["vocab"]
    lens, seqs, nxt = {0: (121, 134), 1: (60, 3)}, {}, {}
    embs, idss, poss = [], [], []
    for slot, (n_v, s_text) in lens.items():
        pool.admit(slot, n_v, 300)
        emb, ids, pos = pair.request_inputs(slot, n_v, s_text)
        seqs[slot] = pair.ora.new_seq(300)
        nxt[slot] = seqs[slot].prefill(emb, ids, pos)
        embs.append(emb)
        idss.append(ids)
        poss.append(pos)
    lg = torch.empty(2, V, dtype=torch.float32, device="cuda")
    toks = pool.prefill_batch([0, 1], torch.cat(embs).cuda(), torch.cat(idss).cuda(), [134, 3],
                              torch.cat(poss, dim=1).contiguous().cuda(), last_logits=lg)
    torch.cuda.synchronize()
    cur = {}
    for k, slot in enumerate([0, 1]):
        ref_logits, ref_tok = nxt[slot]
        assert rel_err(lg[k].cpu().numpy(), ref_logits) <= LOGIT_TOL
        cur[slot] = ref_tok
    tin = torch.zeros(3, dtype=torch.int32, device="cuda")
    tout = torch.zeros(3, dtype=torch.int32, device="cuda")
    logits = torch.empty(2, V, dtype=torch.float32, device="cuda")
    for step in range(6):
        tin.copy_(torch.tensor([cur[0], cur[1], 0], dtype=torch.int32))
        pool.decode(tin, tout, logits)
        torch.cuda.synchronize()
        for k, slot in enumerate([0, 1]):
            r_log, _, r_tok = seqs[slot].decode(cur[slot])
            assert rel_err(logits[k].cpu().numpy(), r_log) <= LOGIT_TOL, (step, slot)
            cur[slot] = r_tok
    assert pool.lengths() == [261, 69, 0]


def test_pool_layer0_rows_bit_identical_to_contiguous_cache():
    """The same requests, prefilled and decoded with the same tokens, in a
    contiguous cache and in a pool: the layer-0 K/V rows (which depend on
    each position's input alone) read back bit for bit equal, across the
    blocks the pool spread them over."""
    import paper_2603_12707_amd as hs
    cfg = small_cfg(n_layers=1, dtype="f16")
    shapes = [(200, 50), (0, 240), (250, 1)]  # contexts 250, 240, 251
    caps = [n + s + 30 for n, s in shapes]
    pair = Pair(cfg, max_batch=3, max_ctx=max(caps))
    kv = hs.KVCache(pair.gpu, [n for n, _ in shapes], caps)
    pool = hs.KVPool(pair.gpu, 3, BT, 6)
    for slot, (n_v, _) in enumerate(shapes):
        pool.admit(slot, n_v, caps[slot])
    inputs = [pair.request_inputs(r, n, s) for r, (n, s) in enumerate(shapes)]
    emb = torch.cat([e for e, _, _ in inputs if e.shape[0]]).cuda()
    ids = torch.cat([i for _, i, _ in inputs]).cuda()
    first_a = kv.prefill_batch([0, 1, 2], emb, ids, [s for _, s in shapes])
    first_b = pool.prefill_batch([0, 1, 2], emb, ids, [s for _, s in shapes])
    torch.cuda.synchronize()
    assert first_a.tolist() == first_b.tolist()
    tin = first_a.clone()
    ta, tb = torch.empty_like(tin), torch.empty_like(tin)
    for _ in range(20):  # every request crosses a block boundary
        kv.decode(tin, ta)
        pool.decode(tin, tb)
        tin = ta.clone()
    torch.cuda.synchronize()
    assert kv.lengths() == pool.lengths()
    hd = cfg["head_dim"]
    for r, n in enumerate(kv.lengths()):
        for sel in (0, 1):
            for h in range(cfg["n_kv_heads"]):
                a = torch.empty(n, hd, dtype=torch.float16)
                b = torch.empty(n, hd, dtype=torch.float16)
                kv.read(r, 0, sel, h, 0, n, a)
                pool.read(r, 0, sel, h, 0, n, b)
                assert torch.equal(a.view(torch.int16), b.view(torch.int16)), (r, sel, h)


def test_pool_graph_replays_take_blocks_on_the_device():
    """Two decode steps captured once, replayed four times: the requests
    cross block boundaries inside the replays, the caches, lengths and free
    blocks match an identical pool driven by eager calls bit for bit, and the
    replayed logits agree with the oracle fed the same tokens."""
    import paper_2603_12707_amd as hs
    cfg = small_cfg(n_layers=1, dtype="bf16")
    pair = Pair(cfg, max_batch=2, max_ctx=400)
    pools = [hs.KVPool(pair.gpu, 2, BT, 8) for _ in range(2)]
    shapes = [(20, 234), (0, 253)]  # contexts 254, 253: blocks end at 256
    inputs = [pair.request_inputs(r, n, s) for r, (n, s) in enumerate(shapes)]
    firsts = []
    for p in pools:
        for slot, (n_v, _) in enumerate(shapes):
            p.admit(slot, n_v, 300)
        firsts.append(p.prefill_batch([0, 1], inputs[0][0].cuda(), torch.cat([inputs[0][1], inputs[1][1]]).cuda(),
                                      [234, 253]))
    torch.cuda.synchronize()
    eager, graphed = pools
    ta, tb = firsts[0].clone(), torch.empty_like(firsts[0])
    ga, gb = firsts[1].clone(), torch.empty_like(firsts[1])
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    V = cfg["vocab"]
    lg1, lg2 = torch.empty(2, V, device="cuda"), torch.empty(2, V, device="cuda")
    with torch.cuda.stream(s):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            graphed.decode(ga, gb, lg1)
            graphed.decode(gb, ga, lg2)
    torch.cuda.current_stream().wait_stream(s)
    graphed.sync()
    assert graphed.lengths() == [254, 253]  # capture ran nothing
    # the oracle, fed the tokens each replayed step was fed
    seqs = []
    for r, (n_v, s_text) in enumerate(shapes):
        emb, ids, _ = inputs[r]
        seqs.append(pair.ora.new_seq(300))
        seqs[-1].prefill(emb if n_v else None, ids)
    near = 0

    def check_oracle(feed, g_log, g_tok):
        nonlocal near
        for r in range(2):
            r_log, _, _ = seqs[r].decode(feed[r])
            assert rel_err(g_log[r], r_log) <= LOGIT_TOL, (r, rel_err(g_log[r], r_log))
            ok, tie = token_ok(g_tok[r], g_log[r], r_log)
            assert ok, r
            near += tie
    for rep in range(4):
        feed0 = ga.tolist()
        g.replay()
        for _ in range(2):
            eager.decode(ta, tb)
            ta, tb = tb, ta
        torch.cuda.synchronize()
        assert ga.tolist() == ta.tolist(), rep
        check_oracle(feed0, lg1.cpu().numpy(), gb.tolist())
        check_oracle(gb.tolist(), lg2.cpu().numpy(), ga.tolist())
    assert near <= 1
    graphed.sync()
    assert graphed.lengths() == eager.lengths() == [262, 261]
    assert graphed.blocks() == eager.blocks() == (8 - 4, 8)
    hd = cfg["head_dim"]
    for r, n in enumerate(eager.lengths()):
        a = torch.empty(n, hd, dtype=torch.bfloat16)
        b = torch.empty(n, hd, dtype=torch.bfloat16)
        eager.read(r, 0, 1, 0, 0, n, a)
        graphed.read(r, 0, 1, 0, 0, n, b)
        assert torch.equal(a.view(torch.int16), b.view(torch.int16)), r


def test_pool_running_dry_inside_replays_is_flagged():
    """A pool with no spare block and a captured decode step replayed until
    request 0's next position needs a block that is not there: that step sets
    status bit 2, every kernel completes, request 0's outputs stay finite (its
    new position unstored and masked from attention), request 1, whose block
    suffices, keeps agreeing with the oracle fed the same tokens, and an eager
    step is then refused by the host-side check."""
    import paper_2603_12707_amd as hs
    cfg = small_cfg(n_layers=1, dtype="bf16")
    pair = Pair(cfg, max_batch=2, max_ctx=400)
    pool = hs.KVPool(pair.gpu, 2, BT, 2)  # one block each after prefill, none free
    shapes = [(20, 230), (0, 100)]  # contexts 250 and 100
    inputs = [pair.request_inputs(r, n, s) for r, (n, s) in enumerate(shapes)]
    for slot, (n_v, s_text) in enumerate(shapes):
        pool.admit(slot, n_v, 300)
    first = pool.prefill_batch([0, 1], inputs[0][0].cuda(), torch.cat([inputs[0][1], inputs[1][1]]).cuda(),
                               [230, 100])
    torch.cuda.synchronize()
    assert pool.blocks() == (0, 2)
    seq1 = pair.ora.new_seq(300)
    seq1.prefill(None, inputs[1][1])
    V = cfg["vocab"]
    ga, gb = first.clone(), torch.empty_like(first)
    lg1, lg2 = torch.empty(2, V, device="cuda"), torch.empty(2, V, device="cuda")
    st = torch.cuda.Stream()
    st.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(st):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=st):
            pool.decode(ga, gb, lg1)
            pool.decode(gb, ga, lg2)
    torch.cuda.current_stream().wait_stream(st)
    assert pair.gpu.status() == 0
    for rep in range(4):  # request 0 writes positions 250 + 2 rep and 251 + 2 rep
        feed0 = ga.tolist()
        g.replay()
        torch.cuda.synchronize()
        feed1 = gb.tolist()
        flags = pair.gpu.status()
        assert flags == (4 if rep == 3 else 0), (rep, flags)
        for feed, lg, out in ((feed0, lg1, feed1), (feed1, lg2, ga.tolist())):
            lg = lg.cpu().numpy()
            assert np.all(np.isfinite(lg))
            assert all(0 <= t < V for t in out)
            r_log, _, _ = seq1.decode(feed[1])
            assert rel_err(lg[1], r_log) <= LOGIT_TOL, (rep, rel_err(lg[1], r_log))
    pool.sync()
    assert pool.lengths() == [258, 108]
    with pytest.raises(hs.HsError):
        pool.decode(ga, gb)


def test_pool_capacity_and_admission_errors():
    import paper_2603_12707_amd as hs
    cfg = small_cfg(n_layers=1, dtype="bf16")
    pair = Pair(cfg, max_batch=3, max_ctx=1024)
    with pytest.raises(hs.HsError) as e:
        hs.KVPool(pair.gpu, 3, 384, 4)                # block size not a power of two
    assert e.value.code == hs.HS_E_INVALID
    with pytest.raises(hs.HsError) as e:
        hs.KVPool(pair.gpu, 3, 128, 4)                # below one batch of attention loads
    assert e.value.code == hs.HS_E_INVALID
    pool = hs.KVPool(pair.gpu, 3, BT, 3)
    ids = torch.randint(0, cfg["vocab"], (800,), dtype=torch.int32).cuda()
    pool.admit(0, 0, 900)
    with pytest.raises(hs.HsError) as e:
        pool.admit(0, 0, 10)                          # slot in use
    assert e.value.code == hs.HS_E_STATE
    with pytest.raises(hs.HsError) as e:
        pool.prefill(1, None, ids[:5])                # slot 1 holds no request
    assert e.value.code == hs.HS_E_STATE
    with pytest.raises(hs.HsError) as e:
        pool.prefill(0, None, ids)                    # 800 positions: 4 blocks > 3
    assert e.value.code == hs.HS_E_CAPACITY
    assert pool.lengths() == [0, 0, 0] and pool.blocks() == (3, 3)
    pool.prefill(0, None, ids[:512])                  # 2 blocks
    pool.admit(1, 0, 400)
    pool.prefill(1, None, ids[:256])                  # 1 block: the pool is full
    assert pool.blocks() == (0, 3)
    tin = torch.zeros(3, dtype=torch.int32, device="cuda")
    tout = torch.zeros(3, dtype=torch.int32, device="cuda")
    with pytest.raises(hs.HsError) as e:
        pool.decode(tin, tout)                        # both enter a new block
    assert e.value.code == hs.HS_E_CAPACITY
    assert pool.lengths() == [512, 256, 0]
    pool.release(1)
    assert pool.blocks() == (1, 3)
    pool.decode(tin, tout)                            # request 0 alone takes the free block
    assert pool.lengths() == [513, 0, 0] and pool.blocks() == (0, 3)
    assert pair.gpu.status() == 0


def test_serving_loop_handoff_pool_continuous_batching():
    """A small serving loop: ten requests arrive over time; the aligned batch
    handoff (B_align = 4, 100 ms timeout) releases them in batches; each
    batch is admitted into free slots of a pool and prefilled in one packed
    call; decode steps run over every live slot, and finished requests leave
    and free their slots for later ones.  Every prefill and step is checked
    against the oracle."""
    import paper_2603_12707_amd as hs
    cfg = small_cfg(n_layers=2, dtype="bf16")
    run = PoolRun(cfg, slots=6, n_blocks=12)  # six live requests of at most 2 blocks each
    rng = np.random.default_rng(7)
    reqs = [dict(n_v=int(rng.integers(0, 200)), s_text=int(rng.integers(1, 90)), n_dec=int(rng.integers(2, 6)),
                 t=float(10 * i + rng.integers(0, 15))) for i in range(10)]
    handoff = hs.Handoff(align=4, timeout_ms=100.0)
    slot_of, left, waiting, arrived, done = {}, {}, [], 0, 0
    now = 0.0
    while done < len(reqs):
        while arrived < len(reqs) and reqs[arrived]["t"] <= now:
            r = reqs[arrived]
            handoff.push(arrived, r["n_v"] + r["s_text"], now_ms=now)
            arrived += 1
        batch, _, _ = handoff.pop(now)
        waiting += batch
        free = [s for s in range(run.slots) if s not in run.seqs]
        admit = []
        while waiting and free:
            q, s = waiting.pop(0), free.pop(0)
            r = reqs[q]
            slot_of[s], left[s] = q, r["n_dec"]
            admit.append((s, r["n_v"], r["s_text"], r["n_v"] + r["s_text"] + r["n_dec"] + 1))
        if admit:
            run.admit_and_prefill(admit, key=1000 + int(now))
        if run.seqs:
            run.decode(1)
            for s in list(run.seqs):
                left[s] -= 1
                if left[s] == 0:
                    run.release(s)
                    done += 1
        now += 10.0
    assert handoff.pending() == 0 and not waiting
    assert run.pool.blocks() == (12, 12) and run.pool.lengths() == [0] * 6
    assert run.pair.gpu.status() == 0
    assert run.near <= 2
