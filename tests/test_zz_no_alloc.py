"""hs_decode_step_static: the decode step with its scratch in the library's
static device array, called through the C ABI, against hs_decode_step on
identical caches.  Tokens, logits and the residual stream after the last
layer must be bit-equal (same kernels, same arithmetic, other buffers), on
consecutive calls with different models and batches sharing the array:
first 20 requests (activations read in the packed layout, with an F that is
not a multiple of 128), then 3 requests (activations staged in LDS, logits
in the scratch).  A step whose scratch would not fit is refused before any
launch."""
from __future__ import annotations

import pytest
import torch

from helpers import Pair, small_cfg

pytestmark = pytest.mark.gpu


def _decode_static(kv, tin, tout, logits, hidden):
    kv.decode_static(tin, tout, logits, hidden)


def _prefilled_pair(pair, n_v, s_text, caps):
    """Two identical caches, every request prefilled; returns them and the first tokens."""
    import paper_2603_12707_amd as hs
    B = len(n_v)
    out = []
    for _ in range(2):
        kv = hs.KVCache(pair.gpu, n_v, caps)
        first = torch.empty(B, dtype=torch.int32, device="cuda")
        for r in range(B):
            emb, ids, pos = pair.request_inputs(r, n_v[r], s_text[r])
            kv.prefill(r, emb.cuda() if n_v[r] else None, ids.cuda(), None if pos is None else pos.cuda(),
                       first_token=first[r:r + 1])
        out.append((kv, first))
    torch.cuda.synchronize()
    return out


def _compare(cfg, n_v, s_text, n_steps, with_logits):
    B = len(n_v)
    caps = [n + s + n_steps + 2 for n, s in zip(n_v, s_text)]
    pair = Pair(cfg, max_batch=B, max_ctx=max(caps))
    (kv_a, ta), (kv_b, tb) = _prefilled_pair(pair, n_v, s_text, caps)
    assert torch.equal(ta, tb)
    V, d = cfg["vocab"], cfg["d_model"]
    la, lb = torch.empty(B, V, device="cuda"), torch.empty(B, V, device="cuda")
    ha, hb = torch.empty(B, d, device="cuda"), torch.empty(B, d, device="cuda")
    oa, ob = torch.empty_like(ta), torch.empty_like(tb)
    for step in range(n_steps):
        kv_a.decode(ta, oa, la, ha)
        _decode_static(kv_b, tb, ob, lb if with_logits else None, hb)
        torch.cuda.synchronize()
        assert torch.equal(oa, ob), step
        assert torch.equal(ha, hb), step
        if with_logits:
            assert torch.equal(la, lb), step
        ta, oa = oa, ta
        tb, ob = ob, tb
    assert kv_a.lengths() == kv_b.lengths()
    assert pair.gpu.status() == 0
    kv_a.close()
    kv_b.close()
    pair.gpu.close()


def test_static_scratch_step_equals_decode_step_on_consecutive_calls():
    # a first user of the array with another model (fp16, MHA)
    _compare(small_cfg(n_layers=1, dtype="f16", seed=9), [7, 0, 12], [3, 9, 4], 2, True)
    # 20 requests: packed activations, F = 1000 (k-blocks past K), GQA-2, bf16
    cfg = small_cfg(n_layers=2, n_heads=6, n_kv_heads=3, ffn_dim=1000, dtype="bf16")
    _compare(cfg, [(7 * b) % 23 for b in range(20)], [2 + b % 5 for b in range(20)], 3, True)
    # then a smaller input: 3 requests, logits kept in the scratch
    _compare(cfg, [30, 0, 11], [4, 20, 1], 3, False)


def test_static_scratch_step_refuses_a_step_that_does_not_fit():
    import paper_2603_12707_amd as hs
    cfg = small_cfg(n_layers=1, d_model=64, n_heads=1, n_kv_heads=1, head_dim=64, ffn_dim=128, vocab=300_000,
                    dtype="bf16")
    B = 64  # B x vocab fp32 logits = 76.8 MB > the 64 MiB array
    pair = Pair(cfg, max_batch=B, max_ctx=8)
    kv = hs.KVCache(pair.gpu, [0] * B, [8] * B)
    tin = torch.zeros(B, dtype=torch.int32, device="cuda")
    tout = torch.zeros(B, dtype=torch.int32, device="cuda")
    with pytest.raises(hs.HsError) as e:
        _decode_static(kv, tin, tout, None, None)
    assert e.value.code == hs.HS_E_INVALID and "scratch" in str(e.value)
    # with a caller logits buffer it fits; the requests are not prefilled
    logits = torch.empty(B, cfg["vocab"], device="cuda")
    with pytest.raises(hs.HsError) as e:
        _decode_static(kv, tin, tout, logits, None)
    assert e.value.code == hs.HS_E_STATE
    assert kv.lengths() == [0] * B
    kv.close()
    pair.gpu.close()
