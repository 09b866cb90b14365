"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every symbol include/hs.h declares, computes Eq. 1 / the embedding size
exactly, and rejects bad arguments before touching a device."""
import ctypes
import json
import os
import re

import pytest

import paper_2603_12707_amd as hs
from paper_2603_12707_amd import hs as H
from workload import configs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    with open(os.path.join(ROOT, "include", "hs.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(hs_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    lib = hs.lib()
    declared = _declared()
    assert set(declared) == set(H.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name


def test_kv_bytes_matches_paper_tables():
    with open(os.path.join(ROOT, "tests", "golden", "transfer_sizes.json")) as f:
        rows = json.load(f)["rows"]
    for row in rows:
        cfg = dict(configs.LLAVA7B, n_layers=row["L"], n_heads=row["n_h"], n_kv_heads=row["n_kv"],
                   head_dim=row["d_h"], d_model=row["d"])
        kv, emb = hs.hs_kv_bytes(cfg, row["n_v"], row["s_text"])
        if "kv_bytes" in row:
            assert kv == row["kv_bytes"]
        if "kv_mib" in row:
            assert round(kv / 2**20) == row["kv_mib"]
        if "emb_mib" in row:
            assert abs(emb / 2**20 - row["emb_mib"]) < 0.05 + 1e-9
        if "r_gqa" in row:
            assert round(kv / emb) == row["r_gqa"]


@pytest.mark.parametrize("name", list(configs.CONFIGS))
def test_kv_bytes_is_eq1(name):
    cfg = configs.get(name)
    b = configs.DTYPE_BYTES[cfg["dtype"]]
    for n_v, s_text in ((0, 1), (576, 64), (1280, 128), (1, 0)):
        kv, emb = hs.hs_kv_bytes(cfg, n_v, s_text)
        assert kv == 2 * cfg["n_layers"] * cfg["n_kv_heads"] * cfg["head_dim"] * (n_v + s_text) * b
        assert emb == n_v * cfg["d_model"] * b


def test_kv_bytes_errors():
    cfg = configs.get("tiny")
    with pytest.raises(hs.HsError) as e:
        hs.hs_kv_bytes(cfg, -1, 0)
    assert e.value.code == hs.HS_E_INVALID
    with pytest.raises(hs.HsError):
        hs.hs_kv_bytes(dict(cfg, n_layers=0), 1, 1)
    with pytest.raises(hs.HsError):  # 2^64 overflow is reported, not wrapped
        hs.hs_kv_bytes(dict(cfg, n_layers=2**30, n_kv_heads=2**30, head_dim=2**30), 2**40, 0)
    assert b"hs_kv_bytes" in hs.lib().hs_last_error()


def test_model_create_rejects_bad_config_on_host():
    lib = hs.lib()
    out = ctypes.c_void_p()
    w = H.hs_weights()
    for bad in (dict(head_dim=48), dict(n_heads=6, n_kv_heads=4), dict(rope_kind=1, mrope_section=(1, 1, 1)),
                dict(ffn_dim=690), dict(dtype="f16", d_model=260)):
        c = H.make_config(dict(configs.get("tiny"), **bad))
        rc = lib.hs_model_create(ctypes.byref(c), ctypes.byref(w), 1, 16, ctypes.byref(out))
        assert rc == hs.HS_E_INVALID, bad
    c = H.make_config(configs.get("tiny"))
    assert lib.hs_model_create(ctypes.byref(c), None, 1, 16, ctypes.byref(out)) == hs.HS_E_INVALID
    assert lib.hs_kv_alloc(None, 1, None, None, None, 0, ctypes.byref(out)) == hs.HS_E_INVALID
    assert lib.hs_decode_step(None, None, None, None, None, None, None) == hs.HS_E_INVALID
    assert lib.hs_kv_free(None) == hs.HS_E_INVALID
