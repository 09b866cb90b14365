"""MI355X (gfx950) language-decode engine for modality-disaggregated MLLM
serving (arXiv 2603.12707): a C-ABI HIP library (libhs.so, include/hs.h) and
its thin Python binding."""
from .hs import (EXPORTS, HS_BF16, HS_E_BUFFER, HS_E_CAPACITY, HS_E_DEVICE, HS_E_INVALID, HS_E_STATE, HS_F16,
                 HS_F32, HS_OK, HS_ROPE_1D, HS_ROPE_M3, Handoff, HsError, KVCache, KVPool, Model, hs_kv_bytes, hs_packed_bytes, lib,
                 pack_matrix, pack_weight, pack_weights, stream_read)

lib()  # the HIP library must be present: there is no other implementation

__all__ = ["EXPORTS", "Handoff", "HsError", "KVCache", "KVPool", "Model", "hs_kv_bytes", "hs_packed_bytes", "lib", "pack_matrix",
           "pack_weight", "pack_weights", "stream_read", "HS_OK", "HS_E_INVALID", "HS_E_CAPACITY",
           "HS_E_BUFFER", "HS_E_STATE", "HS_E_DEVICE", "HS_F32", "HS_F16", "HS_BF16", "HS_ROPE_1D", "HS_ROPE_M3"]
