"""ctypes binding of libfe.so (include/fe.h): argument marshalling only.

Every computation happens in the HIP kernels of the library; this module
mirrors the C structs and calls the C entry points by the same names.  It
raises if the library has not been built: there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
# FE_LIBRARY selects another build of the same library (the host-sanitizer
# build, for host-only test runs); the default is the in-tree libfe.so.
LIB_PATH = os.environ.get("FE_LIBRARY") or os.path.join(HERE, "libfe.so")

FE_OK, FE_E_INVALID, FE_E_UNSUPPORTED, FE_E_ALIGN, FE_E_WORKSPACE, FE_E_HIP = range(6)
FE_F32, FE_BF16 = 0, 1
FE_CTX_CASCADE, FE_CTX_SELF, FE_CTX_PARALLEL = 0, 1, 2
STATUS_NAMES = {0: "FE_OK", 1: "FE_E_INVALID", 2: "FE_E_UNSUPPORTED", 3: "FE_E_ALIGN",
                4: "FE_E_WORKSPACE", 5: "FE_E_HIP"}

# Every function include/fe.h declares.
EXPORTS = ("fe_workspace_bytes", "fe_drafter_create", "fe_draft_forward", "fe_draft_sample",
           "fe_draft_sample_seeded", "fe_build_tree",
           "fe_accept_greedy", "fe_accept_sample", "fe_accept_sample_seeded", "fe_kv_update_workspace_bytes", "fe_kv_update", "fe_kv_update_noalloc", "fe_set_graph_mode", "fe_set_attention_split", "fe_time_stage", "fe_set_pass_mode", "fe_pass_status",
           "fe_drafter_destroy", "fe_last_error", "fe_test_attn_split", "fe_test_philox_uniforms",
           "fe_test_attention", "fe_test_rmsnorm")
FE_STAGE = dict(fuse=0, input=1, qkv=2, attn=3, oproj=4, gateup=5, down=6, lmhead=7, pass_=8)


class fe_config(C.Structure):
    _fields_ = [("hidden", C.c_int32), ("n_q_heads", C.c_int32), ("n_kv_heads", C.c_int32),
                ("head_dim", C.c_int32), ("intermediate", C.c_int32), ("n_layers", C.c_int32),
                ("draft_vocab", C.c_int32), ("target_vocab", C.c_int32),
                ("n_feat_levels", C.c_int32), ("max_batch", C.c_int32), ("max_topk", C.c_int32),
                ("max_prefix", C.c_int32), ("rope_theta", C.c_float), ("rms_eps", C.c_float),
                ("dtype", C.c_int32), ("cascade_ctx", C.c_int32)]


class fe_layer_weights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm",
                                          "w_gate", "w_up", "w_down")]


class fe_weights(C.Structure):
    _fields_ = [("w_fuse", C.c_void_p), ("w_in", C.c_void_p), ("embed", C.c_void_p),
                ("final_norm", C.c_void_p), ("lm_head", C.c_void_p), ("d2t", C.c_void_p),
                ("layers", C.POINTER(fe_layer_weights))]


class fe_kv_view(C.Structure):
    _fields_ = [("k", C.POINTER(C.c_void_p)), ("v", C.POINTER(C.c_void_p)),
                ("cu_prefix", C.c_void_p), ("max_prefix", C.c_int32)]


class fe_kv_cache(C.Structure):
    _fields_ = [("k", C.POINTER(C.c_void_p)), ("v", C.POINTER(C.c_void_p)), ("rows", C.c_int64)]


class fe_tree_out(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("tokens", "parents", "depth", "positions", "mask",
                                          "retrieve")]


class fe_draft_out(C.Structure):
    _fields_ = [("topk_ids", C.c_void_p), ("topk_probs", C.c_void_p), ("topk_draft", C.c_void_p),
                ("logits", C.c_void_p), ("hidden", C.c_void_p),
                ("tree", C.POINTER(fe_tree_out))]


_lib = None


class FeError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


def lib() -> C.CDLL:
    """Load libfe.so; raise if it has not been built (no fallback exists)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2509_20416_amd.build`")
        L = C.CDLL(LIB_PATH)
        L.fe_workspace_bytes.restype = C.c_size_t
        L.fe_workspace_bytes.argtypes = [C.POINTER(fe_config)]
        L.fe_drafter_create.restype = C.c_int
        L.fe_drafter_create.argtypes = [C.POINTER(fe_config), C.POINTER(fe_weights), C.c_void_p,
                                        C.c_size_t, C.c_void_p, C.POINTER(C.c_void_p)]
        L.fe_draft_forward.restype = C.c_int
        L.fe_draft_forward.argtypes = [C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p,
                                       C.POINTER(fe_kv_view), C.c_int32,
                                       C.POINTER(fe_draft_out), C.c_void_p]
        L.fe_draft_sample.restype = C.c_int
        L.fe_draft_sample.argtypes = [C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p,
                                      C.POINTER(fe_kv_view), C.c_int32, C.c_float, C.c_void_p,
                                      C.POINTER(fe_draft_out), C.c_void_p]
        L.fe_draft_sample_seeded.restype = C.c_int
        L.fe_draft_sample_seeded.argtypes = L.fe_draft_sample.argtypes
        L.fe_accept_sample_seeded.restype = C.c_int
        L.fe_test_philox_uniforms.restype = C.c_int
        L.fe_test_philox_uniforms.argtypes = [C.c_void_p, C.c_uint64, C.c_int64, C.c_void_p,
                                              C.c_void_p]
        L.fe_test_attention.restype = C.c_int
        L.fe_test_attention.argtypes = [C.c_int32] * 5 + [C.c_void_p] * 3 + [C.c_int32] + \
            [C.c_void_p] * 3 + [C.c_int32, C.c_int32, C.c_double, C.c_int32, C.c_void_p, C.c_void_p]
        L.fe_test_rmsnorm.restype = C.c_int
        L.fe_test_rmsnorm.argtypes = [C.c_int32, C.c_void_p, C.c_int32, C.c_int32, C.c_void_p,
                                      C.c_float, C.c_void_p, C.c_void_p]
        L.fe_build_tree.restype = C.c_int
        L.fe_build_tree.argtypes = [C.c_void_p, C.c_int32, C.c_int32, C.c_void_p, C.c_void_p,
                                    C.c_void_p, C.POINTER(fe_tree_out), C.c_void_p]
        L.fe_accept_greedy.restype = C.c_int
        L.fe_accept_greedy.argtypes = [C.c_void_p, C.c_int32, C.c_int32] + [C.c_void_p] * 7
        L.fe_accept_sample.restype = C.c_int
        L.fe_accept_sample.argtypes = [C.c_void_p, C.c_int32, C.c_int32] + [C.c_void_p] * 4 + \
            [C.c_float] + [C.c_void_p] * 7
        L.fe_accept_sample_seeded.argtypes = L.fe_accept_sample.argtypes
        L.fe_kv_update_workspace_bytes.restype = C.c_size_t
        L.fe_kv_update_workspace_bytes.argtypes = [C.POINTER(fe_config), C.c_int32]
        L.fe_kv_update.restype = C.c_int
        L.fe_kv_update.argtypes = [C.c_void_p, C.c_int32] + [C.c_void_p] * 4 + \
            [C.POINTER(fe_kv_cache), C.c_void_p, C.c_size_t, C.c_void_p]
        L.fe_kv_update_noalloc.restype = C.c_int
        L.fe_kv_update_noalloc.argtypes = [C.c_void_p, C.c_int32] + [C.c_void_p] * 4 + \
            [C.POINTER(fe_kv_cache), C.c_void_p]
        L.fe_set_graph_mode.restype = C.c_int
        L.fe_set_graph_mode.argtypes = [C.c_void_p, C.c_int32]
        L.fe_set_pass_mode.restype = C.c_int
        L.fe_set_pass_mode.argtypes = [C.c_void_p, C.c_int32]
        L.fe_pass_status.restype = C.c_int
        L.fe_pass_status.argtypes = [C.c_void_p, C.c_void_p, C.POINTER(C.c_int32)]
        L.fe_set_attention_split.restype = C.c_int
        L.fe_set_attention_split.argtypes = [C.c_void_p, C.c_int32]
        L.fe_time_stage.restype = C.c_int
        L.fe_time_stage.argtypes = [C.c_void_p, C.c_int32, C.c_int32, C.c_void_p,
                                    C.POINTER(C.c_float), C.POINTER(C.c_int32)]
        L.fe_test_attn_split.restype = C.c_int
        L.fe_test_attn_split.argtypes = [C.c_void_p] + [C.c_int32] * 5 + [C.c_void_p, C.c_int32,
                                                                         C.c_void_p]
        L.fe_drafter_destroy.restype = None
        L.fe_drafter_destroy.argtypes = [C.c_void_p]
        L.fe_last_error.restype = C.c_char_p
        L.fe_last_error.argtypes = []
        _lib = L
    return _lib


def fe_last_error() -> str:
    return lib().fe_last_error().decode(errors="replace")


def check(status: int) -> None:
    if status != FE_OK:
        raise FeError(status, fe_last_error())


def fe_workspace_bytes(cfg: fe_config) -> int:
    return int(lib().fe_workspace_bytes(C.byref(cfg)))


def fe_drafter_create(cfg: fe_config, w: fe_weights, workspace: int, ws_bytes: int,
                      stream: int = 0) -> int:
    h = C.c_void_p()
    check(lib().fe_drafter_create(C.byref(cfg), C.byref(w), C.c_void_p(workspace),
                                  C.c_size_t(ws_bytes), C.c_void_p(stream), C.byref(h)))
    return h.value


def fe_draft_forward(h: int, batch: int, features: int, next_tokens: int, kv: fe_kv_view,
                     topk: int, out: fe_draft_out, stream: int) -> None:
    check(lib().fe_draft_forward(C.c_void_p(h), batch, C.c_void_p(features),
                                 C.c_void_p(next_tokens), C.byref(kv), topk, C.byref(out),
                                 C.c_void_p(stream)))


def fe_draft_sample(h: int, batch: int, features: int, next_tokens: int, kv: fe_kv_view,
                    topk: int, temperature: float, uniforms, out: fe_draft_out, stream: int) -> None:
    check(lib().fe_draft_sample(C.c_void_p(h), batch, C.c_void_p(features),
                                C.c_void_p(next_tokens), C.byref(kv), topk,
                                C.c_float(temperature), C.c_void_p(uniforms), C.byref(out),
                                C.c_void_p(stream)))


def fe_draft_sample_seeded(h: int, batch: int, features: int, next_tokens: int, kv: fe_kv_view,
                           topk: int, temperature: float, seed_offset: int, out: fe_draft_out,
                           stream: int) -> None:
    check(lib().fe_draft_sample_seeded(C.c_void_p(h), batch, C.c_void_p(features),
                                       C.c_void_p(next_tokens), C.byref(kv), topk,
                                       C.c_float(temperature), C.c_void_p(seed_offset),
                                       C.byref(out), C.c_void_p(stream)))


def fe_test_philox_uniforms(seed_offset: int, first: int, n: int, out: int, stream: int) -> None:
    check(lib().fe_test_philox_uniforms(C.c_void_p(seed_offset), C.c_uint64(int(first)),
                                        C.c_int64(int(n)), C.c_void_p(out), C.c_void_p(stream)))


def fe_build_tree(h: int, batch: int, topk: int, root_tokens: int, topk_ids: int,
                  prefix_lens: int, out: fe_tree_out, stream: int) -> None:
    check(lib().fe_build_tree(C.c_void_p(h), batch, topk, C.c_void_p(root_tokens),
                              C.c_void_p(topk_ids), C.c_void_p(prefix_lens), C.byref(out),
                              C.c_void_p(stream)))


def fe_accept_greedy(h: int, batch: int, topk: int, tokens: int, retrieve: int, target_next: int,
                     accept_len: int, accept_path: int, accepted: int, stream: int) -> None:
    check(lib().fe_accept_greedy(C.c_void_p(h), batch, topk, C.c_void_p(tokens),
                                 C.c_void_p(retrieve), C.c_void_p(target_next),
                                 C.c_void_p(accept_len), C.c_void_p(accept_path),
                                 C.c_void_p(accepted), C.c_void_p(stream)))


def fe_accept_sample(h: int, batch: int, topk: int, tokens: int, retrieve: int, topk_draft: int,
                     draft_logits: int, temperature: float, draft_uniforms, target_probs: int,
                     uniforms: int, accept_len: int, accept_path: int, accepted: int,
                     stream: int) -> None:
    check(lib().fe_accept_sample(C.c_void_p(h), batch, topk, C.c_void_p(tokens),
                                 C.c_void_p(retrieve), C.c_void_p(topk_draft),
                                 C.c_void_p(draft_logits), C.c_float(temperature),
                                 C.c_void_p(draft_uniforms), C.c_void_p(target_probs),
                                 C.c_void_p(uniforms), C.c_void_p(accept_len),
                                 C.c_void_p(accept_path), C.c_void_p(accepted),
                                 C.c_void_p(stream)))


def fe_kv_update_workspace_bytes(cfg: fe_config, chunk_rows: int) -> int:
    return int(lib().fe_kv_update_workspace_bytes(C.byref(cfg), int(chunk_rows)))


def fe_kv_update(h: int, n_rows: int, features: int, tokens: int, positions: int, dst_rows: int,
                 cache: fe_kv_cache, workspace: int, ws_bytes: int, stream: int) -> None:
    check(lib().fe_kv_update(C.c_void_p(h), int(n_rows), C.c_void_p(features),
                             C.c_void_p(tokens), C.c_void_p(positions), C.c_void_p(dst_rows),
                             C.byref(cache), C.c_void_p(workspace), C.c_size_t(ws_bytes),
                             C.c_void_p(stream)))


FE_KV_UPDATE_SCRATCH_BYTES = 8 << 20   # include/fe.h


def fe_kv_update_noalloc(h: int, n_rows: int, features: int, tokens: int, positions: int,
                         dst_rows: int, cache: fe_kv_cache, stream: int) -> None:
    check(lib().fe_kv_update_noalloc(C.c_void_p(h), int(n_rows), C.c_void_p(features),
                                     C.c_void_p(tokens), C.c_void_p(positions),
                                     C.c_void_p(dst_rows), C.byref(cache), C.c_void_p(stream)))


def fe_set_graph_mode(h: int, on: bool) -> None:
    check(lib().fe_set_graph_mode(C.c_void_p(h), 1 if on else 0))


def fe_set_pass_mode(h: int, mode: int) -> None:
    check(lib().fe_set_pass_mode(C.c_void_p(h), int(mode)))


def fe_pass_status(h: int, stream: int) -> int:
    v = C.c_int32()
    check(lib().fe_pass_status(C.c_void_p(h), C.c_void_p(stream), C.byref(v)))
    return int(v.value)


def fe_set_attention_split(h: int, chunks_per_workgroup: int) -> None:
    check(lib().fe_set_attention_split(C.c_void_p(h), int(chunks_per_workgroup)))


def fe_time_stage(h: int, stage: int, repeats: int, stream: int):
    """Mean duration (ms) of one launch of `stage` and launches per pass."""
    ms = C.c_float()
    n = C.c_int32()
    check(lib().fe_time_stage(C.c_void_p(h), int(stage), int(repeats), C.c_void_p(stream),
                              C.byref(ms), C.byref(n)))
    return float(ms.value), int(n.value)


def fe_drafter_destroy(h: int) -> None:
    lib().fe_drafter_destroy(C.c_void_p(h))


def fe_test_attn_split(prefix_lens, ncols: int, nch_ld: int, pmax: int, waves: int):
    """Pieces [n, 7] (wave, sequence, column, first chunk, chunks, slot, pieces of
    the segment or 0) of the persistent attention's split, computed on the host."""
    import numpy as np
    pl = np.ascontiguousarray(prefix_lens, dtype=np.int32)
    n = C.c_int32()
    check(lib().fe_test_attn_split(pl.ctypes.data, len(pl), ncols, nch_ld, pmax, waves, None, 0,
                                   C.byref(n)))
    out = np.zeros((max(1, n.value), 7), np.int32)
    check(lib().fe_test_attn_split(pl.ctypes.data, len(pl), ncols, nch_ld, pmax, waves,
                                   out.ctypes.data, n.value, C.byref(n)))
    return out[:n.value]


def fe_accept_sample_seeded(h: int, batch: int, topk: int, tokens: int, retrieve: int,
                            topk_draft: int, draft_logits: int, temperature: float,
                            draft_seed_offset: int, target_probs: int, uniforms: int,
                            accept_len: int, accept_path: int, accepted: int, stream: int) -> None:
    check(lib().fe_accept_sample_seeded(C.c_void_p(h), batch, topk, C.c_void_p(tokens),
                                        C.c_void_p(retrieve), C.c_void_p(topk_draft),
                                        C.c_void_p(draft_logits), C.c_float(temperature),
                                        C.c_void_p(draft_seed_offset), C.c_void_p(target_probs),
                                        C.c_void_p(uniforms), C.c_void_p(accept_len),
                                        C.c_void_p(accept_path), C.c_void_p(accepted),
                                        C.c_void_p(stream)))


def fe_test_attention(dtype: int, batch: int, n_q_heads: int, n_kv_heads: int, head_dim: int,
                      k_cache: int, v_cache: int, cu_prefix: int, max_prefix: int, q: int,
                      knew: int, vnew: int, nctx: int, cascade: int, rope_theta: float,
                      chunks_per_workgroup: int, out: int, stream: int) -> None:
    check(lib().fe_test_attention(dtype, batch, n_q_heads, n_kv_heads, head_dim,
                                  C.c_void_p(k_cache), C.c_void_p(v_cache), C.c_void_p(cu_prefix),
                                  max_prefix, C.c_void_p(q), C.c_void_p(knew), C.c_void_p(vnew),
                                  nctx, cascade, float(rope_theta), chunks_per_workgroup,
                                  C.c_void_p(out), C.c_void_p(stream)))


def fe_test_rmsnorm(dtype: int, x: int, rows: int, d: int, gamma: int, eps: float, out: int,
                    stream: int) -> None:
    check(lib().fe_test_rmsnorm(dtype, C.c_void_p(x), rows, d, C.c_void_p(gamma), C.c_float(eps),
                                C.c_void_p(out), C.c_void_p(stream)))
