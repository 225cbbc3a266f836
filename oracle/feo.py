"""ctypes wrapper of the C oracle (test infrastructure only).

Marshals numpy arrays (as made by fe_synth) into the oracle's C calls.  No
arithmetic of the drafter is done here.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict, Optional, Sequence

import numpy as np

from . import build as _build

_lib = None


class FeoConfig(C.Structure):
    _fields_ = [("hidden", C.c_int32), ("n_q_heads", C.c_int32), ("n_kv_heads", C.c_int32),
                ("head_dim", C.c_int32), ("intermediate", C.c_int32), ("n_layers", C.c_int32),
                ("draft_vocab", C.c_int32), ("target_vocab", C.c_int32),
                ("n_feat_levels", C.c_int32), ("dtype", C.c_int32), ("cascade_ctx", C.c_int32),
                ("rope_theta", C.c_double), ("rms_eps", C.c_double)]


class FeoLayer(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm",
                                          "w_gate", "w_up", "w_down")]


class FeoWeights(C.Structure):
    _fields_ = [("w_fuse", C.c_void_p), ("w_in", C.c_void_p), ("embed", C.c_void_p),
                ("final_norm", C.c_void_p), ("lm_head", C.c_void_p),
                ("d2t", C.POINTER(C.c_int32)), ("layers", C.POINTER(FeoLayer))]


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        L = C.CDLL(_build.LIB)
        L.feo_draft_forward.restype = C.c_int
        L.feo_draft_sample.restype = C.c_int
        L.feo_build_tree.restype = C.c_int
        L.feo_accept_greedy.restype = C.c_int
        L.feo_kv_update.restype = C.c_int
        L.feo_kv_update_self.restype = C.c_int
        L.feo_accept_sample.restype = C.c_int
        L.feo_get_threads.restype = C.c_int
        _lib = L
    return _lib


def set_threads(n: int) -> None:
    lib().feo_set_threads(int(n))


def get_threads() -> int:
    return int(lib().feo_get_threads())


def _p(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(C.c_void_p)


def _pd(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"] and a.dtype == np.float64
    return a.ctypes.data_as(C.POINTER(C.c_double))


def _pi(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"] and a.dtype == np.int32
    return a.ctypes.data_as(C.POINTER(C.c_int32))


def make_config(cfg) -> FeoConfig:
    return FeoConfig(cfg.hidden, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.intermediate,
                     cfg.n_layers, cfg.draft_vocab, cfg.target_vocab, cfg.n_feat_levels,
                     1 if cfg.dtype == "bf16" else 0,
                     {"cascade": 0, "self": 1, "parallel": 2}[cfg.cascade_ctx],
                     float(cfg.rope_theta), float(cfg.rms_eps))


def rmsnorm(x: np.ndarray, gamma: np.ndarray, dtype: str, eps: float) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float64)
    y = np.empty_like(x)
    lib().feo_rmsnorm(_pd(x), _p(np.ascontiguousarray(gamma)), C.c_int32(1 if dtype == "bf16" else 0),
                      C.c_int32(x.size), C.c_double(eps), _pd(y))
    return y


def rope(v: np.ndarray, pos: int, theta: float) -> np.ndarray:
    y = np.array(v, dtype=np.float64, copy=True)
    lib().feo_rope(_pd(y), C.c_int32(y.size), C.c_int64(pos), C.c_double(theta))
    return y


def attend(q: np.ndarray, keys: np.ndarray, vals: np.ndarray) -> np.ndarray:
    q = np.ascontiguousarray(q, dtype=np.float64)
    keys = np.ascontiguousarray(keys, dtype=np.float64)
    vals = np.ascontiguousarray(vals, dtype=np.float64)
    L, D = keys.shape if keys.ndim == 2 else (0, q.size)
    out = np.empty(q.size, dtype=np.float64)
    lib().feo_attend(_pd(q), _pd(keys), _pd(vals), C.c_int32(L), C.c_int32(D), C.c_int64(D),
                     _pd(out))
    return out


def _weights(w, N):
    """FeoWeights pointing into the numpy arrays of w (plus what must stay alive)."""
    layers = (FeoLayer * N)()
    for i, lw in enumerate(w.layers):
        for f in FeoLayer._fields_:
            setattr(layers[i], f[0], _p(getattr(lw, f[0])))
    d2t = np.ascontiguousarray(w.d2t, dtype=np.int32)
    W = FeoWeights(_p(w.w_fuse), _p(w.w_in), _p(w.embed), _p(w.final_norm), _p(w.lm_head),
                   _pi(d2t), C.cast(layers, C.POINTER(FeoLayer)))
    return W, (layers, d2t)


def draft_forward(cfg, w, inp, topk: Optional[int] = None, want_logits: bool = True,
                  batch_index: Optional[Sequence[int]] = None, temperature: float = 1.0,
                  uniforms: Optional[np.ndarray] = None) -> Dict[str, np.ndarray]:
    """Run the oracle pass.  `batch_index` restricts it to some sequences of the
    batch (sequences are independent), keeping the given order.  With
    `uniforms` [B, N, V] (float32 in (0, 1)) the candidates are sampled at
    `temperature` (see feo_draft_sample in fe_oracle.h)."""
    k = cfg.topk if topk is None else int(topk)
    B_all = len(inp.prefix_lens)
    idx = list(range(B_all)) if batch_index is None else [int(i) for i in batch_index]
    cu = inp.cu_prefix
    feats = np.ascontiguousarray(inp.features[idx])
    toks = np.ascontiguousarray(inp.next_tokens[idx], dtype=np.int32)
    plens = np.ascontiguousarray(inp.prefix_lens[idx], dtype=np.int32)
    # gather the selected sequences' caches into packed arrays
    if idx == list(range(B_all)):
        kc = [np.ascontiguousarray(a) for a in inp.kcache]
        vc = [np.ascontiguousarray(a) for a in inp.vcache]
    else:
        kc = [np.ascontiguousarray(np.concatenate([a[cu[i]:cu[i + 1]] for i in idx])) for a in inp.kcache]
        vc = [np.ascontiguousarray(np.concatenate([a[cu[i]:cu[i + 1]] for i in idx])) for a in inp.vcache]
    B, N, d, V = len(idx), cfg.n_layers, cfg.hidden, cfg.draft_vocab
    W, _keep = _weights(w, N)
    kp = (C.c_void_p * N)(*[a.ctypes.data for a in kc])
    vp = (C.c_void_p * N)(*[a.ctypes.data for a in vc])
    hidden = np.zeros((B, N + 1, d), dtype=np.float64)
    logits = np.zeros((B, N, V), dtype=np.float64) if want_logits else None
    tdraft = np.zeros((B, N, k), dtype=np.int32)
    tids = np.zeros((B, N, k), dtype=np.int32)
    tprob = np.zeros((B, N, k), dtype=np.float64)
    cfgc = make_config(cfg)
    u = None
    if uniforms is not None:
        u = np.ascontiguousarray(np.asarray(uniforms, dtype=np.float32)[idx])
        assert u.shape == (B, N, V), u.shape
    rc = lib().feo_draft_sample(C.byref(cfgc), C.byref(W), C.c_int32(B), _p(feats), _pi(toks),
                                kp, vp, _pi(plens), C.c_int32(k), C.c_double(temperature),
                                _p(u) if u is not None else None, _pd(hidden),
                                _pd(logits) if logits is not None else None,
                                _pi(tdraft), _pi(tids), _pd(tprob))
    if rc != 0:
        raise ValueError("oracle draft_forward rejected its arguments")
    out = dict(hidden=hidden, topk_draft=tdraft, topk_ids=tids, topk_probs=tprob)
    if logits is not None:
        out["logits"] = logits
    return out


def build_tree(n_layers: int, topk: int, root_tokens: np.ndarray, topk_ids: np.ndarray,
               prefix_lens: np.ndarray) -> Dict[str, np.ndarray]:
    root_tokens = np.ascontiguousarray(root_tokens, dtype=np.int32)
    topk_ids = np.ascontiguousarray(topk_ids, dtype=np.int32)
    prefix_lens = np.ascontiguousarray(prefix_lens, dtype=np.int32)
    B, N, k = len(root_tokens), int(n_layers), int(topk)
    T, NL = 1 + N * k, N * (k - 1) + 1
    out = dict(tokens=np.zeros((B, T), np.int32), parents=np.zeros((B, T), np.int32),
               depth=np.zeros((B, T), np.int32), positions=np.zeros((B, T), np.int32),
               mask=np.zeros((B, T, T), np.uint8), retrieve=np.zeros((B, NL, N + 1), np.int32))
    rc = lib().feo_build_tree(C.c_int32(B), C.c_int32(N), C.c_int32(k), _pi(root_tokens),
                              _pi(topk_ids), _pi(prefix_lens), _pi(out["tokens"]),
                              _pi(out["parents"]), _pi(out["depth"]), _pi(out["positions"]),
                              _p(out["mask"]), _pi(out["retrieve"]))
    if rc != 0:
        raise ValueError("oracle build_tree rejected its arguments")
    return out


def accept_greedy(n_layers: int, topk: int, tokens: np.ndarray, retrieve: np.ndarray,
                  target_next: np.ndarray) -> Dict[str, np.ndarray]:
    """Greedy acceptance of one cycle (Section 2.4, temperature 0): see
    feo_accept_greedy in fe_oracle.h."""
    tokens = np.ascontiguousarray(tokens, dtype=np.int32)
    retrieve = np.ascontiguousarray(retrieve, dtype=np.int32)
    target_next = np.ascontiguousarray(target_next, dtype=np.int32)
    B, N = tokens.shape[0], int(n_layers)
    out = dict(accept_len=np.zeros(B, np.int32), accept_path=np.zeros(B, np.int32),
               accepted=np.zeros((B, N + 1), np.int32))
    rc = lib().feo_accept_greedy(C.c_int32(B), C.c_int32(N), C.c_int32(int(topk)), _pi(tokens),
                                 _pi(retrieve), _pi(target_next), _pi(out["accept_len"]),
                                 _pi(out["accept_path"]), _pi(out["accepted"]))
    if rc != 0:
        raise ValueError("oracle accept_greedy rejected its arguments")
    return out


def kv_update(cfg, w, features: np.ndarray, tokens: np.ndarray, positions: np.ndarray):
    """Per-layer cache rows of verified positions (see feo_kv_update in
    fe_oracle.h).  features [M, n_feat_levels*d] in storage precision, tokens
    and positions [M].  Returns (k, v): lists over layers of [M, H_kv, D]
    float64, keys rotated."""
    features = np.ascontiguousarray(features)
    tokens = np.ascontiguousarray(tokens, dtype=np.int32)
    positions = np.ascontiguousarray(positions, dtype=np.int32)
    M, N = len(tokens), cfg.n_layers
    assert features.shape[0] == M and len(positions) == M
    W, _keep = _weights(w, N)
    ks = [np.zeros((M, cfg.n_kv_heads, cfg.head_dim)) for _ in range(N)]
    vs = [np.zeros((M, cfg.n_kv_heads, cfg.head_dim)) for _ in range(N)]
    kp = (C.POINTER(C.c_double) * N)(*[_pd(a) for a in ks])
    vp = (C.POINTER(C.c_double) * N)(*[_pd(a) for a in vs])
    cfgc = make_config(cfg)
    rc = lib().feo_kv_update(C.byref(cfgc), C.byref(W), C.c_int32(M), _p(features), _pi(tokens),
                             _pi(positions), kp, vp)
    if rc != 0:
        raise ValueError("oracle kv_update rejected its arguments")
    return ks, vs


def philox4x64_10(counter, key) -> np.ndarray:
    """One Philox4x64-10 block (see feo_philox4x64_10)."""
    c = np.ascontiguousarray(counter, dtype=np.uint64)
    k = np.ascontiguousarray(key, dtype=np.uint64)
    out = np.zeros(4, np.uint64)
    assert c.shape == (4,) and k.shape == (2,)
    lib().feo_philox4x64_10(C.c_void_p(c.ctypes.data), C.c_void_p(k.ctypes.data),
                            C.c_void_p(out.ctypes.data))
    return out


def philox_uniforms(seed: int, offset: int, first: int, n: int) -> np.ndarray:
    """float32 uniforms first .. first+n-1 of the draw stream (seed, offset)
    (see feo_philox_uniforms)."""
    out = np.zeros(int(n), np.float32)
    lib().feo_philox_uniforms(C.c_uint64(int(seed)), C.c_uint64(int(offset)),
                              C.c_uint64(int(first)), C.c_int64(int(n)), _p(out))
    return out


def kv_update_self(cfg, w, features: np.ndarray, tokens: np.ndarray, positions: np.ndarray,
                   dst_rows: np.ndarray, kcache, vcache):
    """Per-layer cache rows under the self context (see feo_kv_update_self in
    fe_oracle.h): the pass run at each new position in turn.  kcache / vcache:
    per-layer [rows, H_kv, D] caches in storage precision (bf16 as uint16 bit
    patterns) holding the rows written before the call.  Returns (k, v): lists
    over layers of [M, H_kv, D] float64, keys rotated (the rows to write at
    dst_rows)."""
    features = np.ascontiguousarray(features)
    tokens = np.ascontiguousarray(tokens, dtype=np.int32)
    positions = np.ascontiguousarray(positions, dtype=np.int32)
    dst_rows = np.ascontiguousarray(dst_rows, dtype=np.int32)
    M, N = len(tokens), cfg.n_layers
    assert features.shape[0] == M and len(positions) == M and len(dst_rows) == M
    kc = [np.ascontiguousarray(a) for a in kcache]
    vc = [np.ascontiguousarray(a) for a in vcache]
    rows = kc[0].shape[0]
    sdt = np.uint16 if cfg.dtype == "bf16" else np.float32
    for a in kc + vc:
        assert a.dtype == sdt and a.shape == (rows, cfg.n_kv_heads, cfg.head_dim)
    W, _keep = _weights(w, N)
    ks = [np.zeros((M, cfg.n_kv_heads, cfg.head_dim)) for _ in range(N)]
    vs = [np.zeros((M, cfg.n_kv_heads, cfg.head_dim)) for _ in range(N)]
    kp = (C.POINTER(C.c_double) * N)(*[_pd(a) for a in ks])
    vp = (C.POINTER(C.c_double) * N)(*[_pd(a) for a in vs])
    kcp = (C.c_void_p * N)(*[a.ctypes.data for a in kc])
    vcp = (C.c_void_p * N)(*[a.ctypes.data for a in vc])
    cfgc = make_config(cfg)
    rc = lib().feo_kv_update_self(C.byref(cfgc), C.byref(W), C.c_int32(M), _p(features),
                                  _pi(tokens), _pi(positions), _pi(dst_rows), kcp, vcp,
                                  C.c_int64(rows), kp, vp)
    if rc != 0:
        raise ValueError("oracle kv_update_self rejected its arguments")
    return ks, vs


def accept_sample(n_layers: int, topk: int, tokens, retrieve, topk_draft, draft_logits,
                  temperature: float, d2t, target_probs, uniforms,
                  draft_uniforms=None) -> Dict[str, np.ndarray]:
    """Speculative-sampling acceptance of one cycle (see feo_accept_sample)."""
    tokens = np.ascontiguousarray(tokens, dtype=np.int32)
    retrieve = np.ascontiguousarray(retrieve, dtype=np.int32)
    topk_draft = np.ascontiguousarray(topk_draft, dtype=np.int32)
    draft_logits = np.ascontiguousarray(draft_logits, dtype=np.float32)
    target_probs = np.ascontiguousarray(target_probs, dtype=np.float32)
    uniforms = np.ascontiguousarray(uniforms, dtype=np.float32)
    B, N, k = tokens.shape[0], int(n_layers), int(topk)
    V, Vt = draft_logits.shape[-1], target_probs.shape[-1]
    assert draft_logits.shape == (B, N, V) and target_probs.shape == (B, 1 + N * k, Vt)
    assert uniforms.shape == (B, N * k + 1) and topk_draft.shape == (B, N, k)
    d = None if d2t is None else np.ascontiguousarray(d2t, dtype=np.int32)
    du = None
    if draft_uniforms is not None:
        du = np.ascontiguousarray(draft_uniforms, dtype=np.float32)
        assert du.shape == (B, N, V), du.shape
    out = dict(accept_len=np.zeros(B, np.int32), accept_path=np.zeros(B, np.int32),
               accepted=np.zeros((B, N + 1), np.int32), margin=np.zeros(B))
    rc = lib().feo_accept_sample(C.c_int32(B), C.c_int32(N), C.c_int32(k), C.c_int32(V),
                                 C.c_int32(Vt), _pi(tokens), _pi(retrieve), _pi(topk_draft),
                                 _p(draft_logits), C.c_double(temperature),
                                 _p(du) if du is not None else None,
                                 _pi(d) if d is not None else None, _p(target_probs),
                                 _p(uniforms), _pi(out["accept_len"]), _pi(out["accept_path"]),
                                 _pi(out["accepted"]), _pd(out["margin"]))
    if rc != 0:
        raise ValueError("oracle accept_sample rejected its arguments")
    return out
