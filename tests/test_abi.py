"""C-ABI checks that need no GPU: the library loads, exports every function
include/fe.h declares, sizes its workspace, and rejects invalid arguments on
the host before touching the device."""
import ctypes as C
import os
import re

import pytest

from fe_synth import configs as CF

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def fe():
    from paper_2509_20416_amd import fe as _fe
    _fe.lib()
    return _fe


def _cfg(fe, c=CF.LLAMA8B_BF16_B1, **kw):
    v = dict(hidden=c.hidden, n_q_heads=c.n_q_heads, n_kv_heads=c.n_kv_heads,
             head_dim=c.head_dim, intermediate=c.intermediate, n_layers=c.n_layers,
             draft_vocab=c.draft_vocab, target_vocab=c.target_vocab, n_feat_levels=3,
             max_batch=1, max_topk=c.topk, max_prefix=1024, rope_theta=c.rope_theta,
             rms_eps=1e-5, dtype=fe.FE_BF16, cascade_ctx=fe.FE_CTX_CASCADE)
    v.update(kw)
    return fe.fe_config(**v)


def test_exports_match_header(fe):
    hdr = open(os.path.join(ROOT, "include", "fe.h")).read()
    declared = set(re.findall(r"\b(fe_[a-z_]+)\s*\(", hdr))
    assert declared == set(fe.EXPORTS), declared
    for name in declared:
        assert hasattr(fe.lib(), name), name


def test_workspace_bytes(fe):
    n = fe.fe_workspace_bytes(_cfg(fe))
    assert 0 < n < (1 << 30)
    big = fe.fe_workspace_bytes(_cfg(fe, max_batch=32, n_layers=7, max_prefix=8192))
    assert big > n
    assert fe.fe_workspace_bytes(_cfg(fe, head_dim=96)) == 0
    assert "head_dim" in fe.fe_last_error()


@pytest.mark.parametrize("kw,status", [
    (dict(head_dim=96), "FE_E_UNSUPPORTED"), (dict(n_q_heads=30), "FE_E_INVALID"),
    (dict(dtype=7), "FE_E_INVALID"), (dict(cascade_ctx=3), "FE_E_INVALID"),
    (dict(max_topk=17), "FE_E_UNSUPPORTED"), (dict(n_layers=17), "FE_E_UNSUPPORTED"),
    (dict(hidden=4100), "FE_E_UNSUPPORTED"), (dict(hidden=8224), "FE_E_UNSUPPORTED"), (dict(max_batch=64, n_layers=5), "FE_E_UNSUPPORTED"),
    (dict(hidden=0), "FE_E_INVALID"), (dict(rope_theta=0.0), "FE_E_INVALID"),
])
def test_create_rejects_bad_config(fe, kw, status):
    cfg = _cfg(fe, **kw)
    w = fe.fe_weights()
    with pytest.raises(fe.FeError) as e:
        fe.fe_drafter_create(cfg, w, 0, 0)
    assert status in str(e.value)


def _fake_weights(fe, n_layers, base=1 << 20, misalign=None):
    """Plausible (never dereferenced) device addresses: validation only looks at them."""
    layers = (fe.fe_layer_weights * n_layers)()
    addr = [base]

    def nxt():
        addr[0] += 1 << 12
        return addr[0]
    for i in range(n_layers):
        for f, _ in fe.fe_layer_weights._fields_:
            setattr(layers[i], f, nxt())
    w = fe.fe_weights(nxt(), nxt(), nxt(), nxt(), nxt(), None, C.cast(layers, C.POINTER(fe.fe_layer_weights)))
    if misalign:
        setattr(w, misalign, getattr(w, misalign) + 4)
    return w, layers


def test_create_validates_pointers_and_workspace(fe):
    cfg = _cfg(fe)
    need = fe.fe_workspace_bytes(cfg)
    w, keep = _fake_weights(fe, cfg.n_layers)
    with pytest.raises(fe.FeError, match="FE_E_WORKSPACE"):
        fe.fe_drafter_create(cfg, w, 1 << 30, need - 1)
    with pytest.raises(fe.FeError, match="FE_E_ALIGN"):
        fe.fe_drafter_create(cfg, w, (1 << 30) + 64, need)
    wm, keep2 = _fake_weights(fe, cfg.n_layers, misalign="lm_head")
    with pytest.raises(fe.FeError, match="FE_E_ALIGN"):
        fe.fe_drafter_create(cfg, wm, 1 << 30, need)
    keep[2].wk = None
    with pytest.raises(fe.FeError, match="FE_E_INVALID"):
        fe.fe_drafter_create(cfg, w, 1 << 30, need)


def test_forward_and_tree_validate_before_enqueue(fe):
    """A handle over fake addresses: every call below must fail on the host."""
    cfg = _cfg(fe)
    w, keep = _fake_weights(fe, cfg.n_layers)
    h = fe.fe_drafter_create(cfg, w, 1 << 30, fe.fe_workspace_bytes(cfg))
    try:
        N = cfg.n_layers
        kp = (C.c_void_p * N)(*[(1 << 31) + 4096 * i for i in range(N)])
        kv = fe.fe_kv_view(C.cast(kp, C.POINTER(C.c_void_p)), C.cast(kp, C.POINTER(C.c_void_p)),
                           1 << 32, 1024)
        out = fe.fe_draft_out(1 << 33, (1 << 33) + 4096, None, None, None)
        bad = [
            dict(batch=2), dict(batch=-1), dict(topk=0), dict(topk=9), dict(features=(1 << 34) + 2),
            dict(features=0), dict(kv_max_prefix=2048), dict(out_ids=0),
        ]
        for case in bad:
            kv.max_prefix = case.get("kv_max_prefix", 1024)
            o = fe.fe_draft_out(case.get("out_ids", 1 << 33), (1 << 33) + 4096, None, None, None)
            with pytest.raises(fe.FeError):
                fe.fe_draft_forward(h, case.get("batch", 1), case.get("features", 1 << 34),
                                    1 << 35, kv, case.get("topk", 8), o, 0)
        kv.max_prefix = 1024
        with pytest.raises(fe.FeError, match="FE_E_INVALID"):
            fe.fe_draft_forward(h, 1, 1 << 34, 1 << 35, fe.fe_kv_view(), 8, out, 0)
        fe.fe_draft_forward(h, 0, 0, 0, kv, 8, out, 0)       # empty batch: no work, OK
        tout = fe.fe_tree_out(*([1 << 36] * 5 + [0]))
        with pytest.raises(fe.FeError, match="FE_E_INVALID"):
            fe.fe_build_tree(h, 1, 8, 1 << 35, 1 << 33, 1 << 32, tout, 0)
        with pytest.raises(fe.FeError, match="FE_E_INVALID"):
            fe.fe_build_tree(h, 1, 0, 1 << 35, 1 << 33, 1 << 32, fe.fe_tree_out(*([1 << 36] * 6)), 0)
        fe.fe_build_tree(h, 0, 8, 0, 0, 0, tout, 0)
        with pytest.raises(fe.FeError, match="FE_E_INVALID"):
            fe.fe_set_graph_mode(None, 1)
    finally:
        fe.fe_drafter_destroy(h)


def test_binding_fails_loudly_without_library(tmp_path, monkeypatch):
    from paper_2509_20416_amd import fe as _fe
    monkeypatch.setattr(_fe, "_lib", None)
    monkeypatch.setattr(_fe, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="missing"):
        _fe.lib()


def test_kv_update_validates_before_enqueue(fe):
    """fe_kv_update over fake addresses: every bad call fails on the host."""
    cfg = _cfg(fe)
    w, keep = _fake_weights(fe, cfg.n_layers)
    one = fe.fe_kv_update_workspace_bytes(cfg, 1)
    big = fe.fe_kv_update_workspace_bytes(cfg, 1024)
    assert 0 < one < big
    assert fe.fe_kv_update_workspace_bytes(cfg, 0) == 0
    assert fe.fe_kv_update_workspace_bytes(_cfg(fe, head_dim=96), 8) == 0
    h = fe.fe_drafter_create(cfg, w, 1 << 30, fe.fe_workspace_bytes(cfg))
    try:
        N = cfg.n_layers
        kp = (C.c_void_p * N)(*[(1 << 31) + 4096 * i for i in range(N)])
        cache = fe.fe_kv_cache(C.cast(kp, C.POINTER(C.c_void_p)), C.cast(kp, C.POINTER(C.c_void_p)),
                               1 << 20)
        ok = dict(n=3, feat=1 << 34, tok=1 << 35, pos=(1 << 35) + 256, dst=(1 << 35) + 512,
                  cache=cache, ws=1 << 36, wsb=big)
        bad = [(dict(n=-1), "FE_E_INVALID"), (dict(feat=0), "FE_E_INVALID"),
               (dict(feat=(1 << 34) + 8), "FE_E_ALIGN"), (dict(dst=(1 << 35) + 2), "FE_E_ALIGN"),
               (dict(cache=fe.fe_kv_cache()), "FE_E_INVALID"), (dict(ws=0), "FE_E_WORKSPACE"),
               (dict(ws=(1 << 36) + 64), "FE_E_ALIGN"), (dict(wsb=one - 1), "FE_E_WORKSPACE")]
        for case, status in bad:
            a = dict(ok, **case)
            with pytest.raises(fe.FeError, match=status):
                fe.fe_kv_update(h, a["n"], a["feat"], a["tok"], a["pos"], a["dst"], a["cache"],
                                a["ws"], a["wsb"], 0)
        fe.fe_kv_update(h, 0, 0, 0, 0, 0, cache, 0, 0, 0)   # no rows: no work, OK
    finally:
        fe.fe_drafter_destroy(h)
    # the self context's update runs the layers over the rows: more workspace per row
    assert fe.fe_kv_update_workspace_bytes(_cfg(fe, cascade_ctx=fe.FE_CTX_SELF), 8) > \
        fe.fe_kv_update_workspace_bytes(_cfg(fe), 8)
    for kw, status in ((dict(max_prefix=0), "FE_E_INVALID"),):
        c2 = _cfg(fe, **kw)
        h = fe.fe_drafter_create(c2, w, 1 << 30, fe.fe_workspace_bytes(c2))
        try:
            with pytest.raises(fe.FeError, match=status):
                fe.fe_kv_update(h, 3, 1 << 34, 1 << 35, 1 << 35, 1 << 35, cache, 1 << 36, big, 0)
        finally:
            fe.fe_drafter_destroy(h)


def test_accept_sample_validates_before_enqueue(fe):
    cfg = _cfg(fe)
    w, keep = _fake_weights(fe, cfg.n_layers)
    h = fe.fe_drafter_create(cfg, w, 1 << 30, fe.fe_workspace_bytes(cfg))
    try:
        a = [1 << 33] * 7            # tokens .. uniforms (device addresses, never touched)
        o = [(1 << 34) + 256 * i for i in range(3)]
        call = lambda B, k, T, arr, outs: fe.fe_accept_sample(
            h, B, k, arr[0], arr[1], arr[2], arr[3], T, arr[4], arr[5], arr[6], *outs, 0)
        for B, k, T, status in ((2, 8, 1.0, "FE_E_INVALID"), (1, 0, 1.0, "FE_E_INVALID"),
                                (1, 8, 0.0, "FE_E_INVALID"), (1, 8, float("inf"), "FE_E_INVALID"),
                                (1, 8, 1e-39, "FE_E_INVALID")):
            with pytest.raises(fe.FeError, match=status):
                call(B, k, T, a, o)
        with pytest.raises(fe.FeError, match="FE_E_INVALID"):
            call(1, 8, 1.0, a[:5] + [0] + a[6:], o)          # no target distributions
        with pytest.raises(fe.FeError, match="FE_E_ALIGN"):
            call(1, 8, 1.0, a[:4] + [(1 << 33) + 2] + a[5:], o)  # misaligned draft uniforms
        call(0, 8, 1.0, a, o)                                   # empty batch: OK
    finally:
        fe.fe_drafter_destroy(h)
