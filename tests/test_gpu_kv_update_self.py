"""GPU parity of the drafter cache update under the self context (fe_kv_update
with FE_CTX_SELF: the N layers run over the new rows, a multi-position
prefill) against the oracle's feo_kv_update_self on the same seeded rows and
the same cache contents.

Rules: every written K/V row of every layer within the storage tolerance of
tests/parity.py (per row, max|gpu - ref| / max|ref|); rows that are not
destinations unchanged, bit for bit.  The cache rows of positions already
present (the prefix) hold seeded N(0, 1) values, which the new rows attend
to.  Chunk sizes cover one chunk, several chunks (later rows read the earlier
chunks' rows of every layer from the cache), and chunks above 256 rows (the
row-GEMM and attention launches take 256-row slices)."""
import os
import sys

import numpy as np
import pytest

from fe_synth import configs as C
from fe_synth import make_inputs, make_update_rows, make_weights
from fe_synth.gen import float_tensor
from tests.parity import TOL, assert_rows_close

pytestmark = pytest.mark.gpu


def log(*a):
    print("[kv-update-self]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2509_20416_amd import fe
    fe.lib()   # loud failure if the library is missing
    from oracle import feo
    feo.set_threads(min(16, len(os.sched_getaffinity(0))))


def _host(t, dtype):
    import torch
    if dtype == "bf16":
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def _widen(a, dtype):
    from fe_synth import to_f64
    return to_f64(a, dtype)


def _store(a, dtype):
    """fp64 -> storage precision (bf16: round to nearest even, as uint16 bits)."""
    z = np.ascontiguousarray(a, dtype=np.float32)
    if dtype != "bf16":
        return z
    b = z.view(np.uint32).copy()
    b += np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))
    return (b >> np.uint32(16)).astype(np.uint16)


def _prefilled(cfg, rows, seed):
    """Per-layer host caches: every row seeded N(0, 1) in storage precision."""
    shape = (rows, cfg.n_kv_heads, cfg.head_dim)
    ks = [float_tensor(f"self.k{l}", shape, seed, cfg.dtype) for l in range(cfg.n_layers)]
    vs = [float_tensor(f"self.v{l}", shape, seed, cfg.dtype) for l in range(cfg.n_layers)]
    return ks, vs


def _run(cfg, up, chunk_rows, max_prefix, seed=0, order=None):
    import torch
    from oracle import feo
    from paper_2509_20416_amd import Drafter
    from paper_2509_20416_amd.drafter import to_device
    if order is not None:
        up.features, up.tokens = up.features[order], up.tokens[order]
        up.positions, up.dst_rows = up.positions[order], up.dst_rows[order]
    M = len(up.tokens)
    w = make_weights(cfg, seed)
    hk, hv = _prefilled(cfg, up.cache_rows, seed + 1)
    dr = Drafter(cfg, w, max_batch=1, max_prefix=max_prefix, max_topk=cfg.topk)
    dev = dr.device
    ks = [to_device(a, cfg.dtype, dev) for a in hk]
    vs = [to_device(a, cfg.dtype, dev) for a in hv]
    log(f"{cfg.name}: M={M} rows={up.cache_rows} chunk={chunk_rows} max_prefix={max_prefix}")
    dr.kv_update(to_device(up.features, cfg.dtype, dev), to_device(up.tokens, "i32", dev),
                 to_device(up.positions, "i32", dev), to_device(up.dst_rows, "i32", dev),
                 ks, vs, chunk_rows=chunk_rows)
    torch.cuda.synchronize()
    rk, rv = feo.kv_update_self(cfg, w, up.features, up.tokens, up.positions, up.dst_rows, hk, hv)
    tol = TOL[cfg.dtype]
    kvd = cfg.n_kv_heads * cfg.head_dim
    untouched = np.ones(up.cache_rows, bool)
    untouched[up.dst_rows] = False
    worst = 0.0
    for li in range(cfg.n_layers):
        for name, got_t, ref, before in (("k", ks[li], rk[li], hk[li]), ("v", vs[li], rv[li], hv[li])):
            got = _host(got_t, cfg.dtype)
            rows = _widen(got[up.dst_rows], cfg.dtype).reshape(M, kvd)
            worst = max(worst, assert_rows_close(f"layer {li} {name}", rows, ref.reshape(M, kvd), tol))
            assert np.array_equal(got[untouched], before[untouched]), \
                f"layer {li} {name}: a row not updated changed"
    log(f"{cfg.name}: worst per-row error {worst:.2e} (tol {tol:.0e}) over {M} rows")
    dr.close()
    return w, ks, vs


SELF = lambda c: c.with_(cascade_ctx="self", name=c.name + "_self")

CASES = [
    # (config, accepted per sequence, prefix per sequence, chunk rows)
    (SELF(C.SMALL_GQA_BF16), [1], [0], 1024),
    (SELF(C.SMALL_GQA_BF16), [6], [0], 1024),
    (SELF(C.SMALL_GQA_BF16), [4, 6, 1, 3], [17, 0, 64, 130], 1024),
    (SELF(C.SMALL_GQA_BF16), [4, 6, 1, 3], [17, 0, 64, 130], 3),     # chunks of 3 rows
    (SELF(C.SMALL_GQA_F32), [4, 6, 1, 3], [17, 0, 64, 130], 1024),
    (SELF(C.SMALL_GQA_F32), [5, 2], [3, 70], 4),
    (SELF(C.SMALL_MHA_BF16_D128), [9, 7], [65, 5], 1024),
    (SELF(C.SMALL_GQA8_BF16_D128), [5, 5, 5], [0, 200, 511], 1024),  # 8 query heads per KV head
    (SELF(C.SMALL_GQA2_BF16), [8, 3], [40, 0], 5),
    (SELF(C.SMALL_GQA_BF16), [300], [0], 1024),                      # slices of 256 + 44 rows
    (SELF(C.SMALL_GQA_BF16), [280, 20], [0, 100], 150),              # 150-row chunks
    (SELF(C.TINY_F32_B1), [40, 1], [0, 60], 1024),
]


@pytest.mark.parametrize("cfg,acc,plens,chunk", CASES,
                         ids=[f"{c.name}-m{sum(a)}-c{ch}" for c, a, p, ch in CASES])
def test_kv_update_self_parity(cfg, acc, plens, chunk):
    acc = np.asarray(acc, np.int32)
    plens = np.asarray(plens, np.int32)
    cap = int((acc + plens).max()) + 8
    up = make_update_rows(cfg, acc, plens, capacity=cap, seed=int(acc.sum()) + 3)
    _run(cfg, up, chunk, max_prefix=cap)


def test_kv_update_self_interleaved_sequences():
    """Rows of three sequences interleaved (each in increasing position order)."""
    cfg = SELF(C.SMALL_GQA_BF16)
    acc, plens = np.array([5, 4, 3], np.int32), np.array([10, 0, 33], np.int32)
    up = make_update_rows(cfg, acc, plens, capacity=48, seed=41)
    order = np.array([0, 5, 9, 1, 6, 10, 2, 7, 11, 3, 8, 4])
    _run(cfg, up, 1024, max_prefix=48, order=order)


def test_kv_update_self_then_draft():
    """Prefill a sequence's cache with the update, then draft at the grown
    prefix: the library's pass over the library's cache against the oracle's
    pass over the oracle's cache."""
    import torch
    from oracle import feo
    from paper_2509_20416_amd import Drafter
    from paper_2509_20416_amd.drafter import to_device
    from tests.gpu_case import run_case
    cfg = SELF(C.SMALL_GQA_BF16).with_(batch=1)
    P = 50
    up = make_update_rows(cfg, np.array([P + 1]), np.array([0]), capacity=P + 1, seed=43)
    w = make_weights(cfg, 7)
    rows = slice(0, P)
    dr = Drafter(cfg, w, max_batch=1, max_prefix=P + 1, max_topk=cfg.topk)
    dev = dr.device
    z = np.zeros((P + 1, cfg.n_kv_heads, cfg.head_dim), np.uint16)
    ks = [to_device(z, cfg.dtype, dev) for _ in range(cfg.n_layers)]
    vs = [to_device(z, cfg.dtype, dev) for _ in range(cfg.n_layers)]
    dr.kv_update(to_device(up.features[rows], cfg.dtype, dev), to_device(up.tokens[rows], "i32", dev),
                 to_device(up.positions[rows], "i32", dev), to_device(up.dst_rows[rows], "i32", dev),
                 ks, vs, chunk_rows=16)
    torch.cuda.synchronize()
    gk = [_host(k, cfg.dtype)[:P] for k in ks]
    gv = [_host(v, cfg.dtype)[:P] for v in vs]
    dr.close()
    rk, rv = feo.kv_update_self(cfg, w, up.features[rows], up.tokens[rows], up.positions[rows],
                                up.dst_rows[rows], [z] * cfg.n_layers, [z] * cfg.n_layers)
    inp = make_inputs(cfg, seed=0, prefix_lens=np.array([P], np.int32))
    inp.features = np.ascontiguousarray(up.features[P:])
    inp.next_tokens = np.ascontiguousarray(up.tokens[P:])
    inp.kcache, inp.vcache = gk, gv      # the library's cache, for the library's pass
    rep, res, _ = run_case(cfg, seed=7, weights=w, inputs=inp, check_tree_struct=False)
    # and the oracle's pass over the oracle's own cache gives the same states
    inp2 = make_inputs(cfg, seed=0, prefix_lens=np.array([P], np.int32))
    inp2.features, inp2.next_tokens = inp.features, inp.next_tokens
    inp2.kcache = [_store(k, cfg.dtype) for k in rk]
    inp2.vcache = [_store(v, cfg.dtype) for v in rv]
    ref = feo.draft_forward(cfg, w, inp2, topk=cfg.topk)
    got = feo.draft_forward(cfg, w, inp, topk=cfg.topk)
    assert_rows_close("hidden via library cache", got["hidden"][0], ref["hidden"][0], TOL["bf16"])
    log(f"self prefill then draft: {rep}")
