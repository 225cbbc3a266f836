"""GPU parity of the drafter cache update (fe_kv_update, through the C ABI)
against the oracle's feo_kv_update on the same seeded rows.

Rules: every written K/V row within the storage tolerance of tests/parity.py
(per row, max|gpu - ref| / max|ref|); every cache row that is not a
destination is unchanged, bit for bit; out-of-range positions and tokens give
NaN rows, out-of-range destinations write nothing."""
import os
import sys

import numpy as np
import pytest

from fe_synth import configs as C
from fe_synth import make_update_rows, make_weights
from tests.parity import TOL, assert_rows_close

pytestmark = pytest.mark.gpu


def log(*a):
    print("[kv-update]", *a, flush=True)
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


SENTINEL = {"bf16": np.uint16(0x4640), "f32": np.float32(12345.0)}


def _caches(cfg, rows, dev):
    import torch
    from paper_2509_20416_amd.drafter import to_device
    shape = (rows, cfg.n_kv_heads, cfg.head_dim)
    fill = np.full(shape, SENTINEL[cfg.dtype])
    ks = [to_device(fill, cfg.dtype, dev) for _ in range(cfg.n_layers)]
    vs = [to_device(fill, cfg.dtype, dev) for _ in range(cfg.n_layers)]
    torch.cuda.synchronize()
    return ks, vs


def _host(t, dtype):
    import torch
    if dtype == "bf16":
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def _widen(a, dtype):
    from fe_synth import to_f64
    return to_f64(a, dtype)


def _run(cfg, up, chunk_rows, sample=None, seed=0):
    """Update through the library, compare with the oracle on `sample` rows
    (all rows when None) and check the untouched rows."""
    import torch
    from oracle import feo
    from paper_2509_20416_amd import Drafter
    from paper_2509_20416_amd.drafter import to_device
    M = len(up.tokens)
    max_prefix = int(up.positions.max()) + 1 if M else 1
    w = make_weights(cfg, seed)
    dr = Drafter(cfg, w, max_batch=1, max_prefix=max_prefix, max_topk=cfg.topk)
    dev = dr.device
    ks, vs = _caches(cfg, up.cache_rows, dev)
    log(f"{cfg.name}: M={M} rows={up.cache_rows} chunk={chunk_rows}")
    dr.kv_update(to_device(up.features, cfg.dtype, dev), to_device(up.tokens, "i32", dev),
                 to_device(up.positions, "i32", dev), to_device(up.dst_rows, "i32", dev),
                 ks, vs, chunk_rows=chunk_rows)
    torch.cuda.synchronize()
    idx = np.arange(M) if sample is None else np.asarray(sample)
    rk, rv = feo.kv_update(cfg, w, up.features[idx], up.tokens[idx], up.positions[idx])
    tol = TOL[cfg.dtype]
    kvd = cfg.n_kv_heads * cfg.head_dim
    untouched = np.ones(up.cache_rows, bool)
    untouched[up.dst_rows] = False
    worst = 0.0
    for li in range(cfg.n_layers):
        for name, got_t, ref in (("k", ks[li], rk[li]), ("v", vs[li], rv[li])):
            got = _host(got_t, cfg.dtype)
            rows = _widen(got[up.dst_rows[idx]], cfg.dtype).reshape(len(idx), kvd)
            worst = max(worst, assert_rows_close(f"layer {li} {name}", rows,
                                                 ref.reshape(len(idx), kvd), tol))
            rest = got[untouched]
            assert (rest == SENTINEL[cfg.dtype]).all(), f"layer {li} {name}: a row not updated changed"
    log(f"{cfg.name}: worst per-row error {worst:.2e} (tol {tol:.0e}) over {len(idx)} rows")
    dr.close()
    return ks, vs


CASES = [
    # (config, accepted per sequence, chunk rows).  bf16: chunks of up to 16
    # rows fuse the norm into one K/V launch for every layer (the input FC
    # writes the per-layer gamma * x_0 copies); above that one K/V launch over
    # 128-row blocks (32-column tiles below 128 rows, 64 from there on), and
    # the FCs as 256-row launches or, above 256 rows, 2-D tiled GEMMs.  fp32:
    # per-layer launches (row streaming up to 4 rows, 256-row launches above)
    (C.SMALL_GQA_BF16, [1], 1024),
    (C.SMALL_GQA_BF16, [2, 1, 1], 1024),
    (C.SMALL_GQA_BF16, [6], 1024),
    (C.SMALL_MHA_BF16_D128, [3] * 5 + [1], 1024),     # 16 rows: the fused limit
    (C.SMALL_GQA_BF16, [5] * 7 + [2], 9),             # fused chunks of 9 rows and a ragged 1
    (C.SMALL_GQA_BF16.with_(n_layers=10, name="small_gqa_bf16_n10"), [6], 1024),  # 10 layers' copies
    (C.SMALL_GQA_BF16, [4, 6, 1, 3, 5, 2, 7, 9], 1024),
    (C.SMALL_GQA_F32, [4, 6, 1, 3, 5, 2, 7, 9], 1024),
    (C.SMALL_GQA_F32, [2, 1, 1], 1024),
    (C.SMALL_MHA_BF16_D128, [50] * 6 + [13], 1024),   # 2-D tiled GEMMs, ragged row block
    (C.SMALL_MHA_BF16_D128, [50] * 6 + [13], 100),    # chunks of 100 and 13 rows
    (C.SMALL_GQA_BF16, [40] * 8 + [7], 300),          # a tiled chunk of 300 rows, then 27
    (C.SMALL_GQA_BF16, [40] * 8 + [7], 200),          # 200 rows (64-column K/V tiles), then 127
    (C.TINY_F32_B1, [3] * 100 + [1], 40),
]


@pytest.mark.parametrize("cfg,acc,chunk", CASES,
                         ids=[f"{c.name}-m{sum(a)}-c{ch}" for c, a, ch in CASES])
def test_kv_update_parity(cfg, acc, chunk):
    rng = np.random.default_rng(sum(acc) + chunk)
    acc = np.asarray(acc, np.int32)
    cap = int(acc.max()) + 40
    plens = rng.integers(0, cap - acc + 1).astype(np.int32)
    up = make_update_rows(cfg, acc, plens, capacity=cap, seed=int(acc.sum()))
    _run(cfg, up, chunk)


def test_kv_update_full_size_sampled():
    """The 8B shapes at batch 32 with N+1 accepted positions per sequence
    (the largest update a cycle makes), sampled rows through the oracle."""
    cfg = C.LLAMA8B_BF16_B32
    rng = np.random.default_rng(32)
    acc = np.full(32, cfg.n_layers + 1, np.int32)
    plens = rng.integers(256, 8192 - acc[0] + 1, 32).astype(np.int32)
    up = make_update_rows(cfg, acc, plens, capacity=8192, seed=5)
    sample = [0, 1, 7, 100, 129, 255]
    _run(cfg, up, 1024, sample=sample)


def test_kv_update_full_size_prefill_tiled():
    """The 8B shapes over 1000 positions in one chunk: the 2-D tiled GEMMs at
    their full K (12288, 8192, 4096) with a ragged last row block, sampled
    rows (every row block, both ends of the ragged one) through the oracle."""
    cfg = C.LLAMA8B_BF16_B1
    acc = np.array([1000], np.int32)
    up = make_update_rows(cfg, acc, np.array([20], np.int32), capacity=1024, seed=8)
    sample = [0, 1, 127, 128, 383, 640, 895, 896, 999]
    _run(cfg, up, 1024, sample=sample)


def test_kv_update_full_size_b1_cycle():
    """The 8B shapes at batch 1: the N+1 = 6 positions one cycle accepts at
    most, every row through the oracle (the fused-norm path)."""
    cfg = C.LLAMA8B_BF16_B1
    acc = np.array([cfg.n_layers + 1], np.int32)
    up = make_update_rows(cfg, acc, np.array([1000], np.int32), capacity=1024, seed=6)
    _run(cfg, up, 1024)


def test_kv_update_out_of_range_rows():
    """A position past max_prefix or a token outside the vocabulary gives NaN
    rows; destinations outside the cache write nothing; the others are exact
    to the rules."""
    import torch
    from oracle import feo
    from paper_2509_20416_amd import Drafter
    from paper_2509_20416_amd.drafter import to_device
    cfg = C.SMALL_GQA_BF16
    up = make_update_rows(cfg, np.array([6]), np.array([10]), capacity=32, seed=9)
    max_prefix = 16
    pos, tok, dst = up.positions.copy(), up.tokens.copy(), up.dst_rows.copy()
    pos[1] = max_prefix          # row 1: position out of range -> NaN
    tok[2] = cfg.target_vocab    # row 2: token out of range -> NaN
    dst[3] = -1                  # row 3: nowhere to write
    dst[4] = up.cache_rows       # row 4: nowhere to write
    w = make_weights(cfg, 0)
    dr = Drafter(cfg, w, max_batch=1, max_prefix=max_prefix, max_topk=cfg.topk)
    dev = dr.device
    ks, vs = _caches(cfg, up.cache_rows, dev)
    dr.kv_update(to_device(up.features, cfg.dtype, dev), to_device(tok, "i32", dev),
                 to_device(pos, "i32", dev), to_device(dst, "i32", dev), ks, vs)
    torch.cuda.synchronize()
    good = [0, 5]
    rk, rv = feo.kv_update(cfg, w, up.features[good], up.tokens[good], up.positions[good])
    kvd = cfg.n_kv_heads * cfg.head_dim
    for li in range(cfg.n_layers):
        for got_t, ref in ((ks[li], rk[li]), (vs[li], rv[li])):
            got = _widen(_host(got_t, cfg.dtype), cfg.dtype)
            assert_rows_close("good rows", got[dst[good]].reshape(2, kvd), ref.reshape(2, kvd),
                              TOL[cfg.dtype])
            assert np.isnan(got[dst[1]]).all() and np.isnan(got[dst[2]]).all()
            written = set(dst[[0, 1, 2, 5]].tolist())
            rest = [r for r in range(up.cache_rows) if r not in written]
            assert (got[rest] == _widen(np.array(SENTINEL[cfg.dtype]), cfg.dtype)).all()
    dr.close()


def test_kv_update_errors():
    import torch
    from paper_2509_20416_amd import Drafter, fe
    from paper_2509_20416_amd.drafter import to_device
    cfg = C.SMALL_GQA_BF16
    up = make_update_rows(cfg, np.array([2]), np.array([0]), capacity=4, seed=1)
    w = make_weights(cfg, 0)
    dev = torch.device("cuda:0")
    args = (to_device(up.features, cfg.dtype, dev), to_device(up.tokens, "i32", dev),
            to_device(up.positions, "i32", dev), to_device(up.dst_rows, "i32", dev))
    ks, vs = _caches(cfg, 4, dev)
    dr = Drafter(cfg, w, max_batch=1, max_prefix=4, max_topk=cfg.topk)
    with pytest.raises(fe.FeError) as e:   # misaligned features
        dr.kv_update(args[0].view(-1)[1:], *args[1:], ks, vs, n_rows=1)
    assert e.value.status == fe.FE_E_ALIGN
    dr.kv_update(*args, ks, vs, n_rows=0)   # no-op
    torch.cuda.synchronize()
    assert (_host(ks[0], cfg.dtype) == SENTINEL[cfg.dtype]).all()
    dr.close()
