"""fe_kv_update_noalloc (the cache update in the library's own device array,
no allocation) against fe_kv_update given a caller workspace of the same size,
through the C ABI: two calls in a row on one handle, the second with fewer rows
(the array keeps the first call's contents), every cache array bit for bit."""
import ctypes as C
import sys

import numpy as np
import pytest

from fe_synth import configs as CF
from fe_synth import make_update_rows, make_weights

pytestmark = pytest.mark.gpu


def log(*a):
    print("[no-alloc]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2509_20416_amd import fe
    fe.lib()   # loud failure if the library is missing


def _caches(cfg, rows, dev, fill):
    import torch
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    shape = (rows, cfg.n_kv_heads, cfg.head_dim)
    ks = [torch.full(shape, fill, dtype=tdt, device=dev) for _ in range(cfg.n_layers)]
    vs = [torch.full(shape, fill, dtype=tdt, device=dev) for _ in range(cfg.n_layers)]
    return ks, vs


def _view(fe, ks, vs):
    kp = (C.c_void_p * len(ks))(*[k.data_ptr() for k in ks])
    vp = (C.c_void_p * len(vs))(*[v.data_ptr() for v in vs])
    cache = fe.fe_kv_cache(C.cast(kp, C.POINTER(C.c_void_p)), C.cast(vp, C.POINTER(C.c_void_p)),
                           int(ks[0].shape[0]))
    return cache, (kp, vp)


# (config, accepted rows per sequence of call 1, of call 2): several chunks of
# the 8 MiB array in the first call (tiled or split-K launches), a one-cycle
# update (fused norm) in the second
CASES = [(CF.SMALL_GQA_BF16, [200] * 5, [6]),
         (CF.LLAMA8B_BF16_B1, [50, 40, 30], [6]),
         (CF.SMALL_GQA_F32, [90] * 3, [2, 1]),
         # the self context: the layers run over the rows (a prefill)
         (CF.SMALL_GQA_BF16.with_(cascade_ctx="self", name="small_gqa_bf16_self"), [150] * 4, [6]),
         (CF.LLAMA8B_BF16_B1.with_(cascade_ctx="self", name="llama8b_bf16_self"), [40, 30], [6])]


@pytest.mark.parametrize("cfg,acc1,acc2", CASES, ids=[c[0].name for c in CASES])
def test_noalloc_matches_workspace_call(cfg, acc1, acc2):
    import torch
    from paper_2509_20416_amd import Drafter, fe
    from paper_2509_20416_amd.drafter import to_device
    w = make_weights(cfg, 0)
    cap = max(max(acc1), max(acc2)) + 64
    dr = Drafter(cfg, w, max_batch=1, max_prefix=cap, max_topk=cfg.topk)
    dev = dr.device
    ws = torch.empty(fe.FE_KV_UPDATE_SCRATCH_BYTES, dtype=torch.uint8, device=dev)
    rng = np.random.default_rng(len(acc1))
    for call, acc in enumerate((acc1, acc2)):
        acc = np.asarray(acc, np.int32)
        plens = rng.integers(0, cap - acc + 1).astype(np.int32)
        up = make_update_rows(cfg, acc, plens, capacity=cap, seed=100 + call)
        M = len(up.tokens)
        log(f"{cfg.name}: call {call + 1}, {M} rows")
        args = [to_device(up.features, cfg.dtype, dev), to_device(up.tokens, "i32", dev),
                to_device(up.positions, "i32", dev), to_device(up.dst_rows, "i32", dev)]
        ka, va = _caches(cfg, up.cache_rows, dev, 3.0)
        kb, vb = _caches(cfg, up.cache_rows, dev, 3.0)
        ca, keep_a = _view(fe, ka, va)
        cb, keep_b = _view(fe, kb, vb)
        torch.cuda.synchronize()
        fe.fe_kv_update(dr.handle, M, *[a.data_ptr() for a in args], ca, ws.data_ptr(),
                        ws.numel(), dr.stream())
        fe.fe_kv_update_noalloc(dr.handle, M, *[a.data_ptr() for a in args], cb, dr.stream())
        torch.cuda.synchronize()
        for li in range(cfg.n_layers):
            for name, a, b in (("k", ka[li], kb[li]), ("v", va[li], vb[li])):
                assert torch.equal(a.view(torch.int16) if cfg.dtype == "bf16" else a.view(torch.int32),
                                   b.view(torch.int16) if cfg.dtype == "bf16" else b.view(torch.int32)), \
                    f"call {call + 1} layer {li} {name}"
        # the written rows are real updates (not the fill value)
        assert not torch.equal(ka[0][torch.from_numpy(up.dst_rows).long().to(dev)],
                               torch.full_like(ka[0][:M], 3.0))
    dr.close()


def test_noalloc_rejects_bad_arguments():
    from paper_2509_20416_amd import Drafter, fe
    cfg = CF.SMALL_GQA_BF16
    dr = Drafter(cfg, make_weights(cfg, 0), max_batch=1, max_prefix=64, max_topk=cfg.topk)
    cache = fe.fe_kv_cache(None, None, 0)
    with pytest.raises(fe.FeError):
        fe.fe_kv_update_noalloc(dr.handle, 1, 0, 0, 0, 0, cache, dr.stream())
    with pytest.raises(fe.FeError):
        fe.fe_kv_update_noalloc(0, 1, 0, 0, 0, 0, cache, dr.stream())
    dr.close()
