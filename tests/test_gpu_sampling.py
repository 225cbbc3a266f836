"""GPU parity of stochastic drafting (fe_draft_sample, through the C ABI)
against the oracle on the same seeded uniforms.

Rules (extending tests/parity.py to sampled candidates): with zT = z / T and
keys = zT - log(-log(u)) from the oracle's logits, thr = 2 * tol * max|zT|
per row.
* The sampled set is decided when the oracle's k-th and (k+1)-th largest keys
  are more than thr apart: then the GPU set equals the oracle's.  Otherwise
  every GPU candidate's key is within thr of the oracle's k-th key or above.
* Listing order: most probable first, so oracle zT never increases along the
  GPU list by more than thr; with a decided set and gaps above thr the lists
  are equal.
* Probabilities: |log p_gpu - log softmax(zT)(id)| <= 2 * thr."""
import os

import numpy as np
import pytest

from fe_synth import configs as C
from fe_synth import make_inputs, make_uniforms, make_weights
from tests.parity import TOL, assert_rows_close
from tests.treecheck import check_tree

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2509_20416_amd import fe
    fe.lib()
    from oracle import feo
    feo.set_threads(min(16, len(os.sched_getaffinity(0))))


def log(*a):
    print("[sampling]", *a, flush=True)


def check_sampled(gpu_draft, gpu_probs, z, u, T, ref_draft, tol):
    """gpu_draft/ref_draft [rows, k]; z [rows, V] oracle logits; u [rows, V]."""
    rows, k = gpu_draft.shape
    zt = z.reshape(rows, -1) / T
    keys = zt - np.log(-np.log(u.reshape(rows, -1).astype(np.float64)))
    decided = exact = 0
    for r in range(rows):
        thr = 2 * tol * np.abs(zt[r]).max()
        order = np.argsort(-keys[r], kind="stable")
        kth = keys[r, order[k - 1]]
        nxt = keys[r, order[k]] if k < keys.shape[1] else -np.inf
        g = gpu_draft[r]
        assert len(set(g.tolist())) == k, (r, g)
        if kth - nxt > thr:
            decided += 1
            assert set(g.tolist()) == set(ref_draft[r].tolist()), (r, g, ref_draft[r])
            zs = np.sort(zt[r, g])[::-1]
            if k == 1 or np.min(zs[:-1] - zs[1:]) > thr:
                exact += 1
                np.testing.assert_array_equal(g, ref_draft[r])
        else:
            assert (keys[r, g] >= kth - thr).all(), (r, g)
        assert (np.diff(zt[r, g]) <= thr).all(), (r, zt[r, g])
        q = zt[r] - zt[r].max()
        lq = q - np.log(np.exp(q).sum())
        assert np.abs(np.log(gpu_probs[r].astype(np.float64)) - lq[g]).max() <= 2 * thr + 1e-6
    return decided, exact


def _run(cfg, T, seed=1, topk=None, graph=False, prefix_lens=None, philox=None):
    """philox = (seed, offset): the pass draws its uniforms itself
    (fe_draft_sample_seeded); the oracle gets the same stream's uniforms."""
    import torch
    from oracle import feo
    from paper_2509_20416_amd import Drafter
    k = int(topk or cfg.topk)
    w = make_weights(cfg, seed)
    inp = make_inputs(cfg, seed, prefix_lens)
    B, N, V = len(inp.prefix_lens), cfg.n_layers, cfg.draft_vocab
    if philox is None:
        u = make_uniforms((B, N, V), seed=seed + 100)
    else:
        u = feo.philox_uniforms(philox[0], philox[1], 0, B * N * V).reshape(B, N, V)
    log(f"{cfg.name}: T={T} k={k} B={B} graph={graph} philox={philox}")
    dr = Drafter(cfg, w, max_batch=B, max_prefix=int(inp.prefix_lens.max()),
                 max_topk=max(k, cfg.topk), graph=graph)
    di = dr.upload_inputs(inp)
    tree = dr.alloc_tree(B, k)
    if philox is None:
        ud = torch.from_numpy(u).cuda()
        out = dr.forward(di, k, logits=True, temperature=T, uniforms=ud, tree=tree)
    else:
        so = torch.tensor(list(philox), dtype=torch.int64, device="cuda")
        out = dr.forward(di, k, logits=True, temperature=T, seed_offset=so, tree=tree)
    torch.cuda.synchronize()
    got = {n: t.cpu().numpy() for n, t in out.items()}
    tr = {n: t.cpu().numpy() for n, t in tree.items()}
    ref = feo.draft_forward(cfg, w, inp, topk=k, temperature=T, uniforms=u)
    tol = TOL[cfg.dtype]
    assert_rows_close("logits", got["logits"], ref["logits"], tol)
    dec, ex = check_sampled(got["topk_draft"].reshape(B * N, k), got["topk_probs"].reshape(B * N, k),
                            ref["logits"], u, T, ref["topk_draft"].reshape(B * N, k), tol)
    np.testing.assert_array_equal(got["topk_ids"], w.d2t[got["topk_draft"]])
    # the tree hangs the sampled candidates in listing order (backbone = most probable)
    for b in range(B):
        check_tree(tr, b, N, k, inp.next_tokens[b], got["topk_ids"][b], inp.prefix_lens[b])
    log(f"{cfg.name}: sampled sets decided {dec}/{B * N}, lists exact {ex}")
    dr.close()
    return dec, ex, B * N


SAMPLED = [
    (C.SMALL_GQA_F32, 1.0, None),
    (C.SMALL_GQA_F32, 0.6, 16),
    (C.SMALL_GQA_BF16, 1.0, None),
    (C.SMALL_MHA_BF16_D128, 1.3, 1),
    (C.TINY_F32_B1, 1.0, None),
    # more than 16 LM-head rows: the per-row candidate scan
    (C.SMALL_GQA_F32.with_(batch=12, name="small_gqa_f32_b12"), 1.0, 8),
    # more than 128 bf16 LM-head rows: the 256-row tiles' epilogue
    (C.SMALL_GQA_BF16.with_(batch=48, prefix=(0, 300), name="small_gqa_bf16_b48"), 1.0, 8),
]


@pytest.mark.parametrize("cfg,T,k", SAMPLED, ids=[f"{c.name}-T{t}-k{k}" for c, t, k in SAMPLED])
def test_sampled_parity(cfg, T, k):
    dec, ex, rows = _run(cfg, T, topk=k)
    if cfg.dtype == "f32":
        assert dec >= rows // 2, (dec, rows)


def test_sampled_llama8b_b1_full_graph():
    _run(C.LLAMA8B_BF16_B1, 1.0, seed=0, graph=True)


def test_greedy_at_temperature_and_graph_rereads_uniforms():
    """No uniforms: the greedy list at any T, with softmax(z/T) probabilities.
    Graph replay: the captured pass reads the uniforms buffer again on every
    replay (new draws in the same buffer give the eager result for them)."""
    import torch
    from paper_2509_20416_amd import Drafter
    cfg = C.SMALL_GQA_F32
    w, inp = make_weights(cfg, 2), make_inputs(cfg, 2)
    B, N, V = cfg.batch, cfg.n_layers, cfg.draft_vocab
    dr = Drafter(cfg, w, max_batch=B, max_prefix=int(inp.prefix_lens.max()))
    di = dr.upload_inputs(inp)
    g1 = {n: t.cpu().numpy() for n, t in dr.forward(di, logits=True).items()}
    g2 = {n: t.cpu().numpy() for n, t in dr.forward(di, logits=True, temperature=0.5).items()}
    np.testing.assert_array_equal(g1["topk_draft"], g2["topk_draft"])
    zt = g1["logits"] / 0.5
    q = np.exp(zt - zt.max(-1, keepdims=True))
    q /= q.sum(-1, keepdims=True)
    np.testing.assert_allclose(g2["topk_probs"], np.take_along_axis(q, g2["topk_draft"], -1),
                               rtol=1e-4)
    ud = torch.from_numpy(make_uniforms((B, N, V), seed=5)).cuda()
    eager = []
    for s in (5, 6):
        ud.copy_(torch.from_numpy(make_uniforms((B, N, V), seed=s)))
        eager.append(dr.forward(di, temperature=1.0, uniforms=ud)["topk_draft"].cpu().numpy())
    assert not np.array_equal(eager[0], eager[1])
    dr.set_graph_mode(True)
    out = dr.alloc_outputs(B, cfg.topk)
    for rep in range(2):
        for j, s in enumerate((5, 6)):
            ud.copy_(torch.from_numpy(make_uniforms((B, N, V), seed=s)))
            dr.forward(di, out=out, temperature=1.0, uniforms=ud)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(out["topk_draft"].cpu().numpy(), eager[j],
                                          err_msg=f"replay {rep} seed {s}")
    dr.close()


# --- counter-based uniforms (fe_draft_sample_seeded) ------------------------------------

@pytest.mark.parametrize("seed,offset,first,n", [(1, 0, 0, 1000), (0x7EEDFACE1234567, 5, 12345, 777),
                                                 (3, 2**40, 2**41 + 3, 1001)])
def test_philox_uniforms_match_oracle(seed, offset, first, n):
    """The device generator equals the oracle's, bit for bit."""
    import torch
    from oracle import feo
    from paper_2509_20416_amd import fe
    so = torch.tensor([seed, offset], dtype=torch.int64, device="cuda")
    out = torch.empty(n, dtype=torch.float32, device="cuda")
    fe.fe_test_philox_uniforms(so.data_ptr(), first, n, out.data_ptr(),
                               torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(out.cpu().numpy(), feo.philox_uniforms(seed, offset, first, n))


SEEDED = [
    (C.SMALL_GQA_F32, 1.0, None),
    (C.SMALL_GQA_BF16, 1.0, None),
    (C.SMALL_GQA_F32.with_(batch=12, name="small_gqa_f32_b12"), 0.8, 8),
    (C.SMALL_GQA_BF16.with_(batch=48, prefix=(0, 300), name="small_gqa_bf16_b48"), 1.0, 8),
]


@pytest.mark.parametrize("cfg,T,k", SEEDED, ids=[f"{c.name}-T{t}-k{k}" for c, t, k in SEEDED])
def test_seeded_sampling_parity(cfg, T, k):
    dec, ex, rows = _run(cfg, T, topk=k, philox=(2024, 7))
    if cfg.dtype == "f32":
        assert dec >= rows // 2, (dec, rows)


def test_seeded_graph_replays_follow_the_offset():
    """A captured seeded pass reads (seed, offset) from device memory on every
    replay: each replay equals the eager pass at that offset, bit for bit, and
    new offsets draw new candidates."""
    import torch
    from paper_2509_20416_amd import Drafter
    cfg = C.SMALL_GQA_BF16
    w, inp = make_weights(cfg, 3), make_inputs(cfg, 3)
    B = len(inp.prefix_lens)
    dr = Drafter(cfg, w, max_batch=B, max_prefix=int(inp.prefix_lens.max()))
    di = dr.upload_inputs(inp)
    so = torch.tensor([99, 0], dtype=torch.int64, device="cuda")
    eager = []
    for off in range(3):
        so[1] = off
        eager.append(dr.forward(di, temperature=1.0, seed_offset=so)["topk_draft"].cpu().numpy())
    assert not np.array_equal(eager[0], eager[1])
    dr.set_graph_mode(True)
    out = dr.alloc_outputs(B, cfg.topk)
    for rep in range(2):
        for off in range(3):
            so[1] = off
            out["topk_draft"].zero_()
            dr.forward(di, out=out, temperature=1.0, seed_offset=so)
            torch.cuda.synchronize()
            _ = torch.ones(1000, device="cuda").sum().item()
            np.testing.assert_array_equal(out["topk_draft"].cpu().numpy(), eager[off],
                                          err_msg=f"replay {rep} offset {off}")
    dr.close()
