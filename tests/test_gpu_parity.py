"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the
same seeded inputs.  Rules in tests/parity.py."""
import os

import numpy as np
import pytest

from fe_synth import configs as C
from fe_synth import make_inputs, make_weights

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2509_20416_amd import fe
    fe.lib()   # loud failure if the library is missing
    from oracle import feo
    feo.set_threads(min(16, len(os.sched_getaffinity(0))))


def _run(*a, **kw):
    from tests.gpu_case import run_case
    return run_case(*a, **kw)


# --- tree kernel alone: bit-exact on every array -------------------------------------------
@pytest.mark.parametrize("N,k,B", [(1, 1, 1), (3, 1, 2), (5, 8, 1), (7, 8, 32), (5, 10, 3),
                                   (16, 16, 2), (2, 3, 5)])
def test_tree_kernel_bit_exact(N, k, B):
    import torch
    from oracle import feo
    from paper_2509_20416_amd import Drafter
    cfg = C.TINY_F32_B1.with_(n_layers=N, topk=k, batch=B, draft_vocab=max(1024, 16 * k))
    rng = np.random.default_rng(N * 1000 + k * 10 + B)
    ids = np.stack([np.stack([rng.choice(128256, k, replace=False) for _ in range(N)])
                    for _ in range(B)]).astype(np.int32)
    roots = rng.integers(0, 128256, B).astype(np.int32)
    plens = rng.integers(0, 9000, B).astype(np.int32)
    w = make_weights(cfg.with_(n_layers=1), 0)
    w.layers = w.layers * N
    dr = Drafter(cfg, w, max_batch=B, max_prefix=0, max_topk=k)
    inp = make_inputs(cfg.with_(n_layers=N, prefix=0), 0)
    inp.next_tokens = roots
    inp.prefix_lens = plens
    inp.kcache = [np.zeros((0, cfg.n_kv_heads, cfg.head_dim), np.float32)] * N
    inp.vcache = inp.kcache
    di = dr.upload_inputs(inp, max_prefix=0)
    di.next_tokens = torch.from_numpy(roots).cuda()
    tree = dr.build_tree(di, torch.from_numpy(ids).cuda(), k)
    torch.cuda.synchronize()
    ref = feo.build_tree(N, k, roots, ids, plens)
    for n in ref:
        np.testing.assert_array_equal(tree[n].cpu().numpy(), ref[n], err_msg=n)
    dr.close()


# --- greedy acceptance (NEXT-2): bit-exact on every output -----------------------------------
# Trees from the GPU tree kernel; target predictions planted along a random
# walk from the root for a random number of steps, random elsewhere (so every
# accepted length 0..N occurs), plus a batch with nothing accepted.
@pytest.mark.parametrize("N,k,B", [(1, 1, 1), (3, 3, 4), (5, 8, 1), (7, 8, 32), (5, 10, 3),
                                   (16, 16, 2), (4, 1, 5)])
def test_accept_greedy_bit_exact(N, k, B):
    import torch
    from oracle import feo
    from paper_2509_20416_amd import Drafter
    cfg = C.TINY_F32_B1.with_(n_layers=N, topk=k, batch=B, draft_vocab=max(1024, 16 * k))
    rng = np.random.default_rng(N * 1000 + k * 10 + B + 7)
    ids = np.stack([np.stack([rng.choice(1000, k, replace=False) for _ in range(N)])
                    for _ in range(B)]).astype(np.int32)
    roots = rng.integers(0, 1000, B).astype(np.int32)
    w = make_weights(cfg.with_(n_layers=1), 0)
    w.layers = w.layers * N
    dr = Drafter(cfg, w, max_batch=B, max_prefix=0, max_topk=k)
    inp = make_inputs(cfg.with_(n_layers=N, prefix=0), 0)
    inp.next_tokens = roots
    inp.prefix_lens = np.zeros(B, np.int32)
    inp.kcache = [np.zeros((0, cfg.n_kv_heads, cfg.head_dim), np.float32)] * N
    inp.vcache = inp.kcache
    di = dr.upload_inputs(inp, max_prefix=0)
    di.next_tokens = torch.from_numpy(roots).cuda()
    tree = dr.build_tree(di, torch.from_numpy(ids).cuda(), k)
    torch.cuda.synchronize()
    tok, par = tree["tokens"].cpu().numpy(), tree["parents"].cpu().numpy()
    T = 1 + N * k
    for nothing in (False, True):
        nx = rng.integers(1000, 2000, (B, T)).astype(np.int32)   # no node carries these
        if not nothing:
            for b in range(B):
                cur = 0
                for _ in range(rng.integers(0, N + 1)):
                    kids = [n for n in range(T) if par[b, n] == cur]
                    if not kids:
                        break
                    c = kids[rng.integers(0, len(kids))]
                    nx[b, cur] = tok[b, c]
                    cur = c
        got = dr.accept_greedy(tree, torch.from_numpy(nx).cuda(), k)
        torch.cuda.synchronize()
        ref = feo.accept_greedy(N, k, tok, tree["retrieve"].cpu().numpy(), nx)
        for n in ref:
            np.testing.assert_array_equal(got[n].cpu().numpy(), ref[n], err_msg=n)
        if nothing:
            assert (ref["accept_len"] == 0).all()
    dr.close()


# --- small shapes: several tiles, ragged chunks, ragged batch, P = 0 -----------------------
SMALL = [C.SMALL_GQA_BF16, C.SMALL_GQA_F32, C.SMALL_MHA_BF16_D128, C.TINY_F32_B1,
         # 8 query heads per KV head (the attention variant only the 70B shape uses
         # at full size) and 2 per KV head, bf16 and fp32
         C.SMALL_GQA8_BF16_D128, C.SMALL_GQA2_BF16, C.SMALL_GQA2_F32]


@pytest.mark.parametrize("ctx", ["cascade", "self", "parallel"])
@pytest.mark.parametrize("cfg", SMALL, ids=lambda c: c.name)
def test_small_parity(cfg, ctx):
    cfg = cfg.with_(cascade_ctx=ctx)
    plens = None
    if cfg.batch == 3:
        plens = np.array([0, 700, 65], np.int32)   # empty prefix, several chunks, ragged tail
    elif cfg.batch == 2 and cfg.head_dim == 64:
        plens = np.array([400, 1], np.int32)
    rep, _, _ = _run(cfg, seed=1, prefix_lens=plens)
    if cfg.dtype == "f32":
        assert rep["decided"] >= rep["ranks"] // 2, rep


# A deep cascade (N = 10): layers 9 and 10 attend to more than 8 cascade keys
# (the 16-key bound of the attention's cascade loops), every producer writes
# up to 11 normalised copies; batch 3 with the cascade keys in units of their
# own, and batch 20 with the residual row pass.
@pytest.mark.parametrize("cfg", [C.SMALL_GQA_BF16.with_(n_layers=10, name="small_gqa_bf16_n10"),
                                 C.SMALL_GQA_BF16.with_(n_layers=10, batch=20, prefix=(0, 300),
                                                        name="small_gqa_bf16_b20_n10")],
                         ids=lambda c: c.name)
def test_deep_cascade_parity(cfg):
    plens = np.array([0, 700, 65], np.int32) if cfg.batch == 3 else None
    _run(cfg, seed=7, prefix_lens=plens)


# Attention work split: 1 chunk per workgroup (every 128-key chunk its own
# partial, merged by the second launch), 2 and 3 (the sub-chunk loop with a
# ragged last workgroup), 8 (one workgroup per sequence, no merge launch).
@pytest.mark.parametrize("split", [1, 2, 3, 8])
@pytest.mark.parametrize("cfg", [C.SMALL_GQA_BF16, C.SMALL_GQA_F32, C.SMALL_MHA_BF16_D128,
                                 C.SMALL_GQA8_BF16_D128, C.SMALL_GQA2_BF16],
                         ids=lambda c: c.name)
def test_attention_split_parity(cfg, split):
    plens = np.array([0, 700, 65], np.int32) if cfg.batch == 3 else np.array([300, 129], np.int32)
    _run(cfg, seed=4, prefix_lens=plens, attn_split=split)


# More than 32 rows take the batched-rows GEMM (all rows per workgroup, A and
# weights through an LDS ring) and the per-row LM-head top-k: batch 12 x N 3 =
# 36 LM-head rows and up to 36 QKV rows; the MHA config with batch 9 x N 4.
@pytest.mark.parametrize("cfg", [C.SMALL_GQA_BF16.with_(batch=12, name="small_gqa_bf16_b12"),
                                 C.SMALL_GQA_F32.with_(batch=12, name="small_gqa_f32_b12"),
                                 C.SMALL_MHA_BF16_D128.with_(batch=9, name="small_mha_bf16_d128_b9"),
                                 # 36 rows through every GEMM; the down projection's K = 1376
                                 # ends in a ragged 128-byte chunk
                                 C.SMALL_GQA_BF16.with_(batch=36, prefix=(0, 300),
                                                        name="small_gqa_bf16_b36"),
                                 # parallel heads over 12 x 3 rows (normalisation unfused)
                                 C.SMALL_GQA_BF16.with_(batch=12, cascade_ctx="parallel",
                                                        name="small_gqa_bf16_b12_parallel"),
                                 # more than 16 sequences: the residual GEMMs' row pass
                                 # writes the normalised rows of every consumer (fp32 and
                                 # bf16; cascade, parallel and self contexts)
                                 C.SMALL_GQA_F32.with_(batch=20, prefix=(0, 300),
                                                       name="small_gqa_f32_b20"),
                                 C.SMALL_GQA_BF16.with_(batch=20, cascade_ctx="parallel",
                                                        name="small_gqa_bf16_b20_parallel"),
                                 C.SMALL_GQA_BF16.with_(batch=20, cascade_ctx="self",
                                                        name="small_gqa_bf16_b20_self"),
                                 # more than 128 LM-head rows (48 x 3, 60 x 4): every row in
                                 # one 256-row tile per 128 columns (a ragged last column tile
                                 # at V = 1040); Q/K/V over 48..240 rows and the fusion and
                                 # residual GEMMs over more than 32 rows as split-K slices of
                                 # the eight-wave tiles; K = 1376 (not a multiple of 64) keeps
                                 # the down projection on the ring GEMM
                                 C.SMALL_GQA_BF16.with_(batch=48, prefix=(0, 300),
                                                        name="small_gqa_bf16_b48"),
                                 C.SMALL_MHA_BF16_D128.with_(batch=60, prefix=(1, 200),
                                                             name="small_mha_bf16_d128_b60")],
                         ids=lambda c: c.name)
def test_batched_rows_parity(cfg):
    _run(cfg, seed=5)


# More attention work units than resident waves: persistent waves, each taking
# every W-th unit of the dense numbering over ragged sequences (the debug
# forward, and every replay of the captured pass, run it again).  Default split
# and a split of 2 chunks; GQA head dim 64 and MHA head dim 128.
@pytest.mark.parametrize("graph", [False, True])
@pytest.mark.parametrize("cfg,split", [
    (C.SMALL_GQA_BF16.with_(batch=36, prefix=(0, 3000), name="small_gqa_bf16_b36_p3000"), None),
    (C.SMALL_MHA_BF16_D128.with_(batch=24, prefix=(0, 2000), name="small_mha_bf16_d128_b24"), 2),
    (C.SMALL_GQA8_BF16_D128.with_(batch=40, prefix=(0, 3000), name="small_gqa8_bf16_d128_b40"),
     None),
    (C.SMALL_GQA8_BF16_D128.with_(batch=24, prefix=(0, 2000), cascade_ctx="self",
                                  name="small_gqa8_bf16_d128_b24_self"), 2),
    (C.SMALL_GQA2_BF16.with_(batch=48, prefix=(0, 4000), name="small_gqa2_bf16_b48"), None)],
    ids=lambda v: v.name if hasattr(v, "name") else str(v))
def test_attention_queue_parity(cfg, split, graph):
    _run(cfg, seed=6, attn_split=split, graph=graph)


def test_topk_edge_values():
    """k = 1 (chain tree) and k = max (16)."""
    for k in (1, 16):
        _run(C.SMALL_GQA_BF16.with_(topk=k), seed=2, topk=k,
             prefix_lens=np.array([3, 129, 64], np.int32))


def test_planted_topk_is_exact():
    """LM-head rows planted so that one row's top-k has wide, known gaps: every
    rank of that row must be decided and match."""
    from oracle import feo
    from fe_synth import to_f64
    cfg = C.SMALL_GQA_BF16
    w = make_weights(cfg, 3)
    inp = make_inputs(cfg, 3, np.array([10, 0, 300], np.int32))
    ref = feo.draft_forward(cfg, w, inp)
    h = ref["hidden"][0, 1]                                   # x_1 of sequence 0
    g = to_f64(w.final_norm, "bf16")
    hn = g * h / np.sqrt(np.mean(h * h) + cfg.rms_eps)
    ids = np.array([17, 1999, 3, 640, 1024])
    scale = np.array([13.0, 11.0, 9.0, 7.0, 5.0])
    rows = (scale[:, None] * hn[None] / (hn @ hn)).astype(np.float32)
    b = rows.view(np.uint32)
    w.lm_head[ids] = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16).astype(np.uint16)
    rep, res, _ = _run(cfg, seed=3, weights=w, inputs=inp)
    np.testing.assert_array_equal(res["topk_draft"][0, 0], ids)


def test_deterministic_and_graph_replay_bitwise():
    import torch
    from paper_2509_20416_amd import Drafter
    cfg = C.SMALL_GQA_BF16
    w = make_weights(cfg, 4)
    inp = make_inputs(cfg, 4)
    dr = Drafter(cfg, w, max_batch=cfg.batch, max_prefix=int(inp.prefix_lens.max()))
    di = dr.upload_inputs(inp)
    a = {n: t.cpu().numpy() for n, t in dr.forward(di, logits=True, hidden=True).items()}
    b = {n: t.cpu().numpy() for n, t in dr.forward(di, logits=True, hidden=True).items()}
    for n in a:
        np.testing.assert_array_equal(a[n], b[n], err_msg=n)
    dr.set_graph_mode(True)
    out = dr.alloc_outputs(cfg.batch, cfg.topk, logits=True, hidden=True)
    for rep in range(4):                     # replays with eager work in between
        for t in out.values():
            t.zero_()
        dr.forward(di, out=out)
        torch.cuda.synchronize()
        _ = torch.ones(1000, device="cuda").sum().item()
        for n in a:
            np.testing.assert_array_equal(out[n].cpu().numpy(), a[n], err_msg=f"replay {rep} {n}")
    dr.close()


@pytest.mark.parametrize("graph", [False, True])
def test_tree_in_forward_matches_separate_build(graph):
    """The tree built inside fe_draft_forward (P_b from cu_prefix) equals
    fe_build_tree on the same top-k ids, bit for bit, on every replay."""
    import torch
    from paper_2509_20416_amd import Drafter
    cfg = C.SMALL_GQA_BF16
    w, inp = make_weights(cfg, 3), make_inputs(cfg, 3, np.array([0, 700, 65], np.int32))
    dr = Drafter(cfg, w, max_batch=cfg.batch, max_prefix=int(inp.prefix_lens.max()), graph=graph)
    di = dr.upload_inputs(inp)
    for rep in range(3):
        out = dr.alloc_outputs(cfg.batch, cfg.topk)
        t1 = dr.alloc_tree(cfg.batch, cfg.topk)
        dr.forward(di, out=out, tree=t1)
        t2 = dr.build_tree(di, out["topk_ids"])
        torch.cuda.synchronize()
        for n in t1:
            assert torch.equal(t1[n], t2[n]), (rep, n)
    dr.close()


def test_invalid_token_poisons_only_its_sequence():
    import torch
    from paper_2509_20416_amd import Drafter
    cfg = C.SMALL_GQA_BF16
    w = make_weights(cfg, 5)
    inp = make_inputs(cfg, 5)
    dr = Drafter(cfg, w, max_batch=cfg.batch, max_prefix=int(inp.prefix_lens.max()))
    inp.next_tokens = np.array([inp.next_tokens[0], cfg.target_vocab + 7, inp.next_tokens[2]],
                               np.int32)
    di = dr.upload_inputs(inp)
    out = dr.forward(di, hidden=True)
    torch.cuda.synchronize()
    hid = out["hidden"].cpu().numpy()
    assert np.isnan(hid[1]).all() and np.isfinite(hid[[0, 2]]).all()
    dr.close()


@pytest.mark.parametrize("cfg,plens,pmax", [
    (C.SMALL_GQA_BF16, [0, 700, 65], 100),                       # one unit per span
    (C.SMALL_GQA_F32, [0, 700, 65], 100),
    (C.SMALL_GQA_BF16.with_(batch=36, prefix=(0, 3000), name="small_gqa_bf16_b36_p3000"),
     None, 1500)],                                                # persistent waves
    ids=["bf16", "f32", "bf16_persistent"])
def test_prefix_above_bound_poisons_only_its_sequence(cfg, plens, pmax):
    """A P_b above the view's max_prefix (a contract violation the host cannot
    see) reads no cache row: that sequence's states from x_1 on are NaN, and
    every other sequence is unchanged: bit for bit when each sequence has its
    own attention units; with persistent waves the equal-chunk split moves
    (the bad sequence has one chunk left), so the others agree up to rounding."""
    import torch
    from paper_2509_20416_amd import Drafter
    w = make_weights(cfg, 8)
    inp = make_inputs(cfg, 8, None if plens is None else np.array(plens, np.int32))
    P = np.asarray(inp.prefix_lens)
    dr = Drafter(cfg, w, max_batch=cfg.batch, max_prefix=int(P.max()))
    ref = {n: t.cpu().numpy() for n, t in dr.forward(dr.upload_inputs(inp), hidden=True).items()}
    out = {n: t.cpu().numpy()
           for n, t in dr.forward(dr.upload_inputs(inp, max_prefix=pmax), hidden=True).items()}
    torch.cuda.synchronize()
    bad = P > pmax
    assert bad.any() and not bad.all()
    assert np.isnan(out["hidden"][bad][:, 1:]).all()
    np.testing.assert_array_equal(out["hidden"][bad][:, 0], ref["hidden"][bad][:, 0])
    if cfg.batch <= 16:
        for n in ("hidden", "topk_ids", "topk_probs", "topk_draft"):
            np.testing.assert_array_equal(out[n][~bad], ref[n][~bad], err_msg=n)
    else:
        from tests.parity import TOL, assert_rows_close
        assert_rows_close("hidden", out["hidden"][~bad], ref["hidden"][~bad], TOL[cfg.dtype])
        assert (out["topk_ids"][~bad] >= 0).all()
    dr.close()


@pytest.mark.parametrize("batch", [1, 3, 20])
def test_parallel_heads_graph_replays_match_eager(batch):
    """Under FE_CTX_PARALLEL every layer runs on a stream of its own (forked
    from the caller's stream and joined back; a captured pass holds them as
    parallel branches): eager passes and graph replays, with eager work
    between the replays, agree bit for bit, and both match the oracle."""
    import torch
    from paper_2509_20416_amd import Drafter
    cfg = C.SMALL_GQA_BF16.with_(cascade_ctx="parallel", batch=batch,
                                 name=f"small_gqa_bf16_b{batch}_parallel")
    rep, _, _ = _run(cfg, seed=5, graph=True)
    w, inp = make_weights(cfg, 5), make_inputs(cfg, 5)
    dr = Drafter(cfg, w, max_batch=batch, max_prefix=int(inp.prefix_lens.max()))
    di = dr.upload_inputs(inp)
    eager = {n: t.cpu().numpy() for n, t in dr.forward(di, logits=True, hidden=True).items()}
    dr.set_graph_mode(True)
    out = dr.alloc_outputs(batch, cfg.topk, logits=True, hidden=True)
    for r in range(4):
        for t in out.values():
            t.zero_()
        dr.forward(di, out=out)
        torch.cuda.synchronize()
        _ = torch.ones(1000, device="cuda").sum().item()
        for n in eager:
            np.testing.assert_array_equal(out[n].cpu().numpy(), eager[n], err_msg=f"replay {r} {n}")
    dr.close()


# --- paper-shaped workloads at full size, in the configuration the bench times -----------
def _drift_guard(rep, cfg):
    """Full-size errors stay within the drift guard (tests/parity.py DRIFT)."""
    from tests.parity import DRIFT
    for n in ("hidden_err", "logit_err"):
        assert rep[n] <= DRIFT[cfg.dtype], (n, rep[n])


@pytest.mark.timeout(900)
def test_llama8b_b1_full():
    rep, _, _ = _run(C.LLAMA8B_BF16_B1, seed=0, graph=True)
    _drift_guard(rep, C.LLAMA8B_BF16_B1)


@pytest.mark.timeout(900)
def test_llama8b_b1_parallel_heads_full():
    """The ablation without the cascade, at the 8B shapes the bench times it on."""
    cfg = C.LLAMA8B_BF16_B1.with_(cascade_ctx="parallel")
    rep, _, _ = _run(cfg, seed=0, graph=True)
    _drift_guard(rep, cfg)


@pytest.mark.timeout(900)
def test_vicuna13b_b1_full():
    rep, _, _ = _run(C.VICUNA13B_BF16_B1, seed=0, graph=True)
    _drift_guard(rep, C.VICUNA13B_BF16_B1)


@pytest.mark.timeout(1200)
def test_llama70b_b1_full():
    """Element-wise cascade states and logits at the 70B shapes (8 query heads per
    KV head, head dim 128, P = 4096)."""
    rep, _, _ = _run(C.LLAMA70B_BF16_B1, seed=0, graph=True)
    _drift_guard(rep, C.LLAMA70B_BF16_B1)


@pytest.mark.timeout(1200)
def test_llama8b_b32_ragged_all():
    """Batch 32, P_b ~ U[256, 8192], N = 7: every sequence against the oracle."""
    rep, _, _ = _run(C.LLAMA8B_BF16_B32, seed=0, graph=True)
    _drift_guard(rep, C.LLAMA8B_BF16_B32)


def _planted_lm_head(cfg, w, ref_hidden, b, base_ids, top=None):
    """LM-head rows planted so that every level of sequence b has a top-k with wide,
    known gaps: for level l the k rows s_rho * u_l, with u_l the dual basis of the
    N final-normalised cascade states of b (u_l . hn_j = 1 if j = l else 0), so a
    planted row scores s_rho at its own level and about 0 at the others.  Returns
    the planted draft ids [N, k] in rank order."""
    from fe_synth import to_f64
    N, k = cfg.n_layers, cfg.topk
    g = to_f64(w.final_norm, cfg.dtype)
    hs = ref_hidden[b, 1:N + 1]
    hn = g * hs / np.sqrt(np.mean(hs * hs, axis=1, keepdims=True) + cfg.rms_eps)   # [N, d]
    U = np.linalg.pinv(hn)                                                          # [d, N]
    top = top if top is not None else 2.0 * k + 14.0
    scale = top - 2.0 * np.arange(k)                  # gaps of 2, lowest well above random logits
    ids = np.asarray(base_ids, np.int64).reshape(N, k)
    rows = (scale[None, :, None] * U.T[:, None, :]).reshape(N * k, -1).astype(np.float32)
    if cfg.dtype == "bf16":
        bits = rows.view(np.uint32)
        w.lm_head[ids.reshape(-1)] = ((bits + 0x7FFF + ((bits >> 16) & 1)) >> 16).astype(np.uint16)
    else:
        w.lm_head[ids.reshape(-1)] = rows
    return ids


@pytest.mark.timeout(1200)
@pytest.mark.parametrize("cfg", [C.LLAMA8B_BF16_B1, C.LLAMA70B_BF16_B1], ids=lambda c: c.name)
def test_planted_topk_full_size(cfg):
    """At the full 8B / 70B shapes, in graph mode: every level of the sequence gets a
    planted top-k, so every one of the N * k ranks is decided by the oracle and must
    match through the 500-tile LM head and the top-k merge."""
    from oracle import feo
    w = make_weights(cfg, 0)
    inp = make_inputs(cfg, 0)
    ref = feo.draft_forward(cfg, w, inp, want_logits=False)
    rng = np.random.default_rng(11)
    ids = _planted_lm_head(cfg, w, ref["hidden"], 0,
                           rng.choice(cfg.draft_vocab, cfg.n_layers * cfg.topk, replace=False))
    rep, res, _ = _run(cfg, seed=0, graph=True, weights=w, inputs=inp)
    assert rep["decided"] == rep["ranks"] == cfg.n_layers * cfg.topk, rep
    np.testing.assert_array_equal(res["topk_draft"][0], ids)
