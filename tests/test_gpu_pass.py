"""Batch-1 pass shapes (widths multiples of 512, up to eight cascade layers)
through the one-launch-per-stage pass against the oracle, and the persistent
batch-1 pass (stages between attention launches as one launch that hands
results on through tagged words).  Rules in tests/parity.py."""
import os

import numpy as np
import pytest

from fe_synth import configs as C
from fe_synth import make_inputs, make_weights

pytestmark = pytest.mark.gpu

PASS_SMALL = [C.SMALL_PASS_GQA, C.SMALL_PASS_GQA8, C.SMALL_PASS_MHA_N8]

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


@pytest.mark.parametrize("graph", [False, True])
@pytest.mark.parametrize("ctx", ["cascade", "self", "parallel"])
@pytest.mark.parametrize("cfg", PASS_SMALL, ids=lambda c: c.name)
def test_batch1_pass_shapes(cfg, ctx, graph):
    rep, _, _ = _run(cfg.with_(cascade_ctx=ctx), seed=11, graph=graph)
    assert not rep["persistent"]


def test_pass_mode_values():
    from paper_2509_20416_amd import Drafter
    from paper_2509_20416_amd.fe import FeError
    cfg = C.SMALL_PASS_GQA
    dr = Drafter(cfg, make_weights(cfg, 1), max_batch=1, max_prefix=cfg.prefix)
    try:
        with pytest.raises(FeError):
            dr.set_pass_mode(2)
        dr.set_pass_mode(0)
        dr.set_pass_mode(1)
    finally:
        dr.close()


@pytest.mark.parametrize("graph", [False, True])
@pytest.mark.parametrize("ctx", ["cascade", "self", "parallel"])
@pytest.mark.parametrize("cfg", PASS_SMALL, ids=lambda c: c.name)
def test_persistent_pass_parity(cfg, ctx, graph):
    rep, _, _ = _run(cfg.with_(cascade_ctx=ctx), seed=11, graph=graph, pass_mode=0)
    assert rep["persistent"], "the persistent pass did not run"


@pytest.mark.parametrize("P", [0, 1, 64, 65])
def test_persistent_pass_short_prefixes(P):
    """Empty and one-chunk prefixes (the attention's cascade keys alone, one key)."""
    rep, _, _ = _run(C.SMALL_PASS_GQA, seed=12, prefix_lens=np.array([P], np.int32),
                     pass_mode=0)
    assert rep["persistent"]


def test_persistent_matches_per_stage_launches():
    """Same inputs through both pass modes: results agree to the storage tolerance,
    top-k ids wherever the logits are well separated, the tree structure exactly."""
    import torch
    from paper_2509_20416_amd import Drafter
    from tests.parity import TOL, assert_rows_close
    cfg = C.SMALL_PASS_GQA8
    w, inp = make_weights(cfg, 13), make_inputs(cfg, 13)
    res = {}
    for mode in (0, 1):
        dr = Drafter(cfg, w, max_batch=1, max_prefix=int(inp.prefix_lens.max()))
        dr.set_pass_mode(mode)
        di = dr.upload_inputs(inp)
        res[mode] = {n: t.cpu().numpy() for n, t in dr.forward(di, logits=True, hidden=True).items()}
        st = dr.pass_status()
        assert st & 1 == 0
        assert bool(st & (1 << 16)) == (mode == 0)
        dr.close()
    assert_rows_close("hidden", res[0]["hidden"], res[1]["hidden"], TOL["bf16"])
    assert_rows_close("logits", res[0]["logits"], res[1]["logits"], TOL["bf16"])


def test_persistent_pass_inputs_change_between_passes():
    """Three passes with different features and next tokens on one handle (graph
    replay of the same buffers, refilled between passes), each equal bit for bit
    to a fresh handle's pass on the same inputs."""
    import torch
    from paper_2509_20416_amd import Drafter
    import copy
    cfg = C.SMALL_PASS_GQA
    w = make_weights(cfg, 14)
    base = make_inputs(cfg, 21)
    inps = []
    for s in (21, 22, 23):        # same prefix caches, new features and next token
        other = make_inputs(cfg, s)
        inp = copy.copy(base)
        inp.features, inp.next_tokens = other.features, other.next_tokens
        inps.append(inp)
    dr = Drafter(cfg, w, max_batch=1, max_prefix=cfg.prefix, graph=True)
    dr.set_pass_mode(0)
    di = dr.upload_inputs(inps[0])
    out = dr.alloc_outputs(1, cfg.topk, logits=True, hidden=True)
    for i, inp in enumerate(inps):
        d2 = dr.upload_inputs(inp)
        di.features.copy_(d2.features)
        di.next_tokens.copy_(d2.next_tokens)
        for t in out.values():
            t.zero_()
        dr.forward(di, out=out)
        torch.cuda.synchronize()
        assert dr.pass_status() & 1 == 0
        got = {n: t.cpu().numpy() for n, t in out.items()}
        fresh = Drafter(cfg, w, max_batch=1, max_prefix=cfg.prefix)
        fresh.set_pass_mode(0)
        want = {n: t.cpu().numpy()
                for n, t in fresh.forward(fresh.upload_inputs(inp), logits=True, hidden=True).items()}
        fresh.close()
        for n in want:
            np.testing.assert_array_equal(got[n], want[n], err_msg=f"pass {i} {n}")
    dr.close()


def test_persistent_pass_graph_replays_bitwise():
    import torch
    from paper_2509_20416_amd import Drafter
    cfg = C.SMALL_PASS_GQA8
    w, inp = make_weights(cfg, 15), make_inputs(cfg, 15)
    dr = Drafter(cfg, w, max_batch=1, max_prefix=int(inp.prefix_lens.max()))
    dr.set_pass_mode(0)
    di = dr.upload_inputs(inp)
    a = {n: t.cpu().numpy() for n, t in dr.forward(di, logits=True, hidden=True).items()}
    dr.set_graph_mode(True)
    out = dr.alloc_outputs(1, cfg.topk, logits=True, hidden=True)
    tree = dr.alloc_tree(1, cfg.topk)
    for rep in range(4):                     # replays with eager work in between
        for t in out.values():
            t.zero_()
        dr.forward(di, out=out, tree=tree)
        torch.cuda.synchronize()
        _ = torch.ones(1000, device="cuda").sum().item()
        for n in a:
            np.testing.assert_array_equal(out[n].cpu().numpy(), a[n], err_msg=f"replay {rep} {n}")
        t2 = dr.build_tree(di, out["topk_ids"])
        torch.cuda.synchronize()
        for n in tree:
            assert torch.equal(tree[n], t2[n]), (rep, n)
    assert dr.pass_status() == (1 << 16)
    dr.close()


@pytest.mark.timeout(900)
@pytest.mark.parametrize("cfg", [C.LLAMA8B_BF16_B1, C.LLAMA70B_BF16_B1], ids=lambda c: c.name)
def test_persistent_pass_full_size(cfg):
    """The persistent pass at the paper's 8B and 70B batch-1 shapes (one
    workgroup per compute unit handing every stage's rows on through tagged
    words; the 70B activations take the largest workgroup variant), graph
    mode as the bench times it: element-wise cascade states and logits
    against the oracle, the top-k rule, the tree."""
    from tests.parity import DRIFT
    rep, _, _ = _run(cfg, seed=0, graph=True, pass_mode=0)
    assert rep["persistent"], "the persistent pass did not run"
    for n in ("hidden_err", "logit_err"):
        assert rep[n] <= DRIFT[cfg.dtype], (n, rep[n])
