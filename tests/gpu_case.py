"""Runs one seeded workload through the GPU library and through the oracle and
applies the parity rules (used by the GPU tests and the smoke check)."""
from __future__ import annotations

import sys
import time

import numpy as np

from fe_synth import make_inputs, make_weights
from tests.parity import (TOL, assert_rows_close, check_topk, check_topk_self_consistent)
from tests.treecheck import check_tree


def log(*a):
    print("[gpu-case]", *a, flush=True)
    sys.stdout.flush()


def run_case(cfg, seed=0, prefix_lens=None, topk=None, sample=None, graph=False,
             with_debug=True, weights=None, inputs=None, feo=None, check_tree_struct=True,
             attn_split=None, pass_mode=None):
    import torch
    from paper_2509_20416_amd import Drafter
    if feo is None:
        from oracle import feo
    k = int(topk or cfg.topk)
    t0 = time.time()
    w = weights if weights is not None else make_weights(cfg, seed)
    inp = inputs if inputs is not None else make_inputs(cfg, seed, prefix_lens)
    plens = np.asarray(inp.prefix_lens, np.int32)
    B = len(plens)
    log(f"{cfg.name}: ctx={cfg.cascade_ctx} B={B} P=[{plens.min()},{plens.max()}] k={k} "
        f"inputs ready in {time.time() - t0:.1f}s")
    dr = Drafter(cfg, w, max_batch=B, max_prefix=int(plens.max()), max_topk=max(k, cfg.topk),
                 graph=graph)
    if attn_split is not None:
        dr.set_attention_split(attn_split)
    if pass_mode is not None:
        dr.set_pass_mode(pass_mode)
    di = dr.upload_inputs(inp)
    out = dr.forward(di, k)                                   # the benchmarked configuration
    tree = dr.build_tree(di, out["topk_ids"], k)
    torch.cuda.synchronize()
    status = dr.pass_status()
    assert status & 1 == 0, f"persistent pass gave up waiting (status {status:#x})"
    persistent = bool(status & (1 << 16))
    res = {n: t.cpu().numpy() for n, t in out.items()}
    tr = {n: t.cpu().numpy() for n, t in tree.items()}
    if with_debug:
        dbg = dr.forward(di, k, logits=True, hidden=True)
        torch.cuda.synchronize()
        assert dr.pass_status() & 1 == 0
        dbg = {n: t.cpu().numpy() for n, t in dbg.items()}
        for n in ("topk_ids", "topk_probs", "topk_draft"):   # debug outputs change nothing
            np.testing.assert_array_equal(dbg[n], res[n], err_msg=n)
    log(f"{cfg.name}: GPU done in {time.time() - t0:.1f}s")

    idx = list(range(B)) if sample is None else list(sample)
    t1 = time.time()
    ref = feo.draft_forward(cfg, w, inp, topk=k, batch_index=idx)
    log(f"{cfg.name}: oracle on {len(idx)} sequence(s) in {time.time() - t1:.1f}s")
    tol = TOL[cfg.dtype]
    N = cfg.n_layers
    report = {"persistent": persistent}
    if with_debug:
        report["hidden_err"] = assert_rows_close("hidden", dbg["hidden"][idx], ref["hidden"], tol)
        report["logit_err"] = assert_rows_close("logits", dbg["logits"][idx], ref["logits"], tol)
        check_topk_self_consistent(dbg["topk_draft"].reshape(B * N, k),
                                   dbg["logits"].reshape(B * N, -1))
    dec, tot = check_topk(res["topk_draft"][idx].reshape(-1, k),
                          res["topk_probs"][idx].reshape(-1, k),
                          ref["logits"].reshape(len(idx) * N, -1),
                          ref["topk_draft"].reshape(-1, k), tol)
    np.testing.assert_array_equal(res["topk_ids"], w.d2t[res["topk_draft"]])
    report["decided"], report["ranks"] = dec, tot
    # tree: structure bit-exact against the oracle's tree, tokens follow the top-k rule
    rt = feo.build_tree(N, k, inp.next_tokens[idx], ref["topk_ids"], plens[idx])
    for n in ("parents", "depth", "positions", "mask", "retrieve"):
        np.testing.assert_array_equal(tr[n][idx], rt[n], err_msg=f"tree {n}")
    np.testing.assert_array_equal(tr["tokens"][:, 0], inp.next_tokens)
    np.testing.assert_array_equal(tr["tokens"][:, 1:].reshape(B, N, k), res["topk_ids"])
    if check_tree_struct:
        for b in range(B):
            check_tree(tr, b, N, k, inp.next_tokens[b], res["topk_ids"][b], plens[b])
    log(f"{cfg.name}: parity ok {report}")
    dr.close()
    return report, res, tr
