"""GPU parity of the speculative-sampling acceptance (fe_accept_sample,
through the C ABI) against the oracle's feo_accept_sample on the same trees,
distributions and uniforms.

Every decision of the walk (accept tests, draw order of sampled children,
the final inverse-CDF draw) compares floating-point values; the oracle
reports per sequence how close its closest decision came to its threshold
(relative).  Sequences whose margin exceeds 1e-4 (well above fp32 rounding
of the sums involved) must match the oracle exactly; the others must still be a
valid outcome: accepted tokens along one root->leaf path of the tree, its
retrieve row, a final token inside the target vocabulary."""
import os

import numpy as np
import pytest

from fe_synth import configs as C
from fe_synth import make_uniforms, make_weights

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2509_20416_amd import fe
    fe.lib()


def log(*a):
    print("[accept-sample]", *a, flush=True)


def _cycle(cfg, B, k, T, sampled, seed, philox=None):
    """Host arrays of one cycle: draft logits, candidates (drawn or top-k,
    listed most probable first), the tree, target distributions that put part
    of their mass where the draft does, and the uniforms."""
    from oracle import feo
    rng = np.random.default_rng(seed)
    N, V, Vt = cfg.n_layers, cfg.draft_vocab, cfg.target_vocab
    w = make_weights(cfg.with_(n_layers=1), 0)
    d2t = w.d2t
    z = (rng.standard_normal((B, N, V)) * 2.5).astype(np.float32)
    if philox is None:
        ud = make_uniforms((B, N, V), seed=seed + 1)
    else:   # the counter-based stream the seeded pass draws from
        ud = feo.philox_uniforms(philox[0], philox[1], 0, B * N * V).reshape(B, N, V)
    keys = z / T - (np.log(-np.log(ud.astype(np.float64))) if sampled else 0.0)
    cand = np.argsort(-keys, axis=-1, kind="stable")[..., :k]
    zc = np.take_along_axis(z, cand, -1)
    cand = np.take_along_axis(cand, np.argsort(-zc, axis=-1, kind="stable"), -1).astype(np.int32)
    roots = rng.integers(0, Vt, B).astype(np.int32)
    tree = feo.build_tree(N, k, roots, d2t[cand], np.zeros(B, np.int32))
    Tn = 1 + N * k
    q = np.exp(z / T - (z / T).max(-1, keepdims=True))
    q /= q.sum(-1, keepdims=True)
    tp = np.zeros((B, Tn, Vt), np.float32)
    # the rest of the target's mass on 64 ids per row, so that the final
    # inverse-CDF draw has bins far wider than fp32 rounding of the sums
    noise = np.zeros((B, Tn, Vt), np.float32)
    for b in range(B):
        for n in range(Tn):
            ids = rng.choice(Vt, 64, replace=False)
            noise[b, n, ids] = rng.gamma(1.0, size=64)
    noise /= noise.sum(-1, keepdims=True)
    dep = tree["depth"]
    for b in range(B):
        for n in range(Tn):
            lvl = min(dep[b, n] + 1, N)           # the level drafted after this node
            tp[b, n, d2t] = 0.75 * q[b, lvl - 1]
            tp[b, n] += 0.25 * noise[b, n]
    u = make_uniforms((B, N * k + 1), seed=seed + 2)
    return dict(z=z, ud=ud if sampled else None, cand=cand, tree=tree, tp=tp, u=u, d2t=d2t, w=w)


def _run(cfg, B, k, T, sampled, seed, philox=None):
    import torch
    from oracle import feo
    from paper_2509_20416_amd import Drafter
    cfg = cfg.with_(batch=B, topk=k)
    cy = _cycle(cfg, B, k, T, sampled, seed, philox)
    N = cfg.n_layers
    log(f"{cfg.name}: N={N} k={k} B={B} T={T} sampled={sampled} V={cfg.draft_vocab} "
        f"Vt={cfg.target_vocab}")
    dr = Drafter(cfg.with_(n_layers=N), _weights_with_layers(cy["w"], N), max_batch=B,
                 max_prefix=0, max_topk=k)
    dev = dr.device
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    tree = {n: t(a) for n, a in cy["tree"].items()}
    if philox is None:
        got = dr.accept_sample(tree, t(cy["cand"]), t(cy["z"]), t(cy["tp"]), t(cy["u"]),
                               temperature=T,
                               draft_uniforms=t(cy["ud"]) if cy["ud"] is not None else None, topk=k)
    else:
        so = torch.tensor(list(philox), dtype=torch.int64, device=dev)
        got = dr.accept_sample(tree, t(cy["cand"]), t(cy["z"]), t(cy["tp"]), t(cy["u"]),
                               temperature=T, draft_seed_offset=so, topk=k)
    torch.cuda.synchronize()
    got = {n: a.cpu().numpy() for n, a in got.items()}
    ref = feo.accept_sample(N, k, cy["tree"]["tokens"], cy["tree"]["retrieve"], cy["cand"], cy["z"],
                            T, cy["d2t"], cy["tp"], cy["u"], draft_uniforms=cy["ud"])
    dr.close()
    tok, ret = cy["tree"]["tokens"], cy["tree"]["retrieve"]
    firm = ref["margin"] > 1e-4
    for b in range(B):
        L, row = got["accept_len"][b], got["accept_path"][b]
        assert 0 <= L <= N and 0 <= row < ret.shape[1]
        path = ret[b, row, :L + 1]
        assert path[0] == 0 and (path >= 0).all()
        np.testing.assert_array_equal(got["accepted"][b, :L], tok[b, path[1:]])
        assert 0 <= got["accepted"][b, L] < cfg.target_vocab
        assert (got["accepted"][b, L + 1:] == -1).all()
        if firm[b]:
            for n in ("accept_len", "accept_path", "accepted"):
                np.testing.assert_array_equal(got[n][b], ref[n][b], err_msg=f"seq {b} {n}")
    lens = np.bincount(got["accept_len"], minlength=N + 1)
    log(f"{cfg.name}: {int(firm.sum())}/{B} sequences decided and equal; accept lengths {lens.tolist()}")
    assert firm.sum() >= 0.6 * B
    return got


def _weights_with_layers(w, N):
    w.layers = w.layers[:1] * N
    return w


SMALL_V = C.SMALL_GQA_BF16          # draft vocab 2000 inside a 5003-token target vocab
CASES = [
    (SMALL_V, 32, 5, 1.0, True),
    (SMALL_V, 32, 5, 0.7, True),
    (SMALL_V, 16, 1, 1.0, True),
    (SMALL_V, 16, 16, 1.0, True),
    (SMALL_V, 32, 5, 1.0, False),
    (C.TINY_F32_B1.with_(n_layers=6), 8, 4, 1.0, True),   # identity map
    # one sequence: every node's target row reduced by a pre-pass first
    (SMALL_V, 1, 5, 1.0, True),
    (SMALL_V, 1, 4, 1.0, False),
    (C.TINY_F32_B1.with_(n_layers=6), 1, 4, 1.0, True),
    (SMALL_V, 2, 5, 1.0, True),
    (SMALL_V, 4, 16, 0.7, True),
    (SMALL_V, 3, 5, 1.0, False),
    (C.TINY_F32_B1.with_(n_layers=6), 4, 3, 1.0, True),
]


@pytest.mark.parametrize("cfg,B,k,T,sampled", CASES,
                         ids=[f"{c.name}-B{b}-k{k}-T{t}-{'s' if s else 'top'}"
                              for c, b, k, t, s in CASES])
def test_accept_sample_parity(cfg, B, k, T, sampled):
    _run(cfg, B, k, T, sampled, seed=B * 100 + k)


@pytest.mark.parametrize("B,k,T", [(32, 5, 1.0), (16, 16, 0.7), (4, 5, 1.0), (1, 5, 1.0)])
def test_accept_sample_seeded_parity(B, k, T):
    """Children drawn from the counter-based stream (fe_draft_sample_seeded):
    the acceptance recomputes their uniforms from (seed, offset) in device
    memory (fe_accept_sample_seeded); the oracle reads the same stream's
    uniforms from an array."""
    _run(SMALL_V, B, k, T, True, seed=B * 100 + k + 1, philox=(77, 3))


def test_accept_sample_8b_vocabularies():
    """The 8B vocabularies (32000 draft ids in 128256 target ids), N = 5, k = 8."""
    cfg = C.LLAMA8B_BF16_B1.with_(hidden=128, n_q_heads=1, n_kv_heads=1, head_dim=128,
                                  intermediate=256, name="llama8b_vocab_only")
    _run(cfg, 4, 8, 1.0, True, seed=8)
