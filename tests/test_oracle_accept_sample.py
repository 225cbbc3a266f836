"""Pins of the oracle's speculative-sampling acceptance at T > 0 (CPU only).

The property that defines it (Section 2.4: verification is lossless): every
emitted token follows the target's distribution given the tokens before it,
whatever the draft proposed.  Checked by Monte Carlo over many cycles with
candidates drawn without replacement from the draft distribution (the
drafting rule the oracle's sampling pins fix) or taken as the top-k list, on
a 6-token draft vocabulary mapped into an 8-token target vocabulary:
* the first emitted token follows the target's distribution at the root;
* after an accepted first token x, the second follows the target's
  distribution after x;
* with one candidate per level the first test accepts with probability
  sum_x min(p(x), q(x)) (classical speculative sampling).
"""
import numpy as np
import pytest

V, VT = 6, 8
D2T = np.array([0, 2, 3, 5, 6, 7], np.int32)   # target ids 1 and 4 are outside the draft vocab


def _dist(rng, n, conc=1.0):
    p = rng.gamma(conc, size=n)
    return p / p.sum()


def _cycles(feo, N, k, R, T, seed, sampled=True):
    """R independent cycles with fixed draft logits and target tables;
    candidates drawn without replacement (sampled) or the top-k list."""
    rng = np.random.default_rng(seed)
    z = (rng.standard_normal((N, V)) * 1.5).astype(np.float32)
    P1 = _dist(rng, VT)
    P2 = np.stack([_dist(rng, VT) for _ in range(VT)])          # after token x1
    P3 = np.stack([_dist(rng, VT) for _ in range(VT * VT)])     # after (x1, x2)
    # candidates: k draws without replacement from softmax(z / T) (Gumbel-top-k),
    # listed most probable first
    ud = np.clip(rng.uniform(0, 1, (R, N, V)), 2.0 ** -24, 1 - 2.0 ** -24).astype(np.float32)
    g = -np.log(-np.log(ud.astype(np.float64))) if sampled else 0.0
    keys = np.broadcast_to(z[None] / T + g, (R, N, V))
    cand = np.argsort(-keys, axis=-1, kind="stable")[..., :k]
    cand = np.take_along_axis(cand, np.argsort(-z[np.arange(N)[None, :, None], cand], axis=-1,
                                               kind="stable"), -1).astype(np.int32)
    roots = np.full(R, 1, np.int32)
    tree = feo.build_tree(N, k, roots, D2T[cand], np.zeros(R, np.int32))
    tok, par, dep = tree["tokens"], tree["parents"], tree["depth"]
    Tn = 1 + N * k
    tp = np.empty((R, Tn, VT), np.float32)
    tp[:, 0] = P1
    rows = np.arange(R)
    for n in range(1, Tn):
        lvl = dep[:, n]
        x1 = np.where(lvl == 1, tok[:, n], tok[rows, np.clip(par[:, n], 0, None)])
        tp[lvl == 1, n] = P2[tok[lvl == 1, n]]
        m = lvl == 2
        tp[m, n] = P3[x1[m] * VT + tok[m, n]]
    u = np.random.default_rng(seed + 1).uniform(0, 1, (R, N * k + 1)).astype(np.float32)
    u = np.clip(u, 2.0 ** -24, 1 - 2.0 ** -24).astype(np.float32)
    zl = np.repeat(z[None], R, axis=0)
    out = feo.accept_sample(N, k, tok, tree["retrieve"], cand, zl, T, D2T, tp, u,
                            draft_uniforms=ud if sampled else None)
    return out, dict(z=z, P1=P1, P2=P2, cand=cand, tok=tok)


def _check_freq(samples, p, sigmas=5.0):
    n = len(samples)
    freq = np.bincount(samples, minlength=len(p)) / n
    sd = np.sqrt(p * (1 - p) / n)
    assert (np.abs(freq - p) <= sigmas * sd + 1.0 / n).all(), (freq, p)


@pytest.mark.parametrize("k,T,sampled", [(1, 1.0, True), (3, 1.0, True), (3, 0.7, True),
                                         (6, 1.0, True), (3, 1.0, False), (1, 0.5, False)])
def test_emitted_tokens_follow_the_target(feo, k, T, sampled):
    N, R = 2, 60000
    out, ctx = _cycles(feo, N, k, R, T, seed=10 + k, sampled=sampled)
    acc, L = out["accepted"], out["accept_len"]
    assert ((L >= 0) & (L <= N)).all()
    assert (acc[np.arange(R), L] >= 0).all() and (acc[:, :1] < VT).all()
    _check_freq(acc[:, 0], ctx["P1"])
    for x1 in range(VT):
        sel = (L >= 1) & (acc[:, 0] == x1)
        if sel.sum() >= 2000:
            _check_freq(acc[sel, 1], ctx["P2"][x1])
    # accepted tokens are the tree's, along one retrieve path
    assert (out["accept_path"] >= 0).all()


def test_top_k_children_accept_with_their_target_mass(feo):
    """Unsampled children (the top-k list) against point masses: some child is
    accepted exactly with the target's mass on the k listed tokens."""
    N, k, R = 1, 3, 60000
    out, ctx = _cycles(feo, N, k, R, 1.0, seed=31, sampled=False)
    expect = ctx["P1"][D2T[ctx["cand"][0, 0]]].sum()
    got = (out["accept_len"] >= 1).mean()
    assert abs(got - expect) <= 5 * np.sqrt(expect * (1 - expect) / R), (got, expect)


def test_single_candidate_is_classical_speculative_sampling(feo):
    N, k, R, T = 1, 1, 60000, 1.0
    out, ctx = _cycles(feo, N, k, R, T, seed=21)
    z = ctx["z"][0]
    q = np.exp(z - z.max())
    q /= q.sum()
    qt = np.zeros(VT)
    qt[D2T] = q
    expect = np.minimum(ctx["P1"], qt).sum()
    got = (out["accept_len"] >= 1).mean()
    assert abs(got - expect) <= 5 * np.sqrt(expect * (1 - expect) / R), (got, expect)


def test_extreme_uniforms(feo):
    """u -> 0 accepts the first child at every level (the backbone); the last
    uniform then picks the target's first token with mass."""
    N, k = 3, 2
    rng = np.random.default_rng(3)
    z = rng.standard_normal((1, N, V)).astype(np.float32)
    cand = np.argsort(-z[0], axis=-1)[:, :k][None].astype(np.int32)
    tree = feo.build_tree(N, k, np.array([1], np.int32), D2T[cand], np.zeros(1, np.int32))
    tp = np.full((1, 1 + N * k, VT), 1.0 / VT, np.float32)
    u = np.full((1, N * k + 1), 2.0 ** -24, np.float32)
    ud = np.full((1, N, V), 0.5, np.float32)
    out = feo.accept_sample(N, k, tree["tokens"], tree["retrieve"], cand, z, 1.0, D2T, tp, u,
                            draft_uniforms=ud)
    assert out["accept_len"][0] == N
    np.testing.assert_array_equal(out["accepted"][0, :N], D2T[cand[0, :, 0]])
    assert out["accepted"][0, N] == 0
    # leaves in node order: the side branches of levels 1..N-1, then the backbone leaf
    assert out["accept_path"][0] == (N - 1) * (k - 1)
