"""Pins of the oracle's stochastic drafting (CPU only).

Section 2.2 samples k candidates per level from q_{t+i} (Section 3 reports
temperature 1).  The oracle draws them without replacement through the
Gumbel-top-k construction from caller-supplied uniforms.  Pinned against
probability itself, not against the formula:
* the first draw follows softmax(z / T) (binomial bounds over many draws);
* pairs and triples follow successive sampling without replacement
  (Plackett-Luce: P(a then b) = p_a p_b / (1 - p_a), summed over orders);
* constant noise reduces to the greedy top-k; candidates are listed most
  probable first with their softmax(z / T) probabilities.
"""
import itertools

import numpy as np
import pytest

from fe_synth import make_inputs, make_uniforms, make_weights

from tests.test_oracle_pins import PIN


def _same_rows(cfg, R, seed=3, lm_gain=40.0):
    """R identical sequences (prefix 0): every row has the same logits."""
    w = make_weights(cfg, seed)
    w.lm_head = (w.lm_head * np.float32(lm_gain)).astype(np.float32)
    one = make_inputs(cfg.with_(batch=1), seed, prefix_lens=np.zeros(1, np.int32))
    inp = make_inputs(cfg.with_(batch=R), seed, prefix_lens=np.zeros(R, np.int32))
    inp.features = np.ascontiguousarray(np.repeat(one.features, R, axis=0))
    inp.next_tokens = np.repeat(one.next_tokens, R).astype(np.int32)
    return w, inp


def _softmax(z):
    e = np.exp(z - z.max(-1, keepdims=True))
    return e / e.sum(-1, keepdims=True)


def _within(freq, p, R, sigmas=5.0):
    sd = np.sqrt(np.maximum(p * (1 - p), 1e-12) / R)
    return np.abs(freq - p) <= sigmas * sd + 1.0 / R


@pytest.mark.parametrize("T", [1.0, 0.5])
def test_first_draw_follows_softmax(feo, T):
    cfg = PIN.with_(n_layers=2)
    R = 20000
    w, inp = _same_rows(cfg, R)
    u = make_uniforms((R, cfg.n_layers, cfg.draft_vocab), seed=11)
    out = feo.draft_forward(cfg, w, inp, topk=1, temperature=T, uniforms=u)
    z = out["logits"]
    assert np.array_equal(z, np.repeat(z[:1], R, axis=0))
    for i in range(cfg.n_layers):
        p = _softmax(z[0, i] / T)
        assert p.max() > 0.1            # a peaked distribution, not a flat one
        freq = np.bincount(out["topk_draft"][:, i, 0], minlength=cfg.draft_vocab) / R
        assert _within(freq, p, R).all(), np.abs(freq - p).max()


@pytest.mark.parametrize("k", [2, 3])
def test_sets_follow_sampling_without_replacement(feo, k):
    cfg = PIN.with_(n_layers=1, draft_vocab=6, topk=k)
    R = 40000
    w, inp = _same_rows(cfg, R, lm_gain=5.0)
    u = make_uniforms((R, 1, cfg.draft_vocab), seed=12 + k)
    out = feo.draft_forward(cfg, w, inp, topk=k, uniforms=u)
    p = _softmax(out["logits"][0, 0])
    expect = {}
    for combo in itertools.combinations(range(cfg.draft_vocab), k):
        tot = 0.0
        for order in itertools.permutations(combo):
            pr, left = 1.0, 1.0
            for a in order:
                pr *= p[a] / left
                left -= p[a]
            tot += pr
        expect[combo] = tot
    assert abs(sum(expect.values()) - 1.0) < 1e-9
    assert sorted(p)[-k - 1] > 0.02      # every rank has real mass
    sets = [tuple(sorted(r)) for r in out["topk_draft"][:, 0]]
    counts = {c: 0 for c in expect}
    for s in sets:
        counts[s] += 1
    freq = np.array([counts[c] / R for c in expect])
    pe = np.array(list(expect.values()))
    assert _within(freq, pe, R).all(), np.abs(freq - pe).max()


def test_listing_order_and_probabilities(feo):
    cfg = PIN
    T = 0.7
    w = make_weights(cfg, 6)
    inp = make_inputs(cfg, 6)
    u = make_uniforms((cfg.batch, cfg.n_layers, cfg.draft_vocab), seed=6)
    out = feo.draft_forward(cfg, w, inp, temperature=T, uniforms=u)
    z = out["logits"]
    q = _softmax(z / T)
    ids = out["topk_draft"]
    zs = np.take_along_axis(z, ids, -1)
    assert (np.diff(zs, axis=-1) <= 0).all()               # most probable first
    np.testing.assert_allclose(out["topk_probs"], np.take_along_axis(q, ids, -1), rtol=1e-12)
    np.testing.assert_array_equal(out["topk_ids"], w.d2t[ids])
    greedy = feo.draft_forward(cfg, w, inp, temperature=T)
    assert not np.array_equal(greedy["topk_draft"], ids)   # the noise matters here


def test_constant_noise_is_greedy(feo):
    cfg = PIN
    w = make_weights(cfg, 7)
    inp = make_inputs(cfg, 7)
    for T in (1.0, 2.5):
        u = np.full((cfg.batch, cfg.n_layers, cfg.draft_vocab), 0.5, np.float32)
        a = feo.draft_forward(cfg, w, inp, temperature=T, uniforms=u)
        b = feo.draft_forward(cfg, w, inp, temperature=T)
        for n in ("topk_draft", "topk_ids"):
            np.testing.assert_array_equal(a[n], b[n])
        np.testing.assert_allclose(a["topk_probs"], b["topk_probs"], rtol=1e-15)
        q = _softmax(b["logits"] / T)
        np.testing.assert_allclose(b["topk_probs"], np.take_along_axis(q, b["topk_draft"], -1),
                                   rtol=1e-12)
    with pytest.raises(ValueError):
        feo.draft_forward(cfg, w, inp, temperature=0.0)
