"""Pins of the oracle's drafter cache update (CPU only).

The cache row of layer i at a verified position p is layer i's key and value
of the fused input x_0(p) (Section 2.1, Eq. 1; the update step of Section
2.4, read under the cascade context).  Pinned against:
* Hugging Face's LlamaDecoderLayer: its k_proj / v_proj hooks and rotary
  embedding over the rows x_0(p) at positions p give the same keys and values;
* the purpose of the cache: decoding at prefix P from caches written by the
  update equals the textbook layer over the whole causal sequence;
* rotation invariants (norm per head, values free of the position).
"""
import numpy as np
import pytest

from fe_synth import make_inputs, make_update_rows, make_weights

from tests.test_oracle_pins import PIN, _w, _widen


def _x0_rows(feo, cfg, w, feats, toks):
    """x_0 of every row, from the (separately pinned) drafting pass."""
    M = len(toks)
    inp = make_inputs(cfg.with_(batch=M), seed=0, prefix_lens=np.zeros(M, np.int32))
    inp.features = np.ascontiguousarray(feats)
    inp.next_tokens = np.ascontiguousarray(toks, dtype=np.int32)
    return feo.draft_forward(cfg.with_(batch=M), w, inp, want_logits=False)["hidden"][:, 0]


def test_rows_equal_textbook_projections(feo):
    from tests import hf_ref
    cfg = PIN
    w = _w(cfg)
    up = make_update_rows(cfg, np.array([4, 3]), np.array([0, 9]), capacity=16, seed=7)
    ks, vs = feo.kv_update(cfg, w, up.features, up.tokens, up.positions)
    x0 = _x0_rows(feo, cfg, w, up.features, up.tokens)
    for li, lw in enumerate(w.layers):
        layer = hf_ref.decoder_layer(cfg, lw, _widen(cfg))
        _, k_ref, v_ref = hf_ref.run_sequence(cfg, layer, x0, up.positions)
        # HF normalises in float32 and forms the rotary angles in float32
        assert np.abs(ks[li] - k_ref).max() / np.abs(k_ref).max() < 5e-6
        assert np.abs(vs[li] - v_ref).max() / np.abs(v_ref).max() < 1e-6


def test_decode_from_updated_cache_equals_full_sequence(feo):
    """Write the caches of positions 0..P-1 with the update, then draft at
    prefix P: every cascade layer's output is the textbook layer's last row over
    [x_0(0..P-1) ; x_0(P) .. x_{i-1}(P)] at positions 0..P+i-1."""
    from tests import hf_ref
    cfg = PIN.with_(batch=1)
    w = _w(cfg)
    P = 6
    up = make_update_rows(cfg, np.array([P + 1]), np.array([0]), capacity=P + 1, seed=11)
    ks, vs = feo.kv_update(cfg, w, up.features[:P], up.tokens[:P], up.positions[:P])
    inp = make_inputs(cfg, seed=0, prefix_lens=np.array([P], np.int32))
    inp.kcache = [np.ascontiguousarray(k, dtype=np.float32) for k in ks]
    inp.vcache = [np.ascontiguousarray(v, dtype=np.float32) for v in vs]
    inp.features = np.ascontiguousarray(up.features[P:])
    inp.next_tokens = np.ascontiguousarray(up.tokens[P:])
    xs = feo.draft_forward(cfg, w, inp, want_logits=False)["hidden"][0]
    x0 = _x0_rows(feo, cfg, w, up.features[:P], up.tokens[:P])
    worst = 0.0
    for li, lw in enumerate(w.layers):
        i = li + 1
        layer = hf_ref.decoder_layer(cfg, lw, _widen(cfg))
        seq = np.concatenate([x0, xs[:i]])
        ref, _, _ = hf_ref.run_sequence(cfg, layer, seq, np.arange(P + i))
        worst = max(worst, np.abs(ref[-1] - xs[i]).max() / np.abs(ref[-1]).max())
    assert worst < 5e-6, worst


def test_rotation_invariants(feo):
    """One row at several positions: values identical, key norms per head
    identical, keys at distinct positions different."""
    cfg = PIN
    w = make_weights(cfg, 5)
    up = make_update_rows(cfg, np.array([1]), np.array([0]), capacity=1, seed=3)
    pos = np.array([0, 1, 5, 1000, 31], np.int32)
    M = len(pos)
    feats = np.repeat(up.features, M, axis=0)
    toks = np.repeat(up.tokens, M)
    ks, vs = feo.kv_update(cfg, w, feats, toks, pos)
    for k, v in zip(ks, vs):
        assert np.array_equal(v, np.repeat(v[:1], M, axis=0))
        norms = np.linalg.norm(k, axis=-1)
        np.testing.assert_allclose(norms, np.repeat(norms[:1], M, axis=0), rtol=1e-12)
        assert np.abs(k[1] - k[0]).max() > 1e-3


def test_layers_are_independent_and_bf16_widening(feo):
    """Layer i's rows depend on layer i's weights only: an update through a
    one-layer drafter that holds layer i gives the same rows (bf16 storage)."""
    cfg = PIN.with_(dtype="bf16")
    w = make_weights(cfg, 8)
    up = make_update_rows(cfg, np.array([2, 1]), np.array([3, 0]), capacity=8, seed=2)
    ks, vs = feo.kv_update(cfg, w, up.features, up.tokens, up.positions)
    for li in range(cfg.n_layers):
        w1 = make_weights(cfg, 8)
        w1.layers = [w.layers[li]]
        k1, v1 = feo.kv_update(cfg.with_(n_layers=1), w1, up.features, up.tokens, up.positions)
        assert np.array_equal(k1[0], ks[li]) and np.array_equal(v1[0], vs[li])
    assert np.abs(ks[0] - ks[1]).max() > 1e-3


def test_parallel_heads_share_the_cascade_rows(feo):
    """Without the cascade every head keys x_0(p) too: the same rows."""
    cfg = PIN
    w = make_weights(cfg, 4)
    up = make_update_rows(cfg, np.array([3]), np.array([2]), capacity=8, seed=4)
    a = feo.kv_update(cfg, w, up.features, up.tokens, up.positions)
    b = feo.kv_update(cfg.with_(cascade_ctx="parallel"), w, up.features, up.tokens, up.positions)
    for x, y in zip(a[0] + a[1], b[0] + b[1]):
        np.testing.assert_array_equal(x, y)


def test_rejects_self_context_and_bad_tokens(feo):
    cfg = PIN
    w = make_weights(cfg, 1)
    up = make_update_rows(cfg, np.array([2]), np.array([0]), capacity=2, seed=1)
    with pytest.raises(ValueError):
        feo.kv_update(cfg.with_(cascade_ctx="self"), w, up.features, up.tokens, up.positions)
    bad = up.tokens.copy()
    bad[1] = cfg.target_vocab
    with pytest.raises(ValueError):
        feo.kv_update(cfg, w, up.features, bad, up.positions)
    ks, vs = feo.kv_update(cfg, w, up.features[:0], up.tokens[:0], up.positions[:0])
    assert all(k.shape == (0, cfg.n_kv_heads, cfg.head_dim) for k in ks)
