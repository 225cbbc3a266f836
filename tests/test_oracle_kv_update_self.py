"""Pins of the oracle's drafter cache update under the self context (CPU only).

Under FEO_CTX_SELF layer i's context is its prefix plus its own input, so the
cache row of layer i at position p is layer i's key and value of x_{i-1}(p),
the state the pass at prefix p computes (Section 2.1, Eq. 2 read under the
self context; the update step of Section 2.4).  The N layers then form an
ordinary causal decoder stack over the positions, and the update is a
multi-position prefill of that stack.  Pinned against:
* Hugging Face's LlamaDecoderLayer stacked N deep over the whole causal
  sequence of x_0 rows: each layer's k_proj / v_proj (rotated) of its inputs
  are the rows;
* the purpose of the cache: drafting at prefix P from caches written by two
  update calls equals that stack's outputs at position P;
* interleaved sequences in one call equal separate calls, bit for bit.
"""
import numpy as np
import pytest

from fe_synth import make_inputs, make_update_rows

from tests.test_oracle_pins import PIN, _w, _widen
from tests.test_oracle_kv_update import _x0_rows

SELF = PIN.with_(cascade_ctx="self")


def _empty(cfg, rows):
    dt = np.uint16 if cfg.dtype == "bf16" else np.float32
    z = lambda: np.zeros((rows, cfg.n_kv_heads, cfg.head_dim), dt)
    return [z() for _ in range(cfg.n_layers)], [z() for _ in range(cfg.n_layers)]


def _stack(cfg, w, x0, positions):
    """The textbook stack: layer i over the causal sequence of layer i-1's
    outputs.  Returns per layer (outputs, rotated K, V)."""
    from tests import hf_ref
    res, seq = [], x0
    for lw in w.layers:
        layer = hf_ref.decoder_layer(cfg, lw, _widen(cfg))
        out, k, v = hf_ref.run_sequence(cfg, layer, seq, positions)
        res.append((out, k, v))
        seq = out
    return res


def test_self_rows_equal_textbook_stack(feo):
    cfg, L = SELF, 7
    w = _w(cfg)
    up = make_update_rows(cfg, np.array([L]), np.array([0]), capacity=L, seed=21)
    kc, vc = _empty(cfg, L)
    ks, vs = feo.kv_update_self(cfg, w, up.features, up.tokens, up.positions, up.dst_rows, kc, vc)
    x0 = _x0_rows(feo, cfg, w, up.features, up.tokens)
    for li, (_, k_ref, v_ref) in enumerate(_stack(cfg, w, x0, up.positions)):
        assert np.abs(ks[li] - k_ref).max() / np.abs(k_ref).max() < 5e-6, li
        assert np.abs(vs[li] - v_ref).max() / np.abs(v_ref).max() < 5e-6, li
    # the first layer reads x_0 as the cascade context does
    kk, vv = feo.kv_update(PIN, w, up.features, up.tokens, up.positions)
    np.testing.assert_allclose(ks[0], kk[0], rtol=0, atol=1e-12)
    assert np.abs(ks[1] - kk[1]).max() > 1e-3   # deeper layers key their own input


def test_self_decode_from_updated_cache_equals_stack(feo):
    """Rows 0..2 by one call, 3..P-1 by a second that reads the first call's
    rows from the cache; drafting at prefix P then gives every layer's output
    at position P of the stack over positions 0..P."""
    cfg = SELF.with_(batch=1)
    w = _w(cfg)
    P = 6
    up = make_update_rows(cfg, np.array([P + 1]), np.array([0]), capacity=P + 1, seed=23)
    kc, vc = _empty(cfg, P + 1)
    a = slice(0, 3)
    k1, v1 = feo.kv_update_self(cfg, w, up.features[a], up.tokens[a], up.positions[a],
                                up.dst_rows[a], kc, vc)
    for li in range(cfg.n_layers):
        kc[li][:3], vc[li][:3] = k1[li], v1[li]
    b = slice(3, P)
    k2, v2 = feo.kv_update_self(cfg, w, up.features[b], up.tokens[b], up.positions[b],
                                up.dst_rows[b], kc, vc)
    for li in range(cfg.n_layers):
        kc[li][3:P], vc[li][3:P] = k2[li], v2[li]
    inp = make_inputs(cfg, seed=0, prefix_lens=np.array([P], np.int32))
    inp.kcache = [np.ascontiguousarray(k[:P]) for k in kc]
    inp.vcache = [np.ascontiguousarray(v[:P]) for v in vc]
    inp.features = np.ascontiguousarray(up.features[P:])
    inp.next_tokens = np.ascontiguousarray(up.tokens[P:])
    xs = feo.draft_forward(cfg, w, inp, want_logits=False)["hidden"][0]
    x0 = _x0_rows(feo, cfg, w, up.features, up.tokens)
    np.testing.assert_allclose(xs[0], x0[P], rtol=0, atol=1e-12)
    worst = 0.0
    for li, (out, _, _) in enumerate(_stack(cfg, w, x0, np.arange(P + 1))):
        worst = max(worst, np.abs(out[P] - xs[li + 1]).max() / np.abs(out[P]).max())
    assert worst < 5e-6, worst


def test_self_interleaved_sequences_equal_separate_calls(feo):
    """Rows of two sequences interleaved in one call, and a sequence that
    continues a prefix already in the cache."""
    cfg = SELF.with_(dtype="bf16")
    w = _w(cfg)
    cap = 8
    up = make_update_rows(cfg, np.array([4, 3]), np.array([0, 2]), capacity=cap, seed=25)
    kc, vc = _empty(cfg, 2 * cap)
    rng = np.random.default_rng(5)
    for li in range(cfg.n_layers):   # sequence 1's positions 0, 1 are already cached
        kc[li][cap:cap + 2] = rng.integers(0x3c00, 0x3f00, size=kc[li][cap:cap + 2].shape)
        vc[li][cap:cap + 2] = rng.integers(0xbc00, 0xbf00, size=vc[li][cap:cap + 2].shape)
    order = np.array([0, 4, 1, 5, 2, 6, 3])   # A0 B2 A1 B3 A2 B4 A3
    ks, vs = feo.kv_update_self(cfg, w, up.features[order], up.tokens[order], up.positions[order],
                                up.dst_rows[order], kc, vc)
    for sel in (np.arange(4), np.arange(4, 7)):
        k1, v1 = feo.kv_update_self(cfg, w, up.features[sel], up.tokens[sel], up.positions[sel],
                                    up.dst_rows[sel], kc, vc)
        where = np.array([np.where(order == s)[0][0] for s in sel])
        for li in range(cfg.n_layers):
            np.testing.assert_array_equal(ks[li][where], k1[li])
            np.testing.assert_array_equal(vs[li][where], v1[li])


def test_self_update_rejects(feo):
    w = _w(SELF)
    up = make_update_rows(SELF, np.array([2]), np.array([0]), capacity=2, seed=1)
    kc, vc = _empty(SELF, 2)
    with pytest.raises(ValueError):      # another context
        feo.kv_update_self(PIN, w, up.features, up.tokens, up.positions, up.dst_rows, kc, vc)
    with pytest.raises(ValueError):      # position 1 would sit at row -1
        feo.kv_update_self(SELF, w, up.features, up.tokens, up.positions, up.dst_rows - 1, kc, vc)
    with pytest.raises(ValueError):      # row past the cache
        feo.kv_update_self(SELF, w, up.features, up.tokens, up.positions, up.dst_rows + 1, kc, vc)
    ks, _ = feo.kv_update_self(SELF, w, up.features[:0], up.tokens[:0], up.positions[:0],
                               up.dst_rows[:0], kc, vc)
    assert all(k.shape == (0, SELF.n_kv_heads, SELF.head_dim) for k in ks)
