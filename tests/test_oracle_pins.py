"""Pins of the CPU oracle against things other than itself (CPU only).

* Every cascade layer L_i (Section 2.1, Eq. 1-2) is one pre-norm LLaMA decoder
  layer: evaluated by Hugging Face's LlamaDecoderLayer over the full causal
  sequence [prefix ; x_0 .. x_{i-1}], its last row must equal the oracle's
  x_i computed decode-style from a prefix KV cache.
* Feature fusion and input FC (Section 2.1, Eq. 1): special weights that
  select one block of the concatenation fix the concat order and the token
  whose embedding is used; linearity fixes the rest.
* RoPE, RMSNorm, attention, LM head, softmax and top-k: library routines
  (transformers, torch) and closed-form invariants.
"""
import numpy as np
import pytest
import torch

from fe_synth import configs as C
from fe_synth import make_inputs, make_weights, to_f64

PIN = C.DrafterConfig(
    name="pin_f32", hidden=64, n_q_heads=4, n_kv_heads=2, head_dim=16, intermediate=96,
    n_layers=3, draft_vocab=50, target_vocab=70, rope_theta=10000.0, dtype="f32", batch=2,
    prefix=5, topk=3)


def _w(cfg, seed=3, attn_gain=8.0):
    w = make_weights(cfg, seed)
    for lw in w.layers:   # sharper attention so that score mistakes show
        lw.wq = (lw.wq * np.float32(attn_gain)).astype(np.float32) if cfg.dtype == "f32" else lw.wq
        lw.wk = (lw.wk * np.float32(attn_gain)).astype(np.float32) if cfg.dtype == "f32" else lw.wk
    return w


def _widen(cfg):
    return lambda a: to_f64(a, cfg.dtype)


def _caches_from_hf(cfg, w, plens, seed):
    """Prefix K/V for every layer, produced by the HF layer from random prefix
    hidden states Y (the cache a target-prefix pass of that layer would hold)."""
    from tests import hf_ref
    rng = np.random.default_rng(seed)
    Ys, kc, vc = [], [], []
    for li, lw in enumerate(w.layers):
        layer = hf_ref.decoder_layer(cfg, lw, _widen(cfg))
        ks, vs, ys = [], [], []
        for P in plens:
            Y = rng.standard_normal((P, cfg.hidden))
            ys.append(Y)
            if P:
                _, k, v = hf_ref.run_sequence(cfg, layer, Y, np.arange(P))
                ks.append(k)
                vs.append(v)
        Ys.append(ys)
        shape = (0, cfg.n_kv_heads, cfg.head_dim)
        kc.append(np.ascontiguousarray(np.concatenate(ks) if ks else np.zeros(shape), dtype=np.float32))
        vc.append(np.ascontiguousarray(np.concatenate(vs) if vs else np.zeros(shape), dtype=np.float32))
    return Ys, kc, vc


@pytest.mark.parametrize("ctx", ["cascade", "self", "parallel"])
def test_cascade_layers_equal_textbook_llama_layer(feo, ctx):
    from tests import hf_ref
    cfg = PIN.with_(cascade_ctx=ctx)
    w = _w(cfg)
    plens = np.array([5, 0], dtype=np.int32)
    inp = make_inputs(cfg, seed=4, prefix_lens=plens)
    Ys, kc, vc = _caches_from_hf(cfg, w, plens, seed=5)
    inp.kcache, inp.vcache = kc, vc
    out = feo.draft_forward(cfg, w, inp)
    xs = out["hidden"]
    worst = 0.0
    for li, lw in enumerate(w.layers):
        i = li + 1
        layer = hf_ref.decoder_layer(cfg, lw, _widen(cfg))
        for b, P in enumerate(plens):
            Y = Ys[li][b]
            # the HF layer sees the prefix rows in double while the oracle reads
            # the cache rounded to fp32; this bounds the allowed difference
            if ctx == "cascade":
                seq = np.concatenate([Y, xs[b, :i]]) if P else xs[b, :i]
                pos = np.arange(P + i)
            else:   # self: the layer's own input; parallel: x_0 for every layer
                src = i - 1 if ctx == "self" else 0
                seq = np.concatenate([Y, xs[b, src:src + 1]]) if P else xs[b, src:src + 1]
                pos = np.arange(P + 1)
            ref, _, _ = hf_ref.run_sequence(cfg, layer, seq, pos)
            err = np.abs(ref[-1] - xs[b, i]).max() / np.abs(ref[-1]).max()
            worst = max(worst, err)
    assert worst < 2e-6, worst


def test_cascade_and_self_agree_on_first_layer(feo):
    cfg = PIN
    w = _w(cfg)
    inp = make_inputs(cfg, seed=1)
    a = feo.draft_forward(cfg, w, inp)["hidden"]
    b = feo.draft_forward(cfg.with_(cascade_ctx="self"), w, inp)["hidden"]
    c = feo.draft_forward(cfg.with_(cascade_ctx="parallel"), w, inp)["hidden"]
    np.testing.assert_array_equal(a[:, :2], b[:, :2])
    np.testing.assert_array_equal(a[:, :2], c[:, :2])
    assert np.abs(a[:, 2] - b[:, 2]).max() > 1e-6   # deeper layers do differ
    assert np.abs(b[:, 2] - c[:, 2]).max() > 1e-6


def test_parallel_heads_are_independent(feo):
    """Parallel heads (the ablation without the cascade): head i sees x_0, its
    own weights and its own prefix cache only, so reordering the layers (with
    their caches) reorders the outputs, and a one-layer drafter holding layer i
    gives head i."""
    cfg = PIN.with_(cascade_ctx="parallel")
    w = _w(cfg)
    inp = make_inputs(cfg, seed=2)
    out = feo.draft_forward(cfg, w, inp)
    xs, z = out["hidden"], out["logits"]
    perm = [2, 0, 1]
    w2 = _w(cfg)
    w2.layers = [w.layers[p] for p in perm]
    inp2 = make_inputs(cfg, seed=2)   # each layer keeps its own prefix cache
    inp2.kcache = [inp.kcache[p] for p in perm]
    inp2.vcache = [inp.vcache[p] for p in perm]
    xs2 = feo.draft_forward(cfg, w2, inp2)["hidden"]
    np.testing.assert_array_equal(xs2[:, 0], xs[:, 0])
    for i, p in enumerate(perm):
        np.testing.assert_array_equal(xs2[:, 1 + i], xs[:, 1 + p])
    for li in range(cfg.n_layers):
        w1 = _w(cfg)
        w1.layers = [w.layers[li]]
        inp1 = make_inputs(cfg.with_(n_layers=1), 2)
        inp1.kcache, inp1.vcache = [inp.kcache[li]], [inp.vcache[li]]
        one = feo.draft_forward(cfg.with_(n_layers=1), w1, inp1)
        np.testing.assert_array_equal(one["hidden"][:, 1], xs[:, 1 + li])
        np.testing.assert_array_equal(one["logits"][:, 0], z[:, li])


def _eye_block(d, nblk, which):
    W = np.zeros((d, nblk * d), dtype=np.float32)
    W[:, which * d:(which + 1) * d] = np.eye(d, dtype=np.float32)
    return W


def test_fusion_concat_order_and_next_token_embedding(feo):
    cfg = PIN
    w = make_weights(cfg, 2)
    inp = make_inputs(cfg, seed=2)
    d = cfg.hidden
    feats = inp.features.astype(np.float64)
    for lvl in range(3):   # W_fuse selects l_t, m_t or h_t; W_in passes g_t through
        w.w_fuse = _eye_block(d, 3, lvl)
        w.w_in = _eye_block(d, 2, 0)
        x0 = feo.draft_forward(cfg, w, inp)["hidden"][:, 0]
        np.testing.assert_array_equal(x0, feats[:, lvl * d:(lvl + 1) * d])
    w.w_in = _eye_block(d, 2, 1)   # W_in passes e_{t+1} through
    x0 = feo.draft_forward(cfg, w, inp)["hidden"][:, 0]
    np.testing.assert_array_equal(x0, w.embed[inp.next_tokens].astype(np.float64))


def test_fusion_is_affine_in_features(feo):
    cfg = PIN
    w = make_weights(cfg, 2)
    inp = make_inputs(cfg, seed=2)
    x = {}
    for s in (0.0, 1.0, 2.0):
        inp2 = make_inputs(cfg, seed=2)
        inp2.features = (inp.features * np.float32(s)).astype(np.float32)
        x[s] = feo.draft_forward(cfg, w, inp2)["hidden"][:, 0]
    np.testing.assert_allclose(x[2.0] - x[1.0], x[1.0] - x[0.0], rtol=0, atol=1e-12)
    assert np.abs(x[1.0] - x[0.0]).max() > 1e-3


def test_rope_properties_and_library(feo):
    from tests import hf_ref
    from transformers.models.llama.modeling_llama import apply_rotary_pos_emb
    rng = np.random.default_rng(0)
    D, theta = 16, 10000.0
    q, k = rng.standard_normal(D), rng.standard_normal(D)
    np.testing.assert_array_equal(feo.rope(q, 0, theta), q)
    r = feo.rope(q, 37, theta)
    np.testing.assert_allclose(r[:D // 2] ** 2 + r[D // 2:] ** 2, q[:D // 2] ** 2 + q[D // 2:] ** 2,
                               rtol=1e-12)
    # <R(q, p), R(k, p')> depends only on p - p'
    a = feo.rope(q, 11, theta) @ feo.rope(k, 4, theta)
    b = feo.rope(q, 107, theta) @ feo.rope(k, 100, theta)
    assert abs(a - b) < 1e-10
    # library: transformers' rotate-half rotary (angles formed in float32 there)
    cfg = PIN
    rot = hf_ref.rotary(cfg)
    pos = torch.arange(40)[None]
    cos, sin = rot(torch.zeros(1, 40, D, dtype=torch.float64), pos)
    qt = torch.from_numpy(q)[None, None, None].expand(1, 1, 40, D).double()
    qr, _ = apply_rotary_pos_emb(qt, qt, cos.double(), sin.double())
    ours = np.stack([feo.rope(q, p, theta) for p in range(40)])
    np.testing.assert_allclose(ours, qr[0, 0].numpy(), rtol=0, atol=5e-6)


def test_rmsnorm_library_and_closed_form(feo):
    from transformers.models.llama.modeling_llama import LlamaRMSNorm
    rng = np.random.default_rng(1)
    x = rng.standard_normal(64) * 3.0
    g = (1 + 0.02 * rng.standard_normal(64)).astype(np.float32)
    y = feo.rmsnorm(x, g, "f32", 1e-5)
    n = LlamaRMSNorm(64, eps=1e-5).double()
    with torch.no_grad():
        n.weight.copy_(torch.from_numpy(g.astype(np.float64)))
        ref = n(torch.from_numpy(x)[None]).numpy()[0]
    # transformers normalises in float32: agreement to float32 rounding
    np.testing.assert_allclose(y, ref, rtol=5e-7, atol=0)
    u = y / g.astype(np.float64)
    assert abs(np.sqrt(np.mean(u ** 2)) - 1.0) < 1e-5


def test_attention_special_cases_and_library(feo):
    rng = np.random.default_rng(2)
    D = 16
    q = rng.standard_normal(D)
    # one key: output is exactly its value
    K1, V1 = rng.standard_normal((1, D)), rng.standard_normal((1, D))
    np.testing.assert_array_equal(feo.attend(q, K1, V1), V1[0])
    # no keys: zeros
    np.testing.assert_array_equal(feo.attend(q, np.zeros((0, D)), np.zeros((0, D))), np.zeros(D))
    K, V = rng.standard_normal((33, D)) * 2, rng.standard_normal((33, D))
    o = feo.attend(q, K, V)
    perm = rng.permutation(33)
    np.testing.assert_allclose(feo.attend(q, K[perm], V[perm]), o, rtol=1e-12, atol=1e-14)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None, None, None], torch.from_numpy(K)[None, None],
        torch.from_numpy(V)[None, None]).numpy()[0, 0, 0]
    np.testing.assert_allclose(o, ref, rtol=1e-12, atol=1e-14)


def test_gqa_with_replicated_kv_heads_equals_mha(feo):
    """H_kv = H_q with every KV head repeated G times equals the grouped layer."""
    cfg = PIN
    G = cfg.group
    w = _w(cfg)
    inp = make_inputs(cfg, seed=6)
    a = feo.draft_forward(cfg, w, inp)
    mcfg = cfg.with_(n_kv_heads=cfg.n_q_heads)
    D = cfg.head_dim
    for lw in w.layers:
        lw.wk = np.ascontiguousarray(np.repeat(lw.wk.reshape(cfg.n_kv_heads, D, -1), G, 0).reshape(-1, cfg.hidden))
        lw.wv = np.ascontiguousarray(np.repeat(lw.wv.reshape(cfg.n_kv_heads, D, -1), G, 0).reshape(-1, cfg.hidden))
    inp.kcache = [np.ascontiguousarray(np.repeat(k, G, axis=1)) for k in inp.kcache]
    inp.vcache = [np.ascontiguousarray(np.repeat(v, G, axis=1)) for v in inp.vcache]
    b = feo.draft_forward(mcfg, w, inp)
    np.testing.assert_allclose(b["hidden"], a["hidden"], rtol=1e-12, atol=1e-12)


def test_lm_head_softmax_topk_library(feo):
    from transformers.models.llama.modeling_llama import LlamaRMSNorm
    cfg = PIN.with_(topk=7)
    w = _w(cfg)
    inp = make_inputs(cfg, seed=7)
    out = feo.draft_forward(cfg, w, inp)
    n = LlamaRMSNorm(cfg.hidden, eps=cfg.rms_eps).double()
    with torch.no_grad():
        n.weight.copy_(torch.from_numpy(to_f64(w.final_norm, cfg.dtype)))
        h = torch.from_numpy(out["hidden"][:, 1:])
        z = torch.nn.functional.linear(n(h), torch.from_numpy(to_f64(w.lm_head, cfg.dtype)))
    # transformers normalises in float32: agreement to float32 rounding
    np.testing.assert_allclose(out["logits"], z.numpy(), rtol=0, atol=1e-6)
    # selection and softmax: library routines applied to the oracle's logits
    z = torch.from_numpy(out["logits"])
    p = torch.softmax(z, dim=-1)
    assert np.abs(p.sum(-1).numpy() - 1).max() < 1e-12
    order = torch.sort(-z, dim=-1, stable=True).indices[..., :cfg.topk].numpy()
    np.testing.assert_array_equal(out["topk_draft"], order)
    np.testing.assert_array_equal(out["topk_ids"], w.d2t[order])
    np.testing.assert_allclose(out["topk_probs"], np.take_along_axis(p.numpy(), order, -1),
                               rtol=1e-12)
    assert (np.diff(out["topk_probs"], axis=-1) <= 0).all()


def test_topk_ties_go_to_lower_draft_id(feo):
    cfg = PIN.with_(topk=4)
    w = _w(cfg)
    w.lm_head[:] = 0
    w.lm_head[[9, 3, 30, 41]] = w.lm_head[[9, 3, 30, 41]] + np.float32(1.0)   # four equal maxima
    inp = make_inputs(cfg, seed=8)
    out = feo.draft_forward(cfg, w, inp)
    for b in range(cfg.batch):
        for i in range(cfg.n_layers):
            z = out["logits"][b, i]
            top = sorted(range(cfg.draft_vocab), key=lambda v: (-z[v], v))[:4]
            np.testing.assert_array_equal(out["topk_draft"][b, i], top)


def test_cascade_truncation_is_causal(feo):
    cfg = PIN
    w = _w(cfg)
    inp = make_inputs(cfg, seed=9)
    full = feo.draft_forward(cfg, w, inp)
    m = 2
    cfg2 = cfg.with_(n_layers=m)
    w2 = _w(cfg)
    w2.layers = w2.layers[:m]
    inp2 = make_inputs(cfg, seed=9)
    inp2.kcache, inp2.vcache = inp2.kcache[:m], inp2.vcache[:m]
    part = feo.draft_forward(cfg2, w2, inp2)
    np.testing.assert_array_equal(part["hidden"], full["hidden"][:, :m + 1])
    np.testing.assert_array_equal(part["logits"], full["logits"][:, :m])


def test_batched_ragged_equals_per_sequence(feo):
    cfg = C.SMALL_GQA_BF16.with_(hidden=128, intermediate=256, n_q_heads=4, n_kv_heads=2,
                                 head_dim=32, draft_vocab=300, target_vocab=777, batch=4,
                                 prefix=(0, 40))
    w = make_weights(cfg, 11)
    inp = make_inputs(cfg, seed=11)
    allb = feo.draft_forward(cfg, w, inp)
    for b in range(cfg.batch):
        one = feo.draft_forward(cfg, w, inp, batch_index=[b])
        for key in ("hidden", "logits", "topk_ids", "topk_probs"):
            np.testing.assert_array_equal(one[key][0], allb[key][b])


def test_bf16_storage_is_exact_widening(feo):
    """A bf16 run equals an fp32 run on the exactly widened values."""
    cfg = PIN.with_(dtype="bf16")
    w = make_weights(cfg, 12)
    inp = make_inputs(cfg, seed=12)
    a = feo.draft_forward(cfg, w, inp)
    f32 = lambda x: to_f64(x, "bf16").astype(np.float32)
    for name in ("w_fuse", "w_in", "embed", "final_norm", "lm_head"):
        setattr(w, name, f32(getattr(w, name)))
    for lw in w.layers:
        for f in lw.FIELDS:
            setattr(lw, f, f32(getattr(lw, f)))
    inp.features = f32(inp.features)
    inp.kcache = [f32(k) for k in inp.kcache]
    inp.vcache = [f32(v) for v in inp.vcache]
    b = feo.draft_forward(cfg.with_(dtype="f32"), w, inp)
    for key in ("hidden", "logits", "topk_ids", "topk_probs"):
        np.testing.assert_array_equal(a[key], b[key])
