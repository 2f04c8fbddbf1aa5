"""Pins for the oracle's forward pass and vocabulary reduction (CPU only).

Each oracle function is checked against something other than itself: a
library routine (torch float64 CPU ops, scipy), a closed form, or an
invariant that a plausible mistake (dropped term, wrong sign, transposed
operand, wrong index) would break.
"""
import math

import numpy as np
import pytest
import scipy.special
import torch
import torch.nn.functional as F

from oracle import forward as of
from oracle import vocab as ov
from paper_2608_22646_amd import synth

rng = np.random.default_rng(7)


def test_round_bf16_matches_torch():
    # random values over many binades, plus exact ties and specials
    x = rng.standard_normal(200000).astype(np.float32) * np.float32(10.0) ** rng.integers(-30, 30, 200000).astype(np.float32)
    ties = (np.arange(1, 4000, dtype=np.uint32) << 16 | 0x8000).view(np.float32)   # exactly half-way
    special = np.array([0.0, -0.0, np.inf, -np.inf, 3.3895314e38, 1e-40, -1e-41], dtype=np.float32)
    for v in (x, ties, -ties, special):
        want = torch.from_numpy(v).to(torch.bfloat16).to(torch.float32).numpy()
        got = of.round_bf16(v)
        np.testing.assert_array_equal(got.view(np.uint32), want.view(np.uint32))


def test_rmsnorm_matches_torch():
    x = rng.standard_normal((7, 96)) * 3
    g = 1 + 0.1 * rng.standard_normal(96)
    want = F.rms_norm(torch.from_numpy(x), (96,), weight=torch.from_numpy(g), eps=1e-5).numpy()
    np.testing.assert_allclose(of.rmsnorm(x, g, 1e-5), want, rtol=1e-13, atol=1e-13)


def _rope_complex(x, base):
    """RoPE as complex multiplication: (x_j + i x_{j+hd/2}) * exp(i pos base^(-2j/hd))."""
    t = torch.from_numpy(x)
    L, hd = t.shape[-2], t.shape[-1]
    half = hd // 2
    z = torch.complex(t[..., :half], t[..., half:])
    freq = torch.tensor([base ** (-2.0 * j / hd) for j in range(half)], dtype=torch.float64)
    ang = torch.arange(L, dtype=torch.float64)[:, None] * freq[None, :]
    r = z * torch.polar(torch.ones_like(ang), ang)
    return torch.cat([r.real, r.imag], dim=-1).numpy()


@pytest.mark.parametrize("base", [10000.0, 500000.0, 1e6])
def test_rope_matches_complex_rotation(base):
    x = rng.standard_normal((3, 40, 64))
    cos, sin = of.rope_tables(40, 64, base)
    np.testing.assert_allclose(of.rope(x, cos, sin), _rope_complex(x, base), rtol=1e-12, atol=1e-12)


def test_rope_invariants():
    L, hd = 50, 32
    cos, sin = of.rope_tables(L, hd, 10000.0)
    q = rng.standard_normal(hd)
    k = rng.standard_normal(hd)
    # position 0 is the identity; rotation preserves norms
    rq = of.rope(np.tile(q, (L, 1)), cos, sin)
    np.testing.assert_allclose(rq[0], q, atol=1e-15)
    np.testing.assert_allclose(np.linalg.norm(rq, axis=-1), np.linalg.norm(q), rtol=1e-13)
    # <R_m q, R_n k> depends only on m - n
    rk = of.rope(np.tile(k, (L, 1)), cos, sin)
    dots = rq @ rk.T
    for delta in (0, 3, -5, 17):
        vals = [dots[m, m - delta] for m in range(max(0, delta), min(L, L + delta))]
        np.testing.assert_allclose(vals, vals[0], rtol=1e-11, atol=1e-11)


@pytest.mark.parametrize("hq,hkv", [(4, 4), (6, 2), (7, 1)])
def test_attention_matches_sdpa(hq, hkv):
    L, hd = 37, 16
    q = rng.standard_normal((hq, L, hd))
    k = rng.standard_normal((hkv, L, hd))
    v = rng.standard_normal((hkv, L, hd))
    rep = hq // hkv
    want = F.scaled_dot_product_attention(
        torch.from_numpy(q)[None], torch.from_numpy(k).repeat_interleave(rep, 0)[None],
        torch.from_numpy(v).repeat_interleave(rep, 0)[None], is_causal=False)[0].numpy()
    np.testing.assert_allclose(of.attention(q, k, v), want, rtol=1e-12, atol=1e-12)


def test_attention_invariants():
    L, hd = 20, 8
    q = rng.standard_normal((2, L, hd))
    k = rng.standard_normal((1, L, hd))
    v = rng.standard_normal((1, L, hd))
    o = of.attention(q, k, v)
    # GQA == MHA with the KV head duplicated
    np.testing.assert_allclose(o, of.attention(q, np.repeat(k, 2, 0), np.repeat(v, 2, 0)), atol=1e-14)
    # non-causal: permuting the sequence permutes the output the same way
    perm = rng.permutation(L)
    np.testing.assert_allclose(of.attention(q[:, perm], k[:, perm], v[:, perm]), o[:, perm], atol=1e-13)
    # last position sees the first key (no causal mask): changing v[0] moves every output row
    v2 = v.copy()
    v2[0, 0] += 1.0
    assert np.all(np.abs(of.attention(q, k, v2) - o).sum(-1) > 0)
    # identical keys -> uniform weights -> mean of v
    kc = np.tile(k[:, :1], (1, L, 1))
    np.testing.assert_allclose(of.attention(q, kc, v), np.broadcast_to(v.mean(1, keepdims=True), o.shape), atol=1e-13)


def test_silu_softmax():
    x = rng.standard_normal(1000) * 8
    np.testing.assert_allclose(of.silu(x), F.silu(torch.from_numpy(x)).numpy(), rtol=1e-14, atol=1e-15)
    s = rng.standard_normal((5, 300)) * 20
    np.testing.assert_allclose(of.softmax(s), scipy.special.softmax(s, axis=-1), rtol=1e-12, atol=1e-300)


def test_confidence_argmax():
    V, mask = 500, 499
    l = rng.standard_normal((9, V)) * 5
    conf, arg = ov.confidence_argmax(l, mask)
    p = scipy.special.softmax(l[:, :mask], axis=-1)
    np.testing.assert_allclose(conf, p.max(-1), rtol=1e-13)
    np.testing.assert_array_equal(arg, p.argmax(-1))
    # the mask id is never predicted, even when it holds the largest logit
    l[:, mask] = 100.0
    conf2, arg2 = ov.confidence_argmax(l, mask)
    np.testing.assert_array_equal(arg2, arg)
    np.testing.assert_allclose(conf2, conf, rtol=1e-15)
    # ties go to the lowest index; conf = 1/k for k equal maxima and -inf elsewhere
    t = np.full((1, V), -np.inf)
    t[0, [17, 230, 231]] = 2.5
    c, a = ov.confidence_argmax(t, mask)
    assert a[0] == 17 and c[0] == pytest.approx(1 / 3, rel=1e-15)
    # uniform logits -> conf = 1/(V-1)
    c, _ = ov.confidence_argmax(np.zeros((1, V)), mask)
    assert c[0] == pytest.approx(1 / (V - 1), rel=1e-13)


def _gap_by_definition(row, mask):
    """Largest logit minus the largest logit of any other index (mask excluded),
    by a plain scan: the distance by which the argmax leads its runner-up."""
    best, best_i = -math.inf, -1
    for i, v in enumerate(row):
        if i != mask and v > best:
            best, best_i = v, i
    second = -math.inf
    for i, v in enumerate(row):
        if i != mask and i != best_i and v > second:
            second = v
    return best - second


def test_top2_gap():
    V, mask = 12, 11
    # hand rows with a known lead
    row = np.array([0.5, 3.0, -1.0, 2.25, 0.0, 2.9, 1.0, -4.0, 0.0, 0.0, 0.0, 0.0])
    assert ov.top2_gap(row, mask) == pytest.approx(0.1, abs=1e-15)
    row2 = np.zeros(V)
    row2[4] = 7.0
    row2[9] = -3.5
    assert ov.top2_gap(row2, mask) == 7.0          # runner-up is one of the zeros
    # ties at the top: gap 0 (either index is a correct argmax)
    row3 = row.copy()
    row3[5] = 3.0
    assert ov.top2_gap(row3, mask) == 0.0
    # the mask id holding the largest logit is ignored on both places
    row4 = row.copy()
    row4[mask] = 50.0
    assert ov.top2_gap(row4, mask) == pytest.approx(0.1, abs=1e-15)
    row5 = row.copy()
    row5[mask] = 2.95                               # between the leader and the runner-up
    assert ov.top2_gap(row5, mask) == pytest.approx(0.1, abs=1e-15)
    # -inf entries: a single finite candidate leads by +inf; -inf never is the runner-up
    row6 = np.full(V, -np.inf)
    row6[3] = 1.0
    assert ov.top2_gap(row6, mask) == np.inf
    row6[7] = -2.0
    assert ov.top2_gap(row6, mask) == 3.0
    # batched rows, brute force on random logits with planted ties and masks on top
    l = rng.standard_normal((40, 37)) * 3
    l[::5, 8] = l[::5, 20] = l[::5].max(axis=1) + 1.0    # ties at the top
    l[1::7, 36] = 99.0                                     # mask id on top
    g = ov.top2_gap(l, 36)
    assert g.shape == (40,)
    for r in range(40):
        assert g[r] == _gap_by_definition(l[r], 36), r
    # the property the GPU tests rely on: two logit rows within e of each other
    # can only disagree on the argmax where the reference's gap is at most 2 e
    for trial in range(200):
        ref = rng.standard_normal(50) * 2
        e = 10.0 ** rng.uniform(-6, 0)
        got = ref + rng.uniform(-e, e, 50)
        if ov.confidence_argmax(got[None], 49)[1][0] != ov.confidence_argmax(ref[None], 49)[1][0]:
            assert ov.top2_gap(ref, 49) <= 2 * e


def _torch_forward(cfg, weights, tokens, bf16):
    """The same model built from torch float64 library routines (rms_norm,
    complex-rotation RoPE, scaled_dot_product_attention with GQA, silu, linear)."""
    W = [torch.from_numpy(np.asarray(w, dtype=np.float64)) for w in weights]
    r = (lambda t: t.to(torch.bfloat16).to(torch.float64)) if bf16 else (lambda t: t)
    x = torch.from_numpy(np.asarray(tokens, dtype=np.int64))
    B, L = x.shape
    H, Hkv, hd, d = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d_model
    h = F.embedding(x, W[0])
    for l in range(cfg.n_layers):
        an, wq, wk, wv, wo, mn, wg, wu, wd = W[1 + 9 * l: 10 + 9 * l]
        a = r(F.rms_norm(h, (d,), an, cfg.rms_eps))
        q = F.linear(a, wq).view(B, L, H, hd).transpose(1, 2)
        k = F.linear(a, wk).view(B, L, Hkv, hd).transpose(1, 2)
        v = r(F.linear(a, wv).view(B, L, Hkv, hd).transpose(1, 2))
        q = r(torch.from_numpy(_rope_complex(q.numpy(), cfg.rope_base)))
        k = r(torch.from_numpy(_rope_complex(k.numpy(), cfg.rope_base)))
        o = F.scaled_dot_product_attention(q, k, v, is_causal=False, enable_gqa=True)
        h = h + F.linear(r(o.transpose(1, 2).reshape(B, L, H * hd)), wo)
        a = r(F.rms_norm(h, (d,), mn, cfg.rms_eps))
        h = h + F.linear(r(F.silu(F.linear(a, wg)) * F.linear(a, wu)), wd)
    hb = r(F.rms_norm(h, (d,), W[-2], cfg.rms_eps))
    return F.linear(hb, W[-1]).numpy()


TINY_GQA = synth.ModelConfig("t", n_layers=2, d_model=64, n_heads=4, n_kv_heads=2, head_dim=16, d_ff=96,
                             vocab=50, rope_base=10000.0, dtype="f32", lm_head_std=5 / 8, norm_gain_std=0.2,
                             linear_std=0.2)


def _np_weights(cfg):
    return [w.to(torch.float64).numpy() for w in synth.make_weights(cfg)]


def test_forward_f64_matches_torch_library_model():
    w = _np_weights(TINY_GQA)
    tokens = rng.integers(0, TINY_GQA.vocab, (2, 23))
    got = of.forward(TINY_GQA, w, tokens)
    want = _torch_forward(TINY_GQA, w, tokens, bf16=False)
    np.testing.assert_allclose(got, want, rtol=1e-10, atol=1e-10)
    rows = np.array([3, 7, 22])
    np.testing.assert_allclose(of.forward(TINY_GQA, w, tokens, rows=rows), want[:, rows], rtol=1e-10, atol=1e-10)


def test_forward_bf16_matches_torch_library_model():
    # one layer: with more, rounding flips caused by float32-vs-float64
    # accumulation cascade until the two models differ by bf16 noise itself
    cfg = synth.reduced(TINY_GQA, dtype="bf16", n_layers=1)
    w = [t.to(torch.float32).numpy() for t in synth.make_weights(cfg)]
    tokens = rng.integers(0, cfg.vocab, (2, 19))
    got = of.forward(cfg, w, tokens, mode="bf16")
    want = _torch_forward(cfg, w, tokens, bf16=True)
    # Both round the same values to bf16.  float32 (sgemm) against float64
    # accumulation can move an occasional value across a bf16 rounding boundary,
    # whose effect then propagates, so the bound is on the mean with a loose max.
    # A missing or extra rounding point moves the mean by ~1e-2 (the unrounded
    # float64 model differs by ~0.1-0.3 at the max).
    err = np.abs(got - want)
    assert err.mean() < 5e-4 and err.max() < 5e-2, (err.mean(), err.max())
    err64 = np.abs(of.forward(cfg, w, tokens, mode="f64") - want)
    assert err64.mean() > 20 * err.mean()


def test_forward_bf16_f64acc_matches_torch_library_model():
    # the same rounding points as "bf16" with float64 products: the torch float64
    # model with bf16 rounding is that definition, so the two agree to float64
    # rounding through several layers (no bf16 flips at float64 precision)
    cfg = synth.reduced(TINY_GQA, dtype="bf16", n_layers=2)
    w = [t.to(torch.float32).numpy() for t in synth.make_weights(cfg)]
    tokens = rng.integers(0, cfg.vocab, (2, 19))
    want = _torch_forward(cfg, w, tokens, bf16=True)
    got = of.forward(cfg, w, tokens, mode="bf16_f64acc")
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-9)
    # float32 accumulation ("bf16") is a different model at the bf16-flip level
    assert np.abs(of.forward(cfg, w, tokens, mode="bf16") - want).max() > 1e-7


def test_forward_bidirectional_and_position_sensitive():
    w = _np_weights(TINY_GQA)
    tokens = rng.integers(0, TINY_GQA.vocab, (1, 12))
    base = of.forward(TINY_GQA, w, tokens)
    t2 = tokens.copy()
    t2[0, -1] = (t2[0, -1] + 1) % TINY_GQA.vocab
    # a change at the last position changes the logits of the first (no causal mask)
    assert np.abs(of.forward(TINY_GQA, w, t2)[0, 0] - base[0, 0]).max() > 1e-6
