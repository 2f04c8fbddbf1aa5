"""Pins for the oracle's cross-step key/value reuse (CPU only).

The cached forward is pinned against the full forward (itself pinned against a
torch library model): right after a refresh, and for any block tokens in a
one-layer model, the two must agree to rounding; the stored layer-0 keys and
values are checked against torch library calls.  The decode wiring is checked
through the refresh schedule and the refresh-every-step case.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import controller as oc
from oracle import forward as of
from oracle import kvcache as okv
from paper_2608_22646_amd import synth

rng = np.random.default_rng(11)

CFG = synth.ModelConfig("t", n_layers=2, d_model=64, n_heads=4, n_kv_heads=2, head_dim=16, d_ff=96, vocab=50,
                        rope_base=10000.0, dtype="f32", lm_head_std=5 / 8, norm_gain_std=0.2, linear_std=0.2)


def _w(cfg):
    return [w.to(torch.float64).numpy() for w in synth.make_weights(cfg)]


def test_refresh_forward_equals_forward():
    w = _w(CFG)
    x = rng.integers(0, CFG.vocab, (2, 23))
    rows = np.arange(8, 16)
    lg, cache = okv.forward_refresh(CFG, w, x, rows)
    np.testing.assert_allclose(lg, of.forward(CFG, w, x, rows=rows), rtol=1e-12, atol=1e-12)
    assert len(cache) == CFG.n_layers
    for K, V in cache:
        assert K.shape == V.shape == (2, CFG.n_kv_heads, 23, CFG.head_dim)


def test_refresh_layer0_cache_matches_torch():
    """Layer-0 keys and values from torch library calls: rms_norm, linear and
    RoPE as a complex rotation of (x_j, x_{j+hd/2})."""
    w = _w(CFG)
    x = rng.integers(0, CFG.vocab, (2, 19))
    _, cache = okv.forward_refresh(CFG, w, x, np.arange(3))
    W = [torch.from_numpy(t) for t in w]
    hd, half = CFG.head_dim, CFG.head_dim // 2
    e = W[0][torch.from_numpy(x)]
    a = F.rms_norm(e, (CFG.d_model,), W[1], CFG.rms_eps)
    k = F.linear(a, W[3]).view(2, 19, CFG.n_kv_heads, hd).transpose(1, 2)
    v = F.linear(a, W[4]).view(2, 19, CFG.n_kv_heads, hd).transpose(1, 2)
    freq = torch.tensor([CFG.rope_base ** (-2.0 * j / hd) for j in range(half)], dtype=torch.float64)
    ang = torch.arange(19, dtype=torch.float64)[:, None] * freq[None, :]
    z = torch.complex(k[..., :half], k[..., half:]) * torch.polar(torch.ones_like(ang), ang)
    k_rot = torch.cat([z.real, z.imag], dim=-1)
    np.testing.assert_allclose(cache[0][0], k_rot.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(cache[0][1], v.numpy(), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("row0,n", [(8, 8), (0, 4), (15, 8)])
def test_cached_equals_full_right_after_refresh(row0, n):
    w = _w(CFG)
    x = rng.integers(0, CFG.vocab, (2, 23))
    _, cache = okv.forward_refresh(CFG, w, x, np.arange(row0, row0 + n))
    got = okv.forward_cached(CFG, w, x, cache, row0, n)
    np.testing.assert_allclose(got, of.forward(CFG, w, x, rows=np.arange(row0, row0 + n)), rtol=1e-10, atol=1e-10)


def test_cached_one_layer_exact_for_new_block_tokens():
    """One layer: the stored keys/values of the other positions depend only on
    their own tokens, so the cached forward is exact whatever the block holds."""
    cfg = synth.reduced(CFG, n_layers=1)
    w = _w(cfg)
    x = rng.integers(0, cfg.vocab, (2, 21))
    _, cache = okv.forward_refresh(cfg, w, x, np.arange(5, 13))
    x2 = x.copy()
    x2[:, 5:13] = rng.integers(0, cfg.vocab, (2, 8))
    got = okv.forward_cached(cfg, w, x2, cache, 5, 8)
    np.testing.assert_allclose(got, of.forward(cfg, w, x2, rows=np.arange(5, 13)), rtol=1e-10, atol=1e-10)
    # a change outside the block is not seen until the next refresh
    x3 = x2.copy()
    x3[:, 0] = (x3[:, 0] + 1) % cfg.vocab
    np.testing.assert_array_equal(okv.forward_cached(cfg, w, x3, cache, 5, 8), got)


def test_cached_two_layers_is_an_approximation():
    w = _w(CFG)
    x = rng.integers(0, CFG.vocab, (1, 21))
    _, cache = okv.forward_refresh(CFG, w, x, np.arange(5, 13))
    x2 = x.copy()
    x2[:, 5:13] = rng.integers(0, CFG.vocab, (1, 8))
    diff = np.abs(okv.forward_cached(CFG, w, x2, cache, 5, 8) - of.forward(CFG, w, x2, rows=np.arange(5, 13)))
    assert diff.max() > 1e-6


def test_cached_bf16_right_after_refresh():
    cfg = synth.reduced(CFG, dtype="bf16")
    w = [t.to(torch.float32).numpy() for t in synth.make_weights(cfg)]
    x = rng.integers(0, cfg.vocab, (2, 20))
    _, cache = okv.forward_refresh(cfg, w, x, np.arange(4, 12), mode="bf16")
    got = okv.forward_cached(cfg, w, x, cache, 4, 8, mode="bf16")
    want = of.forward(cfg, w, x, rows=np.arange(4, 12), mode="bf16")
    # the same values are rounded to bf16 at the same points; float32 products
    # over fewer rows may still round a value across a bf16 boundary
    err = np.abs(got - want)
    assert err.mean() < 5e-4 and err.max() < 5e-2, (err.mean(), err.max())


def _decode(cfg, w, prompts, G, p, refresh, log=None):
    P = prompts.shape[1]
    pred = okv.cached_predictor(cfg, w, P, p.block_len, cfg.vocab - 1, refresh, log=log)
    return oc.generate(pred, prompts, G, cfg.vocab - 1, p)


def test_cached_decode_refresh_schedule_and_every_step_case():
    w = _w(CFG)
    prompts = rng.integers(0, CFG.vocab - 1, (2, 9))
    p = oc.CaiParams(block_len=8, budgets=False, grinding=False)      # every block runs all T = 8 steps
    log = []
    st = _decode(CFG, w, prompts, 16, p, 3, log)
    assert [r for (_, _, r) in log] == [t % 3 == 0 for _ in range(2) for t in range(8)]
    assert [(b, t) for (b, t, _) in log] == [(b, t) for b in range(2) for t in range(8)]
    assert (st.commit_step >= 0).all() and (st.x[:, 9:] != CFG.vocab - 1).all()
    # refreshing at every step is the no-cache decode
    full = oc.model_predictor(lambda x, rows: of.forward(CFG, w, x, rows=rows), 9, 8, CFG.vocab - 1)
    ref = oc.generate(full, prompts, 16, CFG.vocab - 1, p)
    st1 = _decode(CFG, w, prompts, 16, p, 1)
    np.testing.assert_array_equal(st1.x, ref.x)
    np.testing.assert_array_equal(st1.commit_step, ref.commit_step)
    np.testing.assert_array_equal(st1.reason, ref.reason)
