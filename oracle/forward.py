"""Bidirectional transformer forward of a masked diffusion LM (oracle).

Each denoising step runs the full model on the current partially-masked
sequence (Algorithm 1, "run forward pass"; Section 2: all masked positions are
predicted in one pass, with no causal mask).  The paper names the models
(LLaDA-8B, Dream-7B; Section 5) but prints no architecture; the layer used
here is the one those model families share:

  a   = RMSNorm(h) * g_attn
  q,k = RoPE(a Wq^T), RoPE(a Wk^T);  v = a Wv^T           (rotate-half RoPE)
  o   = softmax(q k^T / sqrt(hd)) v, every query attends to every key (GQA:
        query head j reads kv head j // (Hq / Hkv))
  h  += o Wo^T
  a   = RMSNorm(h) * g_mlp
  h  += (silu(a Wg^T) * (a Wu^T)) Wd^T
and, after the last layer, logits = (RMSNorm(h) * g_final) Wlm^T.

Precision modes
  "f64"  : every operation in float64 (the oracle of an fp32 model).
  "bf16" : the model's stored tensors are bf16.  Reading used for a bf16
           model: every operand of a matrix product is a bf16 value -- the
           normed activations, RoPE'd q/k and v, the attention output, the
           SwiGLU product and the final normed hidden state are rounded to
           bf16 (round-to-nearest-even) where they are produced -- while the
           residual stream, norm statistics, softmax and SiLU stay in float64
           and products accumulate in float32 (BLAS sgemm).
  "bf16_f64acc" : the same rounding points as "bf16", but every matrix
           product accumulates in float64.  Not a model of any kernel: it
           measures how far two correct float32 accumulation orders of one
           bf16 model can drift apart once bf16 rounding of the activations
           turns last-bit differences into whole bf16 steps (the bar that
           end-to-end bf16 logits are held to is set from that drift).

Test infrastructure only; see the package docstring.
"""
import math

import numpy as np


# ---------------------------------------------------------------------------
# bf16 rounding: keep the top 16 bits of the IEEE float32 pattern, rounding the
# dropped 16 bits to nearest with ties to even.
# ---------------------------------------------------------------------------
def round_bf16(x):
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    out = (r & 0xFFFFFFFF).astype(np.uint32).view(np.float32)
    return np.where(np.isnan(f), f, out)


def rmsnorm(x, gain, eps):
    """x / sqrt(mean(x^2) + eps) * gain over the last axis, float64."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(gain, dtype=np.float64)


def rope_tables(seq_len, head_dim, base):
    """cos/sin [L, hd/2] for angle pos * base^(-2j/hd), j = 0..hd/2-1 (float64)."""
    half = head_dim // 2
    j = np.arange(half, dtype=np.float64)
    inv_freq = base ** (-2.0 * j / head_dim)
    ang = np.arange(seq_len, dtype=np.float64)[:, None] * inv_freq[None, :]
    return np.cos(ang), np.sin(ang)


def rope(x, cos, sin):
    """Rotate-half RoPE on x [..., L, hd]: pairs (j, j + hd/2) are rotated by the
    angle of frequency j at the row's position."""
    half = x.shape[-1] // 2
    x1 = x[..., :half]
    x2 = x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def softmax(s, axis=-1):
    s = np.asarray(s, dtype=np.float64)
    m = s.max(axis=axis, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=axis, keepdims=True)


def silu(x):
    x = np.asarray(x, dtype=np.float64)
    return x / (1.0 + np.exp(-x))


def attention(q, k, v, mode="f64"):
    """Non-causal multi-head attention with grouped KV heads.

    q [Hq, L, hd], k/v [Hkv, L, hd] -> o [Hq, L, hd].  No mask: every query
    position attends to every key position of the sequence.
    """
    hq, L, hd = q.shape
    hkv = k.shape[0]
    group = hq // hkv
    scale = 1.0 / math.sqrt(hd)
    dt = np.float32 if mode == "bf16" else np.float64
    out = np.empty((hq, L, hd), dtype=np.float64)
    for h in range(hq):
        kv = h // group
        s = (q[h].astype(dt) @ k[kv].astype(dt).T).astype(np.float64) * scale
        p = softmax(s, axis=-1)
        out[h] = (p.astype(dt) @ v[kv].astype(dt)).astype(np.float64)
    return out


def _matmul(a, w, mode):
    """a [M, K] @ w[N, K]^T: float32 BLAS in "bf16" mode, float64 otherwise."""
    if mode != "bf16":
        return np.asarray(a, np.float64) @ np.asarray(w, np.float64).T
    return (np.asarray(a, np.float32) @ np.asarray(w, np.float32).T).astype(np.float64)


def _op(x, mode):
    """Value handed to a matrix product: bf16-rounded in the bf16 modes."""
    return round_bf16(x).astype(np.float64) if mode != "f64" else np.asarray(x, np.float64)


def norm_in(h, gain, eps, mode):
    """Normed activation handed to the next projections (RMSNorm, then bf16 in "bf16" mode)."""
    return _op(rmsnorm(h, gain, eps), mode)


def qkv_rope(cfg, a, wq, wk, wv, cos, sin, mode):
    """a [L, d] -> q [Hq, L, hd], k [Hkv, L, hd], v [Hkv, L, hd] with RoPE on q, k.
    cos/sin hold the rows' positions."""
    L = a.shape[0]
    H, Hkv, hd = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    q = _matmul(a, wq, mode).reshape(L, H, hd).transpose(1, 0, 2)
    k = _matmul(a, wk, mode).reshape(L, Hkv, hd).transpose(1, 0, 2)
    v = _matmul(a, wv, mode).reshape(L, Hkv, hd).transpose(1, 0, 2)
    return _op(rope(q, cos, sin), mode), _op(rope(k, cos, sin), mode), _op(v, mode)


def attn_out(q, k, v, mode):
    """Attention of q [Hq, Lq, hd] over k/v [Hkv, L, hd] -> o [Lq, Hq*hd] (bf16 in "bf16" mode)."""
    o = attention(q, k, v, mode)
    return _op(o.transpose(1, 0, 2).reshape(q.shape[1], -1), mode)


def swiglu(a, wg, wu, mode):
    """silu(a Wg^T) * (a Wu^T) -> [L, F] (bf16 in "bf16" mode)."""
    return _op(silu(_matmul(a, wg, mode)) * _matmul(a, wu, mode), mode)


def residual(h, x, w, mode):
    """h + x W^T with the residual kept in float64."""
    return np.asarray(h, np.float64) + _matmul(x, w, mode)


def layer(cfg, w, h, cos, sin, mode):
    """One transformer layer on h [B, L, d] (float64 residual); w = the layer's 9 tensors."""
    attn_norm, wq, wk, wv, wo, mlp_norm, wg, wu, wd = w
    out = np.empty(h.shape, dtype=np.float64)
    for b in range(h.shape[0]):
        a = norm_in(h[b], attn_norm, cfg.rms_eps, mode)
        q, k, v = qkv_rope(cfg, a, wq, wk, wv, cos, sin, mode)
        hm = residual(h[b], attn_out(q, k, v, mode), wo, mode)
        a = norm_in(hm, mlp_norm, cfg.rms_eps, mode)
        out[b] = residual(hm, swiglu(a, wg, wu, mode), wd, mode)
    return out


def lm_head(cfg, h, final_norm, lm_head_w, mode):
    """Final RMSNorm and LM head on h [R, d] -> (logits [R, V] float64, normed hidden)."""
    hb = norm_in(h, final_norm, cfg.rms_eps, mode)
    return _matmul(hb, lm_head_w, mode), hb


def forward(cfg, weights, tokens, rows=None, mode="f64", return_hidden=False):
    """Logits of the rows ``rows`` (default: all) for token ids ``tokens`` [B, L].

    cfg: any object with n_layers, d_model, n_heads, n_kv_heads, head_dim,
    rms_eps, rope_base.  weights: the 3 + 9 * n_layers tensors in the fixed
    order (embed, per-layer 9, final_norm, lm_head) as numpy arrays.
    Returns float64 logits [B, len(rows), V] (and the final normed hidden).
    """
    tokens = np.asarray(tokens, dtype=np.int64)
    B, L = tokens.shape
    embed = np.asarray(weights[0])
    h = embed[tokens].astype(np.float64)                          # [B, L, d]
    cos, sin = rope_tables(L, cfg.head_dim, cfg.rope_base)
    for l in range(cfg.n_layers):
        h = layer(cfg, weights[1 + 9 * l: 10 + 9 * l], h, cos, sin, mode)
    rows = np.arange(L) if rows is None else np.asarray(rows)
    logits, hb = lm_head(cfg, h[:, rows, :].reshape(-1, cfg.d_model), weights[-2], weights[-1], mode)
    logits = logits.reshape(B, len(rows), -1)
    if return_hidden:
        return logits, hb.reshape(B, len(rows), -1)
    return logits
