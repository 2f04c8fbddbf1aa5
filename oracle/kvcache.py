"""Cross-step key/value reuse in the denoising loop (oracle).

Section 5 states that the decoder runs on the KV cache backend of the ES-dLLM
codebase, with a cache update frequency of 16 steps for LLaDA and 8 for Dream;
the related-work section describes the cache it stands for (Fast-dLLM's
DualCache: keys/values of the positions outside the current block are reused
across steps).  The paper does not spell the mechanism out; reading taken:

  R22 Local step t of a block is a refresh step when t % R == 0 (R = the update
      frequency; t = 0 always refreshes).  A refresh step runs the full forward
      over all L positions and stores every layer's keys (after RoPE) and
      values for all positions.  Any other step runs only the current block's
      rows through the layers: per layer the block rows' q, k, v come from
      their own hidden states; the keys/values of every other position are the
      stored ones (as of the last refresh); the block rows' fresh k, v take the
      place of the stored ones at the block positions; the block queries attend
      to all L positions (no mask); output projection, MLP, final norm and LM
      head run on the block rows only.  Predictions at a refresh step are those
      of the full forward.

Consequences used by the pins: right after a refresh, the cached forward of
the unchanged sequence equals the full forward on the block rows; in a
one-layer model the stored keys/values of the other positions depend only on
their own tokens, so the cached forward equals the full forward for any block
tokens.  With two or more layers it is an approximation: stored keys/values
of deeper layers still reflect the block tokens of the last refresh.

Test infrastructure only; see the package docstring.
"""
import numpy as np

from . import forward as F


def _layer_capture(cfg, w, h, cos, sin, mode):
    """One layer on h [B, L, d] as forward.layer, also returning the layer's
    keys after RoPE and values, each [B, Hkv, L, hd]."""
    attn_norm, wq, wk, wv, wo, mlp_norm, wg, wu, wd = w
    out = np.empty(h.shape, dtype=np.float64)
    ks, vs = [], []
    for b in range(h.shape[0]):
        a = F.norm_in(h[b], attn_norm, cfg.rms_eps, mode)
        q, k, v = F.qkv_rope(cfg, a, wq, wk, wv, cos, sin, mode)
        ks.append(k)
        vs.append(v)
        hm = F.residual(h[b], F.attn_out(q, k, v, mode), wo, mode)
        a = F.norm_in(hm, mlp_norm, cfg.rms_eps, mode)
        out[b] = F.residual(hm, F.swiglu(a, wg, wu, mode), wd, mode)
    return out, np.stack(ks), np.stack(vs)


def forward_refresh(cfg, weights, tokens, rows, mode="f64"):
    """Full forward (as forward.forward) that also returns the cache: a list over
    layers of (K, V), each [B, Hkv, L, hd].  Returns (logits [B, len(rows), V],
    cache)."""
    tokens = np.asarray(tokens, dtype=np.int64)
    B, L = tokens.shape
    h = np.asarray(weights[0])[tokens].astype(np.float64)
    cos, sin = F.rope_tables(L, cfg.head_dim, cfg.rope_base)
    cache = []
    for l in range(cfg.n_layers):
        h, k, v = _layer_capture(cfg, weights[1 + 9 * l: 10 + 9 * l], h, cos, sin, mode)
        cache.append((k, v))
    rows = np.asarray(rows)
    logits, _ = F.lm_head(cfg, h[:, rows, :].reshape(-1, cfg.d_model), weights[-2], weights[-1], mode)
    return logits.reshape(B, len(rows), -1), cache


def forward_cached(cfg, weights, tokens, cache, row0, nrows, mode="f64"):
    """Forward of rows row0 .. row0 + nrows - 1 only, against the stored keys and
    values of every other position (R22).  Returns logits [B, nrows, V]."""
    tokens = np.asarray(tokens, dtype=np.int64)
    B, L = tokens.shape
    blk = np.arange(row0, row0 + nrows)
    cos, sin = F.rope_tables(L, cfg.head_dim, cfg.rope_base)
    cb, sb = cos[blk], sin[blk]                                   # the block rows' positions
    h = np.asarray(weights[0])[tokens[:, blk]].astype(np.float64)  # [B, nrows, d]
    for l in range(cfg.n_layers):
        attn_norm, wq, wk, wv, wo, mlp_norm, wg, wu, wd = weights[1 + 9 * l: 10 + 9 * l]
        K, V = cache[l]
        out = np.empty(h.shape, dtype=np.float64)
        for b in range(B):
            a = F.norm_in(h[b], attn_norm, cfg.rms_eps, mode)
            q, k, v = F.qkv_rope(cfg, a, wq, wk, wv, cb, sb, mode)
            Kb, Vb = K[b].copy(), V[b].copy()
            Kb[:, blk, :] = k
            Vb[:, blk, :] = v
            hm = F.residual(h[b], F.attn_out(q, Kb, Vb, mode), wo, mode)
            a = F.norm_in(hm, mlp_norm, cfg.rms_eps, mode)
            out[b] = F.residual(hm, F.swiglu(a, wg, wu, mode), wd, mode)
        h = out
    logits, _ = F.lm_head(cfg, h.reshape(-1, cfg.d_model), weights[-2], weights[-1], mode)
    return logits.reshape(B, nrows, -1)


def is_refresh(t, refresh):
    """Whether local step t of a block runs the full forward (R22)."""
    return t % refresh == 0


def cached_predictor(cfg, weights, P, block_len, mask_id, refresh, mode="f64", log=None):
    """predict(x, blk, t) for controller.generate with cross-step KV reuse: the
    full forward (refreshing the cache) at refresh steps, the cached block
    forward otherwise; confidence/argmax of the block rows (Box 1).  log, if
    given, receives (blk, t, refreshed) per call."""
    from .vocab import confidence_argmax
    state = {"cache": None}

    def predict(x, blk, t):
        row0 = P + blk * block_len
        if is_refresh(t, refresh):
            logits, state["cache"] = forward_refresh(cfg, weights, x, np.arange(row0, row0 + block_len), mode)
        else:
            logits = forward_cached(cfg, weights, x, state["cache"], row0, block_len, mode)
        if log is not None:
            log.append((blk, t, is_refresh(t, refresh)))
        conf, arg = confidence_argmax(logits, mask_id)
        return conf.astype(np.float32), arg

    return predict
