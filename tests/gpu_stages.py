"""Stage-by-stage parity of the bf16 forward against the oracle.

In a bf16 model every matrix-product operand is rounded to bf16.  Two correct
implementations that accumulate in a different order round a few values to
the neighbouring bf16 number, and through later layers those differences grow
to the size of bf16 rounding itself, so end-to-end logits of a deep random
model cannot be compared tightly.  Instead each stage of the GPU forward is
compared with the oracle applied to the GPU's own input of that stage: bf16
outputs may differ by one unit in the last place on a small fraction of
elements, float32 outputs only by accumulation-order rounding.
"""
import numpy as np
import torch

from helpers import assert_bf16_flips, bf16_ulp, say, to_np
from oracle import forward as of
from oracle import vocab as ov


def ws_view(ws, off, dtype, shape):
    n = int(np.prod(shape)) * torch.empty((), dtype=dtype).element_size()
    return ws[off:off + n].view(dtype).view(*shape)


def read(ws, off, dtype, shape, rows=None):
    t = ws_view(ws, off, dtype, shape)
    if rows is not None:
        t = t[torch.as_tensor(rows, device=t.device)]
    return to_np(t, np.float64)


def layer_weights(wnp, l):
    return wnp[1 + 9 * l: 10 + 9 * l]


def check_layer(model, cfg, wnp, ws, B, L, l, rows=None, key_rows=None, stats=None):
    """Run layer l on the GPU (both halves) and check every stage.

    rows: sampled flat rows (b*L + pos) checked for row-wise stages (all if None).
    key_rows: sampled positions whose k / v are checked (all if None)."""
    lay = model.layout(B, L, 0)
    d, H, Hkv, hd, F = cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d_ff
    M = B * L
    an, wq, wk, wv, wo, mn, wg, wu, wd = layer_weights(wnp, l)
    cos, sin = of.rope_tables(L, hd, cfg.rope_base)
    allrows = np.arange(M) if rows is None else np.asarray(rows)
    stats = stats if stats is not None else {}

    h_in = read(ws, lay.h, torch.float32, (M, d), allrows)
    model.layer(l, 0, B, L, ws)
    torch.cuda.synchronize()
    a = read(ws, lay.a_attn, torch.bfloat16, (M, d))                      # all rows (q/k/v need them)
    q = read(ws, lay.q, torch.bfloat16, (B, H, L, hd))
    k = read(ws, lay.k, torch.bfloat16, (B, Hkv, L, hd))
    vt = read(ws, lay.vt, torch.float16, (B, Hkv, hd, L))                 # bf16 values held as half
    attn = read(ws, lay.attn, torch.bfloat16, (M, H * hd), allrows)
    h_mid = read(ws, lay.h, torch.float32, (M, d), allrows)
    model.layer(l, 1, B, L, ws)
    torch.cuda.synchronize()
    a2 = read(ws, lay.a_mlp, torch.bfloat16, (M, d), allrows)
    u = read(ws, lay.u, torch.bfloat16, (M, F), allrows)
    h_out = read(ws, lay.h, torch.float32, (M, d), allrows)

    # attention-norm output
    stats["a_attn"] = assert_bf16_flips(a[allrows], of.norm_in(h_in, an, cfg.rms_eps, "bf16"), f"L{l} a_attn")
    # q / k / v with RoPE from the GPU's normed input
    bb, pp = allrows // L, allrows % L
    qr, kr, vr = [], [], []
    for b in range(B):
        sel = allrows[bb == b]
        if len(sel) == 0:
            continue
        pos = sel % L
        q_ref, _, _ = of.qkv_rope(cfg, a[sel], wq, wk, wv, cos[pos], sin[pos], "bf16")
        qr.append((q[b][:, pos], q_ref))
        kp = np.arange(L) if key_rows is None else np.asarray(key_rows)
        _, k_ref, v_ref = of.qkv_rope(cfg, a[b * L + kp], wq, wk, wv, cos[kp], sin[kp], "bf16")
        kr.append((k[b][:, kp], k_ref))
        vr.append((vt[b][:, :, kp].transpose(0, 2, 1), v_ref))
    stats["q"] = assert_bf16_flips(np.concatenate([g for g, _ in qr], 1), np.concatenate([r for _, r in qr], 1),
                                   f"L{l} q")
    stats["k"] = assert_bf16_flips(np.concatenate([g for g, _ in kr], 1), np.concatenate([r for _, r in kr], 1),
                                   f"L{l} k")
    stats["v"] = assert_bf16_flips(np.concatenate([g for g, _ in vr], 1), np.concatenate([r for _, r in vr], 1),
                                   f"L{l} v")
    # attention from the GPU's q / k / v.  The GPU rounds the probabilities to
    # IEEE half (relative error <= 2^-11) for the P.V product, so the bound is
    # 2^-11 * sum_k p_k |v_k| on top of one bf16 ulp of the final rounding.
    o_ref = np.empty_like(attn)
    bound = np.empty_like(attn)
    v_full = vt.transpose(0, 1, 3, 2)
    scale = 1.0 / np.sqrt(hd)
    for b in range(B):
        sel = np.nonzero(bb == b)[0]
        if len(sel) == 0:
            continue
        qs = q[b][:, pp[sel]]
        o_ref[sel] = of.attn_out(qs, k[b], v_full[b], "bf16")
        grp = H // Hkv
        for hh in range(H):
            p = of.softmax(qs[hh] @ k[b][hh // grp].T * scale)
            bound[sel, hh * hd:(hh + 1) * hd] = 2.0 ** -11 * (p @ np.abs(v_full[b][hh // grp]))
    d_att = np.abs(attn - o_ref)
    lim = bound + 1.0001 * np.maximum(bf16_ulp(o_ref), bf16_ulp(attn)) + 1e-6
    assert np.all(d_att <= lim), f"L{l} attn: {int((d_att > lim).sum())} beyond the bound; max {d_att.max():.3g}"
    stats["attn"] = float(np.mean(d_att > 0))
    # output projection + residual (float32)
    hm_ref = of.residual(h_in, attn, wo, "bf16")
    scale = np.abs(hm_ref).max() + 1.0
    err = np.abs(h_mid - hm_ref).max()
    assert err <= 2e-5 * scale, f"L{l} h_mid err {err:.3g} (scale {scale:.3g})"
    stats["h_mid"] = err / scale
    # MLP
    stats["a_mlp"] = assert_bf16_flips(a2, of.norm_in(h_mid, mn, cfg.rms_eps, "bf16"), f"L{l} a_mlp")
    stats["u"] = assert_bf16_flips(u, of.swiglu(a2, wg, wu, "bf16"), f"L{l} u")
    ho_ref = of.residual(h_mid, u, wd, "bf16")
    scale = np.abs(ho_ref).max() + 1.0
    err = np.abs(h_out - ho_ref).max()
    assert err <= 2e-5 * scale, f"L{l} h_out err {err:.3g} (scale {scale:.3g})"
    stats["h_out"] = err / scale
    return stats


def check_head(model, cfg, wnp, ws, B, L, row0, rows, sample=None):
    """Final norm + fused LM head on the GPU's final residual; logits / conf /
    argmax against the oracle on the GPU's normed head rows."""
    lay = model.layout(B, L, rows)
    d, V = cfg.d_model, cfg.vocab
    conf, arg, lg = model.head(B, L, row0, rows, ws, logits=True)
    torch.cuda.synchronize()
    flat = (np.arange(B)[:, None] * L + row0 + np.arange(rows)[None, :]).reshape(-1)
    h = read(ws, lay.h, torch.float32, (B * L, d), flat)
    hb = read(ws, lay.hb, torch.bfloat16, (B * rows, d))
    sel = np.arange(B * rows) if sample is None else np.asarray(sample)
    fa = assert_bf16_flips(hb[sel], of.norm_in(h[sel], wnp[-2], cfg.rms_eps, "bf16"), "head hb")
    lg_ref = hb[sel] @ wnp[-1].astype(np.float64).T                       # exact products, float64 sums
    lg_g = to_np(lg.view(B * rows, V)[torch.as_tensor(sel, device=lg.device)], np.float64)
    err = np.abs(lg_g - lg_ref)
    assert err.max() <= 2e-2, f"logits err {err.max():.3g}"
    conf_ref, arg_ref = ov.confidence_argmax(lg_ref, cfg.mask_id)
    cg = to_np(conf.view(-1), np.float64)[sel]
    ag = arg.view(-1).cpu().numpy()[sel]
    cerr = np.abs(cg - conf_ref).max()
    assert cerr <= 2e-2, f"conf err {cerr:.3g}"
    gap = ov.top2_gap(lg_ref, cfg.mask_id)
    diff = ag != arg_ref
    assert np.all(gap[diff] < 2 * err.max() + 1e-6), "argmax differs away from a near-tie"
    # the fused reduction against the GPU's own logits (same float32 values)
    conf_self, arg_self = ov.confidence_argmax(lg_g, cfg.mask_id)
    assert np.abs(cg - conf_self).max() <= 1e-5
    assert np.array_equal(ag, arg_self)
    return dict(hb_flips=fa, logit_err=float(err.max()), conf_err=float(cerr), argmax_diff=int(diff.sum()))


def kv_views(model, kv, B, L, l):
    """Layer l's cache entries: keys [B, Hkv, L, hd] and values^T [B, Hkv, hd, L]
    (bf16 keys, IEEE-half values for a bf16 model; float32 for fp32)."""
    cfg = model.cfg
    es = 2 if cfg.dtype == "bf16" else 4
    n = B * cfg.n_kv_heads * L * cfg.head_dim
    S = (n * es + 255) // 256 * 256
    kd, vd = (torch.bfloat16, torch.float16) if cfg.dtype == "bf16" else (torch.float32, torch.float32)
    base = l * 2 * S
    K = kv[base:base + n * es].view(kd).view(B, cfg.n_kv_heads, L, cfg.head_dim)
    V = kv[base + S:base + S + n * es].view(vd).view(B, cfg.n_kv_heads, cfg.head_dim, L)
    return K, V


def check_layer_cached(model, cfg, wnp, ws, kv, B, L, row0, Lq, l, stats=None):
    """Run layer l of a cached step (rows row0 .. row0 + Lq - 1 of each sequence,
    keys/values of the other positions from the cache) on the GPU and check every
    stage against the oracle on the GPU's own stage inputs, including that the
    cache changes at the block positions only."""
    lay = model.layout(B, L, Lq)
    d, H, Hkv, hd, F = cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d_ff
    M = B * Lq
    an, wq, wk, wv, wo, mn, wg, wu, wd = layer_weights(wnp, l)
    cos, sin = of.rope_tables(L, hd, cfg.rope_base)
    pos = row0 + np.arange(Lq)
    stats = stats if stats is not None else {}
    Kc, Vc = kv_views(model, kv, B, L, l)
    k_before, v_before = to_np(Kc, np.float64), to_np(Vc, np.float64)

    h_in = read(ws, lay.h, torch.float32, (M, d))
    model.layer_kv(l, 0, B, L, row0, Lq, kv, ws)
    torch.cuda.synchronize()
    a = read(ws, lay.a_attn, torch.bfloat16, (M, d))
    q = read(ws, lay.q, torch.bfloat16, (B, H, Lq, hd))
    K, V = to_np(Kc, np.float64), to_np(Vc, np.float64)
    attn = read(ws, lay.attn, torch.bfloat16, (M, H * hd))
    h_mid = read(ws, lay.h, torch.float32, (M, d))
    model.layer_kv(l, 1, B, L, row0, Lq, kv, ws)
    torch.cuda.synchronize()
    a2 = read(ws, lay.a_mlp, torch.bfloat16, (M, d))
    u = read(ws, lay.u, torch.bfloat16, (M, F))
    h_out = read(ws, lay.h, torch.float32, (M, d))

    stats["a_attn"] = assert_bf16_flips(a, of.norm_in(h_in, an, cfg.rms_eps, "bf16"), f"L{l} a_attn")
    out = np.ones(L, dtype=bool)
    out[pos] = False
    assert np.array_equal(K[:, :, out], k_before[:, :, out]), f"L{l}: cached keys outside the block changed"
    assert np.array_equal(V[:, :, :, out], v_before[:, :, :, out]), f"L{l}: cached values outside the block changed"
    qr, kr, vr = [], [], []
    for b in range(B):
        q_ref, k_ref, v_ref = of.qkv_rope(cfg, a[b * Lq:(b + 1) * Lq], wq, wk, wv, cos[pos], sin[pos], "bf16")
        qr.append((q[b], q_ref))
        kr.append((K[b][:, pos], k_ref))
        vr.append((V[b][:, :, pos].transpose(0, 2, 1), v_ref))
    for name, pairs in (("q", qr), ("k", kr), ("v", vr)):
        stats[name] = assert_bf16_flips(np.concatenate([g for g, _ in pairs], 1),
                                        np.concatenate([r for _, r in pairs], 1), f"L{l} {name}")
    # attention of the block queries over every cached position (bound as in check_layer)
    o_ref = np.empty_like(attn)
    bound = np.empty_like(attn)
    scale = 1.0 / np.sqrt(hd)
    grp = H // Hkv
    for b in range(B):
        vf = V[b].transpose(0, 2, 1)
        sel = slice(b * Lq, (b + 1) * Lq)
        o_ref[sel] = of.attn_out(q[b], K[b], vf, "bf16")
        for hh in range(H):
            p = of.softmax(q[b][hh] @ K[b][hh // grp].T * scale)
            bound[sel, hh * hd:(hh + 1) * hd] = 2.0 ** -11 * (p @ np.abs(vf[hh // grp]))
    d_att = np.abs(attn - o_ref)
    lim = bound + 1.0001 * np.maximum(bf16_ulp(o_ref), bf16_ulp(attn)) + 1e-6
    assert np.all(d_att <= lim), f"L{l} attn: {int((d_att > lim).sum())} beyond the bound; max {d_att.max():.3g}"
    stats["attn"] = float(np.mean(d_att > 0))
    for name, got, ref in (("h_mid", h_mid, of.residual(h_in, attn, wo, "bf16")),):
        sc = np.abs(ref).max() + 1.0
        err = np.abs(got - ref).max()
        assert err <= 2e-5 * sc, f"L{l} {name} err {err:.3g} (scale {sc:.3g})"
        stats[name] = err / sc
    stats["a_mlp"] = assert_bf16_flips(a2, of.norm_in(h_mid, mn, cfg.rms_eps, "bf16"), f"L{l} a_mlp")
    stats["u"] = assert_bf16_flips(u, of.swiglu(a2, wg, wu, "bf16"), f"L{l} u")
    ho_ref = of.residual(h_mid, u, wd, "bf16")
    sc = np.abs(ho_ref).max() + 1.0
    err = np.abs(h_out - ho_ref).max()
    assert err <= 2e-5 * sc, f"L{l} h_out err {err:.3g} (scale {sc:.3g})"
    stats["h_out"] = err / sc
    return stats
