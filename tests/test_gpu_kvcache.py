"""Cross-step key/value reuse on the GPU against the oracle (oracle/kvcache.py).

* tiny fp32 model: the refresh forward equals dllm_forward bit for bit; the
  cached forward of a block whose tokens changed since the refresh agrees with
  the float64 oracle's cached forward (same stale cache) within 1e-5; decodes
  with refresh every 4 and 16 steps: the oracle controller replayed on the
  GPU's predictions reproduces every decision bit for bit, every step's
  confidences agree with the oracle (full forward at refresh steps, cached
  forward from the oracle's own cache otherwise) within 1e-5, and the
  free-running oracle decode equals the GPU decode; refresh every step equals
  dllm_generate;
* small bf16 model: the cache a refresh fills equals the keys/values of the
  plain forward bit for bit; every stage of a cached layer against the oracle
  on the GPU's own stage inputs, also with the packed weight copies
  (dllm_model_pack_weights: at most 64 block rows run the register-direct
  GEMM); decode replay; packed and plain cached forwards bit-identical where
  both run the same tiles (more than 64 rows), close otherwise;
* full-size LLaDA-8B / Dream-7B shapes (packed weights): one cached layer's
  stages and the decode replay with the paper's update frequencies (16 and 8).
"""
import math

import numpy as np
import pytest
import torch

from gpu_stages import check_layer_cached, kv_views, ws_view
from helpers import assert_state_equal, oracle_params, replay, say, tie_aware_predictor, to_np, x_at_step
from oracle import controller as oc
from oracle import forward as of
from oracle import kvcache as okv
from oracle import vocab as ov
from paper_2608_22646_amd import binding as B
from paper_2608_22646_amd import synth

pytestmark = pytest.mark.gpu
WL = synth.WORKLOADS["tiny"]
TOL = 1e-5


@pytest.fixture(scope="module")
def tiny():
    cfg = WL.model
    w_cpu = synth.make_weights(cfg, "cpu")
    model = B.Model(cfg, [w.to("cuda") for w in w_cpu])
    return cfg, model, [w.numpy().astype(np.float64) for w in w_cpu]


def _changed_block(x, row0, n, seed, vocab):
    x2 = x.copy()
    g = np.random.default_rng(seed)
    x2[:, row0:row0 + n] = g.integers(0, vocab - 1, (x.shape[0], n))
    return x2


def test_tiny_refresh_equals_forward(tiny):
    cfg, model, _ = tiny
    P, bl = WL.prompt_len, 32
    x = synth.make_ints((1, P + WL.gen_len), 3, 0, cfg.vocab - 1).cuda()
    say("tiny kv refresh forward")
    kv = model.kv_cache(1, x.shape[1])
    c1, a1, l1 = model.forward(x, P, bl, logits=True)
    c2, a2, l2 = model.forward_kv(x, P, bl, kv, refresh=True, logits=True)
    torch.cuda.synchronize()
    assert torch.equal(l1.view(torch.int32), l2.view(torch.int32))
    assert torch.equal(c1.view(torch.int32), c2.view(torch.int32)) and torch.equal(a1, a2)


@pytest.mark.parametrize("blk", [0, 1])
def test_tiny_cached_forward_matches_oracle(tiny, blk):
    cfg, model, wnp = tiny
    P, bl = WL.prompt_len, 32
    L = P + WL.gen_len
    row0 = P + blk * bl
    x0 = synth.make_ints((2, L), 4, 0, cfg.vocab - 1).numpy().astype(np.int64)
    x1 = _changed_block(x0, row0, bl, 5, cfg.vocab)
    say(f"tiny kv cached forward block {blk}")
    kv = model.kv_cache(2, L)
    ws = model.workspace(2, L, bl)
    model.forward_kv(torch.from_numpy(x0.astype(np.int32)).cuda(), row0, bl, kv, refresh=True, ws=ws)
    conf, arg, lg = model.forward_kv(torch.from_numpy(x1.astype(np.int32)).cuda(), row0, bl, kv, refresh=False,
                                     ws=ws, logits=True)
    torch.cuda.synchronize()
    _, cache = okv.forward_refresh(cfg, wnp, x0, np.arange(row0, row0 + bl))
    lg_ref = okv.forward_cached(cfg, wnp, x1, cache, row0, bl)
    err = np.abs(lg.cpu().numpy() - lg_ref)
    err[..., cfg.mask_id] = 0
    assert err.max() <= TOL, err.max()
    conf_ref, arg_ref = ov.confidence_argmax(lg_ref, cfg.mask_id)
    np.testing.assert_allclose(conf.cpu().numpy(), conf_ref, rtol=0, atol=TOL)
    gap = ov.top2_gap(lg_ref, cfg.mask_id)
    diff = arg.cpu().numpy() != arg_ref
    assert np.all(gap[diff] < 2 * TOL)
    # the cached forward saw the stale cache: it differs from a full forward on x1
    full = of.forward(cfg, wnp, x1, rows=np.arange(row0, row0 + bl))
    assert np.abs(full - lg_ref).max() > 1e-4


@pytest.mark.parametrize("name,refresh", [("cai", 4), ("cai", 16), ("cai_gate_off", 16)])
def test_tiny_generate_kv_matches_oracle(tiny, name, refresh):
    cfg, model, wnp = tiny
    ctl = B.Controller.preset(name)
    prompts = synth.make_prompts(WL)
    P, G, bl = WL.prompt_len, WL.gen_len, ctl.block_len
    say(f"tiny generate_kv {name} refresh {refresh}")
    res = model.generate_kv(ctl, prompts.cuda(), G, refresh, trace=True)
    torch.cuda.synchronize()
    st = res.state
    ct, at = res.conf_trace.cpu().numpy(), res.argmax_trace.cpu().numpy()
    # (1) the controller replayed on the GPU's predictions
    assert_state_equal(st, res.forwards, replay(ct, at, prompts.numpy(), G, cfg.mask_id, ctl))
    # (2) every step against the oracle: the full forward at refresh steps, the
    # cached forward against the oracle's cache of the last refresh otherwise
    fx, cs = st.x.cpu().numpy(), st.commit_step.cpu().numpy()
    near = 0
    for blk, n in enumerate(res.forwards):
        rows = np.arange(P + blk * bl, P + (blk + 1) * bl)
        cache = None
        for t in range(n):
            x = x_at_step(fx, cs, P, bl, blk, t, cfg.mask_id)
            if okv.is_refresh(t, refresh):
                lg_ref, cache = okv.forward_refresh(cfg, wnp, x, rows)
            else:
                lg_ref = okv.forward_cached(cfg, wnp, x, cache, rows[0], bl)
            conf_ref, arg_ref = ov.confidence_argmax(lg_ref, cfg.mask_id)
            np.testing.assert_allclose(ct[blk, t], conf_ref, rtol=0, atol=TOL, err_msg=f"block {blk} step {t}")
            gap = ov.top2_gap(lg_ref, cfg.mask_id)
            diff = at[blk, t] != arg_ref
            assert np.all(gap[diff] < 2 * TOL), (blk, t)
            near += int(diff.sum())
    # (3) the free-running oracle decode, the cache refreshed on the oracle's own
    # schedule (at a logit near-tie the oracle takes the GPU's token)
    state = {"cache": None}

    def logits_at(x, blk, t):
        rows = np.arange(P + blk * bl, P + (blk + 1) * bl)
        if okv.is_refresh(t, refresh):
            lg, state["cache"] = okv.forward_refresh(cfg, wnp, x, rows)
            return lg
        return okv.forward_cached(cfg, wnp, x, state["cache"], rows[0], bl)

    adopted = []
    free = oc.generate(tie_aware_predictor(logits_at, cfg.mask_id, at, TOL, adopted), prompts.numpy(), G,
                       cfg.mask_id, oracle_params(ctl))
    assert_state_equal(st, res.forwards, free, s_tol=TOL)
    assert len(adopted) <= near
    say(f"tiny kv {name}/{refresh}: forwards {res.forwards}, argmax near-ties {near}, adopted {len(adopted)}")


def test_tiny_generate_kv_refresh_every_step_equals_generate(tiny):
    cfg, model, _ = tiny
    ctl = B.Controller()
    prompts = synth.make_prompts(WL).cuda()
    say("tiny generate_kv refresh 1")
    a = model.generate(ctl, prompts, WL.gen_len, trace=True)
    b = model.generate_kv(ctl, prompts, WL.gen_len, 1, trace=True)
    torch.cuda.synchronize()
    assert torch.equal(a.state.x, b.state.x) and torch.equal(a.state.commit_step, b.state.commit_step)
    assert torch.equal(a.conf_trace.view(torch.int32), b.conf_trace.view(torch.int32))
    assert a.forwards == b.forwards


def test_tiny_step_kv_equals_generate_kv(tiny):
    """dllm_step_kv driven from the host with the refresh schedule equals dllm_generate_kv."""
    cfg, model, _ = tiny
    ctl = B.Controller()
    prompts = synth.make_prompts(WL).cuda()
    P, G, bl = WL.prompt_len, WL.gen_len, ctl.block_len
    say("tiny step_kv")
    ref = model.generate_kv(ctl, prompts, G, 8)
    st = B.DecodeState(1, P, G)
    model.state_init(prompts, G, st)
    ws, kv = model.workspace(1, P + G, bl), model.kv_cache(1, P + G)
    for blk in range(G // bl):
        for t in range(ctl.T):
            done, _, _ = model.step_kv(ctl, st, blk, t, t % 8 == 0, kv, ws)
            if done:
                break
    for k in ("x", "commit_step", "reason", "budget"):
        assert torch.equal(getattr(st, k), getattr(ref.state, k)), k


# ----------------------------------------------------------------- bf16 small
SMALL = synth.ModelConfig("small-bf16", n_layers=2, d_model=512, n_heads=4, n_kv_heads=2, head_dim=128, d_ff=768,
                          vocab=4000, rope_base=10000.0, dtype="bf16", lm_head_std=5 / math.sqrt(512),
                          norm_gain_std=0.1)


@pytest.fixture(scope="module")
def small():
    w_cpu = synth.make_weights(SMALL, "cpu")
    return B.Model(SMALL, [w.to("cuda") for w in w_cpu]), [w.to(torch.float32).numpy() for w in w_cpu]


@pytest.fixture(scope="module")
def small_packed(small):
    model, wnp = small
    packed = B.Model(SMALL, model.weights).pack_weights()
    yield packed, wnp
    packed.close()


# one layer of the LLaDA-8B widths with GQA: the register-direct GEMM runs
# 4-group waves (gate/up), 2-group (down) and 1-group (q/k/v, o), with one
# (32 rows) or two (64 rows) row operands
WIDE = synth.ModelConfig("wide-bf16", n_layers=1, d_model=4096, n_heads=32, n_kv_heads=8, head_dim=128,
                         d_ff=12288, vocab=4000, rope_base=500000.0, dtype="bf16", lm_head_std=5 / math.sqrt(4096),
                         norm_gain_std=0.1)


@pytest.fixture(scope="module")
def wide_packed():
    w_cpu = synth.make_weights(WIDE, "cpu")
    model = B.Model(WIDE, [w.to("cuda") for w in w_cpu]).pack_weights()
    yield model, [w.to(torch.float32).numpy() for w in w_cpu]
    model.close()


@pytest.mark.parametrize("which,Bn,P,G,blk,bl", [("small", 2, 40, 64, 1, 32), ("small", 1, 36, 96, 0, 32),
                                                 ("small", 5, 40, 64, 1, 32), ("small", 5, 36, 96, 2, 32),
                                                 ("small_packed", 2, 40, 64, 1, 32),
                                                 ("small_packed", 1, 36, 96, 2, 32),
                                                 ("small_packed", 3, 40, 64, 0, 32),
                                                 ("small_packed", 3, 40, 64, 2, 16),
                                                 ("wide_packed", 1, 40, 64, 1, 32),
                                                 ("wide_packed", 2, 36, 96, 2, 32),
                                                 ("wide_packed", 1, 40, 64, 3, 16)])
def test_bf16_refresh_cache_and_cached_layer_stages(request, which, Bn, P, G, blk, bl):
    """Up to 128 block rows the q/k/v and SwiGLU GEMMs split K and run their
    epilogues on the summed partials; B = 5 (160 rows) runs the fused
    epilogues on the row window.  P = 36: block positions not a multiple of 8
    (the element-wise v^T path).  Packed weights: at most 64 rows (B <= 2) run
    the register-direct GEMM (32 rows: one row operand, 64: two), 96 rows
    (B = 3) the tiled path; 16-row blocks give partial row operands (16 rows,
    and 48 = B 3 x 16: the second operand half past the rows)."""
    model, wnp = request.getfixturevalue(which)
    cfg = model.cfg
    L = P + G
    row0 = P + blk * bl
    say(f"bf16 kv stages {which} B={Bn} L={L} row0={row0}")
    x0 = synth.make_ints((Bn, L), 6, 0, cfg.vocab - 1)
    x1 = torch.from_numpy(_changed_block(x0.numpy(), row0, bl, 7, cfg.vocab).astype(np.int32))
    kv = model.kv_cache(Bn, L)
    ws = model.workspace(Bn, L, bl)
    ws2 = model.workspace(Bn, L, bl)
    # refresh layer by layer; the plain forward's keys/values for comparison
    model.embed(x0.cuda(), ws)
    model.embed(x0.cuda(), ws2)
    lay0 = model.layout(Bn, L, 0)
    for l in range(cfg.n_layers):
        model.layer_kv(l, 2, Bn, L, 0, L, kv, ws)
        model.layer(l, 2, Bn, L, ws2)
        torch.cuda.synchronize()
        K, V = kv_views(model, kv, Bn, L, l)
        k2 = ws_view(ws2, lay0.k, torch.bfloat16, K.shape)
        v2 = ws_view(ws2, lay0.vt, torch.float16, V.shape)
        assert torch.equal(K.view(torch.int16), k2.view(torch.int16)), f"layer {l} keys"
        assert torch.equal(V.view(torch.int16), v2.view(torch.int16)), f"layer {l} values"
    # a cached step on changed block tokens, stage by stage
    model.embed_rows(x1.cuda(), row0, bl, ws)
    for l in range(cfg.n_layers):
        st = check_layer_cached(model, cfg, wnp, ws, kv, Bn, L, row0, bl, l)
        say(f"  layer {l}: " + ", ".join(f"{k}={v:.2e}" for k, v in st.items()))


@pytest.mark.parametrize("Bn", [1, 2, 3, 5])
def test_bf16_packed_weights(small, small_packed, Bn):
    """Above 64 block rows the packed copies change where the block-row GEMMs
    read their weights, not what they compute (same tiles, same k order): the
    logits of a cached forward are bit-identical (B = 3: 96 rows; B = 5: 160
    rows).  At most 64 rows (B <= 2) the
    register-direct GEMM sums k in another order: logits agree to bf16
    rounding of the hidden states (its own parity is the stage test)."""
    model, _ = small
    packed, _ = small_packed
    P, G, bl = 40, 64, 32
    L, row0 = P + G, P + bl
    say(f"bf16 packed weights B={Bn}")
    x0 = synth.make_ints((Bn, L), 12, 0, SMALL.vocab - 1).cuda()
    x1 = torch.from_numpy(_changed_block(x0.cpu().numpy(), row0, bl, 13, SMALL.vocab).astype(np.int32)).cuda()
    out = []
    for mdl in (model, packed):
        kv, ws = mdl.kv_cache(Bn, L), mdl.workspace(Bn, L, bl)
        mdl.forward_kv(x0, row0, bl, kv, refresh=True, ws=ws)
        out.append(mdl.forward_kv(x1, row0, bl, kv, refresh=False, ws=ws, logits=True))
    torch.cuda.synchronize()
    (c0, a0, l0), (c1, a1, l1) = out
    if Bn > 2:
        assert torch.equal(l0.view(torch.int32), l1.view(torch.int32))
        assert torch.equal(c0.view(torch.int32), c1.view(torch.int32)) and torch.equal(a0, a1)
    else:
        err = (l1 - l0).abs()
        say(f"  logits max |diff| {err.max().item():.3e} mean {err.mean().item():.3e} "
            f"(max |logit| {l0.abs().max().item():.2f})")
        assert err.max().item() < 2e-2 * l0.abs().max().item() and err.mean().item() < 1e-2


@pytest.mark.parametrize("which,Bn", [("small", 2), ("small_packed", 2), ("small_packed", 3)])
def test_bf16_generate_kv_replay(request, which, Bn):
    """Cached decodes (refresh every 4 steps) replayed through the oracle
    controller; packed weights: 64 block rows on the register-direct GEMM with
    its partials folded into the next norm, 96 on the tiled path."""
    model, _ = request.getfixturevalue(which)
    ctl = B.Controller()
    P, G = 24, 96
    prompts = synth.make_ints((Bn, P), 21, 0, SMALL.vocab - 1)
    say(f"bf16 generate_kv {which} B={Bn}")
    res = model.generate_kv(ctl, prompts.cuda(), G, 4, trace=True)
    torch.cuda.synchronize()
    ref = replay(res.conf_trace.cpu().numpy(), res.argmax_trace.cpu().numpy(), prompts.numpy(), G, SMALL.mask_id,
                 ctl)
    assert_state_equal(res.state, res.forwards, ref)
    assert (res.state.x[:, P:] != SMALL.mask_id).all()


# ----------------------------------------------------------------- full size
REFRESH = {"llada_b1": 16, "dream_b1": 8}


@pytest.mark.parametrize("name", ["llada_b1", "dream_b1"])
def test_full_size_cached_layer_and_decode(name):
    wl = synth.WORKLOADS[name]
    cfg = wl.model
    Bn, P, G, bl = wl.batch, wl.prompt_len, wl.gen_len, wl.block_len
    L = P + G
    say(f"full-size kv {name}")
    weights = synth.make_weights(cfg, "cuda")
    model = B.Model(cfg, weights).pack_weights()
    # one cached layer (layer 1: its cache was filled from a refresh of layer-0
    # output) on the second block with changed tokens
    lw = [w.to(torch.float32).cpu().numpy() for w in weights[:1 + 9 * 2]] + [None, None]
    x0 = synth.make_prompts(wl).cuda()
    x0 = torch.cat([x0, synth.make_ints((Bn, G), 8, 0, cfg.vocab - 1).cuda()], dim=1)
    row0 = P + bl
    x1 = torch.from_numpy(_changed_block(x0.cpu().numpy(), row0, bl, 9, cfg.vocab).astype(np.int32)).cuda()
    kv = model.kv_cache(Bn, L)
    ws = model.workspace(Bn, L, bl)
    model.embed(x0, ws)
    model.layer_kv(0, 2, Bn, L, 0, L, kv, ws)
    model.layer_kv(1, 2, Bn, L, 0, L, kv, ws)
    model.embed_rows(x1, row0, bl, ws)
    model.layer_kv(0, 2, Bn, L, row0, bl, kv, ws)
    st = check_layer_cached(model, cfg, lw, ws, kv, Bn, L, row0, bl, 1)
    say("  layer 1: " + ", ".join(f"{k}={v:.2e}" for k, v in st.items()))
    # decode with the paper's update frequency; decisions replayed on the oracle
    ctl = B.Controller.gating(wl.gating, block_len=bl)
    prompts = synth.make_prompts(wl).cuda()
    res = model.generate_kv(ctl, prompts, G, REFRESH[name], ws=ws, kv=kv, trace=True)
    torch.cuda.synchronize()
    ref = replay(res.conf_trace.cpu().numpy(), res.argmax_trace.cpu().numpy(), prompts.cpu().numpy(), G,
                 cfg.mask_id, ctl)
    assert_state_equal(res.state, res.forwards, ref)
    say(f"  decode forwards {res.total_forwards} {res.forwards}")
