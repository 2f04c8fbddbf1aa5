"""bf16 path on a small model: every forward stage, the fused LM-head
reduction (exact-logit fixture and random data) and the decode loop."""
import math

import numpy as np
import pytest
import torch

from gpu_stages import check_head, check_layer, ws_view
from helpers import assert_state_equal, replay, say
from oracle import controller as oc
from oracle import vocab as ov
from paper_2608_22646_amd import binding as B
from paper_2608_22646_amd import synth

pytestmark = pytest.mark.gpu

SMALL = synth.ModelConfig("small-bf16", n_layers=2, d_model=512, n_heads=4, n_kv_heads=2, head_dim=128, d_ff=768,
                          vocab=4000, rope_base=10000.0, dtype="bf16", lm_head_std=5 / math.sqrt(512),
                          norm_gain_std=0.1)


# Widths that are multiples of 192 as well as 256, so the GEMMs also run their
# 192-wide tiles: q/k/v = 768 virtual rows (a 192-column tile spans q and k, or
# k and v), gate/up = 2304, and Hq*hd = 256 != d_model.
SMALL192 = synth.ModelConfig("small192-bf16", n_layers=2, d_model=768, n_heads=2, n_kv_heads=2, head_dim=128,
                             d_ff=1152, vocab=3000, rope_base=10000.0, dtype="bf16",
                             lm_head_std=5 / math.sqrt(768), norm_gain_std=0.1)


def _load(cfg):
    w_cpu = synth.make_weights(cfg, "cpu")
    model = B.Model(cfg, [w.to("cuda") for w in w_cpu])
    wnp = [w.to(torch.float32).numpy() for w in w_cpu]
    return model, wnp


@pytest.fixture(scope="module")
def small():
    return _load(SMALL)


@pytest.fixture(scope="module")
def small192():
    return _load(SMALL192)


@pytest.mark.parametrize("Bn,P,G", [(2, 40, 64), (1, 9, 32), (2, 1036, 64), (2, 2936, 64), (2, 16136, 64)])
def test_forward_stages(small, Bn, P, G):
    """Ragged sizes: M = 208 (128-row tiles, ragged), 41 (single partial tile) and
    2200 (256-row tiles, ragged); L not a multiple of the 32- or 64-key attention
    tiles.  L = 3000 runs the key-split attention with 96 queries per workgroup
    (the others with 64) and a partial last query block; L = 16200 the
    8-wave streaming attention (a partial last 64-key tile and a partial
    last 256-query block)."""
    model, wnp = small
    L = P + G
    say(f"bf16 stages B={Bn} L={L}")
    x = synth.make_ints((Bn, L), 5, 0, SMALL.vocab - 1).cuda()
    ws = model.workspace(Bn, L, 32)
    model.embed(x, ws)
    rows = None if Bn * L <= 300 else np.sort(np.random.default_rng(0).choice(Bn * L, 96, replace=False))
    for l in range(SMALL.n_layers):
        st = check_layer(model, SMALL, wnp, ws, Bn, L, l, rows=rows)
        say(f"  layer {l}: " + ", ".join(f"{k}={v:.2e}" for k, v in st.items()))
    hs = check_head(model, SMALL, wnp, ws, Bn, L, P, min(32, G))
    say(f"  head: {hs}")


@pytest.mark.parametrize("Bn,P,G", [(2, 40, 64), (2, 1936, 64)])
def test_forward_stages_192_wide_tiles(small192, Bn, P, G):
    """M = 208 (128 x 192 tiles) and 4000 (256 x 192 tiles for gate/up, ragged in
    M); every q/k/v, SwiGLU and residual epilogue on 192-column tiles."""
    model, wnp = small192
    L = P + G
    say(f"bf16 stages (192-wide tiles) B={Bn} L={L}")
    x = synth.make_ints((Bn, L), 6, 0, SMALL192.vocab - 1).cuda()
    ws = model.workspace(Bn, L, 32)
    model.embed(x, ws)
    rows = None if Bn * L <= 300 else np.sort(np.random.default_rng(1).choice(Bn * L, 96, replace=False))
    for l in range(SMALL192.n_layers):
        st = check_layer(model, SMALL192, wnp, ws, Bn, L, l, rows=rows)
        say(f"  layer {l}: " + ", ".join(f"{k}={v:.2e}" for k, v in st.items()))
    hs = check_head(model, SMALL192, wnp, ws, Bn, L, P, min(32, G))
    say(f"  head: {hs}")


def forward_equals_layer_calls(model, cfg, Bn, P, G, seed):
    """dllm_forward (which folds each residual GEMM's split-K partials into the
    next RMSNorm) against embed + one dllm_layer call per layer + dllm_head
    (every split-K reduction by its own kernel): the same float operations in
    the same order, so conf, argmax and logits must be bitwise identical."""
    L, rows = P + G, min(32, G)
    x = synth.make_ints((Bn, L), seed, 0, cfg.vocab - 1).cuda()
    conf_f, arg_f, lg_f = model.forward(x, P, rows, logits=True)
    ws = model.workspace(Bn, L, rows)
    model.embed(x, ws)
    for l in range(cfg.n_layers):
        model.layer(l, 2, Bn, L, ws)
    conf_l, arg_l, lg_l = model.head(Bn, L, P, rows, ws, logits=True)
    torch.cuda.synchronize()
    assert torch.equal(arg_f, arg_l)
    assert torch.equal(conf_f.view(torch.int32), conf_l.view(torch.int32))
    assert torch.equal(lg_f.view(torch.int32), lg_l.view(torch.int32))


@pytest.mark.parametrize("Bn,P,G", [(2, 40, 64), (1, 9, 32), (2, 1036, 64)])
def test_forward_matches_layer_by_layer(small, Bn, P, G):
    model, _ = small
    say(f"bf16 fused forward vs layer calls B={Bn} L={P + G}")
    forward_equals_layer_calls(model, SMALL, Bn, P, G, seed=9)


@pytest.mark.parametrize("Bn,P,G", [(2, 40, 64), (2, 1936, 64)])
def test_forward_matches_layer_by_layer_192(small192, Bn, P, G):
    model, _ = small192
    say(f"bf16 fused forward vs layer calls (192-wide tiles) B={Bn} L={P + G}")
    forward_equals_layer_calls(model, SMALL192, Bn, P, G, seed=10)


def _head_model(V, d, mask_id_at_top=True):
    cfg = synth.ModelConfig("head-fixture", n_layers=0, d_model=d, n_heads=2, n_kv_heads=2, head_dim=128, d_ff=128,
                            vocab=V, rope_base=1e4, dtype="bf16", rms_eps=1e-30)
    return cfg


# up to 32 head rows use the streaming kernel (R = 32, 20: ragged vocabulary
# tiles; V = 150000: 640-row tiles, five groups per wave, the last one ragged);
# 33..64 use the LDS-ring kernel (R = 64, 60); 65..256 the register-direct
# kernel (R = 96: four 32-row groups, the last past R; R = 150 with V = 150000:
# eight groups, ragged rows and a last vocabulary tile past V; R = 256)
@pytest.mark.parametrize("Bn,rows,V", [(1, 32, 4096), (1, 32, 4000), (1, 20, 2176), (2, 32, 4000), (8, 32, 4096),
                                       (3, 20, 2176), (1, 32, 150000), (3, 32, 4000), (5, 30, 150000)])
def test_head_exact_logit_fixture(Bn, rows, V):
    """Hidden rows of +-1 (RMSNorm is then the identity) and integer weights make
    every logit an exact small integer in float32, so the argmax (with ties going
    to the lowest id, the mask id excluded) must match exactly and the confidence
    to float32 rounding of the sum."""
    d = 512
    cfg = _head_model(V, d)
    L = rows
    say(f"head fixture B={Bn} rows={rows} V={V}")
    h = (synth.make_ints((Bn * L, d), 11, 0, 2) * 2 - 1).to(torch.float32)            # +-1
    W = synth.make_ints((V, d), 12, -3, 4).to(torch.float32)
    # plant exact ties: vocab rows 2*j and 2*j + 1 equal for j < 40
    W[1:80:2] = W[0:80:2]
    # the mask id holds the largest logit of row 0
    W[V - 1] = 3 * h[0]
    weights = [torch.zeros((V, d)), torch.ones(d), W]
    model = B.Model(cfg, [w.to(torch.bfloat16).cuda() for w in weights])
    ws = model.workspace(Bn, L, rows)
    lay = model.layout(Bn, L, rows)
    ws_view(ws, lay.h, torch.float32, (Bn * L, d)).copy_(h.cuda())
    conf, arg, lg = model.head(Bn, L, 0, rows, ws, logits=True)
    torch.cuda.synchronize()
    exact = (h.double() @ W.double().T).numpy()
    np.testing.assert_array_equal(lg.view(Bn * rows, V).cpu().numpy().astype(np.float64), exact)
    c_ref, a_ref = ov.confidence_argmax(exact, V - 1)
    np.testing.assert_array_equal(arg.view(-1).cpu().numpy(), a_ref)
    np.testing.assert_allclose(conf.view(-1).cpu().numpy(), c_ref, rtol=2e-6)
    assert a_ref[0] != V - 1
    # determinism: a second launch (ticket reset by the last workgroup) is identical
    conf2, arg2, _ = model.head(Bn, L, 0, rows, ws, logits=False)
    assert torch.equal(conf2.view(torch.int32), conf.view(torch.int32)) and torch.equal(arg2, arg)


def test_decode_small(small):
    model, wnp = small
    ctl = B.Controller()
    Bn, P, G = 2, 24, 96
    prompts = synth.make_ints((Bn, P), 21, 0, SMALL.vocab - 1)
    say("bf16 small decode")
    res = model.generate(ctl, prompts.cuda(), G, trace=True)
    torch.cuda.synchronize()
    ref = replay(res.conf_trace.cpu().numpy(), res.argmax_trace.cpu().numpy(), prompts.numpy(), G, SMALL.mask_id,
                 ctl)
    assert_state_equal(res.state, res.forwards, ref)
    assert (res.state.commit_step >= 0).all() and (res.state.x[:, P:] != SMALL.mask_id).all()
    res2 = model.generate(ctl, prompts.cuda(), G, trace=True)
    assert torch.equal(res2.state.x, res.state.x)
    assert torch.equal(res2.conf_trace.view(torch.int32), res.conf_trace.view(torch.int32))
    say(f"  forwards {res.forwards}")
