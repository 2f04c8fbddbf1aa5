"""Embedding gather (the state x^(t) of Section 4.1 entering the forward) and the
step's error word.

  * dllm_embed and dllm_embed_rows put E[x] in the workspace's residual rows,
    bit for bit (bf16 -> float32 is exact), for bf16 and float32 models, B > 1,
    and windows starting past position 0;
  * a token id outside [0, vocab) is never used as an address: its row is zero
    and the next commit reports it (dllm_step / dllm_generate return
    DLLM_EINVAL), after which the word is clear again;
  * a v value beyond IEEE half's range is stored as +-65504 for the attention's
    half-precision P.V operand and reported (DLLM_EUNSUPPORTED).
"""
import math

import numpy as np
import pytest
import torch

from helpers import assert_bf16_flips, say, to_np
from oracle import forward as of
from paper_2608_22646_amd import binding as B
from paper_2608_22646_amd import synth

pytestmark = pytest.mark.gpu

SMALL = synth.ModelConfig("embed-bf16", n_layers=1, d_model=512, n_heads=4, n_kv_heads=2, head_dim=128, d_ff=768,
                          vocab=3001, rope_base=1e4, dtype="bf16", lm_head_std=5 / math.sqrt(512))


@pytest.fixture(scope="module")
def models():
    out = {}
    for cfg in (SMALL, synth.TINY):
        w = synth.make_weights(cfg, "cuda")
        out[cfg.dtype] = (cfg, w, B.Model(cfg, w))
    return out


def _h(model, ws, Bn, L, rows):
    lay = model.layout(Bn, L, rows)
    d = model.cfg.d_model
    n = Bn * (rows if rows else L)
    return ws[lay.h:lay.h + n * d * 4].view(torch.float32).view(n, d)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_embed_is_the_table_row(models, dtype):
    cfg, w, model = models[dtype]
    Bn, L = 3, 70
    x = synth.make_ints((Bn, L), 5, 0, cfg.vocab)
    x[0, 0], x[1, -1], x[2, 5] = 0, cfg.vocab - 1, cfg.mask_id      # both ends of the table
    say(f"embed {dtype} B={Bn} L={L}")
    ws = model.workspace(Bn, L, 0)
    model.embed(x.cuda(), ws)
    torch.cuda.synchronize()
    want = w[0].float()[x.view(-1).long().cuda()]
    got = _h(model, ws, Bn, L, 0)
    assert torch.equal(got.view(torch.int32), want.view(torch.int32))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("row0,rows", [(0, 32), (17, 32), (38, 32), (64, 6)])
def test_embed_rows_is_the_table_row(models, dtype, row0, rows):
    cfg, w, model = models[dtype]
    Bn, L = 2, 70
    x = synth.make_ints((Bn, L), 6 + row0, 0, cfg.vocab)
    say(f"embed_rows {dtype} row0={row0} rows={rows}")
    ws = model.workspace(Bn, L, rows)
    model.embed_rows(x.cuda(), row0, rows, ws)
    torch.cuda.synchronize()
    want = w[0].float()[x[:, row0:row0 + rows].reshape(-1).long().cuda()]
    got = _h(model, ws, Bn, L, rows)[:Bn * rows]
    assert torch.equal(got.view(torch.int32), want.view(torch.int32))


def test_out_of_range_token_is_zeroed_and_reported(models):
    cfg, w, model = models["bf16"]
    Bn, L = 2, 40
    x = synth.make_ints((Bn, L), 7, 0, cfg.vocab)
    x[0, 3], x[1, 9] = cfg.vocab, -5
    say("embed out-of-range ids")
    ws = model.workspace(Bn, L, 0)
    model.embed(x.cuda(), ws)
    torch.cuda.synchronize()
    got = _h(model, ws, Bn, L, 0).view(Bn, L, -1)
    assert torch.count_nonzero(got[0, 3]) == 0 and torch.count_nonzero(got[1, 9]) == 0
    ok = torch.ones((Bn, L), dtype=torch.bool)
    ok[0, 3] = ok[1, 9] = False
    want = w[0].float()[x.clamp(0, cfg.vocab - 1).long().cuda()]
    assert torch.equal(got[ok.cuda()], want[ok.cuda()])

    # through a step: the commit reports the error word, then it is clear again
    ctl = B.Controller()
    P, G = 8, 32
    prompt = synth.make_ints((Bn, P), 8, 0, cfg.vocab - 1)
    prompt[1, 2] = cfg.vocab + 100
    st = B.DecodeState(Bn, P, G)
    model.state_init(prompt.cuda(), G, st)
    wss = model.workspace(Bn, P + G, ctl.block_len)
    with pytest.raises(B.DllmError) as e:
        model.step(ctl, st, 0, 0, wss)
    assert e.value.code == -1 and "token id" in str(e.value)
    st.x[1, 2] = 5
    model.step(ctl, st, 0, 1, wss)          # a valid x: no error left over
    with pytest.raises(B.DllmError) as e:
        model.generate(ctl, prompt.cuda(), G)
    assert e.value.code == -1
    model.generate(ctl, prompt.clamp(0, cfg.vocab - 2).cuda(), G)


def test_v_beyond_half_range_is_saturated_and_reported():
    cfg = synth.reduced(SMALL, name="embed-bf16-bigv")
    w = synth.make_weights(cfg, "cuda")
    w[4] = (w[4].float() * 2e5).to(torch.bfloat16)          # wv: |v| ~ 1e5, past half's 65504
    model = B.Model(cfg, w)
    Bn, L = 1, 64
    x = synth.make_ints((Bn, L), 9, 0, cfg.vocab - 1)
    say("v beyond half range")
    ws = model.workspace(Bn, L, 0)
    model.embed(x.cuda(), ws)
    model.layer(0, 0, Bn, L, ws)
    torch.cuda.synchronize()
    lay = model.layout(Bn, L, 0)
    d, Hkv, hd = cfg.d_model, cfg.n_kv_heads, cfg.head_dim
    a = to_np(ws[lay.a_attn:lay.a_attn + L * d * 2].view(torch.bfloat16).view(L, d), np.float64)
    vt = to_np(ws[lay.vt:lay.vt + Hkv * hd * L * 2].view(torch.float16).view(Hkv, hd, L), np.float64)
    wnp = [to_np(t, np.float64) for t in w]
    cos, sin = of.rope_tables(L, hd, cfg.rope_base)
    _, _, v_ref = of.qkv_rope(cfg, a, wnp[2], wnp[3], wnp[4], cos, sin, "bf16")   # bf16-rounded v [Hkv, L, hd]
    g = vt.transpose(0, 2, 1)
    big = np.abs(v_ref) >= 65536
    assert big.any() and (~big).any()
    assert np.all(np.abs(g[big]) == 65504) and np.all(np.sign(g[big]) == np.sign(v_ref[big]))
    sat = np.abs(g) == 65504
    assert np.all(np.abs(v_ref[sat]) >= 65280)                 # saturated only at the range's edge
    assert_bf16_flips(g[~big & ~sat], v_ref[~big & ~sat], "v within range")
    # a step on this model reports it
    ctl = B.Controller()
    P, G = 32, 32
    st = B.DecodeState(1, P, G)
    model.state_init(synth.make_ints((1, P), 10, 0, cfg.vocab - 1).cuda(), G, st)
    with pytest.raises(B.DllmError) as e:
        model.step(ctl, st, 0, 0, model.workspace(1, P + G, ctl.block_len))
    assert e.value.code == -5 and "half" in str(e.value)
