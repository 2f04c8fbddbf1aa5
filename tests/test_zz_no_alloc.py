"""dllm_head_noalloc (the LM head + vocabulary reduction with its scratch in the
library's static device array) against dllm_head (scratch in the workspace),
called through the C ABI: the same kernels on the same residual rows, so conf,
argmax and logits must agree bit for bit.  Two calls in a row, the second on
fewer head rows (256 rows through the LDS-ring head kernel, then 16 through the
streaming kernel), for a bf16 model; a float32 model; and a call whose scratch
would not fit, rejected on the host.
"""
import math

import numpy as np
import pytest
import torch

from helpers import say
from paper_2608_22646_amd import binding as B
from paper_2608_22646_amd import synth

pytestmark = pytest.mark.gpu

BF16 = synth.ModelConfig("noalloc-bf16", n_layers=1, d_model=1024, n_heads=8, n_kv_heads=2, head_dim=128, d_ff=512,
                         vocab=50000, rope_base=1e4, dtype="bf16", lm_head_std=5 / math.sqrt(1024))


def _compare(model, Bn, L, row0, rows, seed):
    cfg = model.cfg
    ws = model.workspace(Bn, L, rows)
    lay = model.layout(Bn, L, rows)
    h = ws[lay.h:lay.h + Bn * L * cfg.d_model * 4].view(torch.float32).view(Bn * L, cfg.d_model)
    h.copy_(synth.make_normal((Bn * L, cfg.d_model), seed, std=2.0).cuda())
    c_ref, a_ref, l_ref = model.head(Bn, L, row0, rows, ws, logits=True)
    c, a, lg = model.head_noalloc(h, Bn, L, row0, rows, logits=True)
    c2, a2, _ = model.head_noalloc(h, Bn, L, row0, rows)          # without the logits output
    torch.cuda.synchronize()
    assert torch.equal(a, a_ref) and torch.equal(a2, a_ref)
    assert torch.equal(c.view(torch.int32), c_ref.view(torch.int32))
    assert torch.equal(c2.view(torch.int32), c_ref.view(torch.int32))
    assert torch.equal(lg.view(torch.int32), l_ref.view(torch.int32))
    return float(c.max()), int(a.min())


def test_head_noalloc_matches_head_bf16():
    w = synth.make_weights(BF16, "cuda")
    model = B.Model(BF16, w)
    say("head_noalloc bf16: 256 head rows")
    _compare(model, 8, 64, 32, 32, seed=1)
    say("head_noalloc bf16: 16 head rows (second, smaller call)")
    _compare(model, 1, 64, 7, 16, seed=2)


def test_head_noalloc_matches_head_f32_and_rejects_oversize():
    cfg = synth.TINY
    model = B.Model(cfg, synth.make_weights(cfg, "cuda"))
    say("head_noalloc fp32: 64 then 32 head rows")
    _compare(model, 2, 96, 32, 32, seed=3)
    _compare(model, 1, 96, 64, 32, seed=4)
    # 16 x 96 rows need (256 + 2048) * 4 bytes each: past the 8 MiB scratch
    h = torch.zeros((16 * 96, cfg.d_model), dtype=torch.float32, device="cuda")
    with pytest.raises(B.DllmError) as e:
        model.head_noalloc(h, 16, 96, 0, 96)
    assert e.value.code == -4 and "static scratch" in str(e.value)
