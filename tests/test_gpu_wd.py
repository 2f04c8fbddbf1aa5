"""The register-direct-weight GEMM (gemm_wd_kernel): q/k/v + RoPE and
gate/up + SwiGLU launches of 129..1024 rows on a model with packed weight
copies, when its tiles fill the compute units.

One layer at the LLaDA-8B widths (d 4096, 32 heads MHA, FFN 12288): q/k/v is
N = 12288 (128 x 192 tiles in two k-groups: 64 column tiles), gate/up N =
24576 (128 x 384 tiles: 64 column tiles); with 4 row tiles either launch is
256 workgroups, so rows 385..512 take it:
  * M = 400, one sequence: the last row tile holds 16 rows (rows past M are
    loaded clamped and never stored);
  * M = 400, two sequences of 200: row tiles straddle the sequence boundary
    (the epilogue's row -> (sequence, position) mapping for q/k/v^T);
  * M = 394, two sequences of 197: as above with L not a multiple of 8, so
    the staged v^T leaves by single positions instead of 16-byte chunks;
  * M = 512: the batch-1 decode shape.
One layer at the Dream-7B widths (d 3584, 28 / 4 heads, FFN 18944): gate/up
is N = 37888 = 148 x 256, which no 192- or 384-wide tile divides, so at 640
rows it runs the 256 x 256 tile (3 x 148 = 444 workgroups, the last row tile
holding 128 rows), and q/k/v (N = 4608) the 128 x 128 two-k-group tile.
Every stage is checked against the oracle on the GPU's own stage inputs (the
bars of gpu_stages), and the fused forward against per-layer calls (bitwise).
"""
import math

import numpy as np
import pytest
import torch

from gpu_stages import check_head, check_layer
from helpers import say
from paper_2608_22646_amd import binding as B
from paper_2608_22646_amd import synth
from test_gpu_bf16 import forward_equals_layer_calls

pytestmark = pytest.mark.gpu

WIDE_MHA = synth.ModelConfig("wide-mha-bf16", n_layers=1, d_model=4096, n_heads=32, n_kv_heads=32, head_dim=128,
                             d_ff=12288, vocab=4000, rope_base=500000.0, dtype="bf16",
                             lm_head_std=5 / math.sqrt(4096), norm_gain_std=0.1)

DREAM_W = synth.ModelConfig("dream-width-bf16", n_layers=1, d_model=3584, n_heads=28, n_kv_heads=4, head_dim=128,
                            d_ff=18944, vocab=4000, rope_base=1000000.0, dtype="bf16", norm_gain_std=0.1)


@pytest.fixture(scope="module")
def wide_mha():
    w_cpu = synth.make_weights(WIDE_MHA, "cpu")
    model = B.Model(WIDE_MHA, [w.to("cuda") for w in w_cpu]).pack_weights()
    yield model, [w.to(torch.float32).numpy() for w in w_cpu]
    model.close()


@pytest.mark.parametrize("Bn,P,G", [(1, 336, 64), (2, 136, 64), (2, 133, 64), (1, 448, 64)])
def test_wd_stages(wide_mha, Bn, P, G):
    model, wnp = wide_mha
    L = P + G
    say(f"register-direct GEMM stages B={Bn} L={L} (M={Bn * L})")
    x = synth.make_ints((Bn, L), 31, 0, WIDE_MHA.vocab - 1).cuda()
    ws = model.workspace(Bn, L, 32)
    model.embed(x, ws)
    rng = np.random.default_rng(3)
    # sampled rows: every 128-row tile, both sequences, the last rows
    rows = np.unique(np.concatenate([rng.choice(Bn * L, 60, replace=False), [0, 127, 128, 199, 200, Bn * L - 1]]))
    st = check_layer(model, WIDE_MHA, wnp, ws, Bn, L, 0, rows=rows)
    say("  " + ", ".join(f"{k}={v:.2e}" for k, v in st.items()))
    hs = check_head(model, WIDE_MHA, wnp, ws, Bn, L, P, 32)
    say(f"  head: {hs}")


@pytest.mark.parametrize("Bn,P,G", [(2, 136, 64), (1, 448, 64)])
def test_wd_forward_matches_layer_by_layer(wide_mha, Bn, P, G):
    model, _ = wide_mha
    say(f"register-direct GEMM: fused forward vs layer calls B={Bn} L={P + G}")
    forward_equals_layer_calls(model, WIDE_MHA, Bn, P, G, seed=33)


def test_wd_dream_widths():
    Bn, P, G = 1, 576, 64
    L = P + G
    say(f"register-direct GEMM stages at the Dream-7B widths B={Bn} L={L}")
    w_cpu = synth.make_weights(DREAM_W, "cpu")
    model = B.Model(DREAM_W, [w.to("cuda") for w in w_cpu]).pack_weights()
    wnp = [w.to(torch.float32).numpy() for w in w_cpu]
    x = synth.make_ints((Bn, L), 37, 0, DREAM_W.vocab - 1).cuda()
    ws = model.workspace(Bn, L, 32)
    model.embed(x, ws)
    rng = np.random.default_rng(5)
    # sampled rows: both 256-row tiles, the ragged last one, the last row
    rows = np.unique(np.concatenate([rng.choice(L, 60, replace=False), [0, 255, 256, 511, 512, L - 1]]))
    st = check_layer(model, DREAM_W, wnp, ws, Bn, L, 0, rows=rows)
    say("  " + ", ".join(f"{k}={v:.2e}" for k, v in st.items()))
    forward_equals_layer_calls(model, DREAM_W, Bn, P, G, seed=35)
    model.close()
