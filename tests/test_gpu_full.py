"""Full-size workloads (LLaDA-8B and Dream-7B shapes) at the launch configuration
the decode uses.

For each workload:
  * the first denoising step's forward runs layer by layer; at the first and
    last layer every stage is checked against the oracle applied to the GPU's
    own stage inputs on sampled rows (all key positions feed the attention
    check), and the fused LM head is checked on sampled block rows;
  * a complete decode (dllm_generate) is replayed through the oracle
    controller on the GPU's recorded predictions: token ids, commit steps,
    reasons, budgets, first-step confidences and forwards per block must be
    bit-identical, and the decode invariants must hold.
Weights are seeded random draws made on the GPU (one 8B-parameter model at a
time); only the layers the oracle needs are copied to the host.
"""
import numpy as np
import pytest
import torch

from gpu_stages import check_head, check_layer
from helpers import assert_state_equal, replay, say, to_np
from paper_2608_22646_amd import binding as B
from paper_2608_22646_amd import synth

pytestmark = pytest.mark.gpu

WORKLOADS = ["llada_b1", "llada_b8", "dream_b1", "dream_long"]


@pytest.fixture(scope="module")
def models():
    cache = {}

    def get(cfg):
        if cfg.name not in cache:
            cache.clear()
            torch.cuda.empty_cache()
            say(f"generating weights for {cfg.name}")
            w = synth.make_weights(cfg, "cuda")
            cache[cfg.name] = (w, B.Model(cfg, w))
        return cache[cfg.name]

    yield get
    cache.clear()


def host_weights(cfg, w, layers):
    out = [None] * len(w)
    for l in layers:
        for i in range(1 + 9 * l, 10 + 9 * l):
            out[i] = to_np(w[i])
    out[-2] = to_np(w[-2])
    out[-1] = to_np(w[-1])
    return out


def check_invariants(st, forwards, P, G, bl, T, mask_id, ctl):
    cs = st.commit_step.cpu().numpy()
    rs = st.reason.cpu().numpy()
    assert (cs >= 0).all() and (cs <= T - 1).all(), "a token was left masked or committed past T"
    assert (rs >= 1).all()
    assert (st.x[:, P:] != mask_id).all().item(), "mask id left in the output"
    if ctl.budgets and not ctl.fixed:
        assert (cs <= st.budget.cpu().numpy()).all(), "a token exceeded its step budget"
    for b in range(cs.shape[0]):
        for blk in range(G // bl):
            assert cs[b, blk * bl:(blk + 1) * bl].max() + 1 <= forwards[blk]


@pytest.mark.parametrize("name,packed", [(n, False) for n in WORKLOADS] + [("llada_b1", True), ("dream_b1", True)])
def test_full_size_stages_and_head(models, name, packed):
    """packed: a second handle on the same weights with the packed copies, so
    the batch-1 q/k/v and gate/up GEMMs (LLaDA-8B shape) and the q/k/v GEMM
    (Dream-7B shape, 128 x 128 tiles) stream their weights register-direct."""
    wl = synth.WORKLOADS[name]
    cfg = wl.model
    w, model = models(cfg)
    if packed:
        model = B.Model(cfg, w).pack_weights()
    Bn, P, G, bl = wl.batch, wl.prompt_len, wl.gen_len, wl.block_len
    L = P + G
    sample_layers = [0, cfg.n_layers - 1]
    wnp = host_weights(cfg, w, sample_layers)
    prompts = synth.make_prompts(wl)
    x = torch.cat([prompts, torch.full((Bn, G), cfg.mask_id, dtype=torch.int32)], 1).cuda()
    ws = model.workspace(Bn, L, bl)
    model.embed(x, ws)
    rng = np.random.default_rng(17)
    rows = np.sort(rng.choice(Bn * L, 64, replace=False))
    keys = np.sort(rng.choice(L, 64, replace=False))
    for l in range(cfg.n_layers):
        if l in sample_layers:
            say(f"{name}{' (packed)' if packed else ''}: stages of layer {l}")
            st = check_layer(model, cfg, wnp, ws, Bn, L, l, rows=rows, key_rows=keys)
            say("  " + ", ".join(f"{k}={v:.2e}" for k, v in st.items()))
        else:
            model.layer(l, 2, Bn, L, ws)
    say(f"{name}: head")
    head_rows = np.sort(rng.choice(Bn * bl, min(16, Bn * bl), replace=False))
    hs = check_head(model, cfg, wnp, ws, Bn, L, P, bl, sample=head_rows)
    say(f"  head {hs}")
    if packed:
        model.close()
        torch.cuda.empty_cache()


@pytest.mark.parametrize("G", [64, 512])
def test_full_size_decode_replay_gen_lengths(models, G):
    # the generation-length sweep's extremes (LLaDA-8B shape, batch 1, prompt 256)
    import dataclasses
    wl = dataclasses.replace(synth.WORKLOADS["llada_b1"], name=f"llada_b1_g{G}", gen_len=G)
    _, model = models(wl.model)
    ctl = B.Controller.gating(wl.gating, block_len=wl.block_len)
    prompts = synth.make_prompts(wl)
    say(f"llada_b1 G={G}: decode")
    res = model.generate(ctl, prompts.cuda(), G, trace=True)
    torch.cuda.synchronize()
    ref = replay(res.conf_trace.cpu().numpy(), res.argmax_trace.cpu().numpy(), prompts.numpy(), G,
                 wl.model.mask_id, ctl)
    assert_state_equal(res.state, res.forwards, ref)
    check_invariants(res.state, res.forwards, wl.prompt_len, G, wl.block_len, ctl.T, wl.model.mask_id, ctl)
    say(f"  forwards per block {res.forwards}")


@pytest.mark.parametrize("name", ["llada_b1", "dream_b1"])
def test_full_size_forward_matches_layer_by_layer(models, name):
    from test_gpu_bf16 import forward_equals_layer_calls
    wl = synth.WORKLOADS[name]
    _, model = models(wl.model)
    say(f"{name}: fused forward vs layer calls")
    forward_equals_layer_calls(model, wl.model, wl.batch, wl.prompt_len, wl.gen_len, seed=23)


@pytest.mark.parametrize("name,preset", [(n, None) for n in WORKLOADS] + [("dream_b1", "cai"),
                                                                          ("llada_b1", "fixed_schedule")])
def test_full_size_decode_replay(models, name, preset):
    wl = synth.WORKLOADS[name]
    cfg = wl.model
    _, model = models(cfg)
    preset = preset or ("cai" if wl.gating else "cai_gate_off")
    ctl = B.Controller.preset(preset, block_len=wl.block_len)
    prompts = synth.make_prompts(wl)
    say(f"{name}: decode, controller {preset}")
    res = model.generate(ctl, prompts.cuda(), wl.gen_len, trace=True)
    torch.cuda.synchronize()
    ref = replay(res.conf_trace.cpu().numpy(), res.argmax_trace.cpu().numpy(), prompts.numpy(), wl.gen_len,
                 cfg.mask_id, ctl)
    assert_state_equal(res.state, res.forwards, ref)
    check_invariants(res.state, res.forwards, wl.prompt_len, wl.gen_len, wl.block_len, ctl.T, cfg.mask_id, ctl)
    say(f"  forwards per block {res.forwards} (total {res.total_forwards})")
    if ctl.fixed:
        assert res.forwards == [ctl.T] * (wl.gen_len // wl.block_len)
