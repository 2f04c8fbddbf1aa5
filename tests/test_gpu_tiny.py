"""Tiny fp32 LLaDA-style model end to end (dllm_generate) against the float64 oracle.

Workload: 2 layers, d 256, 4 heads x 64, FFN 704, vocab 2048 (mask 2047),
prompt 32, 64 generated tokens in 2 blocks of 32, batch 1, under the method
with gating on and off, the fixed-schedule baseline and three ablation presets.
  * every step's logits and confidences, teacher-forced on the token array the
    GPU saw, agree with the oracle within 1e-5; argmax agrees except at a
    logit near-tie (reported);
  * the oracle controller replayed on the GPU's own predictions reproduces the
    GPU's decisions bit for bit;
  * the free-running oracle decode equals the GPU decode (at a logit near-tie
    the oracle takes the GPU's token, equally correct to the tolerance).
"""
import numpy as np
import pytest
import torch

from helpers import assert_state_equal, oracle_params, replay, say, tie_aware_predictor, to_np, x_at_step
from oracle import controller as oc
from oracle import forward as of
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
    w_gpu = [w.to("cuda") for w in w_cpu]
    model = B.Model(cfg, w_gpu)
    wnp = [w.numpy().astype(np.float64) for w in w_cpu]
    return cfg, model, wnp


def _run(model, ctl, prompts, G):
    res = model.generate(ctl, prompts.to("cuda"), G, trace=True)
    torch.cuda.synchronize()
    return res


CONTROLLERS = ["cai", "cai_gate_off", "fixed_schedule", "apd", "apd_block", "fixed_threshold_0.9"]


@pytest.mark.parametrize("name", CONTROLLERS)
def test_tiny_generate_matches_oracle(tiny, name):
    cfg, model, wnp = tiny
    ctl = B.Controller.preset(name)
    prompts = synth.make_prompts(WL)
    P, G, bl = WL.prompt_len, WL.gen_len, ctl.block_len
    say(f"tiny generate {name}")
    res = _run(model, ctl, prompts, G)
    st = res.state
    ct, at = res.conf_trace.cpu().numpy(), res.argmax_trace.cpu().numpy()

    # (1) controller replay on the GPU's predictions: bit-exact
    ref = replay(ct, at, prompts.numpy(), G, cfg.mask_id, ctl)
    assert_state_equal(st, res.forwards, ref)

    # (2) teacher-forced logits / confidences at every step that ran
    fx = st.x.cpu().numpy()
    cs = st.commit_step.cpu().numpy()
    near = 0
    for blk, n in enumerate(res.forwards):
        rows = np.arange(P + blk * bl, P + (blk + 1) * bl)
        for t in range(n):
            x = x_at_step(fx, cs, P, bl, blk, t, cfg.mask_id)
            lg_ref = of.forward(cfg, wnp, x, rows=rows)                    # float64
            conf_ref, arg_ref = ov.confidence_argmax(lg_ref, cfg.mask_id)
            xg = torch.from_numpy(x.astype(np.int32)).cuda()
            conf_g, arg_g, lg_g = model.forward(xg, P + blk * bl, bl, logits=True)
            lg_g = lg_g.cpu().numpy()
            err = np.abs(lg_g - lg_ref)
            err[..., cfg.mask_id] = 0
            assert err.max() <= TOL, (blk, t, err.max())
            np.testing.assert_allclose(conf_g.cpu().numpy(), conf_ref, rtol=0, atol=TOL)
            np.testing.assert_allclose(ct[blk, t], conf_ref, rtol=0, atol=TOL)   # the trace recorded in generate
            gap = ov.top2_gap(lg_ref, cfg.mask_id)
            diff = arg_g.cpu().numpy() != arg_ref
            assert np.all(gap[diff] < 2 * TOL), "argmax differs away from a near-tie"
            near += int(diff.sum())

    # (3) free-running oracle decode (at a logit near-tie the oracle takes the
    # GPU's token, equally correct to the tolerance, so it is never skipped)
    adopted = []
    pred = tie_aware_predictor(
        lambda x, blk, t: of.forward(cfg, wnp, x, rows=np.arange(P + blk * bl, P + (blk + 1) * bl)),
        cfg.mask_id, at, TOL, adopted)
    free = oc.generate(pred, prompts.numpy(), G, cfg.mask_id, oracle_params(ctl))
    assert_state_equal(st, res.forwards, free, s_tol=TOL)
    assert len(adopted) <= near
    say(f"tiny {name}: forwards {res.forwards}, argmax near-ties {near}, adopted in the free run {len(adopted)}")
    if ctl.fixed:
        assert res.forwards == [ctl.T] * (G // bl)


def test_tiny_step_resume_equals_generate(tiny):
    """dllm_step with a host snapshot/restore in the middle equals dllm_generate."""
    cfg, model, _ = tiny
    ctl = B.Controller()
    prompts = synth.make_prompts(WL).cuda()
    P, G, bl = WL.prompt_len, WL.gen_len, ctl.block_len
    say("tiny step/resume")
    ref = _run(model, ctl, prompts, G)
    st = B.DecodeState(1, P, G)
    model.state_init(prompts, G, st)
    ws = model.workspace(1, P + G, bl)
    snap = None
    for blk in range(G // bl):
        for t in range(ctl.T):
            if blk == 0 and t == 1:
                snap = st.snapshot()
                st2 = B.DecodeState(1, P, G)
                st2.restore(snap)
                st = st2          # continue from the restored copy
            done, _, _ = model.step(ctl, st, blk, t, ws)
            if done:
                break
    for k in ("x", "commit_step", "reason", "budget"):
        assert torch.equal(getattr(st, k), getattr(ref.state, k)), k
    assert torch.equal(st.s.view(torch.int32), ref.state.s.view(torch.int32))


def test_tiny_deterministic(tiny):
    cfg, model, _ = tiny
    ctl = B.Controller()
    prompts = synth.make_prompts(WL).cuda()
    say("tiny determinism")
    a = _run(model, ctl, prompts, WL.gen_len)
    b = _run(model, ctl, prompts, WL.gen_len)
    assert torch.equal(a.state.x, b.state.x)
    assert torch.equal(a.conf_trace.view(torch.int32), b.conf_trace.view(torch.int32))
