"""Helpers shared by the GPU parity tests (comparisons, oracle replays)."""
import os
import sys

import numpy as np
import torch

from oracle import controller as oc
from oracle import forward as of
from oracle import vocab as ov
from paper_2608_22646_amd import binding as B


def say(*a):
    """Progress line naming the case before each GPU step (flushed)."""
    print("[gpu-test]", *a, flush=True)


def to_np(t, dtype=np.float32):
    return t.detach().to("cpu").to(torch.float32 if t.dtype in (torch.bfloat16, torch.float16) else t.dtype).numpy().astype(dtype)


def oracle_params(ctl: B.Controller) -> oc.CaiParams:
    """The oracle's parameter object with the same constants as a binding Controller."""
    return oc.CaiParams(block_len=ctl.block_len, steps_per_block=ctl.steps_per_block, theta_s=ctl.theta_s,
                        theta_e=ctl.theta_e, theta_e_step=ctl.theta_e_step, theta_e_floor=ctl.theta_e_floor,
                        warmup=ctl.warmup, pos_edges=tuple(ctl.pos_edges), pos_factors=tuple(ctl.pos_factors),
                        clip_lo=ctl.clip_lo, clip_hi=ctl.clip_hi, s_easy=ctl.s_easy, s_hard=ctl.s_hard,
                        p_easy=ctl.p_easy, p_hard=ctl.p_hard, budget_easy=ctl.budget_easy,
                        budget_mid=ctl.budget_mid, budget_hard=ctl.budget_hard, eta_bar=ctl.eta_bar,
                        patience=ctl.patience, theta_fb=ctl.theta_fb, block_sched=ctl.block_sched,
                        pos_aware=ctl.pos_aware, budgets=ctl.budgets, grinding=ctl.grinding, fixed=ctl.fixed)


def replay(conf_trace, argmax_trace, prompts, G, mask_id, ctl: B.Controller):
    """Run the oracle controller on recorded predictions [nb, T, B, bl]."""
    ct = np.asarray(conf_trace, dtype=np.float32)
    at = np.asarray(argmax_trace)

    def predict(x, blk, t):
        return ct[blk, t], at[blk, t]

    return oc.generate(predict, np.asarray(prompts), G, mask_id, oracle_params(ctl))


def assert_state_equal(gpu_state: B.DecodeState, forwards, ref: oc.DecodeState, s_tol=None):
    """Decisions bit-exact.  s (the step-zero confidences) bit-exact when ref was
    replayed on the GPU's own predictions (s_tol None), else within s_tol.  The
    fixed schedule keeps no s: then both sides still hold their initial values
    (the oracle NaN, the library 0) and s is not compared."""
    np.testing.assert_array_equal(gpu_state.x.cpu().numpy(), ref.x)
    np.testing.assert_array_equal(gpu_state.commit_step.cpu().numpy(), ref.commit_step)
    np.testing.assert_array_equal(gpu_state.reason.cpu().numpy().astype(np.int64), ref.reason)
    np.testing.assert_array_equal(gpu_state.budget.cpu().numpy(), ref.budget)
    if np.all(np.isnan(ref.s)):
        assert np.all(gpu_state.s.cpu().numpy() == 0)
    elif s_tol is None:
        np.testing.assert_array_equal(gpu_state.s.cpu().numpy().view(np.uint32), ref.s.view(np.uint32))
    else:
        np.testing.assert_allclose(gpu_state.s.cpu().numpy(), ref.s, rtol=0, atol=s_tol)
    assert list(forwards) == list(ref.forwards)


def x_at_step(final_x, commit_step, P, bl, blk, t, mask_id):
    """The token array the forward of (blk, t) saw, rebuilt from the final state:
    earlier blocks fully committed, this block's tokens committed before t."""
    x = np.array(final_x, dtype=np.int64, copy=True)
    Bn, L = x.shape
    G = L - P
    g = np.arange(G)
    blk_of = g // bl
    keep = (blk_of < blk)[None, :] | ((blk_of == blk)[None, :] & (commit_step < t) & (commit_step >= 0))
    x[:, P:] = np.where(keep, x[:, P:], mask_id)
    return x


def bf16_ulp(ref):
    """One bf16 unit in the last place of |ref| (normal range)."""
    a = np.maximum(np.abs(np.asarray(ref, dtype=np.float64)), 1e-30)
    return 2.0 ** (np.floor(np.log2(a)) - 7)


def assert_bf16_flips(gpu, ref, what, max_frac=2e-3, max_ulps=1.0, rel_floor=3e-5):
    """gpu holds bf16 values rounded from a float32 computation; ref is the oracle's
    bf16-rounded value of the same quantity from the same (GPU) inputs.  Different
    float32 accumulation order may move a value across a rounding boundary, so a
    small fraction of elements may differ by one bf16 ulp; nothing may differ more.
    Values produced by cancellation (RoPE, SwiGLU near 0) carry the float32 error of
    their inputs, so an absolute floor of rel_floor * max|ref| is allowed as well."""
    g = np.asarray(gpu, dtype=np.float64)
    r = np.asarray(ref, dtype=np.float64)
    d = np.abs(g - r)
    ulp = np.maximum(bf16_ulp(r), bf16_ulp(g))
    bad = d > max_ulps * ulp * 1.0001 + rel_floor * np.abs(r).max()
    frac = float(np.mean(d > 0))
    assert not bad.any(), f"{what}: {int(bad.sum())} elements off by more than {max_ulps} ulp; max {d.max():.3g}"
    assert frac <= max_frac, f"{what}: {frac:.2e} of elements differ (limit {max_frac})"
    return frac


def tie_aware_predictor(logits_at, mask_id, gpu_argmax, tol, adopted):
    """predict(x, blk, t) for the oracle controller from logits_at(x, blk, t) ->
    [B, bl, V] (the oracle's logits).  Where the GPU recorded another argmax
    whose oracle logit lies within 2 tol of the oracle's largest one (a logit
    near-tie: both tokens are correct predictions to the tolerance), the GPU's
    choice is taken, so the free-running decodes stay comparable; each such
    adoption is appended to ``adopted`` as (blk, t, b, i)."""
    def predict(x, blk, t):
        lg = np.array(logits_at(x, blk, t), dtype=np.float64, copy=True)
        conf, arg = ov.confidence_argmax(lg, mask_id)
        g = np.asarray(gpu_argmax[blk, t])
        lm = lg.copy()
        lm[..., mask_id] = -np.inf
        top = lm.max(axis=-1)
        for b, i in zip(*np.nonzero(g != arg)):
            gi = int(g[b, i])
            if 0 <= gi < lg.shape[-1] and gi != mask_id and lm[b, i, gi] >= top[b, i] - 2 * tol:
                arg[b, i] = gi
                adopted.append((blk, t, int(b), int(i)))
        return conf.astype(np.float32), arg

    return predict
