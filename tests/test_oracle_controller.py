"""Pins for the oracle's controller (Boxes 2-7, Algorithm 1), CPU only.

Pinned by: the values the paper prints (block end thresholds, position
factors, budget tiers), closed-form properties of the cosine schedule, traces
worked out by hand from the rules (the derivations are in the comments), and
invariants on random confidence traces.
"""
import math

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import controller as oc
from oracle.controller import BUDGET, FLUSH, GRIND_FB, THRESH, CaiParams

P0 = CaiParams()


# ---------------------------------------------------------------- schedules
def test_block_end_thresholds_printed_values():
    # Box 4: theta_e^(b) = 0.70, 0.60, 0.50, 0.40 for b = 1..4
    assert [oc.block_end_threshold(b, P0) for b in (1, 2, 3, 4)] == pytest.approx([0.70, 0.60, 0.50, 0.40], abs=1e-15)
    # beyond the printed range: held at the floor, never increasing
    vals = [oc.block_end_threshold(b, P0) for b in range(1, 20)]
    assert all(a >= b for a, b in zip(vals, vals[1:]))
    assert vals[-1] == pytest.approx(0.40)
    assert oc.block_end_threshold(7, CaiParams(block_sched=False)) == 0.70


@pytest.mark.parametrize("T", [32, 64, 20, 7])
@pytest.mark.parametrize("b", [1, 2, 4, 9])
def test_cosine_schedule_closed_form_properties(T, b):
    p = CaiParams(block_len=T)
    te = oc.block_end_threshold(b, p)
    wT = 0.15 * T
    th = [oc.block_threshold(t, b, p) for t in range(T)]
    # warm-up: exactly theta_s while t < wT (Box 3)
    for t in range(T):
        if t < wT:
            assert th[t] == 0.90
    # at u = 0 the cosine branch equals theta_s (continuity), at u = 1 it equals theta_e
    assert oc.block_threshold(wT, b, p) == pytest.approx(0.90, abs=1e-15)
    assert oc.block_threshold(T, b, p) == pytest.approx(te, abs=1e-15)
    # at u = 1/2 it is the midpoint (cos(pi/2) = 0)
    assert oc.block_threshold(wT + 0.5 * (T - wT), b, p) == pytest.approx((0.90 + te) / 2, abs=1e-15)
    # point symmetry about the midpoint: theta(u) + theta(1-u) = theta_s + theta_e
    for u in (0.1, 0.25, 0.37):
        a = oc.block_threshold(wT + u * (T - wT), b, p)
        c = oc.block_threshold(wT + (1 - u) * (T - wT), b, p)
        assert a + c == pytest.approx(0.90 + te, abs=1e-14)
    # non-increasing in t and bounded by [theta_e, theta_s]
    assert all(x >= y for x, y in zip(th, th[1:]))
    assert all(te <= x <= 0.90 for x in th)


@pytest.mark.parametrize("b,t,expect", [(1, 8, 0.89325), (1, 16, 0.82737), (1, 24, 0.73974), (1, 31, 0.70067),
                                         (4, 16, 0.71842), (4, 31, 0.40167)])
def test_cosine_schedule_hand_values(b, t, expect):
    # Box 3 at T = 32, w = 0.15 (wT = 4.8): theta = theta_e + (theta_s - theta_e)(1 + cos(pi u)) / 2 with
    # u = (t - 4.8) / 27.2, worked by hand: t = 8 -> u = 0.11765, cos(pi u) = 0.93247; t = 16 -> 0.41176,
    # 0.27366; t = 24 -> 0.70588, -0.60263; t = 31 -> 0.96324, -0.99334.  theta_e = 0.70 (b = 1), 0.40
    # (b = 4, Box 4): 0.70 + 0.10 (1.93247) = 0.89325, ..., 0.40 + 0.25 (1.27366) = 0.71842.
    assert oc.block_threshold(t, b, P0) == pytest.approx(expect, abs=6e-6)


def test_position_factors_and_clip():
    # Box 6: r = 0.80 (p<16), 0.90 (16<=p<32), 1.05 (32<=p<48), 1.10 (p>=48)
    want = {0: 0.80, 15: 0.80, 16: 0.90, 31: 0.90, 32: 1.05, 47: 1.05, 48: 1.10, 63: 1.10}
    for pos, r in want.items():
        assert oc.position_factor(pos, P0) == r
    # t = 0 thresholds: 0.9 * r, with 0.9 * 1.10 = 0.99 capped at 0.98
    got = [float(oc.token_threshold(0, 1, pos, P0)) for pos in (0, 16, 32, 48)]
    assert got == pytest.approx([0.72, 0.81, 0.945, 0.98], abs=1e-7)
    # clip floor: a threshold schedule ending at 0.1 is clipped to 0.20
    low = CaiParams(theta_e=0.1, theta_s=0.2, theta_e_floor=0.0)
    assert float(oc.token_threshold(31, 1, 0, low)) == pytest.approx(0.20, abs=1e-7)
    # thresholds are float32
    assert isinstance(oc.token_threshold(5, 1, 3, P0), np.float32)


def test_budget_truth_table():
    # Eq. token_budget, cases top to bottom:
    #   8 if s > 0.50 and p < 32; else 64 if s < 0.25 or p >= 48; else 32
    f32 = np.float32
    cases = [
        (0.51, 0, 8), (0.51, 31, 8), (0.51, 32, 32), (0.51, 47, 32), (0.51, 48, 64),
        (0.50, 0, 32), (0.50, 31, 32), (0.50, 48, 64),            # s = 0.5 is not > 0.5
        (0.25, 0, 32), (0.25, 47, 32),                              # s = 0.25 is not < 0.25
        (0.2499, 0, 64), (0.2499, 31, 64), (0.10, 40, 64),
        (0.99, 15, 8), (0.99, 16, 8), (0.99, 63, 64),
        (np.nextafter(f32(0.5), f32(1)), 3, 8), (np.nextafter(f32(0.25), f32(0)), 3, 64),
    ]
    for s, pos, want in cases:
        assert oc.token_budget(s, pos, P0) == want, (s, pos)
    # NaN confidence fails every comparison: budget from position alone
    assert oc.token_budget(float("nan"), 3, P0) == 32
    assert oc.token_budget(float("nan"), 50, P0) == 64


# ---------------------------------------------------------------- hand traces
def _run_one_block(conf_fn, p, blk=0, bl=32):
    """Run the controller on a single block whose confidences are conf_fn(t, i);
    every prediction is token 7 + i.  Returns the decode state."""
    G = bl * (blk + 1)

    def predict(x, b, t):
        if b < blk:                                      # earlier blocks: commit at once
            return np.full((1, bl), 0.999, np.float32), np.zeros((1, bl), np.int64)
        return (np.array([[conf_fn(t, i) for i in range(bl)]], np.float32),
                np.array([[7 + i for i in range(bl)]], np.int64))

    return oc.generate(predict, np.zeros((1, 4), np.int64), G, 99, p)


def _expect(stt, blk, n, per_pos, bl=32):
    """per_pos: list of (reason, step) for positions 0..bl-1."""
    assert stt.forwards[blk] == n
    g0 = blk * bl
    got = [(int(stt.reason[0, g0 + i]), int(stt.commit_step[0, g0 + i])) for i in range(bl)]
    assert got == per_pos
    assert all(stt.x[0, 4 + g0 + i] == 7 + i for i in range(bl))


ON = CaiParams()
OFF = CaiParams(budgets=False, grinding=False)


def test_trace_all_confident():
    # S1: c = 0.99 everywhere.  t = 0 thresholds are 0.72 / 0.81 -> every token
    # commits at t = 0 by threshold; no mask left -> one forward.
    _expect(_run_one_block(lambda t, i: 0.99, ON), 0, 1, [(THRESH, 0)] * 32)


def test_trace_all_hopeless_gating_on():
    # S2: c = 0.001.  s < 0.25 -> B = 64 (never reached).  No commit ever, so
    # eta = 0 < 1.5 each step: ell = 1, 2, 3, 4 -> grinding at t = 3; nothing
    # passes c > 0.40, so all 32 are flushed at t = 3 (4 forwards).
    _expect(_run_one_block(lambda t, i: 0.001, ON), 0, 4, [(FLUSH, 3)] * 32)


def test_trace_all_hopeless_gating_off():
    # S2': no budgets, no grinding; lowest threshold is 0.8 * 0.7007 > 0.001,
    # so every token is flushed at the last step t = 31 (32 forwards).
    _expect(_run_one_block(lambda t, i: 0.001, OFF), 0, 32, [(FLUSH, 31)] * 32)


def test_trace_medium_gating_on():
    # S3: c = 0.6.  s > 0.5 and p < 32 -> B = 8.  t = 0..3 thresholds 0.72 / 0.81
    # (warm-up, t < 4.8) block everything; ell hits 4 at t = 3 -> grinding
    # commits every c = 0.6 > 0.40 token at t = 3; B = 8 is never reached.
    _expect(_run_one_block(lambda t, i: 0.6, ON), 0, 4, [(GRIND_FB, 3)] * 32)


def test_trace_medium_gating_off():
    # S3': p < 16 needs 0.8 * theta_1(t) <= 0.6, i.e. theta_1(t) <= 0.75:
    # 0.70 + 0.10 (1 + cos(pi u)) <= 0.75 -> u >= 2/3 -> t >= 4.8 + 27.2 * 2/3
    # = 22.93, so t = 23 (0.8 * theta(23) = 0.5994; at t = 22 it is 0.6077).
    # p >= 16 needs theta_1(t) <= 0.667 < 0.70: never -> flushed at t = 31.
    _expect(_run_one_block(lambda t, i: 0.6, OFF), 0, 32, [(THRESH, 23)] * 16 + [(FLUSH, 31)] * 16)


def test_trace_split_grinding_fallback():
    # S4: c = 0.6 for p < 16 (B = 8) and 0.3 for p >= 16 (0.25 <= s <= 0.5 -> B = 32).
    # Nothing passes 0.72 / 0.81 in t = 0..3 -> grinding at t = 3: the 0.6 tokens
    # pass c > 0.40 (fallback), the 0.3 tokens do not and are flushed.
    _expect(_run_one_block(lambda t, i: 0.6 if i < 16 else 0.3, ON), 0, 4,
            [(GRIND_FB, 3)] * 16 + [(FLUSH, 3)] * 16)


def test_trace_staircase_budget():
    # S5: c_i(t) = 0.99 once t >= i // 2, else 0.6.  Every s_i > 0.5 with p < 32
    # -> B = 8.  Two tokens pass the threshold per step (eta = 2 keeps ell = 0)
    # for t = 0..8; at t = 8 every token still masked (i >= 18, c = 0.6 below
    # 0.9 * 0.893) hits its budget.  No mask left -> 9 forwards.
    want = [(THRESH, i // 2) for i in range(18)] + [(BUDGET, 8)] * 14
    _expect(_run_one_block(lambda t, i: 0.99 if t >= i // 2 else 0.6, ON), 0, 9, want)


@pytest.mark.parametrize("blk", [3, 7])
def test_trace_late_block_lower_end_threshold(blk):
    # S6: block 4 (theta_e = 0.40) and block 8 (held at the 0.40 floor), c = 0.6, OFF.
    # p < 16: 0.4 + 0.25 (1 + cos(pi u)) <= 0.75 -> cos(pi u) <= 0.4 -> u >= 0.36901
    #   -> t >= 14.84 -> t = 15 (0.8 * theta(15) = 0.5965; t = 14 gives 0.6174).
    # p >= 16: theta <= 0.6667 -> cos(pi u) <= 0.06667 -> u >= 0.47877 -> t >= 17.82
    #   -> t = 18 (0.9 * theta(18) = 0.5954; t = 17 gives 0.6212).  Block done at t = 18.
    stt = _run_one_block(lambda t, i: 0.6, OFF, blk=blk)
    _expect(stt, blk, 19, [(THRESH, 15)] * 16 + [(THRESH, 18)] * 16)
    assert stt.forwards[:blk] == [1] * blk


def test_trace_low_yield_counter_resets():
    # S8: token i becomes confident (0.99) at step sched[i], else 0.3.
    # sched = 0,1,2,2,3,4,5,6,...: eta = 1,1,2,1,1,1,1 for t = 0..6 ->
    # ell = 1,2,0,1,2,3,4 -> grinding at t = 6 (7 forwards).  The 0.3 tokens fail
    # the 0.40 fallback and are flushed at t = 6.  Token 0 has s = 0.99 -> B = 8,
    # the others s = 0.3 -> B = 32; neither budget is reached.
    sched = [0, 1, 2, 2, 3, 4, 5, 6] + [100] * 24
    stt = _run_one_block(lambda t, i: 0.99 if t >= sched[i] else 0.3, ON)
    want = [(THRESH, sched[i]) for i in range(8)] + [(FLUSH, 6)] * 24
    _expect(stt, 0, 7, want)
    assert list(stt.budget[0, :3]) == [8, 32, 32]


def test_quarter_scaled_position_edges():
    # R6 alternative: edges 8/16/24 for 32-token blocks.  c = 0.6, OFF, block 1:
    # p < 8 commit at t = 23 (r = 0.8, as S3'), the rest (r >= 0.9) are flushed.
    p = CaiParams(budgets=False, grinding=False, pos_edges=(8, 16, 24), p_easy=16, p_hard=24)
    _expect(_run_one_block(lambda t, i: 0.6, p), 0, 32, [(THRESH, 23)] * 8 + [(FLUSH, 31)] * 24)


def test_nan_confidence_never_passes_a_threshold():
    # NaN fails c >= theta and c > theta_fb; it is committed by budget or flush.
    stt = _run_one_block(lambda t, i: float("nan") if i == 5 else 0.99, ON)
    # t = 0: 31 threshold commits (ell = 0); t = 1..4: eta = 0 -> ell = 1..4 -> grinding at t = 4
    assert stt.reason[0, 5] == FLUSH and stt.commit_step[0, 5] == 4
    stt = _run_one_block(lambda t, i: float("nan"), OFF)
    assert set(stt.reason[0].tolist()) == {FLUSH} and stt.forwards == [32]


# ---------------------------------------------------------------- invariants
def _check_invariants(stt, trace, p, G, P):
    """Invariants any controller run must satisfy: committed tokens are never
    re-masked, every block ends with no mask left, no token exceeds its step
    budget, the block-end threshold never rises over blocks; plus the
    recurrences the decode's records obey."""
    bl, T = p.block_len, p.T
    B = stt.x.shape[0]
    # no mask left at the end; prompt untouched; every token committed once
    assert np.all(stt.commit_step >= 0) and np.all(stt.commit_step <= T - 1)
    assert np.all(stt.reason >= 1)
    # theta_e^(b) non-increasing over blocks
    te = [oc.block_end_threshold(b, p) for b in range(1, G // bl + 1)]
    assert all(a >= b for a, b in zip(te, te[1:]))
    if p.budgets:
        assert np.all(stt.commit_step <= stt.budget)
    prev = None
    for (blk, t, x, conf, arg) in trace:
        if prev is not None and prev[0] == blk:
            px = prev[1]
            committed = px != 99
            # committed tokens never change and are never re-masked
            assert np.all(x[committed] == px[committed])
        prev = (blk, x)
    for seq in range(B):
        for blk in range(G // bl):
            sl = slice(blk * bl, (blk + 1) * bl)
            cs, rs = stt.commit_step[seq, sl], stt.reason[seq, sl]
            last = cs.max()
            # threshold/budget commits at step t give eta(t); the counter ell follows
            # its recurrence, and grinding (reason 3) only happens at the exit step
            assert np.all(cs[rs == GRIND_FB] == last) and np.all(cs[rs == FLUSH] == last)
            ell = 0
            for t in range(last + 1):
                eta = int(np.sum((cs == t) & ((rs == THRESH) | (rs == BUDGET))))
                ell = ell + 1 if eta < p.eta_bar else 0
                if t < last:
                    assert not (p.grinding and ell >= p.patience)
            # exit reasons are consistent with the last step
            if np.any(rs == GRIND_FB):
                assert p.grinding and ell >= p.patience
            if np.any(rs == FLUSH):
                assert last == T - 1 or (p.grinding and ell >= p.patience)
            assert stt.forwards[blk] >= last + 1
    assert np.all(stt.x[:, P:] != 99)


@settings(max_examples=60, deadline=None)
@given(seed=st.integers(0, 2**31 - 1), gating=st.booleans(), bl=st.sampled_from([4, 8, 32]),
       B=st.integers(1, 3), nb=st.integers(1, 3), grid=st.booleans())
def test_random_trace_invariants(seed, gating, bl, B, nb, grid):
    rng = np.random.default_rng(seed)
    p = CaiParams(block_len=bl, budgets=gating, grinding=gating)
    G, P = bl * nb, 3
    trace = []

    def predict(x, blk, t):
        if grid:   # values on a coarse grid hit the comparison boundaries
            c = rng.choice(np.float32([0.0, 0.25, 0.4, 0.5, 0.6, 0.72, 0.81, 0.9, 1.0]), (B, bl))
        else:
            c = rng.random((B, bl)).astype(np.float32) ** 0.5
        return c, rng.integers(0, 99, (B, bl))

    stt = oc.generate(predict, rng.integers(0, 99, (B, P)), G, 99, p,
                      on_step=lambda *a: trace.append((a[0], a[1], a[2], a[3], a[4])))
    _check_invariants(stt, trace, p, G, P)


def test_batch_lockstep_equals_per_sequence_runs():
    rng = np.random.default_rng(11)
    B, bl, nb, P = 3, 32, 3, 5
    G = bl * nb
    p = CaiParams()
    # confidence of (seq, block, step, pos) fixed in advance; argmax fixed too
    C = rng.random((B, nb, 32, bl)).astype(np.float32) ** 0.7
    A = rng.integers(0, 99, (B, nb, bl))

    def pred_for(seqs):
        return lambda x, blk, t: (C[seqs, blk, t], A[seqs, blk])

    prompts = rng.integers(0, 99, (B, P))
    batch = oc.generate(pred_for(list(range(B))), prompts, G, 99, p)
    for s in range(B):
        one = oc.generate(pred_for([s]), prompts[s:s + 1], G, 99, p)
        np.testing.assert_array_equal(one.x[0], batch.x[s])
        np.testing.assert_array_equal(one.commit_step[0], batch.commit_step[s])
        np.testing.assert_array_equal(one.reason[0], batch.reason[s])
    # the lockstep block runs as many forwards as its slowest sequence
    per = [oc.generate(pred_for([s]), prompts[s:s + 1], G, 99, p).forwards for s in range(B)]
    assert batch.forwards == [max(f[b] for f in per) for b in range(nb)]


# ------------------------------------------------ fixed-schedule baseline (R19)
FIXED = oc.FIXED


def test_fixed_schedule_hand_trace():
    # S9, block of 4, one token per step.  t0: c = (.1 .5 .3 .5): the tie at .5
    # goes to position 1.  t1: masked 0, 2, 3 with (.9 .2 .1): position 0 (the .9
    # at the already committed position 1 is not eligible).  t2: masked 2, 3 with
    # (.1 .4): position 3.  t3: position 2.  Four forwards, all reason FIXED.
    p = CaiParams(block_len=4, fixed=True)
    confs = [[.1, .5, .3, .5], [.9, .9, .2, .1], [.3, .2, .1, .4], [0., 0., 0., 0.]]
    stt = oc.generate(lambda x, blk, t: (np.array([confs[t]], np.float32), np.array([[10 + t, 20 + t, 30 + t, 40 + t]])),
                      np.zeros((1, 2), np.int64), 4, 99, p)
    assert stt.forwards == [4]
    assert stt.commit_step[0].tolist() == [1, 0, 3, 2]
    assert stt.reason[0].tolist() == [FIXED] * 4
    assert stt.x[0, 2:].tolist() == [11, 20, 33, 42]      # each token takes the argmax of its commit step


@pytest.mark.parametrize("bl,T,expect", [(32, 32, [1] * 32), (32, 16, [2] * 16), (4, 3, [2, 1, 1]),
                                         (32, 12, [3] * 8 + [2] * 4), (8, 8, [1] * 8)])
def test_fixed_schedule_commit_counts(bl, T, expect):
    p = CaiParams(block_len=bl, steps_per_block=T, fixed=True)
    got = [oc.fixed_commits(t, p) for t in range(T)]
    assert got == expect and sum(got) == bl


@settings(max_examples=60, deadline=None)
@given(seed=st.integers(0, 2**31 - 1), bl=st.sampled_from([4, 8, 32]), div=st.sampled_from([1, 2, 3]),
       B=st.integers(1, 3), nb=st.integers(1, 2), grid=st.booleans())
def test_fixed_schedule_commits_dominate_the_rest(seed, bl, div, B, nb, grid):
    # Brute-force restatement: after every step, each token committed in that
    # step beats every token still masked (higher confidence, or equal and a
    # lower position); the step commits k_t tokens; every block takes T forwards.
    rng = np.random.default_rng(seed)
    T = max(1, bl // div)
    p = CaiParams(block_len=bl, steps_per_block=T, fixed=True)
    G, P = bl * nb, 2
    trace = []

    def predict(x, blk, t):
        if grid:
            c = rng.choice(np.float32([0.1, 0.5, 0.9]), (B, bl))
        else:
            c = rng.random((B, bl)).astype(np.float32)
        return c, rng.integers(0, 99, (B, bl))

    stt = oc.generate(predict, rng.integers(0, 99, (B, P)), G, 99, p,
                      on_step=lambda *a: trace.append((a[0], a[1], a[3])))
    assert stt.forwards == [T] * nb
    assert np.all(stt.reason == FIXED)
    for blk, t, conf in trace:
        sl = slice(blk * bl, (blk + 1) * bl)
        for seq in range(B):
            cs = stt.commit_step[seq, sl]
            now = [i for i in range(bl) if cs[i] == t]
            later = [i for i in range(bl) if cs[i] > t]
            assert len(now) == oc.fixed_commits(t, p)
            for i in now:
                for j in later:
                    assert conf[seq, i] > conf[seq, j] or (conf[seq, i] == conf[seq, j] and i < j)
