"""CAI-dLLM confidence-aware controller (oracle).

Restates Boxes 2-7 and Algorithm 1 (Section 4.7) for one block, and the
semi-autoregressive outer loop over blocks (Section 4.3).  Readings taken
where the paper is silent or inconsistent:

  R1  A block that exits (grinding, all-steps-used) with tokens still masked
      commits each of them with its current argmax at the exit step ("flush",
      as Box 5 does for an exhausted budget); no extra forward.
  R2  eta is a count of tokens committed by the threshold/budget rule in the
      step; "low yield" is eta < eta_bar with eta_bar = 1.5 (Algorithm 1 counts
      tokens; the fraction form in Section 4.5 is not used).
  R3  Gating OFF (Section 4.6) disables the token budgets and the grinding
      detector with its fallback; the cosine and block schedules stay on.
  R4  T, the per-block step limit, defaults to the block length.
  R5  theta_e^(b) = max(theta_e - step*(b-1), floor) with floor 0.40, the
      last value Box 4 prints, for blocks past the fourth.
  R6  Position bands use absolute in-block positions 16/32/48 (Boxes 5, 6).
  R7  s_i and B_i are set from each block's own step-zero forward.
  R8  Local steps t = 0..T-1; a budget B_i forces commit at t = B_i.
  R9  Only masked positions of the current block are eligible.
  R12 Thresholds are evaluated in float64 (cos from libm), clipped, then
      rounded to float32; confidences are float32; every comparison is made
      in float32.  The warm-up test t < w*T is made in float64.
  R13 Order inside a step: threshold/budget commits, eta, ell update,
      grinding fallback, no-mask check, flush.
  R14 A batch advances in lockstep: each sequence keeps its own s, B, ell and
      done flag; a finished sequence is frozen; the block ends when every
      sequence has finished.
  R19 The fixed-schedule baseline (the "Fixed" column of the step-reduction
      table, Section 6: as many denoising steps as generated tokens) commits,
      at local step t, the k_t masked tokens of highest confidence (lowest
      position first on equal confidence), k_t = floor(bl/T) plus one in the
      first bl mod T steps; with T = block_len that is one token per step.
      A NaN confidence ranks below every number.  It keeps no s, B or ell.

Reason codes per committed token: 1 threshold, 2 budget, 3 grinding
fallback, 4 flush, 5 fixed schedule.

Test infrastructure only; see the package docstring.
"""
import math
from dataclasses import dataclass, field

import numpy as np

THRESH, BUDGET, GRIND_FB, FLUSH, FIXED = 1, 2, 3, 4, 5


@dataclass
class CaiParams:
    """Controller constants, defaults as printed in Boxes 3-7 and Section 5."""
    block_len: int = 32
    steps_per_block: int = 0          # T; 0 means block_len (R4)
    theta_s: float = 0.90             # Box 3
    theta_e: float = 0.70             # Box 3
    theta_e_step: float = 0.10        # Box 4
    theta_e_floor: float = 0.40       # R5
    warmup: float = 0.15              # Box 3
    pos_edges: tuple = (16, 32, 48)   # Box 6
    pos_factors: tuple = (0.80, 0.90, 1.05, 1.10)
    clip_lo: float = 0.20
    clip_hi: float = 0.98
    s_easy: float = 0.50              # Box 5
    s_hard: float = 0.25
    p_easy: int = 32
    p_hard: int = 48
    budget_easy: int = 8
    budget_mid: int = 32
    budget_hard: int = 64
    eta_bar: float = 1.5              # Box 7 (R2)
    patience: int = 4
    theta_fb: float = 0.40
    block_sched: bool = True          # Box 4 on (else theta_e for every block)
    pos_aware: bool = True            # Box 6 on (else theta_i = theta_b(t), no clip)
    budgets: bool = True              # Box 5 on   } confidence gating (Section 4.6)
    grinding: bool = True             # Box 7 on   }
    fixed: bool = False               # fixed-schedule baseline instead (R19)

    @property
    def T(self):
        return self.steps_per_block or self.block_len


def fixed_commits(t, p: CaiParams):
    """k_t, the tokens the fixed schedule commits at local step t (R19)."""
    base, extra = divmod(p.block_len, p.T)
    return base + (1 if t < extra else 0)


def block_end_threshold(b, p: CaiParams):
    """theta_e^(b) for 1-based block index b (Box 4, R5)."""
    if not p.block_sched:
        return p.theta_e
    return max(p.theta_e - p.theta_e_step * (b - 1), p.theta_e_floor)


def block_threshold(t, b, p: CaiParams):
    """theta^(b)(t) in float64 (Boxes 3 and 4)."""
    T = p.T
    wT = p.warmup * T
    if t < wT:
        return p.theta_s
    te = block_end_threshold(b, p)
    u = (t - wT) / (T - wT)
    return te + 0.5 * (p.theta_s - te) * (1.0 + math.cos(math.pi * u))


def position_factor(pos, p: CaiParams):
    """r_pos(i) for in-block position pos (Box 6)."""
    e0, e1, e2 = p.pos_edges
    if pos < e0:
        return p.pos_factors[0]
    if pos < e1:
        return p.pos_factors[1]
    if pos < e2:
        return p.pos_factors[2]
    return p.pos_factors[3]


def token_threshold(t, b, pos, p: CaiParams):
    """theta_i(t) as float32 (Box 6, Eq. position_threshold; R12)."""
    tb = block_threshold(t, b, p)
    if p.pos_aware:
        tb = min(max(tb * position_factor(pos, p), p.clip_lo), p.clip_hi)
    return np.float32(tb)


def token_budget(s, pos, p: CaiParams):
    """B_i from the float32 first-step confidence s (Box 5, Eq. token_budget)."""
    s = np.float32(s)
    if s > np.float32(p.s_easy) and pos < p.p_easy:
        return p.budget_easy
    if s < np.float32(p.s_hard) or pos >= p.p_hard:
        return p.budget_hard
    return p.budget_mid


@dataclass
class DecodeState:
    """Complete decoding state of a batch (the quantities Algorithm 1 keeps)."""
    x: np.ndarray              # int64 [B, P+G]   token ids; mask id where masked
    commit_step: np.ndarray    # int64 [B, G]     local step of commit, -1 while masked
    reason: np.ndarray         # int64 [B, G]
    s: np.ndarray              # float32 [B, G]   first-step confidence (Box 2)
    budget: np.ndarray         # int64 [B, G]     B_i (Box 5)
    forwards: list = field(default_factory=list)   # forwards run per block


def init_state(prompts, gen_len, mask_id):
    prompts = np.asarray(prompts, dtype=np.int64)
    B, P = prompts.shape
    x = np.concatenate([prompts, np.full((B, gen_len), mask_id, dtype=np.int64)], axis=1)
    return DecodeState(x=x,
                       commit_step=np.full((B, gen_len), -1, dtype=np.int64),
                       reason=np.zeros((B, gen_len), dtype=np.int64),
                       s=np.full((B, gen_len), np.nan, dtype=np.float32),
                       budget=np.zeros((B, gen_len), dtype=np.int64))


def step_sequence(st: DecodeState, seq, P, blk, t, conf, arg, ell, p: CaiParams):
    """Algorithm 1's body for one sequence at local step t of block blk (0-based).

    conf (float32) and arg (int) hold the prediction for each in-block position
    from the forward on x^(t).  Updates st in place.  Returns (ell, exited).
    """
    bl = p.block_len
    g0 = blk * bl
    b1 = blk + 1
    conf = np.asarray(conf, dtype=np.float32)
    masked = [st.commit_step[seq, g0 + i] < 0 for i in range(bl)]

    def commit(i, why):
        st.x[seq, P + g0 + i] = int(arg[i])
        st.commit_step[seq, g0 + i] = t
        st.reason[seq, g0 + i] = why
        masked[i] = False

    if p.fixed:                                           # fixed-schedule baseline (R19)
        key = lambda i: (-(float(conf[i]) if conf[i] == conf[i] else -math.inf), i)   # NaN ranks lowest
        order = sorted((i for i in range(bl) if masked[i]), key=key)
        for i in order[:fixed_commits(t, p)]:
            commit(i, FIXED)
        exited = not any(masked)
        if not exited and t == p.T - 1:                   # flush (R1), unreachable when sum k_t = bl
            for i in range(bl):
                if masked[i]:
                    commit(i, FLUSH)
            exited = True
        return ell, exited

    if t == 0:                                            # step-zero init (Boxes 2, 5)
        for i in range(bl):
            st.s[seq, g0 + i] = conf[i]
            st.budget[seq, g0 + i] = token_budget(conf[i], i, p)

    eta = 0                                               # threshold / budget commits
    for i in range(bl):
        if not masked[i]:
            continue
        if conf[i] >= token_threshold(t, b1, i, p):
            commit(i, THRESH)
            eta += 1
        elif p.budgets and t >= st.budget[seq, g0 + i]:
            commit(i, BUDGET)
            eta += 1

    ell = ell + 1 if eta < p.eta_bar else 0               # low-yield counter

    exited = False
    if p.grinding and ell >= p.patience:                  # grinding-phase fallback
        for i in range(bl):
            if masked[i] and conf[i] > np.float32(p.theta_fb):
                commit(i, GRIND_FB)
        exited = True
    if not any(masked):
        exited = True
    if exited or t == p.T - 1:                            # flush (R1)
        for i in range(bl):
            if masked[i]:
                commit(i, FLUSH)
        exited = True
    return ell, exited


def generate(predict, prompts, gen_len, mask_id, p: CaiParams, on_step=None):
    """Decode gen_len tokens after the prompts, block by block.

    predict(x, blk, t) -> (conf float32 [B, bl], argmax int [B, bl]) for the
    current block's positions given the full token array x [B, P+G].
    on_step(blk, t, x, conf, arg) is called after each prediction (tracing).
    Returns the final DecodeState.
    """
    st = init_state(prompts, gen_len, mask_id)
    B, P = st.x.shape[0], st.x.shape[1] - gen_len
    if gen_len % p.block_len:
        raise ValueError("gen_len must be a multiple of block_len")
    for blk in range(gen_len // p.block_len):
        ell = [0] * B
        done = [False] * B
        n = 0
        for t in range(p.T):
            conf, arg = predict(st.x.copy(), blk, t)
            conf = np.asarray(conf, dtype=np.float32)
            arg = np.asarray(arg)
            if on_step is not None:
                on_step(blk, t, st.x.copy(), conf, arg)
            n += 1
            for seq in range(B):
                if done[seq]:
                    continue
                ell[seq], done[seq] = step_sequence(st, seq, P, blk, t, conf[seq], arg[seq], ell[seq], p)
            if all(done):
                break
        st.forwards.append(n)
    return st


def model_predictor(forward_fn, P, block_len, mask_id):
    """Wrap a logits function forward_fn(x, rows) -> [B, len(rows), V] into a
    predict callback: confidence/argmax of the current block's rows (Box 1)."""
    from .vocab import confidence_argmax

    def predict(x, blk, t):
        rows = np.arange(P + blk * block_len, P + (blk + 1) * block_len)
        logits = forward_fn(x, rows)
        conf, arg = confidence_argmax(logits, mask_id)
        return conf.astype(np.float32), arg

    return predict
