"""End-to-end bf16 parity by depth: the LLaDA-8B- and Dream-7B-shaped forwards
on the GPU against the oracle's bf16 forward (float32 products), logits and
confidences of the first block (Box 1), teacher-forced on the workload's first
input (prompt set 0 + the generation length of masks), after 1, 2, 4, 8, 16
layers and the last (32 / 28).  The batch-8 LLaDA-8B workload (8 x 1024
tokens: the large-row GEMM tiles, batched attention and the many-row LM head)
runs its whole batch on the GPU; the oracle follows its sequence 5 (sequences
of a batch do not interact).  The Dream-7B long-context workload (8448 tokens)
runs all 28 layers as well, in four tests of at most eight layers.
The batch-1 workloads run twice: on the plain weights (the LDS-staged GEMM
tiles) and with the packed weight copies the bench decodes with (the
register-direct tiles at these row counts).

Two correct float32 accumulation orders of a bf16 model drift apart by bf16
rounding flips that later layers carry forward; the oracle's own float32 and
float64 runs of each model and input differ by the amounts in
tests/golden/bf16_drift_*.json (one table per workload, written by
make_drift_table.py from the oracle alone).  The bars are derived from that table: the
GPU may differ from the float32 oracle by at most twice the oracle's own
spread (logits), and by at most 2e-2 or twice the table's spread, whichever is
larger (confidences), where the spread at a depth is the largest the table
shows at that depth or any shallower one: rounding drift accumulates with
depth, and the maximum over 32 rows at a single depth is one noisy extreme
(the batch-8 table's confidence spread is 0.014 at depth 4 and 0.011 at 8).
An argmax may differ only where the oracle's top-two logit gap is within twice
the measured logit error.
"""
import json
import os

import numpy as np
import pytest
import torch

from helpers import say, to_np
from oracle import forward as of
from oracle import vocab as ov
from paper_2608_22646_amd import binding as B
from paper_2608_22646_amd import synth

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
CASES = {"llada_b1": ("bf16_drift_llada.json", (1, 2, 4, 8, 16, 32), 0),
         "dream_b1": ("bf16_drift_dream.json", (1, 2, 4, 8, 16, 28), 0),
         "llada_b8": ("bf16_drift_llada_b8.json", (1, 2, 4, 8, 16, 32), 5),
         "dream_long": ("bf16_drift_dream_long.json", (1, 2, 4, 8, 16, 28), 0)}


def drift_table(name):
    path = os.path.join(HERE, "golden", CASES[name][0])
    return {r["depth"]: r for r in json.load(open(path))["rows"]}


def bars(drift, depth):
    rows = [r for d, r in drift.items() if d <= depth]
    logit = max(r["logit_max_abs_diff"] for r in rows)
    conf = max(r["conf_max_abs_diff"] for r in rows)
    return 2.0 * logit, max(2e-2, 2.0 * conf)


class DepthRun:
    """One workload's forward on the GPU (layer calls into one workspace) and
    the oracle's float32 forward of the followed sequence, advanced together;
    the head is compared at every depth of the workload's table."""

    def __init__(self, name, packed):
        self.name, self.packed = name, packed
        self.drift, self.depths, self.seq = drift_table(name), CASES[name][1], CASES[name][2]
        wl = synth.WORKLOADS[name]
        self.cfg = cfg = wl.model
        self.Bn, self.P, G, self.bl = wl.batch, wl.prompt_len, wl.gen_len, wl.block_len
        self.L = L = self.P + G
        say(f"{name} depth parity: weights")
        self.w = w = synth.make_weights(cfg, "cuda")
        self.model = B.Model(cfg, w)
        if packed:
            self.model.pack_weights()
        x = np.concatenate([synth.make_prompts(wl).numpy().astype(np.int64), np.full((self.Bn, G), cfg.mask_id)],
                           axis=1)
        self.ws = self.model.workspace(self.Bn, L, self.bl)
        # layer calls (rows 0) and head calls (rows bl) share h and the RoPE tables
        l0, lb = self.model.layout(self.Bn, L, 0), self.model.layout(self.Bn, L, self.bl)
        assert [getattr(l0, f) for f in ("h", "a_attn", "q", "k", "vt", "attn", "a_mlp", "u")] == \
            [getattr(lb, f) for f in ("h", "a_attn", "q", "k", "vt", "attn", "a_mlp", "u")]
        self.model.embed(torch.from_numpy(x.astype(np.int32)).cuda(), self.ws)
        self.h = to_np(w[0], np.float32)[x[self.seq:self.seq + 1]].astype(np.float64)
        self.cos, self.sin = of.rope_tables(L, cfg.head_dim, cfg.rope_base)
        self.final_norm, self.lm = to_np(w[-2]), to_np(w[-1])
        self.rows = np.arange(self.P, self.P + self.bl)
        self.layers_done = 0
        self.report = []

    def advance(self, to_depth):
        cfg, seq = self.cfg, self.seq
        for l in range(self.layers_done, to_depth):
            self.model.layer(l, 2, self.Bn, self.L, self.ws)
            lw = [to_np(t) for t in self.w[1 + 9 * l: 10 + 9 * l]]
            self.h = of.layer(cfg, lw, self.h, self.cos, self.sin, "bf16")
            del lw
            self.layers_done = depth = l + 1
            if depth not in self.depths:
                continue
            say(f"{self.name}{' packed' if self.packed else ''} depth {depth}: head")
            conf_g, arg_g, lg_g = self.model.head(self.Bn, self.L, self.P, self.bl, self.ws, logits=True)
            torch.cuda.synchronize()
            lg_ref, _ = of.lm_head(cfg, self.h[0, self.rows, :], self.final_norm, self.lm, "bf16")
            conf_ref, arg_ref = ov.confidence_argmax(lg_ref, cfg.mask_id)
            lg = to_np(lg_g[seq], np.float64)
            err = np.abs(lg - lg_ref)
            err[:, cfg.mask_id] = 0
            cerr = np.abs(to_np(conf_g[seq], np.float64) - conf_ref).max()
            bar_l, bar_c = bars(self.drift, depth)
            diff = arg_g[seq].cpu().numpy() != arg_ref
            gap = ov.top2_gap(lg_ref, cfg.mask_id)
            rec = dict(depth=depth, logit_err=float(err.max()), logit_bar=bar_l, conf_err=float(cerr), conf_bar=bar_c,
                       argmax_diff=int(diff.sum()))
            self.report.append(rec)
            say("  " + json.dumps(rec))
            assert err.max() <= bar_l, rec
            assert cerr <= bar_c, rec
            assert np.all(gap[diff] <= 2 * err.max()), rec


@pytest.mark.parametrize("name,packed", [("dream_b1", False), ("dream_b1", True), ("llada_b1", False),
                                         ("llada_b1", True), ("llada_b8", False)])
def test_forward_against_oracle_by_depth(name, packed):
    run = DepthRun(name, packed)
    run.advance(max(run.depths))
    assert [r["depth"] for r in run.report] == list(run.depths)


# The long-context forward in segments of at most eight layers (the oracle
# takes ~11 s per layer there), each its own test, so that every test ends
# within two minutes; a segment whose predecessor did not finish is skipped.
LONG_SEGMENTS = [8, 16, 22, 28]


@pytest.fixture(scope="module")
def long_run():
    state = {}
    yield state
    state.clear()


@pytest.mark.parametrize("to_depth", LONG_SEGMENTS)
def test_long_context_forward_against_oracle_by_depth(long_run, to_depth):
    k = LONG_SEGMENTS.index(to_depth)
    if k == 0:
        long_run["run"] = DepthRun("dream_long", False)
    elif long_run.get("done") != LONG_SEGMENTS[k - 1]:
        pytest.skip("the previous segment of the long-context forward did not finish")
    run = long_run["run"]
    run.advance(to_depth)
    long_run["done"] = to_depth
    if to_depth == LONG_SEGMENTS[-1]:
        assert [r["depth"] for r in run.report] == list(run.depths)
        long_run.clear()
