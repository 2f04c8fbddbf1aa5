"""Writes tests/golden/bf16_drift_llada.json (bf16_drift_dream.json with
--workload dream_b1, bf16_drift_llada_b8.json with --workload llada_b8,
bf16_drift_dream_long.json with --workload dream_long): how
far the oracle's own bf16 forward moves between float32 and float64
accumulation, by depth, at the LLaDA-8B (Dream-7B) shape.

A bf16 model rounds every matrix-product operand to bf16 (the oracle's "bf16"
mode).  Two correct implementations whose float32 sums differ in the last bit
round a few activations to the neighbouring bf16 value; later layers carry
those steps forward.  This script measures that spread with the oracle alone:
the same model and input through mode "bf16" (float32 products) and mode
"bf16_f64acc" (float64 products, same rounding points), the block's logits and
confidences (Box 1) compared after 1, 2, 4, 8, 16 and 32 layers.  The GPU's
end-to-end bar is derived from this table.

Input: the workload's model with weights drawn by torch's CPU generator
(seed 1234 + tensor index; the GPU tests draw theirs with the GPU generator, a
different stream of the same distribution), one sequence of its prompt set 0
(the first; sequence 5 of the eight for llada_b8) followed by its generation
length of mask tokens (LLaDA-8B: 256 + 256, batch 8: 512 + 512; Dream-7B: 512 +
256), the head on the first generated block (32 rows).  Sequences of a batch
do not interact, so one sequence stands for the batch.  Calls only oracle/ and
the seeded input generators.

  python tests/golden/make_drift_table.py [--workload llada_b1] [--depths 1,2,4,8,16,32]
  python tests/golden/make_drift_table.py --workload dream_b1 --depths 1,2,4,8,16,28
  python tests/golden/make_drift_table.py --workload llada_b8
  python tests/golden/make_drift_table.py --workload dream_long --depths 1,2
"""
import argparse
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from oracle import forward as of  # noqa: E402
from oracle import vocab as ov  # noqa: E402
from paper_2608_22646_amd import synth  # noqa: E402

OUTS = {"llada_b1": os.path.join(HERE, "bf16_drift_llada.json"),
        "dream_b1": os.path.join(HERE, "bf16_drift_dream.json"),
        "llada_b8": os.path.join(HERE, "bf16_drift_llada_b8.json"),
        "dream_long": os.path.join(HERE, "bf16_drift_dream_long.json")}
SEQ = {"llada_b1": 0, "dream_b1": 0, "llada_b8": 5, "dream_long": 0}  # the sequence of the batch the table follows
OUT = OUTS["llada_b1"]
MODES = ("bf16", "bf16_f64acc")
DEFAULT_DEPTHS = "1,2,4,8,16,32"


def drift(depths, log=print, workload="llada_b1", checkpoint=None):
    wl = synth.WORKLOADS[workload]
    cfg = wl.model
    P, G, bl = wl.prompt_len, wl.gen_len, wl.block_len
    L = P + G
    seq = SEQ[workload]
    x = np.concatenate([synth.make_prompts(wl).numpy().astype(np.int64)[seq:seq + 1], np.full((1, G), cfg.mask_id)],
                       axis=1)
    host = lambda i: synth.make_weight(cfg, i).float().numpy()  # noqa: E731
    h0 = host(0)[x].astype(np.float64)
    h = {m: h0.copy() for m in MODES}
    cos, sin = of.rope_tables(L, cfg.head_dim, cfg.rope_base)
    final_norm, lm = host(cfg.n_weights - 2), host(cfg.n_weights - 1)
    rows = np.arange(P, P + bl)
    out = []
    t0 = time.time()
    for l in range(max(depths)):
        w = [host(i) for i in range(1 + 9 * l, 10 + 9 * l)]
        for m in MODES:
            h[m] = of.layer(cfg, w, h[m], cos, sin, m)
        del w
        if l + 1 not in depths:
            continue
        lg, conf, arg = {}, {}, {}
        for m in MODES:
            lg[m], _ = of.lm_head(cfg, h[m][0, rows, :], final_norm, lm, m)
            conf[m], arg[m] = ov.confidence_argmax(lg[m], cfg.mask_id)
        d = np.abs(lg["bf16"] - lg["bf16_f64acc"])
        d[:, cfg.mask_id] = 0
        hd = np.abs(h["bf16"][0] - h["bf16_f64acc"][0])
        rec = {
            "depth": l + 1,
            "logit_max_abs_diff": float(d.max()),
            "logit_p999_abs_diff": float(np.quantile(d, 0.999)),
            "logit_std": float(lg["bf16_f64acc"].std()),
            "conf_max_abs_diff": float(np.abs(conf["bf16"] - conf["bf16_f64acc"]).max()),
            "argmax_differs": int((arg["bf16"] != arg["bf16_f64acc"]).sum()),
            "hidden_max_abs_diff": float(hd.max()),
            "hidden_max_abs": float(np.abs(h["bf16_f64acc"][0]).max()),
        }
        out.append(rec)
        log(f"[drift] {time.time() - t0:.0f}s " + json.dumps(rec))
        if checkpoint:
            checkpoint(out)
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="llada_b1", choices=sorted(OUTS))
    ap.add_argument("--depths", default=DEFAULT_DEPTHS)
    a = ap.parse_args()
    depths = sorted({int(v) for v in a.depths.split(",")})
    wl = synth.WORKLOADS[a.workload]

    def write(table):  # after every depth, so that a long run keeps what it has measured
        doc = {
            "what": ("max |difference| between the oracle's bf16-model forward with float32 and with float64 "
                     f"accumulation (same bf16 rounding points), {shape} shape, sequence {SEQ[a.workload]} of prompt "
                     f"set 0 + {wl.gen_len} masks, first block's 32 rows; logits exclude the mask column"),
            "generator": "tests/golden/make_drift_table.py" + ("" if a.workload == "llada_b1" else
                                                                f" --workload {a.workload}")
                         + ("" if a.depths == DEFAULT_DEPTHS else f" --depths {a.depths}"),
            "rows": table,
        }
        with open(OUTS[a.workload], "w") as f:
            json.dump(doc, f, indent=1)

    shape = {"llada_b1": "LLaDA-8B", "dream_b1": "Dream-7B", "llada_b8": "LLaDA-8B", "dream_long": "Dream-7B"}[
        a.workload]
    drift(depths, log=lambda s: print(s, flush=True), workload=a.workload, checkpoint=write)
    print(OUTS[a.workload])


if __name__ == "__main__":
    main()
