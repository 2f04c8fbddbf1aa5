"""Token confidence and greedy prediction over the vocabulary (oracle).

Box 1 (Token Confidence) defines c_i = max_v p(x_i = v | x); Box 5 and
Algorithm 1 commit x_i = argmax_v p(x_i = v | x) at temperature 0 (Section 5).
Reading used here: the mask token itself is never a prediction (its logit is
removed before the softmax), and ties go to the lowest vocabulary index.

Test infrastructure only; see the package docstring.
"""
import numpy as np


def confidence_argmax(logits, mask_id):
    """logits [..., V] -> (conf float64 [...], argmax int64 [...]).

    softmax over v != mask_id, evaluated in float64:
      m = max_v l_v,  conf = max_v p_v = exp(m - m) / sum_v exp(l_v - m) = 1 / sum_v exp(l_v - m).
    """
    l = np.array(logits, dtype=np.float64, copy=True)
    l[..., mask_id] = -np.inf
    m = l.max(axis=-1, keepdims=True)
    z = np.exp(l - m).sum(axis=-1)
    conf = 1.0 / z
    arg = np.argmax(l, axis=-1)          # first maximal index
    return conf, arg.astype(np.int64)


def top2_gap(logits, mask_id):
    """logits [..., V] -> float64 [...]: the largest logit over v != mask_id minus
    the largest logit of any other index v != mask_id (0 at a tie for the top,
    +inf when only one finite candidate exists).

    Used to excuse near-ties: if two logit rows differ by at most e in every
    entry, their argmaxes can differ only where this gap is at most 2 e."""
    l = np.array(logits, dtype=np.float64, copy=True)
    l[..., mask_id] = -np.inf
    part = np.sort(l, axis=-1)
    return part[..., -1] - part[..., -2]
