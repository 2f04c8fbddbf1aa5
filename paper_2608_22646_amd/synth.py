"""Seeded synthetic inputs shared by the HIP path, the tests and the oracle.

This module holds model shapes, workload shapes and seeded random draws only:
no step of the decoding method is computed here.  Both sides of every parity
check receive the tensors made here; neither side generates its own.

Shapes follow the two model families the paper evaluates (LLaDA-8B and
Dream-7B, Section 5 "Setup"); the paper prints no architecture, so the
dimensions are the public shapes of those checkpoints.  Weights are random
(no checkpoint is available), drawn from N(0, std^2) per tensor with a seed
derived from the tensor's index in the fixed weight order below.  The paper
fixes NumPy/torch seeds at 1234 (Appendix A, "Benchmark Sample Sizes" and
seeds paragraph); tensor i uses seed 1234 + i.  Prompts are uniform token ids
in [0, vocab-2] (the mask id is vocab-1), seeded 0 + sequence index.

Weight order (``weight_specs``): embed [V,d]; per layer: attn_norm [d],
wq [Hq*hd, d], wk [Hkv*hd, d], wv [Hkv*hd, d], wo [d, Hq*hd], mlp_norm [d],
w_gate [F, d], w_up [F, d], w_down [d, F]; then final_norm [d], lm_head [V, d].
Linear weights are [out, in] row-major (the reduction dimension contiguous).
"""
from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass, field

import torch

WEIGHT_SEED_BASE = 1234
PROMPT_SEED_BASE = 0
PER_LAYER = ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "w_gate", "w_up", "w_down")


@dataclass(frozen=True)
class ModelConfig:
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    rope_base: float
    dtype: str                # "f32" or "bf16": storage type of weights and GEMM operands
    rms_eps: float = 1e-5
    linear_std: float = 0.02
    lm_head_std: float = 0.02
    norm_gain_std: float = 0.0  # 0: gains are exactly 1; >0: 1 + N(0, std^2) (tests only)

    @property
    def mask_id(self) -> int:
        return self.vocab - 1

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    @property
    def n_weights(self) -> int:
        return 3 + len(PER_LAYER) * self.n_layers

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    def param_count(self) -> int:
        return sum(math.prod(s) for _, s, _ in weight_specs(self))


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelConfig
    batch: int
    prompt_len: int
    gen_len: int
    block_len: int = 32
    gating: bool = True        # confidence gating (token budgets + grinding fallback)

    @property
    def seq_len(self) -> int:
        return self.prompt_len + self.gen_len

    @property
    def n_blocks(self) -> int:
        return self.gen_len // self.block_len


def weight_specs(cfg: ModelConfig):
    """[(name, shape, std)] in the fixed weight order; std None means a norm gain."""
    d, F, V = cfg.d_model, cfg.d_ff, cfg.vocab
    specs = [("embed", (V, d), cfg.linear_std)]
    for l in range(cfg.n_layers):
        specs += [
            (f"l{l}.attn_norm", (d,), None),
            (f"l{l}.wq", (cfg.q_dim, d), cfg.linear_std),
            (f"l{l}.wk", (cfg.kv_dim, d), cfg.linear_std),
            (f"l{l}.wv", (cfg.kv_dim, d), cfg.linear_std),
            (f"l{l}.wo", (d, cfg.q_dim), cfg.linear_std),
            (f"l{l}.mlp_norm", (d,), None),
            (f"l{l}.w_gate", (F, d), cfg.linear_std),
            (f"l{l}.w_up", (F, d), cfg.linear_std),
            (f"l{l}.w_down", (d, F), cfg.linear_std),
        ]
    specs += [("final_norm", (d,), None), ("lm_head", (V, d), cfg.lm_head_std)]
    return specs


def make_weight(cfg: ModelConfig, i: int, device="cpu"):
    """Tensor i of the fixed order (seed 1234 + i), stored in ``cfg.torch_dtype``.

    Draws use torch's generator for ``device`` (the CPU and GPU generators give
    different streams; a parity test always hands the same tensors to both
    sides).  bf16 storage rounds the fp32 draw to nearest-even.
    """
    _, shape, std = weight_specs(cfg)[i]
    g = torch.Generator(device=device)
    g.manual_seed(WEIGHT_SEED_BASE + i)
    if std is None:
        if cfg.norm_gain_std > 0:
            w = 1.0 + cfg.norm_gain_std * torch.randn(shape, generator=g, device=device)
        else:
            w = torch.ones(shape, device=device)
    else:
        w = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
        w.mul_(std)
    return w.to(cfg.torch_dtype).contiguous()


def make_weights(cfg: ModelConfig, device="cpu"):
    """Every tensor of the fixed order (make_weight)."""
    return [make_weight(cfg, i, device) for i in range(cfg.n_weights)]


def make_prompts(wl: Workload, device="cpu", first=0):
    """int32 [B, P]: sequence b drawn uniformly from [0, vocab-2] with seed first + b
    (first = 0: the workload's prompts; other values give further prompt sets)."""
    rows = []
    for b in range(wl.batch):
        g = torch.Generator(device="cpu")
        g.manual_seed(PROMPT_SEED_BASE + first + b)
        rows.append(torch.randint(0, wl.model.vocab - 1, (wl.prompt_len,), generator=g, dtype=torch.int64))
    return torch.stack(rows).to(torch.int32).to(device)


def make_uniform(shape, seed, lo=0.0, hi=1.0, dtype=torch.float32, device="cpu"):
    """Seeded uniform draws (controller traces, kernel parity inputs)."""
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    return (lo + (hi - lo) * torch.rand(shape, generator=g, dtype=torch.float64)).to(dtype).to(device)


def make_normal(shape, seed, std=1.0, dtype=torch.float32, device="cpu"):
    """Seeded normal draws for kernel parity inputs (generated on the CPU)."""
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    return (std * torch.randn(shape, generator=g, dtype=torch.float32)).to(dtype).to(device)


def make_ints(shape, seed, lo, hi, device="cpu"):
    """Seeded uniform integers in [lo, hi) as int32."""
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    return torch.randint(lo, hi, shape, generator=g, dtype=torch.int64).to(torch.int32).to(device)


# ---------------------------------------------------------------------------
# The five workloads.  LLaDA-style heads use an LM-head std of 5/sqrt(d) so that
# logits have std ~5 and first-step confidences spread over all three budget
# tiers; the Dream-shaped models use N(0, 0.02^2) for every linear, lm_head
# included, as their description states.
# ---------------------------------------------------------------------------
TINY = ModelConfig("tiny-llada", n_layers=2, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64,
                   d_ff=704, vocab=2048, rope_base=10000.0, dtype="f32",
                   lm_head_std=5.0 / math.sqrt(256))
LLADA_8B = ModelConfig("llada-8b-shape", n_layers=32, d_model=4096, n_heads=32, n_kv_heads=32,
                       head_dim=128, d_ff=12288, vocab=126464, rope_base=500000.0, dtype="bf16",
                       lm_head_std=5.0 / math.sqrt(4096))
DREAM_7B = ModelConfig("dream-7b-shape", n_layers=28, d_model=3584, n_heads=28, n_kv_heads=4,
                       head_dim=128, d_ff=18944, vocab=152064, rope_base=1000000.0, dtype="bf16",
                       lm_head_std=0.02)

WORKLOADS = {
    "tiny": Workload("tiny", TINY, batch=1, prompt_len=32, gen_len=64, gating=True),
    "llada_b1": Workload("llada_b1", LLADA_8B, batch=1, prompt_len=256, gen_len=256, gating=True),
    "llada_b8": Workload("llada_b8", LLADA_8B, batch=8, prompt_len=512, gen_len=512, gating=True),
    "dream_b1": Workload("dream_b1", DREAM_7B, batch=1, prompt_len=512, gen_len=256, gating=False),
    "dream_long": Workload("dream_long", DREAM_7B, batch=1, prompt_len=8192, gen_len=256, gating=False),
}


def reduced(cfg: ModelConfig, **kw) -> ModelConfig:
    """A copy of ``cfg`` with some fields replaced (fewer layers for sampled parity runs)."""
    return dataclasses.replace(cfg, **kw)
