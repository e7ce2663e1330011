"""The five synthetic workloads, named by what they are.

Each entry fixes shapes, group size, budget law, temperature and seed key.
Projection shapes are (d_out, d_in) in the nn.Linear convention; groups are
1 x g blocks of consecutive input columns of one output row (Sec. 2.1).
"""
from __future__ import annotations

LLAMA2_7B_LINEARS = [  # one decoder layer, (name, d_out, d_in)
    ("q", 4096, 4096), ("k", 4096, 4096), ("v", 4096, 4096), ("o", 4096, 4096),
    ("gate", 11008, 4096), ("up", 11008, 4096), ("down", 4096, 11008),
]
LLAMA2_13B_LINEARS = [
    ("q", 5120, 5120), ("k", 5120, 5120), ("v", 5120, 5120), ("o", 5120, 5120),
    ("gate", 13824, 5120), ("up", 13824, 5120), ("down", 5120, 13824),
]

CONFIGS = {
    # Single masked linear, fwd + bwd, hard mask with exactly half the groups kept.
    "single_1024": dict(id=1, T=128, linears=[("w", 1024, 1024)], g=256, tau=0.5,
                        law=("fixed", 0.5), layers=1),
    # LLaMA-2-7B attention-projection shape, 2 sequences x 2048 tokens.
    "attn_4096": dict(id=2, T=4096, linears=[("q", 4096, 4096)], g=256, tau=0.4,
                      law=("fixed", 0.5), layers=1),
    # LLaMA-2-7B MLP trio with per-matrix sparsity ~ U(0.3, 0.7).
    "mlp_trio_7b": dict(id=3, T=4096, linears=LLAMA2_7B_LINEARS[4:], g=256, tau=0.4,
                        law=("uniform", 0.3, 0.7), layers=1),
    # Every masked linear of LLaMA-2-7B (32 layers x 7), Beta(2,2) budgets rescaled to 50 %.
    "llama2_7b_step": dict(id=4, T=4096, linears=LLAMA2_7B_LINEARS, g=256, tau=0.4,
                           law=("beta", 0.5), layers=32),
    # LLaMA-2-13B shapes for the pruned-model inference path and the group-size sweep.
    "llama2_13b_infer": dict(id=5, T_decode=(1, 8, 16, 512), T_sweep=8192,
                             linears=LLAMA2_13B_LINEARS, g=256, g_sweep=(64, 128, 256, 512),
                             tau=0.4, law=("fixed", 0.5), layers=40),
}


def config(name: str) -> dict:
    return dict(CONFIGS[name])
