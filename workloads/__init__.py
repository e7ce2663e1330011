"""Seeded synthetic inputs for the group-masked linear layer.

This module is shared by the tests, the benchmark and the oracle checks.  It
holds no arithmetic of the method itself: it only draws random numbers,
rounds them to the storage formats the layer consumes (bf16 bit patterns,
fp32) and picks which groups are kept.  Gate noise is drawn as the uniform
variate ``u`` that the gate consumes, never transformed here.

Shapes follow the paper's workloads: LLaMA-2-7B / 13B projection shapes, token
counts that are multiples of the 2048-token calibration length (Appendix A),
1x256 groups along the input dimension (Table 5) and a 50 % budget (Table 5),
with per-matrix budgets that vary around the global one (layer-adaptive
allocation, Sec. 2.3).
"""
from .gen import (  # noqa: F401
    SEED,
    bf16_bits_from_f32,
    f32_from_bf16_bits,
    draw_uniform_noise,
    budgeted_gate_inputs,
    independent_gate_inputs,
    random_kept_mask,
    kept_counts_uniform_law,
    kept_counts_beta_law,
    LinearCase,
    make_linear_case,
    DistillCase,
    make_distill_case,
    HyperCase,
    make_hyper_case,
)
from .configs import CONFIGS, LLAMA2_7B_LINEARS, LLAMA2_13B_LINEARS, config  # noqa: F401
