"""Seeded synthetic workloads shared by the oracle tests, the GPU tests and the benchmark.

This package holds shapes, random draws and input synthesis only (Gaussian Q/K/V, 3D rotary
position embedding, bf16 rounding, uniform stripe-parameter draws).  It contains none of the
stripe-mask or attention arithmetic: density-targeted stripe parameters are read from
``stripe_params.json``, which ``make_stripe_params.py`` writes by calling the oracle.
"""
from .configs import CONFIGS, Config, get_config  # noqa: F401
from .inputs import bf16_round, bf16_bits, make_head_qkv, make_qkv  # noqa: F401
from .params import STRIDE_INF, stripe_params  # noqa: F401
