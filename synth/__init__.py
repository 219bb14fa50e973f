"""Seeded synthetic models and request inputs shared by the oracle and the HIP path.

This package only draws numbers and lays bytes out. It holds none of the method's
arithmetic: no layer, no activation, no swap or placement rule. Both sides of a
parity test receive exactly the bytes produced here.
"""
from .models import (  # noqa: F401
    ALIGN, Tensor, Model, mlp, resnet50, bert, config_model, CONFIG_SEEDS,
    bf16_round, bf16_to_f32, mlp_input, resnet_input, bert_input, config_input,
)
from .tenants import tenant_models, tenant_trace, build_models, request_input  # noqa: F401,E402
