"""Seeded synthetic workloads for the DASC checkpoint path.

This package only draws random numbers and shapes them into the tensors both
sides consume (the oracle on the host, the HIP library on the device).  It holds
none of the method's arithmetic: no horizon, no selection, no packing, no
recurrence.  See ``workloads.synth`` for the recipes.
"""

from .synth import (  # noqa: F401
    Workload,
    WORKLOADS,
    bf16_bits_from_f32,
    f32_from_bf16_bits,
    log_lambda,
    refresh_inputs,
    refresh_inputs_device,
    states_host,
    states_device,
    streams,
)
