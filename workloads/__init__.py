"""Seeded synthetic inputs shared by the oracle tests, the GPU tests and the bench.

This package holds only input generation: network shapes, seeded weight blobs,
latents, contexts and timestep schedules. None of the method's arithmetic (the
velocity network, the Euler update, the queue shift) lives here; the oracle and
the HIP library each implement that on their own.
"""
from .configs import CONFIGS, Config, get_config
from .blob import HEADER_FMT, HEADER_SIZE, MAGIC, VERSION, tensor_specs, write_blob
from .gen import (make_weights, make_blob, latents, z_new_for_image, context,
                  null_context, schedule, slot_times)

__all__ = [
    "CONFIGS", "Config", "get_config", "HEADER_FMT", "HEADER_SIZE", "MAGIC", "VERSION",
    "tensor_specs", "write_blob", "make_weights", "make_blob", "latents",
    "z_new_for_image", "context", "null_context", "schedule", "slot_times",
]
