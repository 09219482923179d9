"""MI355X (gfx950) ROCKET transform: HIP kernels behind a C ABI (include/rocket.h).

Python-side entry points (argument marshalling over ctypes):
    generate_kernels(seed, n_kernels, input_length) -> dict of numpy arrays
    Plan(kernels, L)  .transform(X) / .transform_into(X, F) / .info()
    transform(X, kernels)  one-shot
The seeded synthetic series live in ``paper_2601_17091_amd.workloads``.
"""
from .rocket import (EXPORTED, Plan, RocketError, generate_kernels, generate_kernels_multi, library,  # noqa: F401
                     status_string,
                     plan_tables, transform, transform_batched)
