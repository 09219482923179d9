"""MI355X (gfx950) ROCKET transform: HIP kernels behind a C ABI (include/rocket.h).

Python-side entry points (argument marshalling over ctypes):
    generate_kernels(seed, n_kernels, input_length) -> dict of numpy arrays
    Plan(kernels, L)  .transform(X) / .transform_into(X, F) / .info()
    transform(X, kernels)  one-shot
    minirocket_fit(X_train, num_features, seed) -> MINIROCKET parameters
    MiniRocketPlan(params)  .transform(X): PPV features [n, n_features]
The seeded synthetic series live in ``paper_2601_17091_amd.workloads``.
With ROCKET_DEBUG=1 in the environment the checked build is loaded
(librocket_checked.so: device-side bounds checks, see check_flags).
"""
from .rocket import (EXPORTED, MiniRocketPlan, Plan, RocketError, check_flags, checked_build,  # noqa: F401
                     generate_kernels, generate_kernels_multi, library, library_at, minirocket_fit,
                     plan_tables, status_string, transform, transform_batched)
