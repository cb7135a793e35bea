"""Seeded synthetic inputs shared by the tests, the smoke check and the bench.

Holds no attention arithmetic: only forest structure, page placement, random
values and NaN poisoning of memory the method must never read.
"""

from .synth import (  # noqa: F401
    CONFIG_NAMES,
    Workload,
    build_workload,
    make_config,
    random_forest,
)
