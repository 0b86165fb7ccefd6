"""Seeded synthetic workloads and inputs shared by the oracle tests, the GPU
tests and the benchmark.  Input generation only: no arithmetic of the
training step lives here."""
from .workloads import Workload, PartySpec, TopSpec, get, ALL  # noqa: F401
from .data import generate, init_params, group_rows, to_bf16_values  # noqa: F401
