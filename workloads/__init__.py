"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle checks."""
from .synth import (Workload, WorkloadSpec, build_workload, config_spec, gather_unit,  # noqa: F401
                    make_workload)
