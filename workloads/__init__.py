"""Seeded synthetic inputs shared by the oracle and the HIP path (no method arithmetic)."""
from .gen import (Workload, WorkloadSpec, TaskSpec, config, config_spec, config_seed, make,
                  build_structure, build_tensors, small_spec, bernoulli, uniform01, normal,
                  constant)
