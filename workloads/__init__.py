"""Seeded synthetic workloads shared by the tests, the bench and the oracle checks."""
from .synth import (CONFIGS, DESCRIPTIONS, GENERATOR_VERSION, Config, Workload,
                    get_config, input_digest, make_logp_pair, make_workload)

__all__ = ["CONFIGS", "DESCRIPTIONS", "GENERATOR_VERSION", "Config", "Workload",
           "get_config", "input_digest", "make_logp_pair", "make_workload"]
