"""Seeded synthetic inputs (no method arithmetic) for tests, bench and smoke."""
from .workloads import (WORKLOADS, LayerInputs, Layout, Workload, bf16_bits,  # noqa: F401
                        bf16_bits_to_f32, make_layer, make_layout, make_scores,
                        scaled)
