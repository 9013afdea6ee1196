"""Seeded synthetic inputs (scenes, query banks, decoder weights) for the Rift
hot path.  Shared by the GPU tests, the bench and the oracle's tests; holds no
arithmetic of the method itself."""
from .configs import WORKLOADS, Workload, ModelShape, get  # noqa: F401
from .scene import (Scene, make_scene, make_query_bank, make_layer, weight_shapes,  # noqa: F401
                    WEIGHT_NAMES, round_bf16, bf16_to_f32, to_f64, store)
