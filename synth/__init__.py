"""Seeded synthetic inputs shared by the oracle and the GPU path (random draws only)."""
from .workloads import (WORKLOADS, Arenas, Layer, Model, Params, Payload, Queue, Trace, Workload,
                        arenas, model_params, next_version, poisson_arrivals, request_payload, trace, workload)
