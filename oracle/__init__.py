"""CPU oracle of request batching (paper section 2.2.1): test infrastructure.

Plain, slow, fp64 reference of what the batched inference path computes:
batch formation, padding, round-robin dispatch on a simulated clock, row
routing, and the served models' forward passes run one request at a time.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this package. The product path (the HIP library and its binding) never
imports, links or runs it, and shares no code with it; the two meet only in
the seeded input generators of the `synth` package.
"""
from . import batching, models, numerics  # noqa: F401
