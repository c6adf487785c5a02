"""Seeded synthetic inputs for the KV-cache reconstruction path.

This package holds the model-shape presets and the deterministic input
generators (weights, token ids, block tables, synthetic KV pools).  It holds
none of the method's arithmetic: no normalisation, projection, attention,
copy or assembly.  Both the HIP path (through ``paper_2608_16477_amd``) and
the CPU oracle (through the tests) consume the tensors it produces.
"""
from .configs import ModelConfig, Workload, PRESETS, preset, workload  # noqa: F401
from . import gen  # noqa: F401
