"""Seeded synthetic inputs for the BinaryPC decode path.

This package only draws random numbers and lays them out; it holds none of
the method's arithmetic, so both the CPU oracle (through the tests) and the
HIP path (through the tests and the benchmark) consume the same inputs.
"""

from .synth import (  # noqa: F401
    CONFIGS,
    DecodeConfig,
    config_by_name,
    make_calibration_keys,
    make_gaussian_directions,
    make_layer,
)
