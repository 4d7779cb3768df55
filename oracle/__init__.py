"""Float64 CPU oracle of the encoder layer (test infrastructure only).

Only the tests, the smoke check and the CPU-baseline leg of the benchmark
import this package.  The product library never does.
"""
from .encoder_layer import *  # noqa: F401,F403
from .encoder_layer import __all__ as _layer_all
from .parallel_layer import *  # noqa: F401,F403
from .parallel_layer import __all__ as _parallel_all
from . import schedule, vit_encoder  # noqa: F401

__all__ = list(_layer_all) + list(_parallel_all) + ["schedule", "vit_encoder"]
