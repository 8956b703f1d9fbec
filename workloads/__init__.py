"""Seeded synthetic inputs for the verification step: model shapes, random-init
bf16 weights, contexts and drafts with planted acceptance.

This package holds no arithmetic of the method itself (no forward pass, no
argmax, no acceptance rule).  It only draws numbers and arranges tokens.  Both
the CPU oracle and the GPU library consume what it produces; neither imports
the other.
"""

from .configs import ModelConfig, TINY, SHAPE_8B, SHAPE_32B, config_by_name  # noqa: F401
from .weights import (  # noqa: F401
    canonical_tensors,
    make_tensor,
    make_weights,
    f32_to_bf16_bits,
)
from . import tokens  # noqa: F401
from . import batches  # noqa: F401
from . import trees  # noqa: F401
