"""SkewAdam optimizer step for AMD Instinct MI355X (gfx950): HIP kernels behind a C ABI."""
from .skewadam import (BACKBONE, EXPERT, ROUTER, TIERS, STATE_MOMENTUM, STATE_FACTORED,  # noqa: F401
                       SkewAdam, SkewError, HParams, TensorDesc, lib, make_desc, state_bytes)
