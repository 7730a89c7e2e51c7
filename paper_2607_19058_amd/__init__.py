"""SkewAdam optimizer step for AMD Instinct MI355X (gfx950): HIP kernels behind a C ABI."""
from .skewadam import (BACKBONE, EXPERT, ROUTER, TIERS, SkewAdam, SkewError, HParams, TensorDesc,  # noqa: F401
                       lib, make_desc, state_bytes)
