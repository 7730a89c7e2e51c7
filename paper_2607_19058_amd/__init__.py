"""SkewAdam optimizer step for AMD Instinct MI355X (gfx950): HIP kernels behind a C ABI."""
from .skewadam import (BACKBONE, EXPERT, ROUTER, TIERS, STATE_MOMENTUM, STATE_FACTORED, STATE_FP32,  # noqa: F401
                       FLAG_EXACT_CLIP, FLAG_EXACT_ULP, SkewAdam, SkewError, HParams, TensorDesc, lib, make_desc,
                       state_bytes)
