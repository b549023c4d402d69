"""MI355X (gfx950) implementation of the GPU-resident query path of Chimera's
multi-vector retrieval: IVF probe on MFMA, candidate generation, partial-score
refinement, residual-code document scoring and top-k, behind the C ABI in
``include/chimera.h``."""
from .chimera import (BF16, F32, Builder, ChimeraError, Index, build_index, last_error, lib)  # noqa: F401
