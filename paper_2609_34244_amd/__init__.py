"""MI355X (gfx950) batched plan pricing: PartitionLayers + Evaluate + argmin
of Heddle's profile-based cost model, as hand-written HIP kernels behind a C
ABI (include/heddle.h). ``heddle`` is the ctypes binding."""
from . import heddle  # noqa: F401
