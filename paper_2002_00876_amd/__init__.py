"""MI355X-native batched linear-chain CRF inference (log-partition, edge marginals,
Viterbi) as a log-depth tree of semiring matrix products, after Torch-Struct
(Rush 2020, Sec. 5.2 and 6a).  The compute runs in hand-written HIP kernels for
gfx950 behind the C ABI declared in include/ts_chain.h; ``binding`` is the thin
Python layer over that library (it imports torch lazily)."""
from . import workloads  # noqa: F401
