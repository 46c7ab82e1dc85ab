"""MI355X (gfx950) streaming-MoE decode hot path: HIP kernels behind a C ABI.

``libmoe.so`` (built from ``csrc/`` by :mod:`.build`) holds every step of the
path; :mod:`.binding` marshals torch device tensors into its C calls.
"""

from . import binding  # noqa: F401
from .binding import MoeError, SlotTable, make_spec, spec_from_workload  # noqa: F401
