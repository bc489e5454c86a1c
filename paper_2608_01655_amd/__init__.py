"""MI355X (gfx950) implementation of the PrefixPlace planner hot path.

The compute path is libprefixplace.so (HIP kernels + C ABI, see
include/prefixplace.h); `binding` marshals arguments to it and `workloads`
draws seeded synthetic inputs.
"""

from . import binding  # noqa: F401
