"""Cross-mesh resharding on one MI355X: C-ABI library + thin binding.

See include/reshard.h for the boundary.  ``binding`` wraps libreshard.so,
``workloads`` holds the seeded synthetic inputs, ``build`` compiles the
library in-tree for gfx950.
"""

__version__ = "0.1.0"
