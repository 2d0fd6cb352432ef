"""SideQuest KV-cache hot path for MI355X (gfx950).

The library (``libsq.so``: C++ host code plus hand-written HIP kernels,
declared in ``include/sq.h``) holds a paged KV cache shared by a main
reasoning thread and its forked auxiliary threads, evicts the token spans of
stale tool responses, and runs decode-step attention over the result.
``sq`` is its ctypes binding; ``workload`` builds seeded synthetic
agent-shaped inputs; ``build_lib`` compiles the library in-tree.
"""

__all__ = ["sq", "workload", "build_lib"]
