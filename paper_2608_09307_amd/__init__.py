"""MI355X-native LinSimp (Linearized 2-Simplicial Attention) core.

``linsimp`` is the ctypes binding of the HIP library built by ``build``;
``workloads`` draws the seeded synthetic inputs.
"""

__all__ = ["linsimp", "workloads", "build"]
