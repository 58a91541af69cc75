"""libmesa: the chunkwise-parallel Mesa layer (MesaNet, arXiv 2506.05233) on MI355X.

The layer runs in hand-written HIP kernels behind the C ABI of
``include/libmesa.h``; ``paper_2506_05233_amd.libmesa`` is its thin Python
binding and ``paper_2506_05233_amd.workloads`` the seeded input generator.
"""
from . import libmesa, workloads  # noqa: F401
from .libmesa import decode_step, forward, prefill_states  # noqa: F401

__all__ = ["libmesa", "workloads", "forward", "decode_step", "prefill_states"]
