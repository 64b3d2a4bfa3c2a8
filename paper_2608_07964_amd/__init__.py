"""EasyBalance hot path on AMD Instinct MI355X (gfx950).

Cross-layer load balancing for expert-parallel MoE inference (arXiv
2608.07964): a greedy scheduler picks which micro-batches run their MoE layer
now and which wait, and the chosen micro-batches -- each at its own layer --
run their expert FFNs jointly in one grouped launch.

* ``binding``  -- ctypes binding of libeasybalance.so (include/easybalance.h)
* ``driver``   -- Algorithm 1 on one GPU over the C ABI
* ``build``    -- hipcc build of the library
"""
from . import binding  # noqa: F401

__all__ = ["binding"]
