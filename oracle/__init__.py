"""CPU oracle for the centroid + residual LoRA apply (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline``
leg may import this package.  The product path never imports or calls it.
"""
from .ref import (adapter_bytes, align_loss, apply, decode, fuse_centroid, plan, route,  # noqa: F401
                  route_decide, update_terms)
