"""CPU oracle for the JAGG group backward (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It is a plain numpy implementation,
fp64 by default, written from the paper: ``mmdit`` holds the network forward
and its parameter VJP, ``jagg`` the interpolation weights, composites, group
gradients, routing, group scores and the linear toy of Theorem 1, ``grpo``
the per-step GRPO upstream gradients of Phase 2 and their composites.  It shares
no code with the HIP library and imports nothing from it.

Parity status: every function is pinned by the oracle tests except the
forward values of the random MMDiT as a whole, which no paper value fixes
("parity unpinned" beyond the per-operator library checks, the closed-form
special cases and finite-difference consistency of the VJP).
"""
from . import grpo, jagg, mmdit  # noqa: F401
