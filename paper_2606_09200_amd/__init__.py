"""MI355X-native hot path of resource-aware computation/communication overlap.

The product is the C-ABI library ``libocc.so`` (``include/occ.h``) built from
``csrc/`` for gfx950; :mod:`.binding` exposes its entry points to Python with
the same names.  :mod:`.inputs` draws the seeded synthetic operands and
:mod:`.workloads` names the measured configurations.
"""
__all__ = ["binding", "inputs", "workloads"]
