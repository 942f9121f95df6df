"""MI355X-native (gfx950) implementation of the reconcile hot path of
Controlled Periodic Data Parallelism (CPDP) with SlowMo.

Submodules
  cpdp   ctypes binding of the C ABI in include/cpdp.h (libcpdp.so)
  state  HBM-resident replica state (flat layout), the host cadence driving
         it, step tables and HIP-graph capture, checkpoint/resume
  multi  the same for a model held as separate tensors (multi-tensor plans)
  build  hipcc build of the shared libraries

Importing ``cpdp`` (directly or through ``state``) raises ImportError when the
HIP library is not built: there is no CPU fallback.
"""
__all__ = ["cpdp", "state", "multi", "build"]
