"""MI355X-native SOMA SPSA hot path (arXiv 2609.37899).

The compute path is the C-ABI library ``libsoma.so`` (hand-written HIP for
gfx950) behind the thin ctypes binding in :mod:`paper_2609_37899_amd.soma`.
PyTorch supplies device memory and streams only.
"""
__all__ = ["soma", "synth", "workloads"]
