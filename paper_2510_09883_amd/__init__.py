"""DELTA decode-step attention hot path for MI355X (gfx950).

The compute path is the HIP library built from ``csrc/``; ``paper_2510_09883_amd.delta`` is
its Python binding (argument marshalling only) and raises if the library is not built.
``configs`` and ``synth`` describe and generate the synthetic workloads.
"""
__all__ = ["configs", "synth", "delta"]
