"""Per-use backward-state checks of emulated FP8 rounding on MI355X (gfx950).

The compute path is libbsp.so (HIP kernels behind the C-ABI of include/bsp.h);
``paper_2609_39813_amd.bsp`` is its Python binding and ``paper_2609_39813_amd.synth``
the seeded synthetic inputs. Build with ``python -m paper_2609_39813_amd.build``.
"""
__all__ = ["bsp", "synth", "build"]
