"""VBQ on MI355X: packed variable-bit-width weights and the fused
dequantize-and-multiply of autoregressive decode (arxiv 2607.02893, section 6),
as a C-ABI library (libvbq.so: host packer + gfx950 HIP kernels) with a thin
ctypes binding.

    from paper_2607_02893_amd import vbq      # loads libvbq.so, raises if not built
    blob, desc = vbq.pack_codes(q, scales, bits)
    Wp = vbq.PackedMatrix(blob, desc)
    y = Wp.gemv(x)

`synth` draws the seeded synthetic inputs; `build` compiles the library.
"""

__all__ = ["vbq", "synth", "build"]


def __getattr__(name):
    if name in __all__:
        import importlib
        return importlib.import_module(f"{__name__}.{name}")
    raise AttributeError(name)
