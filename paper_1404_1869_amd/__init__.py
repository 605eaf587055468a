"""DenseNet conv5 descriptor pyramids (Iandola et al., arXiv 1404.1869) on one MI355X.

The computation lives in ``libdensenet.so`` (HIP for gfx950, C ABI declared in ``include/densenet.h``);
``paper_1404_1869_amd.densenet`` is the thin ctypes binding with the same entry-point names.  The
binding is imported lazily so that the input generators and configs can be used without a GPU.
"""
__all__ = ["configs", "synth", "workmodel"]
