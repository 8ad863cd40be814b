"""MI355X-native per-stream phrase boosting for batched Transducer decoding.

The hot path (TurboBias 2.0, Sec. II) lives in libtbias.so: a host graph
compiler (C++) and HIP kernels for gfx950. ``capi`` is the thin ctypes
binding; ``decoder`` a small convenience layer over it. Importing ``capi``
requires the built library (``python -m paper_2608_21343_amd.build``).
"""

__all__ = ["capi", "decoder", "build"]
