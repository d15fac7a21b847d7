"""FlashNorm on MI355X: the deferred RMSNorm/LayerNorm -> linear hot path of
"FlashNorm: Fast Normalization for Transformers" (arXiv 2407.09577) as hand-written
HIP kernels for gfx950 behind a C ABI (``include/flashnorm.h``).

``paper_2407_09577_amd.flashnorm`` is the thin ctypes binding to ``libflashnorm.so``;
``paper_2407_09577_amd.workloads`` draws the seeded synthetic inputs.  The binding is
imported lazily so that the input generators work on machines without the library.
"""
__all__ = ["flashnorm", "workloads"]


def __getattr__(name):
    if name in __all__:
        import importlib
        return importlib.import_module(f"{__name__}.{name}")
    raise AttributeError(name)
