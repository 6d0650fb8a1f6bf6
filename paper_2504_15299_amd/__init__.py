"""MI355X (gfx950) MoE-layer hot path of D^2MoE: dual routing (top-k expert
IDs plus a bit-width per activated expert) over matryoshka-quantized (MWQ)
expert weights.  The compute runs in ``libd2moe.so`` (hand-written HIP kernels
behind the C ABI in ``include/d2moe.h``); ``api`` is its ctypes binding and
``workloads`` draws seeded synthetic inputs."""

__all__ = ["api", "workloads", "build"]


def __getattr__(name):
    if name in __all__:
        import importlib
        return importlib.import_module(f"{__name__}.{name}")
    raise AttributeError(name)
