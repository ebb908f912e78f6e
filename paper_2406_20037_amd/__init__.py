"""MI355X (gfx950) implementation of the schedule-tuning hot path of the
combined Ansor + Droplet Search approach: a schedule-parameterised fp32
conv2d / matmul kernel family in HIP, a hipEvent measurement harness, a seeded
exploration sampler and Droplet Search coordinate descent, behind the C ABI
of ``include/droplet.h``.  ``_lib`` is the Python binding of that ABI; it is
loaded on first use of any name below, and raises if the library is missing.
"""
_EXPORTS = ["DS_OP_CONV2D_NCHW", "DS_OP_MATMUL_RM", "Space", "ansor_sample", "droplet_tune",
            "droplet_tune_ex", "ds_empty_kernel_floor", "ds_measure", "ds_tune", "kernel_run",
            "kernel_run_reference", "make_io", "measure_cfg", "tune_cfg"]

__all__ = _EXPORTS + ["_lib"]


def __getattr__(name):
    if name == "_lib" or name in _EXPORTS:
        import importlib
        lib = importlib.import_module("._lib", __name__)
        return lib if name == "_lib" else getattr(lib, name)
    raise AttributeError(name)
