"""MI355X (gfx950) dense GEMM: int8 -> int32 and bf16 -> fp32 behind a C ABI.

The GPU entry points live in ``paper_2512_13282_amd.binding`` (a thin ctypes
layer over ``libgemm_mi355x.so``); they are imported lazily so that the input
generators can be used on machines without the built library.
"""
__all__ = ["gemm_i8_i32", "gemm_bf16_f32", "gemm_plan", "gemm_status_string"]


def __getattr__(name):
    if name in __all__:
        from . import binding
        return getattr(binding, name)
    raise AttributeError(name)
