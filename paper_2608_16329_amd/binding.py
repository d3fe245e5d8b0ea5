"""ctypes binding of libmlip.so (C ABI in include/mlip.h).

Functions carry the C names and only marshal arguments: device buffers are
passed as raw pointers (for example `tensor.data_ptr()` of contiguous
PyTorch-ROCm tensors), host arrays as NumPy float64/int32/int64 buffers.
Every step of the computation runs in the library's HIP kernels; there is no
fallback.  Importing this module raises if the library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmlip.so")

MLIP_OK = 0
STATUS = {0: "MLIP_OK", -1: "MLIP_E_ARG", -2: "MLIP_E_OOM", -3: "MLIP_E_HIP", -4: "MLIP_E_BOX",
          -5: "MLIP_E_NBR_CAP", -6: "MLIP_E_STATE", -7: "MLIP_E_TYPE"}

# Every symbol include/mlip.h declares.
EXPORTED = ["mlip_weight_count", "mlip_create", "mlip_build_neighbors", "mlip_compute", "mlip_get_neighbors",
            "mlip_memory_bytes", "mlip_get_stats", "mlip_last_error", "mlip_destroy", "mlip_md_set_masses",
            "mlip_md_first_half", "mlip_md_second_half", "mlip_md_kinetic", "mlip_set_fusion",
            "mlip_get_neighbor_rows", "mlip_compute_noalloc", "mlip_set_scatter", "mlip_set_list_format"]

MLIP_STATIC_SCRATCH_BYTES = 256 * 1024 * 1024

MLIP_FUSION_CACHED, MLIP_FUSION_RECOMPUTE, MLIP_FUSION_PARTIAL, MLIP_FUSION_UNFUSED = 0, 1, 2, 3
MLIP_SCATTER_ATOMIC, MLIP_SCATTER_TILE = 0, 1
MLIP_LIST_AUTO, MLIP_LIST_INDEX = 0, 1


class mlip_hparams(ctypes.Structure):
    _fields_ = [("n_species", ctypes.c_int32), ("cutoff", ctypes.c_double), ("skin", ctypes.c_double),
                ("k", ctypes.c_int32), ("lmax", ctypes.c_int32), ("angular", ctypes.c_int32),
                ("enc_cond", ctypes.c_int32), ("reg_cond", ctypes.c_int32), ("enc_width", ctypes.c_int32),
                ("enc_hidden", ctypes.c_int32), ("reg_width", ctypes.c_int32), ("reg_hidden", ctypes.c_int32),
                ("precision", ctypes.c_int32)]


class mlip_stats(ctypes.Structure):
    _fields_ = [("n_atoms", ctypes.c_int64), ("n_listed_pairs", ctypes.c_int64),
                ("n_active_pairs", ctypes.c_int64), ("max_row", ctypes.c_int32), ("tile_atoms", ctypes.c_int32),
                ("n_tiles", ctypes.c_int64), ("n_blocks", ctypes.c_int32), ("n_cells", ctypes.c_int32),
                ("n_builds", ctypes.c_int64), ("device_bytes", ctypes.c_size_t),
                ("list_entry_bytes", ctypes.c_int32)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


class MlipError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with paper_2608_16329_amd/build.py "
                          "(or __graft_entry__.build())")
    lib = ctypes.CDLL(LIB_PATH)
    vp, dp, ip32, ip64 = ctypes.c_void_p, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int32), \
        ctypes.POINTER(ctypes.c_int64)
    st = ctypes.c_int
    sig = {
        "mlip_weight_count": (ctypes.c_size_t, [ctypes.POINTER(mlip_hparams)]),
        "mlip_create": (st, [ctypes.POINTER(mlip_hparams), dp, ctypes.c_size_t, vp, ctypes.POINTER(vp)]),
        "mlip_build_neighbors": (st, [vp, ctypes.c_int64, vp, vp, dp]),
        "mlip_compute": (st, [vp, vp, vp, vp, vp, dp]),
        "mlip_compute_noalloc": (st, [vp, vp, vp, vp, vp, dp]),
        "mlip_get_neighbors": (st, [vp, ip64, ip32]),
        "mlip_get_neighbor_rows": (st, [vp, ip64, ctypes.c_int64, ip64, ip32, ctypes.c_int64]),
        "mlip_memory_bytes": (st, [vp, ctypes.POINTER(ctypes.c_size_t)]),
        "mlip_get_stats": (st, [vp, ctypes.POINTER(mlip_stats)]),
        "mlip_last_error": (ctypes.c_char_p, [vp]),
        "mlip_destroy": (None, [vp]),
        "mlip_md_set_masses": (st, [vp, dp]),
        "mlip_md_first_half": (st, [vp, vp, vp, vp, ctypes.c_double, vp, dp]),
        "mlip_md_second_half": (st, [vp, vp, vp, ctypes.c_double]),
        "mlip_md_kinetic": (st, [vp, vp, dp]),
        "mlip_set_fusion": (st, [vp, ctypes.c_int32]),
        "mlip_set_scatter": (st, [vp, ctypes.c_int32]),
        "mlip_set_list_format": (st, [vp, ctypes.c_int32]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_lib = _load()


def _dp(a: Optional[np.ndarray]):
    if a is None:
        return None
    assert a.dtype == np.float64 and a.flags.c_contiguous
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _check(ctx, status: int):
    if status != MLIP_OK:
        # with no context (mlip_create) the library keeps the reason per thread
        raise MlipError(status, _lib.mlip_last_error(ctx).decode())


def hparams_from(hp) -> mlip_hparams:
    """mlip_hparams from any object with the same attribute names."""
    return mlip_hparams(*(getattr(hp, name) for name, _ in mlip_hparams._fields_))


def mlip_weight_count(hp) -> int:
    h = hp if isinstance(hp, mlip_hparams) else hparams_from(hp)
    return int(_lib.mlip_weight_count(ctypes.byref(h)))


def mlip_create(hp, weights: np.ndarray, hip_stream: int = 0) -> int:
    h = hp if isinstance(hp, mlip_hparams) else hparams_from(hp)
    w = np.ascontiguousarray(weights, dtype=np.float64)
    ctx = ctypes.c_void_p()
    _check(None, _lib.mlip_create(ctypes.byref(h), _dp(w), w.size, ctypes.c_void_p(hip_stream or None),
                                  ctypes.byref(ctx)))
    return ctx.value


def mlip_build_neighbors(ctx: int, n_atoms: int, pos_ptr: int, types_ptr: int, box) -> None:
    b = np.ascontiguousarray(box, dtype=np.float64)
    _check(ctx, _lib.mlip_build_neighbors(ctx, int(n_atoms), pos_ptr, types_ptr, _dp(b)))


def mlip_compute(ctx: int, pos_ptr: int, energy_ptr: Optional[int], forces_ptr: int, virial_ptr: Optional[int],
                 want_totals: bool = False) -> Optional[np.ndarray]:
    tot = np.zeros(10) if want_totals else None
    _check(ctx, _lib.mlip_compute(ctx, pos_ptr, energy_ptr or None, forces_ptr, virial_ptr or None, _dp(tot)))
    return tot


def mlip_compute_noalloc(ctx: int, pos_ptr: int, energy_ptr: Optional[int], forces_ptr: int,
                         virial_ptr: Optional[int], want_totals: bool = False) -> Optional[np.ndarray]:
    tot = np.zeros(10) if want_totals else None
    _check(ctx, _lib.mlip_compute_noalloc(ctx, pos_ptr, energy_ptr or None, forces_ptr, virial_ptr or None,
                                          _dp(tot)))
    return tot


def mlip_get_stats(ctx: int) -> dict:
    s = mlip_stats()
    _check(ctx, _lib.mlip_get_stats(ctx, ctypes.byref(s)))
    return s.as_dict()


def mlip_get_neighbors(ctx: int):
    n = mlip_get_stats(ctx)
    off = np.zeros(n["n_atoms"] + 1, dtype=np.int64)
    idx = np.zeros(max(n["n_listed_pairs"], 1), dtype=np.int32)
    _check(ctx, _lib.mlip_get_neighbors(ctx, off.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                                        idx.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))))
    return off, idx[:n["n_listed_pairs"]]


def mlip_get_neighbor_rows(ctx: int, atoms, cap: int):
    """Rows of the given atoms (caller indices): (counts int64 [n_rows], idx int32
    [sum counts]) with cap entries of room."""
    a = np.ascontiguousarray(atoms, dtype=np.int64)
    counts = np.zeros(len(a), dtype=np.int64)
    idx = np.zeros(max(int(cap), 1), dtype=np.int32)
    _check(ctx, _lib.mlip_get_neighbor_rows(ctx, a.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), len(a),
                                            counts.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                                            idx.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), int(cap)))
    return counts, idx[:int(counts.sum())]


def mlip_set_fusion(ctx: int, fusion: int) -> None:
    _check(ctx, _lib.mlip_set_fusion(ctx, int(fusion)))


def mlip_set_scatter(ctx: int, scatter: int) -> None:
    _check(ctx, _lib.mlip_set_scatter(ctx, int(scatter)))


def mlip_set_list_format(ctx: int, fmt: int) -> None:
    _check(ctx, _lib.mlip_set_list_format(ctx, int(fmt)))


def mlip_memory_bytes(ctx: int) -> int:
    b = ctypes.c_size_t()
    _check(ctx, _lib.mlip_memory_bytes(ctx, ctypes.byref(b)))
    return int(b.value)


def mlip_last_error(ctx: int) -> str:
    return _lib.mlip_last_error(ctx).decode()


def mlip_destroy(ctx: int) -> None:
    _lib.mlip_destroy(ctx)


def mlip_md_set_masses(ctx: int, masses) -> None:
    m = np.ascontiguousarray(masses, dtype=np.float64)
    _check(ctx, _lib.mlip_md_set_masses(ctx, _dp(m)))


def mlip_md_first_half(ctx: int, pos_ptr: int, vel_ptr: int, forces_ptr: int, dt: float,
                       ref_ptr: Optional[int] = None, track: bool = False) -> Optional[float]:
    out = np.zeros(1) if (ref_ptr or track) else None
    _check(ctx, _lib.mlip_md_first_half(ctx, pos_ptr, vel_ptr, forces_ptr, float(dt), ref_ptr or None, _dp(out)))
    return float(out[0]) if out is not None else None


def mlip_md_second_half(ctx: int, vel_ptr: int, forces_ptr: int, dt: float) -> None:
    _check(ctx, _lib.mlip_md_second_half(ctx, vel_ptr, forces_ptr, float(dt)))


def mlip_md_kinetic(ctx: int, vel_ptr: int) -> float:
    out = np.zeros(1)
    _check(ctx, _lib.mlip_md_kinetic(ctx, vel_ptr, _dp(out)))
    return float(out[0])


def exported_symbols():
    """Names of the library's exported symbols that the header declares."""
    return [name for name in EXPORTED if hasattr(_lib, name)]
