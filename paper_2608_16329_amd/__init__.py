"""MI355X-native small-footprint MLIP energy/force/virial path (arXiv 2608.16329).

The compute lives in libmlip.so (HIP for gfx950, C ABI in include/mlip.h);
`binding` marshals arguments to it, and `Potential` wraps one context around
PyTorch-ROCm device tensors.  PyTorch supplies device memory and the stream.
"""
from __future__ import annotations

from typing import Optional

import numpy as np

from . import binding
from .binding import MlipError, mlip_hparams

__all__ = ["binding", "MlipError", "mlip_hparams", "Potential"]


class Potential:
    """One library context bound to the current PyTorch stream.

    hp: object with the mlip_hparams field names (for example synth.HParams);
    weights: flat float64 blob in the layout of include/mlip.h."""

    def __init__(self, hp, weights: np.ndarray, stream=None):
        import torch
        if not torch.cuda.is_available():
            raise RuntimeError("no GPU visible: the MLIP library runs only on the GPU")
        self.torch = torch
        self.stream = stream if stream is not None else torch.cuda.current_stream()
        self.ctx = binding.mlip_create(hp, weights, self.stream.cuda_stream)
        self.n = 0

    def close(self):
        if self.ctx:
            binding.mlip_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def build_neighbors(self, pos, types, box) -> None:
        assert pos.is_cuda and pos.dtype == self.torch.float64 and pos.is_contiguous()
        assert types.is_cuda and types.dtype == self.torch.int32 and types.is_contiguous()
        self.n = pos.shape[0]
        binding.mlip_build_neighbors(self.ctx, self.n, pos.data_ptr(), types.data_ptr(), np.asarray(box, float))

    def compute(self, pos, forces, energy=None, virial=None, totals: bool = False) -> Optional[np.ndarray]:
        assert pos.is_cuda and pos.dtype == self.torch.float64 and pos.is_contiguous()
        assert forces.is_cuda and forces.dtype == self.torch.float64 and forces.is_contiguous()
        return binding.mlip_compute(self.ctx, pos.data_ptr(), energy.data_ptr() if energy is not None else None,
                                    forces.data_ptr(), virial.data_ptr() if virial is not None else None, totals)

    def compute_noalloc(self, pos, forces, energy=None, virial=None, totals: bool = False) -> Optional[np.ndarray]:
        """compute() with the library's fixed per-device scratch instead of
        context buffers (mlip_compute_noalloc: no device allocation)."""
        assert pos.is_cuda and pos.dtype == self.torch.float64 and pos.is_contiguous()
        assert forces.is_cuda and forces.dtype == self.torch.float64 and forces.is_contiguous()
        return binding.mlip_compute_noalloc(self.ctx, pos.data_ptr(),
                                            energy.data_ptr() if energy is not None else None, forces.data_ptr(),
                                            virial.data_ptr() if virial is not None else None, totals)

    def set_fusion(self, fusion: int) -> None:
        """binding.MLIP_FUSION_CACHED (default), _RECOMPUTE, _PARTIAL or _UNFUSED."""
        binding.mlip_set_fusion(self.ctx, fusion)

    def set_scatter(self, scatter: int) -> None:
        """binding.MLIP_SCATTER_ATOMIC (default) or MLIP_SCATTER_TILE."""
        binding.mlip_set_scatter(self.ctx, scatter)

    def set_list_format(self, fmt: int) -> None:
        """binding.MLIP_LIST_AUTO (2-byte coded entries where possible, default)
        or MLIP_LIST_INDEX (4-byte indices); applies from the next build."""
        binding.mlip_set_list_format(self.ctx, fmt)

    def neighbors(self):
        return binding.mlip_get_neighbors(self.ctx)

    def neighbor_rows(self, atoms, cap=None):
        """Neighbour rows (caller indices) of the given atoms, one array each."""
        atoms = np.asarray(atoms, dtype=np.int64)
        cap = cap if cap is not None else 4096 * max(len(atoms), 1)
        counts, idx = binding.mlip_get_neighbor_rows(self.ctx, atoms, cap)
        ends = np.cumsum(counts)
        return [idx[e - c:e] for c, e in zip(counts, ends)]

    def stats(self) -> dict:
        return binding.mlip_get_stats(self.ctx)

    def memory_bytes(self) -> int:
        return binding.mlip_memory_bytes(self.ctx)

    def set_masses(self, masses) -> None:
        binding.mlip_md_set_masses(self.ctx, masses)

    def md_first_half(self, pos, vel, forces, dt, ref=None, track: bool = False) -> Optional[float]:
        """Half kick + drift; returns the largest squared displacement since
        `ref` (or, with track=True and no ref, since the last neighbour build)."""
        return binding.mlip_md_first_half(self.ctx, pos.data_ptr(), vel.data_ptr(), forces.data_ptr(), dt,
                                          ref.data_ptr() if ref is not None else None, track)

    def md_second_half(self, vel, forces, dt) -> None:
        binding.mlip_md_second_half(self.ctx, vel.data_ptr(), forces.data_ptr(), dt)

    def kinetic(self, vel) -> float:
        return binding.mlip_md_kinetic(self.ctx, vel.data_ptr())
