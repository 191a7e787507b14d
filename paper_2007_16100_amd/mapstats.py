"""Kernel-map statistics and the MAC count of sparse convolutions.

A sparse convolution computes only over its active synapses, so its MAC count
depends on the input's sparsity pattern as well as on the layer shape.  The
paper's resource model (Sec. 4.3, "Resource Constraints") averages each
convolution layer's kernel-map size over the data and multiplies by the layer
width:

    MACs(layer) = sum_k E[|map_k|] * C_in * C_out

This module records |map_k| per offset from the CSR offsets `off[K^3 + 1]` that
`spv_kernel_map` writes (|map_k| = off[k + 1] - off[k]), averages them over
scans, and evaluates that sum for a list of layers.  Host-side bookkeeping only:
the maps themselves come from the library.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, Iterable, List, Sequence, Tuple

import numpy as np


def map_sizes(off) -> np.ndarray:
    """|map_k| for every offset k from a CSR offset array (device tensor or array)."""
    try:
        import torch
        if isinstance(off, torch.Tensor):
            off = off.detach().cpu().numpy()
    except ImportError:  # pragma: no cover - torch is part of the environment
        pass
    o = np.asarray(off, dtype=np.int64)
    if o.ndim != 1 or o.size < 2:
        raise ValueError("off must be a 1-D array of K^3 + 1 offsets")
    d = np.diff(o)
    if (d < 0).any():
        raise ValueError("off is not non-decreasing")
    return d


@dataclass
class MapStats:
    """Running per-offset map sizes of named map kinds (e.g. "s1k3", "s2k2") over scans."""
    sums: Dict[str, np.ndarray] = field(default_factory=dict)
    scans: Dict[str, int] = field(default_factory=dict)

    def add(self, name: str, off) -> np.ndarray:
        """Record one scan's map of kind `name`; returns its |map_k|."""
        s = map_sizes(off)
        if name in self.sums and self.sums[name].shape != s.shape:
            raise ValueError(f"{name}: {s.size} offsets, earlier scans had {self.sums[name].size}")
        self.sums[name] = self.sums.get(name, np.zeros_like(s)) + s
        self.scans[name] = self.scans.get(name, 0) + 1
        return s

    def mean(self, name: str) -> np.ndarray:
        """E[|map_k|] over the recorded scans of kind `name`."""
        if not self.scans.get(name):
            raise KeyError(name)
        return self.sums[name] / self.scans[name]


def conv_macs(layers: Sequence[Tuple[str, int, int]], stats: MapStats) -> Tuple[float, List[float]]:
    """MACs of a list of convolution layers (map kind, C_in, C_out), each
    sum_k E[|map_k|] * C_in * C_out; returns the total and the per-layer values."""
    per = [float(stats.mean(kind).sum()) * cin * cout for kind, cin, cout in layers]
    return float(sum(per)), per


def flops_of_map(off, cin: int, cout: int) -> float:
    """Effective FLOPs of one convolution on one map: 2 * C_in * C_out * sum_k |map_k|."""
    return 2.0 * cin * cout * float(map_sizes(off).sum())


__all__ = ["map_sizes", "MapStats", "conv_macs", "flops_of_map"]
