"""Dynamic voxels of the decoded occupancy grid (Eq. 1) -- test infrastructure.

The oracle of the path: plain NumPy, no shared code with the HIP library.
Only the tests, the package's smoke check and the benchmark's CPU baseline use
it.

Eq. (1) counts the voxels whose binary occupancy differs between the grids
decoded at two consecutive steps: the number of positions where O_{t+1} XOR
O_t is 1, i.e. the Hamming distance of the two grids. Readings:
* the decoder returns one logit per voxel and a voxel is occupied when its
  logit is > 0 (occupancy probability above one half); NaN is unoccupied;
* the grid is flattened row-major, voxel n = (i * N + j) * N + k, and packed
  32 voxels per little-endian 32-bit word, voxel n in bit n % 32 of word
  n // 32; a tail word is padded with zero bits.
"""
from __future__ import annotations

import numpy as np


def occupancy(logits: np.ndarray) -> np.ndarray:
    """Binary occupancy of each voxel: logit > 0 (NaN compares false)."""
    return np.asarray(logits) > 0


def pack(occ: np.ndarray) -> np.ndarray:
    """Flattened boolean grid -> uint32 words, voxel n in bit n % 32 of word n // 32."""
    flat = np.asarray(occ, dtype=bool).reshape(-1)
    n_words = (flat.size + 31) // 32
    padded = np.zeros(n_words * 32, dtype=bool)
    padded[:flat.size] = flat
    bits = padded.reshape(n_words, 32).astype(np.uint64)
    return (bits << np.arange(32, dtype=np.uint64)).sum(axis=1).astype(np.uint32)


def dynamic_voxels(occ_next: np.ndarray, occ_prev: np.ndarray) -> int:
    """Eq. (1): sum over voxels of O_{t+1} XOR O_t."""
    a = np.asarray(occ_next, dtype=bool)
    b = np.asarray(occ_prev, dtype=bool)
    return int(np.count_nonzero(a ^ b))
