"""Per-token record buffers of the GPU (64-token tiles, 8-byte chunks
outermost: [B, T/64, S/8, 64, 8]) to and from the oracle's [B, T, C] records.
Test helper: a layout conversion, no arithmetic of the method."""

import numpy as np


def to_tiles(rec: np.ndarray, S: int) -> np.ndarray:
    """[B, T, C] records -> the GPU buffer layout, zero-padded to S bytes."""
    B, T, C = rec.shape
    full = np.zeros((B, T, S), dtype=np.uint8)
    full[..., :C] = rec
    return np.ascontiguousarray(full.reshape(B, T // 64, 64, S // 8, 8).transpose(0, 1, 3, 2, 4))


def from_tiles(tiles: np.ndarray) -> np.ndarray:
    """GPU buffer [B, T/64, S/8, 64, 8] -> [B, T, S] (record slots in token order)."""
    B, NT, NC, _, _ = tiles.shape
    return np.ascontiguousarray(tiles.transpose(0, 1, 3, 2, 4)).reshape(B, NT * 64, NC * 8)
