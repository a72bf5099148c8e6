"""Append-only upsert on a host model of the index.  Test infrastructure only.

Op_upsert (Section 3.2, "Upsert") inserts new embeddings into the index, I' = Op_upsert(I, E; b_u).
The reading here is append-only: the new rows take ids n_rows .. n_rows + m - 1 in order,
existing rows are unchanged, and a batch that does not fit the capacity changes nothing.
Rows given in fp32 are rounded to the index dtype with round-to-nearest-even.
"""
from __future__ import annotations

import numpy as np

from .storage import round_f32_to_bf16, round_f32_to_f16


class HostIndex:
    def __init__(self, dim: int, capacity: int, dtype: str):
        self.dim, self.capacity, self.dtype = dim, capacity, dtype
        self.bits = np.zeros((capacity, dim), dtype=np.uint32 if dtype == "f32" else np.uint16)
        self.n_rows = 0

    def append_bits(self, rows_bits: np.ndarray) -> int:
        m = rows_bits.shape[0]
        if self.n_rows + m > self.capacity:
            raise OverflowError("capacity")
        first = self.n_rows
        self.bits[first:first + m] = rows_bits
        self.n_rows += m
        return first

    def append_f32(self, rows_f32: np.ndarray) -> int:
        x = np.asarray(rows_f32, dtype=np.float32)
        if self.dtype == "f32":
            return self.append_bits(x.view(np.uint32))
        if self.dtype == "bf16":
            return self.append_bits(round_f32_to_bf16(x))
        return self.append_bits(round_f32_to_f16(x))

    def valid_bits(self) -> np.ndarray:
        return self.bits[:self.n_rows]
