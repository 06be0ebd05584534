"""The paper's MatMul 2 work split (Section IV-E, Algorithm 2), as a partition model -- TEST ONLY.

Test infrastructure: used by tests/ only, never by the product path, which partitions for 256
compute units instead (its own plan, in the library).

What the section describes, restated here in this module's own terms:

* The weight [K, N] is cut into blocks of ``k_slice`` = 1024 rows by ``col_block`` = 16
  columns: ``n_slices`` = K // k_slice row slices times ``n_col_blocks`` = N // col_block column
  blocks, ``n_blocks`` blocks in all.
* The blocks are dealt to ``n_units`` vector units -- the largest count not above two per core
  (2P) that divides ``n_blocks`` evenly -- each unit taking one contiguous run of
  ``blocks_per_unit`` blocks, numbered slice-major (block b is column block b % n_col_blocks of
  row slice b // n_col_blocks).  ``units_per_slice`` = n_units // n_slices is how many units
  share one row slice when the runs line up with slices.
* Each block yields 16 fp32 partial dot products of the token's row slice with the block's
  columns; they go to a [n_slices, N] fp32 buffer.  After every unit has stored its blocks,
  each column block sums its partials over the row slices in slice order, and the sum is cast
  to bf16.

Reading of the section's indexing: the listing gives a unit one token offset, derived from its
unit number.  That is only well defined when a unit's run of blocks stays inside one row slice,
which holds at the paper's N = 576 but not at N = 2112 (44 units over 7 slices).  This model
takes the block numbering above, under which a run may straddle two slices, and every block
reads its own slice of the token.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

COL_BLOCK = 16
K_SLICE = 1024


@dataclass(frozen=True)
class Partition:
    K: int
    N: int
    cores: int            # P
    col_block: int
    k_slice: int
    n_slices: int
    n_col_blocks: int
    n_blocks: int
    n_units: int
    blocks_per_unit: int
    units_per_slice: int

    def blocks_of(self, unit: int) -> range:
        """The contiguous run of block numbers that ``unit`` computes."""
        return range(unit * self.blocks_per_unit, (unit + 1) * self.blocks_per_unit)

    def slice_and_cols(self, block: int) -> tuple[int, int]:
        """(row slice, column block) of a block number."""
        return divmod(block, self.n_col_blocks)

    def slices_of(self, unit: int) -> set[int]:
        """The row slices that ``unit``'s run touches."""
        return {self.slice_and_cols(b)[0] for b in self.blocks_of(unit)}


def partition(K: int, N: int, cores: int = 24) -> Partition:
    """The split of T[1, K] x W[K, N] over ``cores`` cores (two vector units each)."""
    n_slices, n_col_blocks = K // K_SLICE, N // COL_BLOCK
    n_blocks = n_slices * n_col_blocks
    if n_blocks == 0:
        raise ValueError("the split needs K >= 1024 and N >= 16")
    n_units = next(u for u in range(2 * cores, 0, -1) if n_blocks % u == 0)
    return Partition(K, N, cores, COL_BLOCK, K_SLICE, n_slices, n_col_blocks, n_blocks, n_units,
                     n_blocks // n_units, n_units // n_slices)


def evaluate(T: np.ndarray, W: np.ndarray, part: Partition, decode) -> tuple[np.ndarray, np.ndarray]:
    """Run the split in fp32.  ``T`` [1, K] and ``W`` [K, N] are bf16 bit patterns and ``decode``
    turns bits into float64.  Returns (the gathered fp32 sums [N'], the partial-sum buffer
    [n_slices, N']) for the N' = n_col_blocks * 16 columns the split covers."""
    t = decode(T, 2).astype(np.float32).reshape(-1)            # widening is exact
    w = decode(W, 2).astype(np.float32)
    width = part.n_col_blocks * part.col_block
    partials = np.full((part.n_slices, width), np.nan, dtype=np.float32)
    for unit in range(part.n_units):
        for block in part.blocks_of(unit):
            s, c = part.slice_and_cols(block)
            rows = slice(s * part.k_slice, (s + 1) * part.k_slice)
            cols = slice(c * part.col_block, (c + 1) * part.col_block)
            partials[s, cols] = np.dot(t[rows], w[rows, cols]).astype(np.float32)
    # every unit has stored its blocks: sum each column's partials over the slices, in order
    total = np.zeros(width, dtype=np.float32)
    for s in range(part.n_slices):
        total = total + partials[s]
    return total, partials
