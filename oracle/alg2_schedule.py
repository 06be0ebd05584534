"""Model of the paper's specialised MatMul 2 partition (Algorithm 2, Section IV-E) -- TEST ONLY.

This is the oracle's model of *how the paper splits the work*, written in the paper's notation
(fractalSize, kSplitSize, kParts, fractalNum, S, V, nPart_W, groupSize, off_T, fracId, tmpBuf,
Acc).  It is used to pin the reading of Algorithm 2's indexing and its worked constants; the HIP
path does not follow it (its partition is sized for 256 compute units, not 2P vector units).

Steps, in the order Algorithm 2 takes them:

* Init: fractalSize = 16, kSplitSize = 1024, kParts = K DIV kSplitSize,
  fractalNum = N DIV fractalSize, S = fractalNum * kParts; V is the largest divisor of S that is
  at most 2P; nPart_W = S DIV V; groupSize = V DIV kParts.
* Compute: executor v processes fracId = v * nPart_W + w for w < nPart_W.  Each fracId is one
  block of kSplitSize rows by fractalSize columns; the block's 16 partial sums are fp32 dot
  products of the token slice with the block's columns (Transpose + Cast + Mul + ReduceSum).
  They are stored to the fp32 partial-sum buffer tmpBuf.
* Gather (after WaitAllVectors): executor v < fractalNum sums the kParts partials of column
  fractal v in order i = 0..kParts-1 into the fp32 accumulator Acc, then casts Acc to bf16.

Reading of the garbled/ambiguous indexing (Algorithm 2): the printed token offset
off_T = (v DIV groupSize) * kSplitSize only holds when every executor's nPart_W blocks sit in one
k-part (true for the paper's N = 576, false e.g. for N = 2112 where V = 44 is not a multiple of
kParts = 7).  The reading used here: block fracId has k-part ``fracId DIV fractalNum`` and column
fractal ``fracId MOD fractalNum``; tmpBuf is laid out [kParts][N] in fp32, so block fracId's 16
floats start at element fracId * fractalSize, which is the gather's ``off_C + i * N``.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

FRACTAL_SIZE = 16
K_SPLIT_SIZE = 1024


@dataclass(frozen=True)
class Alg2Plan:
    K: int
    N: int
    P: int
    fractalSize: int
    kSplitSize: int
    kParts: int
    fractalNum: int
    S: int
    V: int
    nPart_W: int
    groupSize: int

    def frac_ids(self, v: int) -> list[int]:
        """Blocks of executor v (compute stage)."""
        return [v * self.nPart_W + w for w in range(self.nPart_W)]

    def block(self, fracId: int) -> tuple[int, int]:
        """(k-part, column fractal) of a block under the reading above."""
        return fracId // self.fractalNum, fracId % self.fractalNum

    def literal_off_T(self, v: int) -> int:
        """The token offset exactly as printed: (v DIV groupSize) * kSplitSize."""
        return (v // self.groupSize) * self.kSplitSize


def plan(K: int, N: int, P: int = 24) -> Alg2Plan:
    """Init stage of Algorithm 2 for T[1,K] x W[K,N] on P cores (2P vector units)."""
    kParts = K // K_SPLIT_SIZE
    fractalNum = N // FRACTAL_SIZE
    S = fractalNum * kParts
    if S == 0:
        raise ValueError("Algorithm 2 needs K >= kSplitSize and N >= fractalSize")
    V = max(d for d in range(1, 2 * P + 1) if S % d == 0)
    nPart_W = S // V
    groupSize = V // kParts
    return Alg2Plan(K, N, P, FRACTAL_SIZE, K_SPLIT_SIZE, kParts, fractalNum, S, V, nPart_W,
                    groupSize)


def run(T: np.ndarray, W: np.ndarray, p: Alg2Plan, decode) -> tuple[np.ndarray, np.ndarray]:
    """Execute the compute and gather stages in fp32.

    ``T`` is [1,K] and ``W`` is [K,N] bf16 bit patterns; ``decode`` turns bits into float64 (the
    oracle's decoder).  Returns (Acc as fp32 [N'], tmpBuf [kParts, N']) where
    N' = fractalNum * fractalSize.
    """
    fs, ks = p.fractalSize, p.kSplitSize
    Tf = decode(T, 2).astype(np.float32).reshape(-1)          # Cast (exact widening)
    Wf = decode(W, 2).astype(np.float32)
    Np = p.fractalNum * fs
    tmpBuf = np.full((p.kParts, Np), np.nan, dtype=np.float32)
    for v in range(p.V):                                       # compute stage, executor v
        for fracId in p.frac_ids(v):
            kpart, cf = p.block(fracId)
            Tv = Tf[kpart * ks:(kpart + 1) * ks]
            Wvw = Wf[kpart * ks:(kpart + 1) * ks, cf * fs:(cf + 1) * fs]
            partSum = np.array([np.dot(Tv, Wvw[:, j]) for j in range(fs)], dtype=np.float32)
            tmpBuf.reshape(-1)[fracId * fs:(fracId + 1) * fs] = partSum
    # WaitAllVectors: every block above has been stored.
    Acc = np.zeros(Np, dtype=np.float32)
    for v in range(p.fractalNum):                              # gather stage, executor v
        off_C = v * fs
        acc = np.zeros(fs, dtype=np.float32)
        for i in range(p.kParts):
            acc = acc + tmpBuf.reshape(-1)[off_C + i * Np: off_C + i * Np + fs]
        Acc[off_C:off_C + fs] = acc
    return Acc, tmpBuf
