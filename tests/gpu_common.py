"""Helpers shared by the GPU parity tests (inputs, row sampling, tolerances)."""
from __future__ import annotations

import math
import sys

import numpy as np

from oracle import partir_oracle as O
from paper_2401_11202_amd import inputs as I

# Tolerances: max over elements of |gpu - oracle| / (|A|.|B|) of the last
# contraction -- 1e-4 for fp32 inputs, 2e-2 for bf16 inputs with fp32
# accumulation.
TOL_F32 = 1e-4
TOL_BF16 = 2e-2
# Chained products (backward passes) round several bf16 intermediates
# (2^-8 relative each); the error normalised by the whole gradient's size,
# ||got - ref||_F / ||ref||_F, must stay at the level of a few such roundings.
# This catches a wrong factor that the elementwise |A|.|B| normaliser, loose
# by ~sqrt(K) per contraction, would let through.
TOL_REL_FRO = 1e-2


def rel_fro(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = float(np.linalg.norm(ref))
    return float(np.linalg.norm(got - ref)) / den if den > 0 else float(np.linalg.norm(got))


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def host(t):
    """Device tensor -> float64 numpy."""
    return t.float().cpu().numpy().astype(np.float64)


def sample_rows(T: int, R_batch: int, n: int, seed: int, S: int | None = None,
                max_pos: int | None = None, full_seq_rows: int = 0):
    """Seeded output-row sample: the first and last row of every batch shard
    (or, for sequence workloads, positions 0 and S-1 / max_pos of sequences),
    plus uniformly drawn rows."""
    rng = np.random.default_rng(seed)
    Tb = T // R_batch
    rows = set()
    if S is None:
        for b in range(R_batch):
            rows.update((b * Tb, (b + 1) * Tb - 1))
        while len(rows) < n:
            rows.add(int(rng.integers(0, T)))
        return sorted(rows)
    nseq = T // S
    lim = S if max_pos is None else max_pos
    for s in range(nseq):
        rows.add(s * S)
    # last position of a few sequences needs the whole sequence as keys
    for s in range(min(full_seq_rows, nseq)):
        rows.add(s * S + S - 1)
    for b in range(R_batch):
        rows.add(b * Tb)
    while len(rows) < n:
        s = int(rng.integers(0, nseq))
        rows.add(s * S + int(rng.integers(0, lim)))
    return sorted(rows)


def every_block_rows(B: int, S: int, seqs, seed: int, block: int = 128):
    """One seeded row in every `block`-query block of each sequence in
    `seqs` (so late blocks with long causal key loops are compared too), plus
    positions 0 and S-1 of those sequences and position 0 of every sequence."""
    rng = np.random.default_rng(seed)
    rows = {s * S for s in range(B)}
    for s in seqs:
        rows.update((s * S, s * S + S - 1))
        for b0 in range(0, S, block):
            rows.add(s * S + b0 + int(rng.integers(0, block)))
    return sorted(rows)


def accum_bound(K: int) -> float:
    """Higham-style bound for fp32 accumulation of K exact products."""
    u = 2.0 ** -24
    return K * u / (1 - K * u)
