"""Seeded synthetic inputs shared by the oracle tests, the GPU tests and the bench.

This module only draws random numbers.  It holds none of the method's
arithmetic: every value it returns is a random draw that the method takes as
an input (the weight matrix, the client's plaintext queries, the random code
description, the sparse noise of Encrypt and the sparse challenges of Verify).
Both the CPU oracle and the HIP library receive these arrays as explicit
inputs, so the two sides never need a shared sampler.

Field: p = 2^31 - 1 by default; the draws that depend on the field take it as
``p`` (the BabyBear prime 15 * 2^27 + 1 is ``P_BABYBEAR``).  All field arrays
are uint32 in canonical form [0, p).

Distributions (paper notation):
  * W: i.i.d. uniform int8 in [-127, 127] (integer-quantised weights that the
    method embeds into F_p, Sec. 7.2 "Model quantization").
  * X: i.i.d. uniform in F_p.
  * RAA code (App. B): two uniform permutations pi1, pi2 of [0, N) and two
    diagonals v1, v2 uniform in F_p^* = [1, p-1].
  * Sparse vectors of E_t^N (Sec. 3 notation; Lemma 5.1 samples them this
    way): support a uniform t-subset of [0, N) (distinct positions, in draw
    order), values uniform in F_p^*.

Seeds follow ``seed = 1000 * config_id + purpose`` with purposes
1=W, 2=X, 3=code x, 4=code y, 5=noise, 6=challenge, 7=tamper.
"""
from __future__ import annotations

import numpy as np

P = 2**31 - 1
P_BABYBEAR = 15 * 2**27 + 1

PURPOSE_W = 1
PURPOSE_X = 2
PURPOSE_CX = 3
PURPOSE_CY = 4
PURPOSE_NOISE = 5
PURPOSE_CHAL = 6
PURPOSE_TAMPER = 7
PURPOSE_C2 = 8      # secondary code of batch verification
PURPOSE_CHAL2 = 9   # secondary challenges of batch verification


def rng(seed: int) -> np.random.Generator:
    """Counter-based Philox stream keyed by ``seed``."""
    return np.random.Generator(np.random.Philox(key=int(seed)))


def seed_for(config_id: int, purpose: int, sub: int = 0) -> int:
    return 1000 * int(config_id) + int(purpose) + 1_000_000 * int(sub)


def weights(seed: int, m: int, n: int, lo: int = -127, hi: int = 127) -> np.ndarray:
    """int8 m x n row-major, uniform in [lo, hi]."""
    g = rng(seed)
    return g.integers(lo, hi + 1, size=(m, n), dtype=np.int16).astype(np.int8)


def field_uniform(seed: int, shape, p: int = P) -> np.ndarray:
    """uint32 array uniform in [0, p)."""
    g = rng(seed)
    return g.integers(0, p, size=shape, dtype=np.uint32)


def field_nonzero(seed: int, shape, p: int = P) -> np.ndarray:
    """uint32 array uniform in [1, p-1]."""
    g = rng(seed)
    return g.integers(1, p, size=shape, dtype=np.uint32)


def permutation(g: np.random.Generator, N: int) -> np.ndarray:
    return g.permutation(N).astype(np.uint32)


def raa_code(seed: int, k: int, r: int, p: int = P) -> dict:
    """Random description of an RAA code of dimension k and block length N = r*k.

    Returns dict(k, r, N, pi1, pi2, v1, v2) with uint32 arrays of length N.
    """
    N = int(k) * int(r)
    g = rng(seed)
    pi1 = permutation(g, N)
    pi2 = permutation(g, N)
    v1 = g.integers(1, p, size=N, dtype=np.uint32)
    v2 = g.integers(1, p, size=N, dtype=np.uint32)
    return dict(k=int(k), r=int(r), N=N, pi1=pi1, pi2=pi2, v1=v1, v2=v2)


def identity_code(k: int, r: int) -> dict:
    """Degenerate code with identity permutations and unit diagonals (test use)."""
    N = int(k) * int(r)
    ident = np.arange(N, dtype=np.uint32)
    ones = np.ones(N, dtype=np.uint32)
    return dict(k=int(k), r=int(r), N=N, pi1=ident.copy(), pi2=ident.copy(), v1=ones.copy(), v2=ones.copy())


def sparse(seed: int, count: int, N: int, t: int, p: int = P) -> tuple[np.ndarray, np.ndarray]:
    """``count`` independent draws from E_t^N.

    Returns (idx, val), each uint32 of shape (count, t).  idx rows hold t
    distinct positions in [0, N); val entries are uniform in [1, p-1].
    """
    if t > N:
        raise ValueError("sparsity t exceeds length N")
    g = rng(seed)
    idx = np.empty((count, t), dtype=np.uint32)
    for c in range(count):
        if t * 4 < N:
            # rejection of repeats in draw order (cheap when t << N)
            seen: set[int] = set()
            out = []
            while len(out) < t:
                cand = g.integers(0, N, size=2 * (t - len(out)) + 4)
                for v in cand.tolist():
                    if v not in seen:
                        seen.add(v)
                        out.append(v)
                        if len(out) == t:
                            break
            idx[c] = np.asarray(out, dtype=np.uint32)
        else:
            idx[c] = g.choice(N, size=t, replace=False).astype(np.uint32)
    val = g.integers(1, p, size=(count, t), dtype=np.uint32)
    return idx, val


def tamper_delta(seed: int, count: int, m: int, p: int = P) -> tuple[np.ndarray, np.ndarray]:
    """Per tampered response: a coordinate in [0, m) and a nonzero additive delta."""
    g = rng(seed)
    pos = g.integers(0, m, size=count, dtype=np.uint32)
    delta = g.integers(1, p, size=count, dtype=np.uint32)
    return pos, delta


# ---------------------------------------------------------------------------
# Workload shapes (LLM-layer shaped matrices; parameters per configuration)
# ---------------------------------------------------------------------------
# Each entry: m x n, B query columns, code rate r (Nx = r*n, Ny = r*m),
# noise weight tx, challenge weight ty and repetitions ell.
CONFIGS = {
    "tiny": dict(cid=0, m=256, n=256, B=1, r=2, tx=8, ty=31, ell=2),
    "attn4096": dict(cid=1, m=4096, n=4096, B=1, r=3, tx=64, ty=31, ell=2),
    "mlp_up_11008x4096": dict(cid=2, m=11008, n=4096, B=16, r=3, tx=64, ty=31, ell=2),
    "mlp_large_28672x8192": dict(cid=3, m=28672, n=8192, B=64, r=4, tx=128, ty=31, ell=2),
}

# The pvMVMD evaluation of Sec. 7.1: square n x n matrices, one query, over
# BabyBear, RAA rate 1/8 for both codes (r = 8), noise weight t_x from Eq. (1)
# for the block length 8n, t_y = 31 and ell = 2.
PAPER_EVAL = dict(cid=6, r=8, ty=31, ell=2, B=1, p=P_BABYBEAR,
                  tx={1024: 160, 2048: 159, 4096: 157, 8192: 156, 16384: 154})

# 32-layer stack: per layer the seven projections of a 4096-wide decoder block
# (q, k, v, o: 4096x4096; up, gate: 11008x4096; down: 4096x11008), 8 columns.
STACK = dict(cid=4, layers=32, B=8, r=3, tx=64, ty=31, ell=2,
             mats=[("q", 4096, 4096), ("k", 4096, 4096), ("v", 4096, 4096), ("o", 4096, 4096),
                   ("up", 11008, 4096), ("gate", 11008, 4096), ("down", 4096, 11008)])
