"""Helpers for the GPU parity tests: move synth arrays to the device and back."""
from __future__ import annotations

import numpy as np
import torch

import paper_2609_10264_amd as mvk
import synth


def dev(a: np.ndarray) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype == np.int8:
        return torch.from_numpy(a).cuda()
    assert a.dtype in (np.uint32, np.int32, np.int64)
    assert int(a.max(initial=0)) < 2**31
    return torch.from_numpy(a.astype(np.int32)).cuda()


def host(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().astype(np.uint32)


def code(c: dict, p: int = synth.P) -> mvk.Code:
    return mvk.Code(c["k"], c["r"], dev(c["pi1"]), dev(c["pi2"]), dev(c["v1"]), dev(c["v2"]), p)


class Instance:
    """One seeded pvMVMD instance: W, X, the two codes, noise and challenges."""

    def __init__(self, cid: int, m: int, n: int, B: int, r: int, tx: int, ty: int = 31, ell: int = 2,
                 ry: int | None = None, sub: int = 0, p: int = synth.P):
        self.m, self.n, self.B, self.p = m, n, B, p
        sd = lambda purpose: synth.seed_for(cid, purpose, sub)  # noqa: E731
        self.W = synth.weights(sd(synth.PURPOSE_W), m, n)
        self.X = synth.field_uniform(sd(synth.PURPOSE_X), (B, n), p=p)
        self.cx = synth.raa_code(sd(synth.PURPOSE_CX), n, r, p=p)
        self.cy = synth.raa_code(sd(synth.PURPOSE_CY), m, ry or r, p=p)
        self.exi, self.exv = synth.sparse(sd(synth.PURPOSE_NOISE), B, self.cx["N"], tx, p=p)
        self.eyi, self.eyv = synth.sparse(sd(synth.PURPOSE_CHAL), ell, self.cy["N"], ty, p=p)

    def to_device(self):
        self.dW = dev(self.W)
        self.dX = dev(self.X)
        self.key = mvk.Key.allocate(self.m, self.n, code(self.cx, self.p), code(self.cy, self.p))
        self.dexi, self.dexv = dev(self.exi), dev(self.exv)
        self.deyi, self.deyv = dev(self.eyi), dev(self.eyv)
        return self
