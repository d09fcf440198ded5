"""Product-quantisation codes for the compressed traversal (input preparation).

The paper traverses with product-quantised asymmetric distances and
re-ranks exactly at the end (Alg. 2 "PQDist"; Sec. III-B, steps 2, 6 and
8). Codebooks are trained offline, like the graph; this module trains and
encodes, and holds none of the search arithmetic.

Layout shared by every consumer:
  * M subspaces of ds = d / M consecutive dimensions (M even, d % M == 0);
  * 16 centroids per subspace (4-bit codes): codebook float32 M x 16 x ds;
  * codes: n x M/2 bytes, byte b holding subspace 2b in its low nibble and
    subspace 2b + 1 in its high nibble.

Training: k-means (Lloyd, a fixed number of iterations) per subspace on a
seeded sample, initialised from seeded sample points; encoding: the nearest
centroid in float64, ties to the lowest index.
"""
from __future__ import annotations

import numpy as np

K = 16


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0x50])))


def train(vectors: np.ndarray, M: int, seed: int = 0, sample: int = 65536, iters: int = 16) -> np.ndarray:
    """Codebook (M x 16 x ds float32) by k-means per subspace."""
    n, d = vectors.shape
    assert d % M == 0 and M % 2 == 0
    ds = d // M
    g = _rng(seed)
    idx = np.sort(g.choice(n, min(sample, n), replace=False))
    X = vectors[idx].astype(np.float64).reshape(len(idx), M, ds)
    cb = np.empty((M, K, ds), dtype=np.float64)
    for m in range(M):
        x = X[:, m, :]
        c = x[g.choice(len(x), K, replace=len(x) < K)].copy()
        for _ in range(iters):
            d2 = ((x[:, None, :] - c[None, :, :]) ** 2).sum(-1)
            a = d2.argmin(1)
            for j in range(K):
                sel = a == j
                if sel.any():
                    c[j] = x[sel].mean(0)
        cb[m] = c
    return cb.astype(np.float32)


def encode(vectors: np.ndarray, codebook: np.ndarray, chunk: int = 1 << 16) -> np.ndarray:
    """n x M/2 packed 4-bit codes: the nearest centroid per subspace (float64,
    ties to the lowest index)."""
    n, d = vectors.shape
    M, k, ds = codebook.shape
    cb = codebook.astype(np.float64)
    out = np.empty((n, M // 2), dtype=np.uint8)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        x = vectors[s:e].astype(np.float64).reshape(e - s, M, ds)
        codes = np.empty((e - s, M), dtype=np.uint8)
        for m in range(M):
            d2 = ((x[:, m, None, :] - cb[m][None, :, :]) ** 2).sum(-1)
            codes[:, m] = d2.argmin(1)
        out[s:e] = codes[:, 0::2] | (codes[:, 1::2] << 4)
    return out


def unpack(codes: np.ndarray) -> np.ndarray:
    """n x M centroid indices from packed codes."""
    n, h = codes.shape
    out = np.empty((n, 2 * h), dtype=np.uint8)
    out[:, 0::2] = codes & 15
    out[:, 1::2] = codes >> 4
    return out


def decode(codes: np.ndarray, codebook: np.ndarray) -> np.ndarray:
    """The reconstructed vectors (float64): each subspace's centroid."""
    c = unpack(codes)
    M = codebook.shape[0]
    return np.concatenate([codebook[m][c[:, m]].astype(np.float64) for m in range(M)], axis=1)
