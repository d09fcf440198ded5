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
seeded sample, initialised from seeded sample points (torch, all subspaces
at once); encoding: the nearest centroid, ties to the lowest index.
"""
from __future__ import annotations

import numpy as np

K = 16


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0x50])))


def _torch_dev(device):
    import torch
    dev = torch.device(device)
    return torch, dev, (torch.float64 if dev.type == "cpu" else torch.float32)


def train(vectors: np.ndarray, M: int, seed: int = 0, sample: int = 65536, iters: int = 16,
          device: str = "cpu") -> np.ndarray:
    """Codebook (M x 16 x ds float32) by k-means, all subspaces at once
    (float64 on the CPU, float32 on a GPU)."""
    torch, dev, dt = _torch_dev(device)
    n, d = vectors.shape
    assert d % M == 0 and M % 2 == 0
    ds = d // M
    g = _rng(seed)
    idx = np.sort(g.choice(n, min(sample, n), replace=False))
    S = len(idx)
    X = torch.from_numpy(vectors[idx].astype(np.float32)).to(dev).to(dt).reshape(S, M, ds)
    init = g.choice(S, K, replace=S < K)
    C = X[torch.from_numpy(init).to(dev)].permute(1, 0, 2).contiguous()    # M x K x ds
    ar = torch.arange(M, device=dev)
    for _ in range(iters):
        d2 = ((X[:, :, None, :] - C[None, :, :, :]) ** 2).sum(-1)          # S x M x K
        a = d2.argmin(-1)                                                   # S x M
        flat = (ar[None, :] * K + a).reshape(-1)
        sums = torch.zeros((M * K, ds), dtype=dt, device=dev).index_add_(0, flat, X.reshape(-1, ds))
        cnt = torch.zeros(M * K, dtype=dt, device=dev).index_add_(0, flat, torch.ones_like(flat, dtype=dt))
        upd = sums / cnt.clamp_min(1)[:, None]
        keep = (cnt == 0)[:, None]
        C = torch.where(keep, C.reshape(M * K, ds), upd).reshape(M, K, ds)
    return C.cpu().numpy().astype(np.float32)


def encode(vectors: np.ndarray, codebook: np.ndarray, chunk: int = 1 << 14, device: str = "cpu") -> np.ndarray:
    """n x M/2 packed 4-bit codes: the nearest centroid per subspace (ties
    to the lowest index; float64 on the CPU, float32 on a GPU)."""
    torch, dev, dt = _torch_dev(device)
    n, d = vectors.shape
    M, k, ds = codebook.shape
    cb = torch.from_numpy(codebook).to(dev).to(dt)
    out = np.empty((n, M // 2), dtype=np.uint8)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        x = torch.from_numpy(vectors[s:e].astype(np.float32)).to(dev).to(dt).reshape(e - s, M, ds)
        c = ((x[:, :, None, :] - cb[None]) ** 2).sum(-1).argmin(-1).to(torch.uint8).cpu().numpy()
        out[s:e] = c[:, 0::2] | (c[:, 1::2] << 4)
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
