"""Shared helpers of the GPU parity tests (no method arithmetic here)."""
import numpy as np
import torch

from paper_2203_10428_amd.step import ld_of

# tolerances: max |gpu - oracle| / max |oracle| per tensor
TOL = {"f32": {"act": 1e-4, "grad": 1e-3}, "bf16": {"act": 2e-2, "grad": 3e-2}}


def rel_err(gpu: np.ndarray, ref: np.ndarray) -> float:
    ref = np.asarray(ref, dtype=np.float64)
    gpu = np.asarray(gpu, dtype=np.float64)
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    if ref.size == 0:
        return 0.0
    den = np.abs(ref).max()
    num = np.abs(gpu - ref).max()
    return float(num / den) if den > 0 else float(num)


def dev(x: np.ndarray, f: int = None, dtype=torch.float32) -> torch.Tensor:
    """Upload a [rows, f] array into a zero-padded [rows, ld_of(f)] device matrix."""
    x = np.asarray(x)
    rows, f = x.shape
    t = torch.zeros((rows, ld_of(f)), dtype=dtype, device="cuda")
    t[:, :f] = torch.from_numpy(x.astype(np.float32)).to("cuda").to(dtype)
    return t


def host(t: torch.Tensor, f: int) -> np.ndarray:
    torch.cuda.synchronize()
    return t[:, :f].float().cpu().numpy().astype(np.float64)


def random_partition_graph(n_inner, n_pool, nparts, mean_deg, seed, hub_deg=0):
    """A symmetric random graph whose first n_inner nodes are partition 0."""
    rng = np.random.default_rng(seed)
    n = n_inner + n_pool
    m = int(n_inner * mean_deg / 2)
    u = rng.integers(0, n_inner, m)
    v = rng.integers(0, n, m)
    if hub_deg:
        u = np.concatenate([u, np.zeros(hub_deg, np.int64)])
        v = np.concatenate([v, rng.integers(1, n, hub_deg)])
    keep = u != v
    u, v = u[keep], v[keep]
    src, dst = np.concatenate([u, v]), np.concatenate([v, u])
    key = np.unique(src * n + dst)
    src, dst = key // n, key % n
    rowptr = np.zeros(n + 1, np.int64)
    np.cumsum(np.bincount(src, minlength=n), out=rowptr[1:])
    owner = np.zeros(n, np.int32)
    owner[n_inner:] = 1 + rng.integers(0, nparts - 1, n_pool)
    return n, rowptr, dst.astype(np.int32), owner
