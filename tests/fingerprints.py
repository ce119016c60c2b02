"""Whole-array and hit-set fingerprints computed with plain torch ops, for
comparing the GPU's full-size outputs with the oracle's references without
moving the arrays to the host.  Same definitions as the oracle's:

* array fingerprint: sum over t of mix64(mix64(t + 1) + a[t]) mod 2^64
  (uint32 arrays zero-extended);
* hit-set fingerprint at capacity c: sum of mix64(t + 1) over the accesses
  t with dist[t] < c.

mix64 is splitmix64's finalizer.  torch has no uint64 arithmetic, so the
values live in int64 tensors: addition and multiplication wrap mod 2^64 the
same way, and right shifts are made logical with a mask."""
import torch

_C1 = 0xBF58476D1CE4E5B9 - (1 << 64)
_C2 = 0x94D049BB133111EB - (1 << 64)
CHUNK = 1 << 26


def _shr(z, k):
    return (z >> k) & ((1 << (64 - k)) - 1)


def mix64(z):
    z = z ^ _shr(z, 30)
    z = z * _C1
    z = z ^ _shr(z, 27)
    z = z * _C2
    return z ^ _shr(z, 31)


def to_u64(v):
    """python int of an int64 value's bit pattern"""
    return int(v) & ((1 << 64) - 1)


def _as_u64_values(a):
    if a.dtype == torch.int32:
        return a.to(torch.int64) & 0xFFFFFFFF
    assert a.dtype == torch.int64
    return a


def array_fp(a, t0=0):
    """Fingerprint of an int32 (uint32 bits) or int64 (uint64 bits) tensor."""
    n = a.numel()
    s = torch.zeros((), dtype=torch.int64, device=a.device)
    for lo in range(0, n, CHUNK):
        hi = min(n, lo + CHUNK)
        pos = torch.arange(t0 + lo + 1, t0 + hi + 1, dtype=torch.int64, device=a.device)
        s += (mix64(mix64(pos) + _as_u64_values(a[lo:hi]))).sum()
    return to_u64(s.item())


def hit_fps(dist, caps):
    """Per capacity edge: (hits, hit-set fingerprint) from uint32 distances
    (int32 tensor, NONE = 0xFFFFFFFF never hits) and the edges (int64
    tensor on the same device, ascending)."""
    k = caps.numel()
    n = dist.numel()
    cnt = torch.zeros(k + 1, dtype=torch.int64, device=dist.device)
    fp = torch.zeros(k + 1, dtype=torch.int64, device=dist.device)
    for lo in range(0, n, CHUNK):
        hi = min(n, lo + CHUNK)
        d = dist[lo:hi].to(torch.int64) & 0xFFFFFFFF
        b = torch.bucketize(d, caps, right=True)
        b[d == 0xFFFFFFFF] = k
        cnt += torch.bincount(b, minlength=k + 1)
        pos = torch.arange(lo + 1, hi + 1, dtype=torch.int64, device=dist.device)
        fp.scatter_add_(0, b, mix64(pos))
    hits = torch.cumsum(cnt[:k], 0).cpu().tolist()
    fps = torch.cumsum(fp[:k], 0).cpu().tolist()
    return [(int(h), to_u64(f)) for h, f in zip(hits, fps)]
