"""Shared helpers of the GPU parity tests (host <-> device marshalling and
the comparison metrics).  No arithmetic of the method lives here."""
import numpy as np


def to_dev(x, dtype):
    """numpy storage array (uint16 bf16 bits or float32) -> CUDA tensor."""
    import torch
    x = np.ascontiguousarray(x)
    if dtype == "bf16":
        return torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(x.astype(np.float32)).cuda()


def to_host(t, dtype):
    """CUDA tensor -> numpy storage array (uint16 bf16 bits or float32)."""
    import torch
    t = t.detach().cpu().contiguous()
    if dtype == "bf16":
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy().astype(np.float32)


def empty(shape, dtype):
    import torch
    return torch.empty(shape, dtype=torch.bfloat16 if dtype == "bf16" else torch.float32, device="cuda")


def rel_l2(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def pair_norm(x):
    """Per-element norm of the rotary pair the element belongs to, [..., D]."""
    P = x.shape[-1] // 2
    pn = np.hypot(x[..., :P], x[..., P:])
    return np.concatenate([pn, pn], axis=-1)


def ulp(x, dtype):
    """Spacing of the storage format at |x| (bf16: 8 significant bits, float32: 24)."""
    mant, emin = (7, -126) if dtype == "bf16" else (23, -126)
    _, e = np.frexp(np.abs(np.asarray(x, dtype=np.float64)))
    lead = np.maximum(e.astype(np.int64) - 1, emin)
    return np.ldexp(1.0, lead - mant)


def log(*a):
    print(*a, flush=True)
