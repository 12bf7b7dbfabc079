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


def check_scores_and_selection(got_scores, ref_scores, got_sel, k, cs1, select_top):
    """Scores: float32, equal to the oracle's or one ulp away (the GPU sums the
    float64 squares in another order; the two roundings to float32 can land on
    adjacent values within ~1e-16 of a midpoint).  Selection: identical to the
    oracle's when the scores are; otherwise exact on the GPU's own scores, and
    every index in one set but not the other within a relative score gap of
    1e-6 of its counterpart (the tie window of the selection bar)."""
    g = np.asarray(got_scores, np.float32)
    r = np.asarray(ref_scores, np.float32)
    d = np.abs(g.view(np.int32).astype(np.int64) - r.view(np.int32).astype(np.int64))
    assert d.max(initial=0) <= 1, f"scores differ by {d.max()} float32 ulps"
    sel = np.asarray(got_sel[:k], np.int64)
    want = select_top(r, k, cs1)
    if not d.any():
        assert sel.tolist() == want.tolist()
        return 0
    assert sel.tolist() == select_top(g, k, cs1).tolist()
    extra, missing = sorted(set(sel.tolist()) - set(want.tolist())), sorted(set(want.tolist()) - set(sel.tolist()))
    assert len(extra) == len(missing)
    sc = r.astype(np.float64)
    for i, j in zip(extra, missing):
        a, b = sc[i - cs1], sc[j - cs1]
        assert abs(a - b) < 1e-6 * max(a, b), (i, j, a, b)
    return int(d.sum())
