"""The work plan the planning workgroup writes into the workspace, read back
after a call and compared with the host mirror of its integer formulas
(tests/test_plan_host.py): piece size, cut row tiles, pieces per row tile,
partial-slot prefixes, piece sections and every item descriptor.  The
reordered last quarter of a queue holds the same descriptors as the mirror's
(its order among equal lengths is free), longest first.

Ascending selections only: the device is never given an out-of-contract
selection (the mirror covers those)."""
import collections

import numpy as np
import pytest

from tests.gpu_util import log
from tests.test_plan_host import GEOS, check

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

HDR, SORT_CAP, MAGIC = 32, 2048, 0x43530231


@pytest.fixture(scope="module", autouse=True)
def _gpu(built_lib):
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")


def B():
    from paper_2607_19547_amd import binding
    return binding


@pytest.mark.parametrize("G,hkv,T,k", GEOS)
def test_device_plan_matches_mirror(G, hkv, T, k):
    b = B()
    rng = np.random.default_rng(T + k)
    cs1 = T // 16
    sel = np.sort(rng.choice(np.arange(cs1, T), size=k, replace=False))
    log(f"case device plan G={G} Hkv={hkv} T={T} k={k}")
    D, hq = 128, G * hkv
    cs = np.array([0, cs1, T], dtype=np.int64)
    geo = b.Geo(1, hq, hkv, D, (16, 24, 24), "bf16", cs)
    n = T - cs1
    z = lambda *s: torch.zeros(*s, dtype=torch.bfloat16, device="cuda")
    K, V, Q, KF, VF = z(1, hkv, T, D), z(1, hkv, T, D), z(1, hq, n, D), z(1, hkv, n, D), z(1, hkv, n, D)
    S_dev = torch.from_numpy(sel.astype(np.int32)).cuda()
    out = torch.empty((1, hq, k, D), dtype=torch.bfloat16, device="cuda")
    # (zeroed: a block the allocator hands back may hold a matching plan, which the call would keep)
    ws = torch.zeros(b.selective_attend_scatter_workspace(geo, k, 1), dtype=torch.uint8, device="cuda")
    b.selective_attend_scatter(geo, K, V, 0, 1, S_dev, k, Q, KF, VF, out, None, ws)
    torch.cuda.synchronize()
    plan = ws.view(torch.int32).cpu().numpy()

    want = check(sel, k, G, T, hkv)
    nt = want["n_tiles"]
    nsp_w = want["nsp"]
    n_cut = sum(1 for x in nsp_w if x > 1)
    nj = max(nsp_w) if max(nsp_w) > 1 else 0
    hdr = plan[:HDR]
    assert hdr[8] == want["nq"] and hdr[9] == want["S"], (hdr[8:10], want["nq"], want["S"])
    assert hdr[10] == n_cut and hdr[11] == nj and hdr[12] == want["per_q"], (hdr[10:13], n_cut, nj, want["per_q"])
    nsp = plan[HDR + nt:HDR + 2 * nt]
    ppre = plan[HDR + 2 * nt:HDR + 3 * nt + 1]
    assert list(nsp) == nsp_w
    assert list(ppre) == want["ppre"]
    # what the plan was made from (a later call compares it), and a fresh plan's mark
    assert list(hdr[16:22]) == [MAGIC, nt, 256 // G, hkv, hdr[20], hdr[14]] and hdr[24] == 0
    assert list(plan[HDR:HDR + nt]) == list(want["nu"])
    # its checksum: two position-weighted sums (mod 2^32) over the header's [8, 16), pieces and
    # partial-slot prefixes, piece sections and item descriptors
    pj0 = HDR + 3 * nt + 1
    idx = np.concatenate([np.arange(8, 16), np.arange(HDR + nt, pj0), np.arange(pj0, pj0 + nj + 1),
                          np.arange(int(hdr[14]), int(hdr[14]) + 4 * want["per_q"])]).astype(np.uint64)
    v = plan.view(np.uint32)[idx.astype(np.int64)].astype(np.uint64)
    m32 = np.uint64(0xFFFFFFFF)
    c1 = int(np.sum((v * (2 * idx + 1)) & m32) & m32)
    c2 = int(np.sum((((v ^ ((idx * 0x9E3779B9) & m32)) * 0x85EBCA6B) & m32) + idx) & m32)
    assert (c1, c2) == (int(np.uint32(hdr[22])), int(np.uint32(hdr[23]))), "checksum words"
    # descriptors: {row tile, KV head in the queue | piece << 16, first and end key tile}
    per_q, off = want["per_q"], int(hdr[14])
    d = plan[off:off + 4 * per_q].reshape(per_q, 4)
    got = [(int(r[0]), int(r[1]) & 0xffff, int(r[1]) >> 16, int(r[2]), int(r[3])) for r in d]
    exp = [want["desc"][p] for p in range(per_q)]
    r0 = per_q - (per_q + 3) // 4
    head = r0 if per_q - r0 <= SORT_CAP else per_q
    assert got[:head] == exp[:head], "descriptors before the reordered tail"
    assert collections.Counter(got[head:]) == collections.Counter(exp[head:]), "the tail's descriptors"
    lens = [e - b_ for (_, _, _, b_, e) in got[head:]]
    shift = 0
    while (want["S"] >> shift) > 255:
        shift += 1
    buckets = [min(x >> shift, 255) for x in lens]
    assert all(x >= y for x, y in zip(buckets, buckets[1:])), "the tail is ordered longest first"
    log(f"  {nt} row tiles, {n_cut} cut, most pieces {nj}, {per_q} positions per queue: plan matches")
