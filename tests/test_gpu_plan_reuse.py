"""The work plan kept in the workspace from one selective-attention call to
the next.  The layer calls of one composition share their selection, so the
planning kernel keeps the plan it finds when that plan was made from the same
key-tile counts and sizes and its checksum holds (header word 24 says which
happened).  Reused or made afresh, the plan gives the same outputs bit for
bit; any change of the selection, the geometry or the stored plan makes a new
one."""
import numpy as np
import pytest

from tests.gpu_util import log

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

REUSED = 24  # header word: 1 when the last planning launch kept the stored plan


@pytest.fixture(scope="module", autouse=True)
def _gpu(built_lib):
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")


def B():
    from paper_2607_19547_amd import binding
    return binding


class Case:
    """A small cache (3 layers, H_q 16, D 128) with random K/V/Q and fresh rows."""

    def __init__(self, T, k, seed, layers=3, hkv=2):
        b = B()
        g = torch.Generator(device="cpu").manual_seed(seed)
        self.T, self.k, self.L, self.hq, self.hkv = T, k, layers, 16, hkv
        cs1 = T // 8
        self.cs = np.array([0, cs1, T], dtype=np.int64)
        self.geo = b.Geo(layers, self.hq, self.hkv, 128, (16, 24, 24), "bf16", self.cs)
        n = T - cs1
        r = lambda *s: torch.randn(*s, generator=g).to(torch.bfloat16).cuda()
        self.K0, self.V0 = r(layers, self.hkv, T, 128), r(layers, self.hkv, T, 128)
        self.Q, self.KF, self.VF = r(layers, self.hq, n, 128), r(layers, self.hkv, n, 128), r(layers, self.hkv, n, 128)
        rng = np.random.default_rng(seed)
        self.sel = self.selection(rng)

    def selection(self, rng):
        s = np.sort(rng.choice(np.arange(int(self.cs[1]), self.T), size=self.k, replace=False))
        return torch.from_numpy(s.astype(np.int32)).cuda()

    def workspace(self, seed):
        """A workspace holding arbitrary bytes (a plan is made in it on first use)."""
        b = B()
        nbytes = b.selective_attend_scatter_workspace(self.geo, self.k, 1)
        g = torch.Generator(device="cpu").manual_seed(seed)
        return torch.randint(0, 256, (nbytes,), dtype=torch.uint8, generator=g).cuda()

    def outputs(self):
        """out [L][H_q][n_sel][128] and lse [L][H_q][n_sel]: a call writes the rows of its layers."""
        return (torch.zeros((self.L, self.hq, self.k, 128), dtype=torch.bfloat16, device="cuda"),
                torch.zeros((self.L, self.hq, self.k), dtype=torch.float32, device="cuda"))

    def call(self, K, V, layer, sel, ws):
        b = B()
        out, lse = self.outputs()
        b.selective_attend_scatter(self.geo, K, V, layer, layer + 1, sel, self.k, self.Q, self.KF, self.VF, out, lse, ws)
        torch.cuda.synchronize()
        return out[layer], lse[layer]


def reused(ws):
    return int(ws[:128].view(torch.int32)[REUSED].item())


# (T, n_sel): cut row tiles with several pieces (and a sorted tail), and uncut ones only
CASES = [(20000, 2500), (1024, 100)]


@pytest.mark.parametrize("T,k", CASES)
def test_layer_calls_reuse_the_plan(T, k):
    c = Case(T, k, seed=T + k)
    log(f"case plan reuse over layer calls T={T} n_sel={k}")
    K, V = c.K0.clone(), c.V0.clone()
    ws = c.workspace(1)
    K2, V2 = c.K0.clone(), c.V0.clone()
    for layer in range(c.L):
        out, lse = c.call(K, V, layer, c.sel, ws)
        assert reused(ws) == (1 if layer > 0 else 0), (layer, reused(ws))
        fresh = c.workspace(100 + layer)  # a plan made afresh for the same call
        out_f, lse_f = c.call(K2, V2, layer, c.sel, fresh)
        assert reused(fresh) == 0
        assert torch.equal(out, out_f) and torch.equal(lse, lse_f), f"layer {layer}"
    assert torch.equal(K, K2) and torch.equal(V, V2)
    log(f"  {c.L} layer calls: the first plans, the others reuse; outputs identical to fresh plans")


def test_changed_selection_is_replanned():
    c = Case(20000, 2500, seed=7)
    log("case plan reuse: a new selection of the same size")
    K, V = c.K0.clone(), c.V0.clone()
    ws = c.workspace(2)
    c.call(K, V, 0, c.sel, ws)
    sel2 = c.selection(np.random.default_rng(99))
    assert not torch.equal(sel2, c.sel)
    Ka, Va = K.clone(), V.clone()
    out, lse = c.call(K, V, 1, sel2, ws)
    assert reused(ws) == 0
    out_f, lse_f = c.call(Ka, Va, 1, sel2, c.workspace(3))
    assert torch.equal(out, out_f) and torch.equal(lse, lse_f)
    # and the same selection again keeps the new plan
    Kb, Vb = K.clone(), V.clone()
    out2, _ = c.call(K, V, 1, sel2, ws)
    assert reused(ws) == 1
    out2_f, _ = c.call(Kb, Vb, 1, sel2, c.workspace(4))
    assert torch.equal(out2, out2_f)


def test_longer_cache_keeps_the_plan():
    """The same selection with a cache one key tile longer: every count and
    size the plan is made from is unchanged (keys past a row's last token are
    never read), so the stored plan is kept, and the outputs are those of a
    fresh plan."""
    b = B()
    c = Case(20000, 2500, seed=11)
    log("case plan reuse: the cache grows by one key tile")
    ws = c.workspace(5)
    c.call(c.K0.clone(), c.V0.clone(), 0, c.sel, ws)
    T2 = c.T + 64
    geo2 = b.Geo(c.L, c.hq, c.hkv, 128, (16, 24, 24), "bf16", np.array([0, c.cs[1], T2], dtype=np.int64))
    assert b.selective_attend_scatter_workspace(geo2, c.k, 1) == ws.numel()
    pad = lambda x: torch.cat([x, torch.zeros_like(x[:, :, :64])], dim=2)
    K2, V2, Q2, KF2, VF2 = pad(c.K0), pad(c.V0), pad(c.Q), pad(c.KF), pad(c.VF)
    outs = []
    for w, want in ((ws, 1), (c.workspace(6), 0)):
        out, _ = c.outputs()
        b.selective_attend_scatter(geo2, K2.clone(), V2.clone(), 0, 1, c.sel, c.k, Q2, KF2, VF2, out, None, w)
        torch.cuda.synchronize()
        assert reused(w) == want
        outs.append(out)
    assert torch.equal(outs[0], outs[1])


def test_changed_geometry_is_replanned():
    """The same workspace and selection size for a cache with four KV heads
    instead of two (64 selected rows per row tile instead of 32: the row tiles
    and the queues change): the stored plan does not match, and a new one is
    made."""
    a = Case(20000, 2500, seed=19)
    c = Case(20000, 2500, seed=19, hkv=4)
    log("case plan reuse: H_kv changes from 2 to 4")
    nbytes = max(B().selective_attend_scatter_workspace(x.geo, x.k, 1) for x in (a, c))
    ws = torch.randint(0, 256, (nbytes,), dtype=torch.uint8, device="cuda")
    a.call(a.K0.clone(), a.V0.clone(), 0, a.sel, ws)
    out, lse = c.call(c.K0.clone(), c.V0.clone(), 0, c.sel, ws)
    assert reused(ws) == 0
    out_f, lse_f = c.call(c.K0.clone(), c.V0.clone(), 0, c.sel, c.workspace(9))
    assert torch.equal(out, out_f) and torch.equal(lse, lse_f)


@pytest.mark.parametrize("where", ["descriptor", "count"])
def test_modified_workspace_is_replanned(where):
    """An int of the stored plan changed between calls: the checksum or the
    stored key-tile counts no longer match, and the plan is made again."""
    c = Case(20000, 2500, seed=13)
    log(f"case plan reuse: the workspace's stored {where} changed")
    K, V = c.K0.clone(), c.V0.clone()
    ws = c.workspace(7)
    c.call(K, V, 0, c.sel, ws)
    plan = ws.view(torch.int32)
    hdr = plan[:32].cpu().numpy()
    if where == "descriptor":
        i = int(hdr[14]) + 4 * (int(hdr[12]) // 2) + 3  # the end key tile of a mid-queue item
        plan[i] += 1
    else:
        plan[32 + 3] += 1  # the stored key-tile count of row tile 3
    Ka, Va = K.clone(), V.clone()
    out, lse = c.call(K, V, 1, c.sel, ws)
    assert reused(ws) == 0
    out_f, lse_f = c.call(Ka, Va, 1, c.sel, c.workspace(8))
    assert torch.equal(out, out_f) and torch.equal(lse, lse_f)


def test_fused_rope_calls_reuse_the_plan():
    """The fused-RoPE call plans in the same kernel: repeated calls over the
    same selection give the outputs of calls with a fresh workspace."""
    b = B()
    c = Case(20000, 2500, seed=17)
    log("case plan reuse: fused RoPE layer calls")
    coords = torch.from_numpy(np.stack([np.arange(c.T)] * 3, axis=1).astype(np.int32)).cuda()
    nbytes = b.selective_attend_scatter_rope_workspace(c.geo, c.k, 1)
    g = torch.Generator(device="cpu").manual_seed(3)
    ws = torch.randint(0, 256, (nbytes,), dtype=torch.uint8, generator=g).cuda()
    K, V = c.K0.clone(), c.V0.clone()
    K2, V2 = c.K0.clone(), c.V0.clone()
    for layer in range(c.L):
        outs = []
        for (KK, VV, w) in ((K, V, ws), (K2, V2, torch.randint(0, 256, (nbytes,), dtype=torch.uint8,
                                                                generator=g).cuda())):
            out, _ = c.outputs()
            b.selective_attend_scatter_rope(c.geo, KK, VV, layer, layer + 1, c.sel, c.k, c.Q, c.KF, c.VF, coords,
                                            out, None, w)
            torch.cuda.synchronize()
            outs.append(out[layer])
        assert torch.equal(outs[0], outs[1]), f"layer {layer}"
    assert torch.equal(K, K2) and torch.equal(V, V2)


def test_batched_call_keeps_the_per_layer_plan():
    """A call over all layers finds the plan the per-layer calls left (the plan
    does not depend on the layer count) and gives the outputs of a batched call
    with a fresh workspace."""
    b = B()
    c = Case(20000, 2500, seed=29)
    log("case plan reuse: a batched call after per-layer calls")
    nbytes = b.selective_attend_scatter_workspace(c.geo, c.k, c.L)
    ws = torch.randint(0, 256, (nbytes,), dtype=torch.uint8, device="cuda")
    K, V = c.K0.clone(), c.V0.clone()
    for layer in range(c.L):
        c.call(K, V, layer, c.sel, ws)
    outs = []
    for w, want in ((ws, 1), (torch.randint(0, 256, (nbytes,), dtype=torch.uint8, device="cuda"), 0)):
        out, lse = c.outputs()
        b.selective_attend_scatter(c.geo, c.K0.clone(), c.V0.clone(), 0, c.L, c.sel, c.k, c.Q, c.KF, c.VF, out, lse,
                                   w)
        torch.cuda.synchronize()
        assert reused(w) == want
        outs.append((out, lse))
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])
