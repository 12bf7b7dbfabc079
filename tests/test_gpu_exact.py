"""Exact-answer attention checks on the timed geometry (65,536 tokens in 32
chunks of 2,048, 16 query / 2 KV heads, head_dim 128, bf16), through the C ABI.

Inputs with a known answer (Eq. 1 over the post-scatter cache, the repair
step of Section 2) catch structural errors that a rel-L2 bar over a whole
layer cannot see: a dropped or repeated 64-key tile, a causal boundary off by
one, a lost key piece.
  * zero query: every score is 0, so every visible key has probability 1:
    lse = ln(t + 1) and the output is the mean of V[0..t] of the post-scatter
    cache (expected values from float64 prefix sums on the host);
  * identical keys (all rows of a head equal, fresh rows too): every score
    equals q.k0 / sqrt(D), so lse = q.k0 / sqrt(D) + ln(t + 1) and the output
    is again the mean of V[0..t];
  * constant values (every stored and fresh V row of a head equal to u, with
    |u_d| in [1/4, 2]): the output is u exactly, whatever the weights.
Each at rho = 0.1 and 1 (cut row tiles and their combine), one call per layer,
on the contiguous cache and on 32 chunk buffers.

Full-size bit-identity: the batched 36-layer call and a HIP-graph replay of
the 36 per-layer calls against the per-layer calls, and the fused-rotary call
against the oracle's rotation on sampled rows."""
import math

import numpy as np
import pytest

import oracle
from oracle import bf16 as obf
from paper_2607_19547_amd import synth
from tests.gpu_util import log, pair_norm, rel_l2, ulp
from tests.test_plan_host import check as plan_check

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

L, HQ, HKV, D, CH, NCH = 2, 16, 2, 128, 2048, 32
G = HQ // HKV


@pytest.fixture(scope="module", autouse=True)
def _gpu(built_lib):
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")


def B():
    from paper_2607_19547_amd import binding
    return binding


def _geo(layers=L):
    cs = np.arange(NCH + 1, dtype=np.int64) * CH
    return B().Geo(layers, HQ, HKV, D, (16, 24, 24), "bf16", cs), cs


def _sel(rho, seed):
    T, cs1 = NCH * CH, CH
    n = T - cs1
    k = int(math.ceil(rho * n - 1e-9))
    rng = np.random.default_rng(seed)
    return np.sort(rng.choice(np.arange(cs1, T), size=k, replace=False)).astype(np.int64)


def _randn(shape, seed, lo=None):
    g = torch.Generator(device="cuda").manual_seed(seed)
    x = torch.randn(shape, generator=g, device="cuda", dtype=torch.float32)
    if lo is not None:  # magnitudes in [lo, 2], random signs
        x = torch.sign(x) * (lo + (2 - lo) * torch.rand(shape, generator=g, device="cuda"))
    return x.to(torch.bfloat16)


def _run(geo, cs, K, V, Q, KF, VF, sel_np, paged):
    b = B()
    S = torch.from_numpy(sel_np.astype(np.int32)).cuda()
    k = len(sel_np)
    out = torch.empty((L, HQ, k, D), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((L, HQ, k), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(1, b.selective_attend_scatter_workspace(geo, k, 1)), dtype=torch.uint8, device="cuda")
    if paged:
        kc = [K[:, :, cs[c]:cs[c + 1]].contiguous() for c in range(NCH)]
        vc = [V[:, :, cs[c]:cs[c + 1]].contiguous() for c in range(NCH)]
        for l in range(L):
            b.selective_attend_scatter_paged(geo, kc, vc, l, l + 1, S, k, Q, KF, VF, out, lse, ws)
        torch.cuda.synchronize()
        K = torch.cat(kc, dim=2)
        V = torch.cat(vc, dim=2)
    else:
        for l in range(L):
            b.selective_attend_scatter(geo, K, V, l, l + 1, S, k, Q, KF, VF, out, lse, ws)
        torch.cuda.synchronize()
    return K, V, out, lse


def _post_scatter_mean(V_host, VF_host, sel, cs1):
    """Mean of V[0..t] of the post-scatter cache for every selected t: [L][H_kv][k][D] float64."""
    Vp = np.array(V_host, dtype=np.float64)
    Vp[:, :, sel, :] = VF_host[:, :, sel - cs1, :]
    cum = np.cumsum(Vp, axis=2)
    return cum[:, :, sel, :] / (sel + 1)[None, None, :, None], Vp


def _host(x):
    return x.float().cpu().numpy().astype(np.float64)


# A row tile cut into key pieces keeps each piece's O / sum in fp16, scaled so
# that the largest of its 128 elements lies in [0.5, 1): 2^-12 of that
# element, absolute, per piece.  A piece spans at least 4,096 keys, so with
# V ~ N(0, 1) the largest element of a piece's mean stays below 0.1 (about 6
# standard deviations of a 4,096-key mean), and the merged output is within
# 2^-12 x 0.1 < 3e-5 of the float32 result.  A dropped or repeated 64-key
# tile moves the mean of a 35,000-key prefix by ~sqrt(64) / 35,000 = 2.3e-4,
# far outside this bar (and moves lse by ~64 / 35,000 = 1.8e-3).
PIECE_ABS = 3e-5


def _check_mean(out, mean, tag):
    """out [L][HQ][k][D] (device) against the per-KV-head mean [L][HKV][k][D] (host float64)."""
    k = out.shape[2]
    exp = torch.from_numpy(mean).cuda()[:, :, None]                          # [L][HKV][1][k][D]
    _, e = torch.frexp(exp.abs())
    tol = torch.ldexp(torch.ones_like(exp), (e - 8).clamp(min=-133)) + PIECE_ABS  # 1 bf16 ulp at |mean| + pieces
    err = (out.view(L, HKV, G, k, D).double() - exp).abs()
    ratio = float((err / tol).max())
    bad = int((err > tol).sum())
    emax = float(err.max())
    log(f"  {tag}: output vs mean of V[0..t]: max abs err {emax:.2e}, max err/tol {ratio:.3f}, {bad} outside")
    assert bad == 0


@pytest.mark.parametrize("paged", [False, True], ids=["contiguous", "paged"])
@pytest.mark.parametrize("rho", [0.1, 1.0])
def test_zero_query_gives_prefix_mean(rho, paged):
    geo, cs = _geo()
    T, cs1, n = int(cs[-1]), CH, int(cs[-1]) - CH
    sel = _sel(rho, seed=11)
    log(f"case zero query rho={rho} paged={paged} k={len(sel)}")
    K, V = _randn((L, HKV, T, D), 1), _randn((L, HKV, T, D), 2)
    KF, VF = _randn((L, HKV, n, D), 3), _randn((L, HKV, n, D), 4)
    Q = torch.zeros((L, HQ, n, D), dtype=torch.bfloat16, device="cuda")
    mean, Vp = _post_scatter_mean(_host(V), _host(VF), sel, cs1)
    Kp, Vg, out, lse = _run(geo, cs, K, V, Q, KF, VF, sel, paged)
    assert np.array_equal(_host(Vg), Vp), "scattered values"
    want = torch.from_numpy(np.log(sel + 1.0)).cuda()
    lerr = float((lse.double() - want[None, None, :]).abs().max())
    log(f"  lse vs ln(t+1): max abs {lerr:.2e}")
    assert lerr <= 1e-5
    _check_mean(out, mean, f"zero query rho={rho}")


@pytest.mark.parametrize("paged", [False, True], ids=["contiguous", "paged"])
@pytest.mark.parametrize("rho", [0.1, 1.0])
def test_identical_keys_give_prefix_mean(rho, paged):
    geo, cs = _geo()
    T, cs1, n = int(cs[-1]), CH, int(cs[-1]) - CH
    sel = _sel(rho, seed=12)
    log(f"case identical keys rho={rho} paged={paged} k={len(sel)}")
    k0 = _randn((L, HKV, 1, D), 5)
    K = k0.expand(L, HKV, T, D).contiguous()
    KF = k0.expand(L, HKV, n, D).contiguous()
    V, VF = _randn((L, HKV, T, D), 6), _randn((L, HKV, n, D), 7)
    Q = _randn((L, HQ, n, D), 8)
    mean, _ = _post_scatter_mean(_host(V), _host(VF), sel, cs1)
    # q . k0 / sqrt(D) of every selected row and head, in float64
    qs = Q[:, :, torch.from_numpy(sel - cs1).cuda()].double().view(L, HKV, G, len(sel), D)
    dots = ((qs * k0.double()[:, :, None]).sum(-1) / math.sqrt(D)).view(L, HQ, len(sel)).cpu().numpy()
    del qs
    Kp, _, out, lse = _run(geo, cs, K, V, Q, KF, VF, sel, paged)
    assert torch.equal(Kp, K), "every key row equals k0 after the scatter"
    want = dots + np.log(sel + 1.0)[None, None, :]
    lerr = float(np.max(np.abs(lse.cpu().numpy() - want)))
    log(f"  lse vs q.k0/sqrt(D) + ln(t+1): max abs {lerr:.2e}")
    assert lerr <= 1e-4
    _check_mean(out, mean, f"identical keys rho={rho}")


@pytest.mark.parametrize("paged", [False, True], ids=["contiguous", "paged"])
@pytest.mark.parametrize("rho", [0.1, 1.0])
def test_constant_values_give_that_value(rho, paged):
    geo, cs = _geo()
    T, n = int(cs[-1]), int(cs[-1]) - CH
    sel = _sel(rho, seed=13)
    log(f"case constant values rho={rho} paged={paged} k={len(sel)}")
    u = _randn((L, HKV, 1, D), 9, lo=0.25)
    V = u.expand(L, HKV, T, D).contiguous()
    VF = u.expand(L, HKV, n, D).contiguous()
    K, KF, Q = _randn((L, HKV, T, D), 10), _randn((L, HKV, n, D), 11), _randn((L, HQ, n, D), 12)
    _, _, out, lse = _run(geo, cs, K, V, Q, KF, VF, sel, paged)
    want = u.repeat_interleave(G, dim=1).expand(L, HQ, len(sel), D)
    diff = int((out != want).sum())
    log(f"  output == u: {diff} elements differ")
    assert diff == 0
    assert bool(torch.isfinite(lse).all())


def test_zero_query_many_pieces():
    """Row tiles cut into many key pieces: 301,056 tokens, 32 query heads on
    one KV head, 40 selected rows near the end (five row tiles of ~4,700 key
    tiles, cut into pieces of the smallest size: 294 per row tile, the host
    mirror's count).  Zero query: lse = ln(t + 1) and the output is the mean
    of V[0..t] after the merge of every piece."""
    b = B()
    hq, hkv, nch = 32, 1, 147
    cs = np.arange(nch + 1, dtype=np.int64) * CH
    geo = b.Geo(1, hq, hkv, D, (16, 24, 24), "bf16", cs)
    T, cs1 = int(cs[-1]), CH
    n = T - cs1
    rng = np.random.default_rng(21)
    sel = np.sort(rng.choice(np.arange(T - 20000, T), size=40, replace=False)).astype(np.int64)
    log(f"case zero query, many pieces: T={T} k={len(sel)}")
    K, V = _randn((1, hkv, T, D), 31), _randn((1, hkv, T, D), 32)
    KF, VF = _randn((1, hkv, n, D), 33), _randn((1, hkv, n, D), 34)
    Q = torch.zeros((1, hq, n, D), dtype=torch.bfloat16, device="cuda")
    mean, _ = _post_scatter_mean(_host(V), _host(VF), sel, cs1)
    S = torch.from_numpy(sel.astype(np.int32)).cuda()
    k = len(sel)
    out = torch.empty((1, hq, k, D), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((1, hq, k), dtype=torch.float32, device="cuda")
    ws = torch.empty(b.selective_attend_scatter_workspace(geo, k, 1), dtype=torch.uint8, device="cuda")
    b.selective_attend_scatter(geo, K, V, 0, 1, S, k, Q, KF, VF, out, lse, ws)
    torch.cuda.synchronize()
    most = int(ws[:64].view(torch.int32)[11])  # the plan's header: most pieces of a row tile
    want_most = max(plan_check(sel, k, hq // hkv, T, hkv)["nsp"])
    log(f"  most pieces of a row tile: {most} (host mirror {want_most})")
    assert most == want_most and most > 60
    want = torch.from_numpy(np.log(sel + 1.0)).cuda()
    lerr = float((lse.double() - want[None, None, :]).abs().max())
    log(f"  lse vs ln(t+1): max abs {lerr:.2e}")
    assert lerr <= 1e-5
    exp = torch.from_numpy(mean).cuda()[:, :, None]                          # [1][1][1][k][D]
    _, e = torch.frexp(exp.abs())
    tol = torch.ldexp(torch.ones_like(exp), (e - 8).clamp(min=-133)) + PIECE_ABS
    err = (out.view(1, hkv, hq, k, D).double() - exp).abs()
    log(f"  output vs mean of V[0..t]: max abs err {float(err.max()):.2e}, max err/tol {float((err / tol).max()):.3f}")
    assert int((err > tol).sum()) == 0


# ------------------------------------------------------------ full-size bit identity
def test_batched_and_graph_equal_per_layer_36_layers():
    """The timed composition's attention stage at full size (36 layers): one
    batched call over all layers, and the 36 per-layer calls captured into a
    HIP graph and replayed, are bit-identical to the 36 eager per-layer calls
    (rho = 0.1 and 1)."""
    b = B()
    Lf = 36
    geo, cs = _geo(Lf)
    T, cs1, n = int(cs[-1]), CH, int(cs[-1]) - CH
    K0, V0 = _randn((Lf, HKV, T, D), 21), _randn((Lf, HKV, T, D), 22)
    KF, VF, Q = _randn((Lf, HKV, n, D), 23), _randn((Lf, HKV, n, D), 24), _randn((Lf, HQ, n, D), 25)
    for rho in (0.1, 1.0):
        sel = _sel(rho, seed=14)
        k = len(sel)
        log(f"case 36 layers rho={rho} k={k}")
        S = torch.from_numpy(sel.astype(np.int32)).cuda()
        res = {}
        for mode in ("per_layer", "batched", "graph"):
            K, V = K0.clone(), V0.clone()
            out = torch.empty((Lf, HQ, k, D), dtype=torch.bfloat16, device="cuda")
            lse = torch.empty((Lf, HQ, k), dtype=torch.float32, device="cuda")
            per = 1 if mode != "batched" else Lf
            ws = torch.empty(b.selective_attend_scatter_workspace(geo, k, per), dtype=torch.uint8, device="cuda")
            ranges = [(0, Lf)] if mode == "batched" else [(l, l + 1) for l in range(Lf)]
            if mode == "graph":
                torch.cuda.synchronize()
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g):  # the calls enqueue on the capturing stream
                    for lb, le in ranges:
                        b.selective_attend_scatter(geo, K, V, lb, le, S, k, Q, KF, VF, out, lse, ws)
                torch.cuda.synchronize()
                out.fill_(0)
                lse.fill_(0)
                g.replay()
                torch.cuda.synchronize()
            else:
                for lb, le in ranges:
                    b.selective_attend_scatter(geo, K, V, lb, le, S, k, Q, KF, VF, out, lse, ws)
                torch.cuda.synchronize()
            res[mode] = (K, V, out, lse)
            del ws
        for mode in ("batched", "graph"):
            for name, x, y in zip(("K", "V", "out", "lse"), res[mode], res["per_layer"]):
                assert torch.equal(x, y), f"{mode} {name} differs from the per-layer calls"
        log("  batched and graph replay bit-identical to the per-layer calls")
        del res
        torch.cuda.empty_cache()


@pytest.mark.parametrize("rho", [0.1, 1.0])
def test_fused_rope_full_size_sampled(rho):
    """selective_attend_scatter_rope on the timed geometry (2 layers): every
    scattered K row of sampled selected tokens against the oracle's rotation at
    the global coordinates (1 bf16 ulp + 2^-20 |pair|), V rows exact, rows not
    selected untouched, and sampled output slots against the oracle's
    attention over the oracle-rotated rows."""
    b = B()
    w = synth.WORKLOADS["long65k"]
    geo, cs = _geo()
    T, cs1, n = int(cs[-1]), CH, int(cs[-1]) - CH
    glob = (synth.local_coords(w) + np.repeat(synth.chunk_offsets(w), CH, axis=0)).astype(np.int32)
    sel = _sel(rho, seed=15)
    k = len(sel)
    log(f"case fused rope full size rho={rho} k={k}")
    K, V = _randn((L, HKV, T, D), 31), _randn((L, HKV, T, D), 32)
    QP, KP, VF = _randn((L, HQ, n, D), 33), _randn((L, HKV, n, D), 34), _randn((L, HKV, n, D), 35)
    K_host, V_host, VF_host = K.cpu(), V.cpu(), VF.cpu()
    C = torch.from_numpy(glob).cuda()
    S = torch.from_numpy(sel.astype(np.int32)).cuda()
    out = torch.empty((L, HQ, k, D), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((L, HQ, k), dtype=torch.float32, device="cuda")
    ws = torch.empty(b.selective_attend_scatter_rope_workspace(geo, k, 1), dtype=torch.uint8, device="cuda")
    for l in range(L):
        b.selective_attend_scatter_rope(geo, K, V, l, l + 1, S, k, QP, KP, VF, C, out, lse, ws)
    torch.cuda.synchronize()
    th, sg = oracle.rope.inv_freq(D, 1.0e6), oracle.rope.axis_of_pair((16, 24, 24))

    def bits(t):
        return t.contiguous().view(torch.int16).numpy().view(np.uint16)

    # every selected row's key, oracle-rotated (Eq. 2 at p', one rounding to bf16)
    kp_sel = obf.decode(bits(KP[:, :, torch.from_numpy(sel - cs1).cuda()].cpu()))   # [L][HKV][k][D]
    k_rot = obf.encode(oracle.rope.apply_mrope(kp_sel, glob[sel], th, sg))
    Kg, Vg = K.cpu(), V.cpu()
    rt = 8 * (32 // G)
    rng = np.random.default_rng(int(rho * 100))
    slots = np.unique(np.concatenate([[0, k - 1, rt - 1, rt, k // 2], rng.choice(k, size=min(24, k), replace=False)]))
    for l in range(L):
        kg = bits(Kg[l])
        assert np.array_equal(bits(Vg[l])[:, sel], bits(VF_host[l])[:, sel - cs1]), "scattered values"
        other = np.ones(T, bool)
        other[sel] = False
        assert np.array_equal(kg[:, other], bits(K_host[l])[:, other]), "rows not selected untouched"
        g_, o_ = obf.decode(kg[:, sel]), obf.decode(k_rot[l])
        assert np.all(np.abs(g_ - o_) <= ulp(o_, "bf16") + 2.0 ** -20 * pair_norm(o_)), "rotated keys"
        # sampled output slots: oracle attention of the oracle-rotated query over the post-scatter cache
        kpost = obf.decode(bits(K_host[l])).copy()
        kpost[:, sel] = o_
        vpost = obf.decode(bits(V_host[l])).copy()
        vpost[:, sel] = obf.decode(bits(VF_host[l]))[:, sel - cs1]
        qs = obf.decode(bits(QP[l][:, torch.from_numpy(sel[slots] - cs1).cuda()].cpu()))
        q_rot = obf.decode(obf.encode(oracle.rope.apply_mrope(qs, glob[sel[slots]], th, sg)))
        o_ref = np.zeros((HQ, len(slots), D))
        lse_ref = np.zeros((HQ, len(slots)))
        for i, t in enumerate(sel[slots]):
            o1, l1 = oracle.attention.attend_rows(q_rot[:, i:i + 1], kpost, vpost, [t], int(t))
            o_ref[:, i], lse_ref[:, i] = o1[:, 0], l1[:, 0]
        og = out[l][:, torch.from_numpy(slots).cuda()].float().cpu().numpy()
        err = rel_l2(og, o_ref)
        lerr = float(np.max(np.abs(lse[l][:, torch.from_numpy(slots).cuda()].cpu().numpy() - lse_ref)))
        log(f"  layer {l}: {len(slots)} sampled slots, rel-L2 {err:.2e}, lse max abs {lerr:.2e}")
        assert err <= 1e-2 and lerr <= 1e-2
