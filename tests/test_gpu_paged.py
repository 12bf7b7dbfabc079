"""GPU parity of the paged cache: every chunk's keys and values in buffers of
their own ([L][H_kv][len_c][D] each, allocated separately and out of order),
reached through the *_paged entry points.

Bars: the paged calls give results bit-identical to the contiguous calls on
the concatenated cache (the same kernels' arithmetic on the same rows), and,
stage-isolated on the oracle's inputs, the bars of the contiguous parity
tests against the oracle: scores and selection bit-exact, scattered rows
bit-exact, attention rel-L2 <= 1e-2 (bf16) / 1e-5 (float32), lse within
1e-2 / 1e-5.
"""
import dataclasses

import numpy as np
import pytest

import oracle
from oracle import bf16 as obf
from paper_2607_19547_amd import synth
from tests.gpu_util import check_scores_and_selection, empty, log, pair_norm, rel_l2, to_dev, to_host, ulp

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu(built_lib):
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")


def B():
    from paper_2607_19547_amd import binding
    return binding


def dec(x, dtype):
    return obf.decode(x) if dtype == "bf16" else np.asarray(x, np.float64)


def workload(lens, G=8, Hkv=2, n_layers=2, dtype="bf16", head_dim=128, sections=(16, 24, 24), seed=11):
    base = synth.WORKLOADS["qwen8k"]
    return dataclasses.replace(base, name="paged", n_layers=n_layers, n_q_heads=G * Hkv, n_kv_heads=Hkv,
                               n_chunks=len(lens), chunk_lens=tuple(lens), offsets="random_all_axes",
                               seed=seed, score_layer=1 if n_layers > 1 else 0, dtype=dtype,
                               head_dim=head_dim, sections=sections)


def split(x, cs):
    """One separately allocated tensor per chunk, allocated last chunk first
    with spacer allocations between them, so that no two chunks are adjacent."""
    parts, spacers = [None] * (len(cs) - 1), []
    for c in reversed(range(len(cs) - 1)):
        parts[c] = x[:, :, cs[c]:cs[c + 1]].clone().contiguous()
        spacers.append(torch.empty(4096 + 256 * c, dtype=torch.uint8, device=x.device))
    return parts


def joined(parts, dtype):
    return to_host(torch.cat(parts, dim=2), dtype)


def run_both(w, d, rho, per_layer=True):
    """The whole path on a contiguous cache and on the same cache paged;
    returns the two sets of host results."""
    b = B()
    geo = b.Geo.from_workload(w)
    dt, cs = w.dtype, w.chunk_start
    Q, KF, VF = to_dev(d["q_fresh"], dt), to_dev(d["k_fresh"], dt), to_dev(d["v_fresh"], dt)
    n, L = w.n_candidates, w.n_layers
    ranges = [(l, l + 1) for l in range(L)] if per_layer else [(0, L)]
    res = {}
    for paged in (False, True):
        K, V = to_dev(d["k_stored"], dt), to_dev(d["v_stored"], dt)
        if paged:
            K, V = split(K, cs), split(V, cs)
            b.compose_rebase_k_paged(geo, K, d["chunk_offsets"])
            k_reb = joined(K, dt)
        else:
            b.compose_rebase_k(geo, K, d["chunk_offsets"])
            k_reb = to_host(K, dt)
        scores = torch.empty(n, dtype=torch.float32, device="cuda")
        sel = torch.empty(max(n, 1), dtype=torch.int32, device="cuda")
        score = b.score_deviation_topk_paged if paged else b.score_deviation_topk
        k = score(geo, K, w.score_layer, KF[w.score_layer], rho, scores, sel)
        out = empty((L, w.n_q_heads, max(k, 1), w.head_dim), dt)
        lse = torch.empty((L, w.n_q_heads, max(k, 1)), dtype=torch.float32, device="cuda")
        ws = torch.empty(max(b.selective_attend_scatter_workspace(geo, k, ranges[0][1] - ranges[0][0]), 1),
                         dtype=torch.uint8, device="cuda")
        attend = b.selective_attend_scatter_paged if paged else b.selective_attend_scatter
        for lb, le in ranges:
            attend(geo, K, V, lb, le, sel, k, Q, KF, VF, out, lse, ws)
        torch.cuda.synchronize()
        res[paged] = dict(k_rebased=k_reb, scores=scores.cpu().numpy(), sel=sel[:k].cpu().numpy(),
                          k_post=joined(K, dt) if paged else to_host(K, dt),
                          v_post=joined(V, dt) if paged else to_host(V, dt),
                          out=to_host(out, dt)[:, :, :k], lse=lse.cpu().numpy()[:, :, :k], k=k)
    return res[False], res[True]


CASES = [
    ((256, 320, 192, 440), 8, 2, 0.2, "bf16"),             # MFMA path, ragged last chunk
    ((1024, 1536, 1664, 832), 8, 2, 0.05, "bf16"),         # long rows cut into key pieces + combine
    ((128, 192, 64), 2, 8, 1.0, "bf16"),                   # rho = 1, one queue per XCD
    ((64,) * 40, 4, 4, 0.3, "bf16"),                       # many short chunks: tiles cross chunk ends every step
    ((100, 130, 103, 167), 4, 2, 0.3, "bf16-d32"),         # generic kernels, unaligned chunks
    ((32, 32), 2, 2, 0.25, "f32"),                         # float32, generic kernels
]


def _w(lens, G, Hkv, kind):
    if kind == "bf16-d32":
        return workload(lens, G, Hkv, head_dim=32, sections=(4, 6, 6))
    if kind == "f32":
        return workload(lens, G, Hkv, dtype="f32", head_dim=16, sections=(2, 3, 3), n_layers=1)
    return workload(lens, G, Hkv)


@pytest.mark.parametrize("lens,G,Hkv,rho,kind", CASES)
def test_paged_compose_equals_contiguous(lens, G, Hkv, rho, kind):
    w = _w(lens, G, Hkv, kind)
    log(f"case paged compose lens={lens[:6]}{'...' if len(lens) > 6 else ''} G={G} Hkv={Hkv} rho={rho} {kind}")
    d = oracle.inputs.build(w)
    flat, paged = run_both(w, d, rho)
    for key in ("k_rebased", "scores", "sel", "k_post", "v_post", "out", "lse"):
        assert np.array_equal(flat[key], paged[key]), key
    # and the batched call over every layer
    flat2, paged2 = run_both(w, d, rho, per_layer=False)
    assert np.array_equal(paged2["out"], paged["out"]) and np.array_equal(flat2["out"], paged["out"])


def _random_paged(n=6, seed=77):
    """Seeded paged geometries for the MFMA path: 2-12 chunks of 64-1024 tokens
    in whole 64-token tiles, a ragged last chunk, every GQA group."""
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        G = (1, 2, 4, 8, 16, 32)[i % 6]
        Hkv = int(rng.choice([1, 2, 4])) if G <= 8 else 1
        nch = int(rng.integers(2, 13))
        lens = [64 * int(x) for x in rng.integers(1, 17, nch - 1)] + [int(rng.integers(1, 700))]
        cases.append((tuple(lens), G, Hkv, float(np.round(rng.uniform(0.02, 1.0), 3)), "bf16"))
    return cases


@pytest.mark.parametrize("lens,G,Hkv,rho,kind", _random_paged())
def test_paged_random_equals_contiguous(lens, G, Hkv, rho, kind):
    test_paged_compose_equals_contiguous(lens, G, Hkv, rho, kind)


@pytest.mark.parametrize("lens,G,Hkv,rho,kind", CASES[:2] + CASES[4:])
def test_paged_isolated_against_oracle(lens, G, Hkv, rho, kind):
    """Each paged stage from the oracle's inputs, against the oracle."""
    w = _w(lens, G, Hkv, kind)
    log(f"case paged isolated lens={lens} G={G} Hkv={Hkv} rho={rho} {kind}")
    d = oracle.inputs.build(w)
    ref = oracle.compose.compose(w.dtype, w.head_dim, w.sections, w.base, d["chunk_start"], d["chunk_offsets"],
                                 d["k_stored"], d["v_stored"], d["q_fresh"], d["k_fresh"], d["v_fresh"],
                                 rho, w.score_layer)
    b = B()
    geo = b.Geo.from_workload(w)
    dt, cs = w.dtype, w.chunk_start
    # rebase: the rebase bound against the oracle
    K = split(to_dev(d["k_stored"], dt), cs)
    b.compose_rebase_k_paged(geo, K, d["chunk_offsets"])
    got, want = dec(joined(K, dt), dt), dec(ref["k_rebased"], dt)
    assert np.all(np.abs(got - want) <= ulp(want, dt) + 2.0 ** -20 * pair_norm(want))
    # score + select on the oracle's rebased keys: bit-exact
    K = split(to_dev(ref["k_rebased"], dt), cs)
    n = w.n_candidates
    scores = torch.empty(n, dtype=torch.float32, device="cuda")
    sel = torch.empty(n, dtype=torch.int32, device="cuda")
    k = b.score_deviation_topk_paged(geo, K, w.score_layer, to_dev(d["k_fresh"][w.score_layer], dt), rho, scores, sel)
    torch.cuda.synchronize()
    check_scores_and_selection(scores.cpu().numpy(), ref["scores"], sel.cpu().numpy(), k, w.cs1,
                               oracle.select.select_top)
    # scatter + attention on the oracle's caches and selection
    V = split(to_dev(d["v_stored"], dt), cs)
    Q, KF, VF = to_dev(d["q_fresh"], dt), to_dev(d["k_fresh"], dt), to_dev(d["v_fresh"], dt)
    S = torch.from_numpy(ref["sel"].astype(np.int32)).cuda()
    out = empty((w.n_layers, w.n_q_heads, k, w.head_dim), dt)
    lse = torch.empty((w.n_layers, w.n_q_heads, k), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(b.selective_attend_scatter_workspace(geo, k, 1), 1), dtype=torch.uint8, device="cuda")
    for layer in range(w.n_layers):
        b.selective_attend_scatter_paged(geo, K, V, layer, layer + 1, S, k, Q, KF, VF, out, lse, ws)
    torch.cuda.synchronize()
    assert np.array_equal(joined(K, dt), ref["k_post"]) and np.array_equal(joined(V, dt), ref["v_post"])
    o, ls = to_host(out, dt), lse.cpu().numpy()
    tol = 1e-2 if dt == "bf16" else 1e-5
    for layer in range(w.n_layers):
        o_ref, lse_ref = ref["attn"][layer]
        err = rel_l2(dec(o[layer], dt), o_ref)
        log(f"  layer {layer}: rel-L2 {err:.3e}")
        assert err <= tol
        assert np.max(np.abs(ls[layer] - lse_ref)) <= tol


def test_paged_128_chunks():
    """The largest chunk table (128 chunks), every stage, against the contiguous calls."""
    w = workload((64,) * 127 + (100,), G=8, Hkv=2, n_layers=2)
    log("case paged 128 chunks")
    d = oracle.inputs.build(w)
    flat, paged = run_both(w, d, 0.1)
    for key in ("k_rebased", "scores", "sel", "k_post", "v_post", "out", "lse"):
        assert np.array_equal(flat[key], paged[key]), key


@pytest.mark.parametrize("lens,G,Hkv,kind", [
    ((256, 320, 192, 440), 8, 2, "bf16"),        # bf16 / D = 128 kernels
    ((100, 130, 103, 167), 4, 2, "bf16-d32"),    # generic kernels, bf16
    ((32, 32), 2, 2, "f32"),                     # generic kernels, float32
])
def test_paged_rebase_tokens_and_fused_rope(lens, G, Hkv, kind):
    """The per-token re-basing and the fused-rotary scatter on a paged cache
    give the contiguous calls' bits."""
    w = _w(lens, G, Hkv, kind)
    log(f"case paged per-token rebase + fused rope {kind}")
    d = oracle.inputs.build(w)
    b = B()
    geo = b.Geo.from_workload(w)
    dt, cs = w.dtype, w.chunk_start
    toff = oracle.policies.token_offsets("scalar1d", d["local_coords"], cs, d["chunk_offsets"])
    O = torch.from_numpy(np.ascontiguousarray(toff, dtype=np.int32)).cuda()
    K = to_dev(d["k_stored"], dt)
    Kp = split(K, cs)
    b.compose_rebase_k_tokens(geo, K, O)
    b.compose_rebase_k_tokens_paged(geo, Kp, O)
    torch.cuda.synchronize()
    assert np.array_equal(to_host(K, dt), joined(Kp, dt))
    want = oracle.rebase.rebase_tokens_stored(d["k_stored"], dt, toff, oracle.rope.inv_freq(w.head_dim, w.base),
                                              oracle.rope.axis_of_pair(w.sections))
    g_, o_ = dec(joined(Kp, dt), dt), dec(want, dt)
    assert np.all(np.abs(g_ - o_) <= ulp(o_, dt) + 2.0 ** -20 * pair_norm(o_))
    # fused rotary scatter + attention
    sel = np.sort(np.random.default_rng(5).choice(np.arange(w.cs1, w.n_tokens), size=min(97, w.n_candidates // 2),
                                                  replace=False))
    S = torch.from_numpy(sel.astype(np.int32)).cuda()
    C = torch.from_numpy(np.ascontiguousarray(d["global_coords"], dtype=np.int32)).cuda()
    Q, KF, VF = to_dev(d["q_fresh"], dt), to_dev(d["k_fresh"], dt), to_dev(d["v_fresh"], dt)
    outs = {}
    for paged in (False, True):
        K, V = to_dev(d["k_stored"], dt), to_dev(d["v_stored"], dt)
        if paged:
            K, V = split(K, cs), split(V, cs)
        out = empty((w.n_layers, w.n_q_heads, len(sel), w.head_dim), dt)
        lse = torch.empty((w.n_layers, w.n_q_heads, len(sel)), dtype=torch.float32, device="cuda")
        ws = torch.empty(b.selective_attend_scatter_rope_workspace(geo, len(sel), 1), dtype=torch.uint8,
                         device="cuda")
        f = b.selective_attend_scatter_rope_paged if paged else b.selective_attend_scatter_rope
        for layer in range(w.n_layers):
            f(geo, K, V, layer, layer + 1, S, len(sel), Q, KF, VF, C, out, lse, ws)
        torch.cuda.synchronize()
        outs[paged] = (joined(K, dt) if paged else to_host(K, dt), joined(V, dt) if paged else to_host(V, dt),
                       to_host(out, dt), lse.cpu().numpy())
    for a, c in zip(outs[False], outs[True]):
        assert np.array_equal(a, c)


def test_paged_long65k_equals_contiguous():
    """The timed cache geometry (65,536 tokens in 32 chunk buffers of 2048) at rho = 0.1, first
    two layers: the paged composition gives the contiguous one's bits in every output."""
    import bench
    w = dataclasses.replace(synth.WORKLOADS["long65k"], n_layers=2)
    log("case paged long65k, two layers")
    b = B()
    inp = bench.Inputs(w, torch, b, synth)
    cs, n = w.chunk_start, w.n_candidates
    res = []
    for paged in (False, True):
        K, V = inp.K0.clone(), inp.V0.clone()
        if paged:
            K, V = split(K, cs), split(V, cs)
            b.compose_rebase_k_paged(inp.geo, K, inp.offsets)
        else:
            b.compose_rebase_k(inp.geo, K, inp.offsets)
        scores = torch.empty(n, dtype=torch.float32, device="cuda")
        sel = torch.empty(n, dtype=torch.int32, device="cuda")
        score = b.score_deviation_topk_paged if paged else b.score_deviation_topk
        k = score(inp.geo, K, w.score_layer, inp.KF[w.score_layer], 0.1, scores, sel)
        out = torch.empty((w.n_layers, w.n_q_heads, k, w.head_dim), dtype=torch.bfloat16, device="cuda")
        lse = torch.empty((w.n_layers, w.n_q_heads, k), dtype=torch.float32, device="cuda")
        ws = torch.empty(b.selective_attend_scatter_workspace(inp.geo, k, 1), dtype=torch.uint8, device="cuda")
        attend = b.selective_attend_scatter_paged if paged else b.selective_attend_scatter
        for layer in range(w.n_layers):
            attend(inp.geo, K, V, layer, layer + 1, sel, k, inp.QF, inp.KF, inp.VF, out, lse, ws)
        torch.cuda.synchronize()
        Kh = torch.cat(K, dim=2) if paged else K
        Vh = torch.cat(V, dim=2) if paged else V
        res.append([scores.cpu(), sel[:k].cpu(), Kh.cpu(), Vh.cpu(), out.cpu(), lse.cpu()])
    for x, y in zip(*res):
        assert torch.equal(x, y)
