"""GPU parity: the HIP library, called through its C ABI, against the CPU
oracle on the same seeded inputs.

Bars (floating point, from the arithmetic of each stage):
  rebased K      per element |gpu - oracle| <= 1 ulp of the storage format at
                 the oracle's value + 2^-20 |pair|: both sides round once to
                 the storage format (which can land on adjacent values), and
                 the GPU's float32 rotation with float32 cos/sin tables adds an
                 absolute error of a few 2^-24 |pair|.  Also max abs
                 <= 2^-8 |k| with |k| the norm of the whole key row.  Chunks
                 with Delta = 0 are bit-exact
  scores         float32, bit-exact when both sides read the same keys
  selection      index work: bit-exact on the same scores
  scatter        K/V rows bit-exact
  attention O    rel-L2 <= 1e-2 per layer (bf16 MFMA path), <= 1e-5 (float32)
  lse            |gpu - oracle| <= 1e-2 (bf16) / 1e-5 (float32)
Stage-isolated tests feed both sides the same oracle-made inputs; chained
tests run the whole GPU path and compare each stage against the oracle's own
chain.
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
    from paper_2607_19547_amd import binding
    binding.lib()


def B():
    from paper_2607_19547_amd import binding
    return binding


def dec(x, dtype):
    return obf.decode(x) if dtype == "bf16" else np.asarray(x, np.float64)


def theta_sigma(w):
    return oracle.rope.inv_freq(w.head_dim, w.base), oracle.rope.axis_of_pair(w.sections)


def assert_rebase_close(w, got, want, stored):
    """got/want/stored: storage arrays [L, H, T, D]."""
    g, o = dec(got, w.dtype), dec(want, w.dtype)
    err = np.abs(g - o)
    tol = ulp(o, w.dtype) + 2.0 ** -20 * pair_norm(o)
    bad = err > tol
    assert not bad.any(), (f"{bad.sum()} elements outside the rebase bound; worst err/ulp "
                           f"{np.max(err / ulp(o, w.dtype)):.3f}")
    row = np.sqrt(np.sum(o * o, axis=-1, keepdims=True))
    assert np.all(err <= 2.0 ** -8 * row + 2.0 ** -126)
    off = synth.chunk_offsets(w)
    cs = w.chunk_start
    for c in range(w.n_chunks):
        if not off[c].any():
            assert np.array_equal(got[:, :, cs[c]:cs[c + 1]], stored[:, :, cs[c]:cs[c + 1]])
    return int((got != want).sum())


def gpu_compose(w, d, rho, per_layer=True):
    """Runs the whole GPU path; returns host copies of every stage output."""
    b = B()
    geo = b.Geo.from_workload(w)
    dt = w.dtype
    K, V = to_dev(d["k_stored"], dt), to_dev(d["v_stored"], dt)
    Q, KF, VF = to_dev(d["q_fresh"], dt), to_dev(d["k_fresh"], dt), to_dev(d["v_fresh"], dt)
    b.compose_rebase_k(geo, K, d["chunk_offsets"])
    k_reb = to_host(K, dt)
    n = w.n_candidates
    scores = torch.empty(n, dtype=torch.float32, device="cuda")
    sel = torch.empty(max(n, 1), dtype=torch.int32, device="cuda")
    k = b.score_deviation_topk(geo, K, w.score_layer, KF[w.score_layer], rho, scores, sel)
    out = empty((w.n_layers, w.n_q_heads, max(k, 1), w.head_dim), dt)
    lse = torch.empty((w.n_layers, w.n_q_heads, max(k, 1)), dtype=torch.float32, device="cuda")
    L = w.n_layers
    ranges = [(l, l + 1) for l in range(L)] if per_layer else [(0, L)]
    ws_bytes = b.selective_attend_scatter_workspace(geo, k, ranges[0][1] - ranges[0][0])
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device="cuda")
    for lb, le in ranges:
        b.selective_attend_scatter(geo, K, V, lb, le, sel, k, Q, KF, VF, out, lse, ws)
    torch.cuda.synchronize()
    return dict(k_rebased=k_reb, scores=scores.cpu().numpy(), sel=sel[:k].cpu().numpy().astype(np.int64),
                k_post=to_host(K, dt), v_post=to_host(V, dt), out=to_host(out, dt)[:, :, :k],
                lse=lse.cpu().numpy()[:, :, :k], k=k)


def gpu_attend(w, k_cache, v_cache, d, sel, layers=None, per_layer=True):
    """Stage-isolated scatter + attention on the given (oracle-made) caches."""
    b = B()
    geo = b.Geo.from_workload(w)
    dt = w.dtype
    K, V = to_dev(k_cache, dt), to_dev(v_cache, dt)
    Q, KF, VF = to_dev(d["q_fresh"], dt), to_dev(d["k_fresh"], dt), to_dev(d["v_fresh"], dt)
    S = torch.from_numpy(np.asarray(sel, np.int32)).cuda()
    k = len(sel)
    out = empty((w.n_layers, w.n_q_heads, max(k, 1), w.head_dim), dt)
    lse = torch.full((w.n_layers, w.n_q_heads, max(k, 1)), float("nan"), dtype=torch.float32, device="cuda")
    L = w.n_layers
    ranges = [(l, l + 1) for l in range(L)] if per_layer else [(0, L)]
    ws_bytes = b.selective_attend_scatter_workspace(geo, k, ranges[0][1] - ranges[0][0])
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device="cuda")
    for lb, le in ranges:
        b.selective_attend_scatter(geo, K, V, lb, le, S, k, Q, KF, VF, out, lse, ws)
    torch.cuda.synchronize()
    return to_host(K, dt), to_host(V, dt), to_host(out, dt)[:, :, :k], lse.cpu().numpy()[:, :, :k]


def oracle_attend_layer(w, d, k_post_layer, v_post_layer, sel, layer, rows=None):
    q = dec(d["q_fresh"][layer], w.dtype)
    rows = sel if rows is None else rows
    return oracle.attention.attend_rows(q, dec(k_post_layer, w.dtype), dec(v_post_layer, w.dtype),
                                        rows, w.cs1)


def check_attention(w, out, lse, o_ref, lse_ref, tag):
    tol = 1e-2 if w.dtype == "bf16" else 1e-5
    err = rel_l2(dec(out, w.dtype), o_ref)
    lerr = float(np.max(np.abs(lse - lse_ref))) if lse_ref.size else 0.0
    log(f"  {tag}: attention rel-L2 {err:.3e}, lse max abs {lerr:.2e}")
    assert err <= tol
    assert lerr <= (1e-2 if w.dtype == "bf16" else 1e-5)


# ======================================================================== tiny fp32
def test_tiny_chained_and_isolated():
    w = synth.WORKLOADS["tiny"]
    log(f"case tiny fp32: T={w.n_tokens} rho={w.rho}")
    d = oracle.inputs.build(w)
    th, sg = theta_sigma(w)
    ref = oracle.compose.compose(w.dtype, w.head_dim, w.sections, w.base, d["chunk_start"], d["chunk_offsets"],
                                 d["k_stored"], d["v_stored"], d["q_fresh"], d["k_fresh"], d["v_fresh"],
                                 w.rho, w.score_layer)
    g = gpu_compose(w, d, w.rho)
    assert_rebase_close(w, g["k_rebased"], ref["k_rebased"], d["k_stored"])
    assert g["k"] == len(ref["sel"]) == 8
    assert np.allclose(g["scores"], ref["scores"], rtol=1e-5)
    assert g["sel"].tolist() == ref["sel"].tolist()
    # scatter: selected rows are the fresh rows, every other row is the GPU's rebased row
    sel = g["sel"]
    rest = np.setdiff1d(np.arange(w.n_tokens), sel)
    assert np.array_equal(g["k_post"][:, :, sel], d["k_fresh"][:, :, sel - w.cs1])
    assert np.array_equal(g["v_post"][:, :, sel], d["v_fresh"][:, :, sel - w.cs1])
    assert np.array_equal(g["k_post"][:, :, rest], g["k_rebased"][:, :, rest])
    assert np.array_equal(g["v_post"][:, :, rest], d["v_stored"][:, :, rest])
    o_ref, lse_ref = ref["attn"][0]
    check_attention(w, g["out"][0], g["lse"][0], o_ref, lse_ref, "tiny chained")
    # stage-isolated attention on the oracle's caches and selection
    kp, vp, out, lse = gpu_attend(w, ref["k_rebased"], d["v_stored"], d, ref["sel"])
    assert np.array_equal(kp, ref["k_post"]) and np.array_equal(vp, ref["v_post"])
    check_attention(w, out[0], lse[0], o_ref, lse_ref, "tiny isolated")


# ======================================================================== qwen8k bf16
@pytest.fixture(scope="module")
def qwen8k():
    w = synth.WORKLOADS["qwen8k"]
    log(f"building qwen8k inputs: L={w.n_layers} T={w.n_tokens}")
    d = oracle.inputs.build(w, q_layers=(0, 1, 35))     # attention is compared on these layers
    th, sg = theta_sigma(w)
    k_reb = oracle.rebase.rebase_stored(d["k_stored"], w.dtype, d["chunk_start"], d["chunk_offsets"], th, sg)
    return w, d, k_reb


def test_qwen8k_rebase(qwen8k):
    w, d, k_reb = qwen8k
    b = B()
    K = to_dev(d["k_stored"], w.dtype)
    V = to_dev(d["v_stored"], w.dtype)
    loc = synth.local_coords(w)
    glob = b.compose_rebase_k(b.Geo.from_workload(w), K, d["chunk_offsets"], loc, want_global=True)
    torch.cuda.synchronize()
    assert np.array_equal(glob, d["global_coords"])
    ndiff = assert_rebase_close(w, to_host(K, w.dtype), k_reb, d["k_stored"])
    log(f"  qwen8k rebase: {ndiff} of {k_reb.size} elements differ from the oracle (all within 1 rounding)")
    assert np.array_equal(to_host(V, w.dtype), d["v_stored"])   # values untouched


def test_qwen8k_score_select_isolated(qwen8k):
    w, d, k_reb = qwen8k
    b = B()
    geo = b.Geo.from_workload(w)
    K = to_dev(k_reb, w.dtype)
    KF = to_dev(d["k_fresh"][w.score_layer], w.dtype)
    n = w.n_candidates
    ref_scores = oracle.score.deviation_f32(dec(k_reb[w.score_layer], w.dtype),
                                            dec(d["k_fresh"][w.score_layer], w.dtype), w.cs1)
    for rho in (0.0, 1e-4, 0.1, 0.35, 1.0):
        scores = torch.empty(n, dtype=torch.float32, device="cuda")
        sel = torch.full((n,), -1, dtype=torch.int32, device="cuda")
        k = b.score_deviation_topk(geo, K, w.score_layer, KF, rho, scores, sel)
        torch.cuda.synchronize()
        kk = oracle.select.n_select(rho, n)
        assert k == kk
        got = sel.cpu().numpy()
        check_scores_and_selection(scores.cpu().numpy(), ref_scores, got, k, w.cs1, oracle.select.select_top)
        assert (got[k:] == -1).all()        # nothing written past n_sel
        log(f"  qwen8k select rho={rho}: k={k} identical")
    # without a scores buffer: the workspace holds them
    ws = torch.empty(b.score_deviation_topk_workspace(geo), dtype=torch.uint8, device="cuda")
    sel = torch.empty(n, dtype=torch.int32, device="cuda")
    k = b.score_deviation_topk(geo, K, w.score_layer, KF, 0.1, None, sel, workspace=ws)
    torch.cuda.synchronize()
    assert sel[:k].cpu().numpy().tolist() == oracle.select.select_top(ref_scores, k, w.cs1).tolist()


@pytest.mark.parametrize("n_tok,seed", [(3000, 5), (70000, 6)])
def test_select_heavy_ties(n_tok, seed):
    """Scores from the four values 0, 1, 2, 3 (exactly): every threshold falls
    inside a tie group, so the selection must take the lowest indices of that
    group, across the ranges of several wavefronts."""
    w = ragged(n_layers=1, chunk_lens=(64, n_tok - 64), offsets="none")
    log(f"case select ties n={n_tok}")
    b = B()
    geo = b.Geo.from_workload(w)
    rng = np.random.default_rng(seed)
    H, T, D, cs1 = w.n_kv_heads, w.n_tokens, w.head_dim, w.cs1
    k_cache = obf.encode(rng.standard_normal((1, H, T, D)))
    k_cache[..., 0] = obf.encode(np.zeros(1))[0]
    kf = k_cache[0][:, cs1:].copy()
    v = rng.integers(0, 4, size=T - cs1)
    kf[0, :, 0] = obf.encode(v.astype(np.float64))
    ref = oracle.score.deviation_f32(dec(k_cache[0], w.dtype), dec(kf, w.dtype), cs1)
    assert np.array_equal(ref, v.astype(np.float32))   # delta_t = v_t exactly
    K, KF = to_dev(k_cache, w.dtype), to_dev(kf, w.dtype)
    n = T - cs1
    for rho in (1e-9, 0.1, 0.25, 0.26, 0.5, 0.77, 1.0):
        sel = torch.full((n,), -1, dtype=torch.int32, device="cuda")
        scores = torch.empty(n, dtype=torch.float32, device="cuda")
        k = b.score_deviation_topk(geo, K, 0, KF, rho, scores, sel)
        torch.cuda.synchronize()
        assert np.array_equal(scores.cpu().numpy(), ref)
        want = oracle.select.select_top(ref, oracle.select.n_select(rho, n), cs1)
        got = sel.cpu().numpy()
        assert k == len(want)
        assert got[:k].tolist() == want.tolist()
        assert (got[k:] == -1).all()


def test_qwen8k_attention_isolated(qwen8k):
    w, d, k_reb = qwen8k
    ref_scores = oracle.score.deviation_f32(dec(k_reb[w.score_layer], w.dtype),
                                            dec(d["k_fresh"][w.score_layer], w.dtype), w.cs1)
    sel = oracle.select.select_top(ref_scores, oracle.select.n_select(w.rho, w.n_candidates), w.cs1)
    kp, vp, out, lse = gpu_attend(w, k_reb, d["v_stored"], d, sel)
    for layer in range(w.n_layers):
        assert np.array_equal(kp[layer], oracle.attention.scatter_rows(k_reb[layer], d["k_fresh"][layer], sel, w.cs1))
        assert np.array_equal(vp[layer], oracle.attention.scatter_rows(d["v_stored"][layer], d["v_fresh"][layer], sel, w.cs1))
    for layer in (0, 1, 35):
        o_ref, lse_ref = oracle_attend_layer(w, d, kp[layer], vp[layer], sel, layer)
        check_attention(w, out[layer], lse[layer], o_ref, lse_ref, f"qwen8k layer {layer}")


def test_qwen8k_chained_and_deterministic(qwen8k):
    w, d, k_reb = qwen8k
    g = gpu_compose(w, d, w.rho)
    assert_rebase_close(w, g["k_rebased"], k_reb, d["k_stored"])
    ref_scores = oracle.score.deviation_f32(dec(k_reb[w.score_layer], w.dtype),
                                            dec(d["k_fresh"][w.score_layer], w.dtype), w.cs1)
    k = oracle.select.n_select(w.rho, w.n_candidates)
    ref_sel = oracle.select.select_top(ref_scores, k, w.cs1)
    assert g["k"] == k == 615
    # scores move by at most the norm of the rebase error of the token's key:
    # |delta_gpu - delta_orc| <= ||k_gpu - k_orc|| <= 2^-8 sqrt(2) ||k_orc||
    ko = dec(k_reb[w.score_layer][:, w.cs1:], w.dtype)
    bound = 2.0 ** -8 * np.sqrt(2) * np.sqrt(np.sum(ko * ko, axis=(0, 2))) + 1e-6
    assert np.all(np.abs(g["scores"].astype(np.float64) - ref_scores) <= bound)
    gs, rs = set(g["sel"].tolist()), set(ref_sel.tolist())
    extra, missing = sorted(gs - rs), sorted(rs - gs)
    for i in extra:       # a swapped choice is only allowed within the error bound
        for j in missing:
            bi, bj = bound[i - w.cs1], bound[j - w.cs1]
            assert ref_scores[i - w.cs1] >= ref_scores[j - w.cs1] - bi - bj
    log(f"  qwen8k chained selection: {len(extra)} swaps vs the oracle")
    first_diff = min(extra + missing) if extra or missing else w.n_tokens
    rows = ref_sel[ref_sel < first_diff]
    slots = np.arange(len(rows))
    # the oracle's own chain: scatter its selection, attend its rows
    for layer in (0, 35):
        kp = oracle.attention.scatter_rows(k_reb[layer], d["k_fresh"][layer], ref_sel, w.cs1)
        vp = oracle.attention.scatter_rows(d["v_stored"][layer], d["v_fresh"][layer], ref_sel, w.cs1)
        o_ref, lse_ref = oracle_attend_layer(w, d, kp, vp, ref_sel, layer, rows=rows)
        check_attention(w, g["out"][layer][:, slots], g["lse"][layer][:, slots], o_ref, lse_ref,
                        f"qwen8k chained layer {layer}")
    # determinism: a second run is bit-identical
    g2 = gpu_compose(w, d, w.rho, per_layer=False)
    for key in ("k_rebased", "scores", "sel", "k_post", "v_post", "out"):
        assert np.array_equal(g[key], g2[key]), key


# ======================================================================== ragged / edge geometries
def ragged(n_layers=2, chunk_lens=(100, 130, 103, 167), G=8, Hkv=2, offsets="random_all_axes", seed=7):
    base = synth.WORKLOADS["qwen8k"]
    return dataclasses.replace(base, name="ragged", n_layers=n_layers, n_q_heads=G * Hkv, n_kv_heads=Hkv,
                               n_chunks=len(chunk_lens), chunk_lens=tuple(chunk_lens), offsets=offsets,
                               seed=seed, score_layer=1 if n_layers > 1 else 0)


@pytest.mark.parametrize("G,Hkv,lens,rho", [
    (8, 2, (100, 130, 103, 167), 0.1),
    (8, 2, (100, 130, 103, 167), 1.0),
    (8, 2, (100, 130, 103, 167), 1e-9),          # k = 1
    (1, 2, (64, 64, 70), 0.5),
    (2, 3, (33, 200, 1), 0.3),
    (4, 1, (500, 260, 333), 0.2),
    (16, 1, (70, 190), 0.6),
    (32, 1, (40, 90, 31), 0.45),
    (8, 2, (1000, 1500, 1700, 800), 0.01),      # long rows, few of them: key pieces + combine
    (8, 2, (1000, 1500, 1700, 800), 0.3),
    (4, 4, (200, 260, 333), 0.25),              # one queue per KV head on 2 XCDs each
    (2, 8, (100, 300, 200), 0.3),               # one queue per XCD
    (1, 16, (64, 200, 150), 0.2),               # two KV heads per queue
])
def test_ragged_geometries(G, Hkv, lens, rho):
    w = ragged(G=G, Hkv=Hkv, chunk_lens=lens)
    log(f"case ragged G={G} Hkv={Hkv} lens={lens} rho={rho}")
    d = oracle.inputs.build(w)
    th, sg = theta_sigma(w)
    ref = oracle.compose.compose(w.dtype, w.head_dim, w.sections, w.base, d["chunk_start"], d["chunk_offsets"],
                                 d["k_stored"], d["v_stored"], d["q_fresh"], d["k_fresh"], d["v_fresh"],
                                 rho, w.score_layer)
    g = gpu_compose(w, d, rho)
    assert_rebase_close(w, g["k_rebased"], ref["k_rebased"], d["k_stored"])
    # isolated selection on the oracle's rebased keys must be exact
    b = B()
    geo = b.Geo.from_workload(w)
    n = w.n_candidates
    K = to_dev(ref["k_rebased"], w.dtype)
    KF = to_dev(d["k_fresh"][w.score_layer], w.dtype)
    scores = torch.empty(n, dtype=torch.float32, device="cuda")
    sel = torch.empty(n, dtype=torch.int32, device="cuda")
    k = b.score_deviation_topk(geo, K, w.score_layer, KF, rho, scores, sel)
    torch.cuda.synchronize()
    check_scores_and_selection(scores.cpu().numpy(), ref["scores"], sel.cpu().numpy(), k, w.cs1,
                               oracle.select.select_top)
    # isolated attention on the oracle's caches and selection
    kp, vp, out, lse = gpu_attend(w, ref["k_rebased"], d["v_stored"], d, ref["sel"])
    assert np.array_equal(kp, ref["k_post"]) and np.array_equal(vp, ref["v_post"])
    for layer in range(w.n_layers):
        o_ref, lse_ref = ref["attn"][layer]
        check_attention(w, out[layer], lse[layer], o_ref, lse_ref, f"layer {layer}")
    # the batched multi-layer call gives the same result as per-layer calls
    kp2, vp2, out2, lse2 = gpu_attend(w, ref["k_rebased"], d["v_stored"], d, ref["sel"], per_layer=False)
    assert np.array_equal(out2, out) and np.array_equal(kp2, kp)


def _random_geometries(n=10, seed=2026):
    """Seeded draws of GQA group, KV heads, chunk lengths (1-399 tokens, 2-6
    chunks) and rho, beyond the hand-picked cases above."""
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        G = (1, 2, 4, 8, 16, 32)[i % 6]
        Hkv = int(rng.choice([1, 2, 3, 4])) if G <= 8 else int(rng.choice([1, 2]))
        lens = tuple(int(x) for x in rng.integers(1, 400, int(rng.integers(2, 7))))
        rho = float(np.round(rng.uniform(0.02, 1.0), 3))
        cases.append((G, Hkv, lens, rho))
    return cases


@pytest.mark.parametrize("G,Hkv,lens,rho", _random_geometries())
def test_random_geometries(G, Hkv, lens, rho):
    test_ragged_geometries(G, Hkv, lens, rho)


def test_rho_zero_and_single_chunk():
    w = ragged(chunk_lens=(100, 130, 103, 167))
    d = oracle.inputs.build(w)
    g = gpu_compose(w, d, 0.0)
    assert g["k"] == 0
    # nothing scattered: caches equal the rebased input
    assert np.array_equal(g["k_post"], g["k_rebased"]) and np.array_equal(g["v_post"], d["v_stored"])
    w1 = ragged(chunk_lens=(300,), offsets="none")
    d1 = oracle.inputs.build(w1)
    b = B()
    K = to_dev(d1["k_stored"], w1.dtype)
    k = b.score_deviation_topk(b.Geo.from_workload(w1), K, 1, K, 0.5, None, None)
    assert k == 0


def test_rebase_large_offsets_all_axes():
    """rebase8k: Delta_t up to 1e5 on every chunk and all three axes; the
    float64 angle reduction keeps every element within one rounding."""
    w = synth.WORKLOADS["rebase8k"]
    log(f"case rebase8k offsets {synth.chunk_offsets(w).tolist()}")
    th, sg = theta_sigma(w)
    loc = synth.local_coords(w)
    ks = []
    for layer in range(w.n_layers):
        x = synth.draw_layer(w, layer)["k_pre"]
        ks.append(obf.encode(oracle.rope.apply_mrope(x, loc, th, sg)))
    stored = np.stack(ks)
    want = oracle.rebase.rebase_stored(stored, w.dtype, w.chunk_start, synth.chunk_offsets(w), th, sg)
    b = B()
    K = to_dev(stored, w.dtype)
    b.compose_rebase_k(b.Geo.from_workload(w), K, synth.chunk_offsets(w))
    torch.cuda.synchronize()
    nd = assert_rebase_close(w, to_host(K, w.dtype), want, stored)
    log(f"  rebase8k: {nd} of {want.size} elements differ by one rounding")
    # against the key rotated directly at the global coordinate (Eq. 3, Table 1 layer 0)
    glob = oracle.compose.global_coords(loc, w.chunk_start, synth.chunk_offsets(w))
    x = synth.draw_layer(w, 0)["k_pre"]
    direct = oracle.rope.apply_mrope(x, glob, th, sg)
    got = obf.decode(to_host(K, w.dtype)[0])
    rel = np.sum((got - direct) ** 2) / np.sum(direct ** 2)
    log(f"  rebase8k layer 0 rel-MSE vs direct global rotation: {rel:.2e}")
    assert rel < 2e-5


def test_rebase_extreme_offsets():
    """Offsets of up to 2^30 on every axis (the temporal pairs turn by up to
    1.07e9 rad): the per-chunk and per-token kernels reduce the float64 angle
    on both sides of the Cody-Waite range (|k| < 2^27 turns) and stay within
    one rounding of the oracle's exact rotation."""
    w = ragged(n_layers=2, chunk_lens=(64, 128, 192, 256, 100), offsets="none")
    th, sg = theta_sigma(w)
    off = np.array([[0, 0, 0],
                    [1 << 30, -(1 << 30), 123456789],
                    [-(1 << 30) + 7, 1 << 29, -(1 << 29) - 3],
                    [800000000, -800000001, 799999999],     # just inside |k| < 2^27 for theta_0 = 1
                    [-850000000, 2147483, -17]], dtype=np.int32)
    log(f"case rebase extreme offsets {off.tolist()}")
    rng = np.random.default_rng(13)
    stored = obf.encode(rng.standard_normal((w.n_layers, w.n_kv_heads, w.n_tokens, w.head_dim)))
    want = oracle.rebase.rebase_stored(stored, w.dtype, w.chunk_start, off, th, sg)
    b = B()
    geo = b.Geo.from_workload(w)
    K = to_dev(stored, w.dtype)
    b.compose_rebase_k(geo, K, off)
    torch.cuda.synchronize()
    got = to_host(K, w.dtype)
    g, o = dec(got, w.dtype), dec(want, w.dtype)
    assert np.all(np.abs(g - o) <= ulp(o, w.dtype) + 2.0 ** -20 * pair_norm(o))
    c1 = int(w.chunk_start[1])
    assert np.array_equal(got[:, :, :c1], stored[:, :, :c1])      # chunk 0 has Delta = 0
    log(f"  {int((got != want).sum())} of {want.size} elements differ by one rounding")
    toff = np.repeat(off, np.diff(w.chunk_start), axis=0)
    K2 = to_dev(stored, w.dtype)
    b.compose_rebase_k_tokens(geo, K2, torch.from_numpy(np.ascontiguousarray(toff)).cuda())
    torch.cuda.synchronize()
    assert np.array_equal(to_host(K2, w.dtype), to_host(K, w.dtype))


def test_debug_validation_of_the_selection(monkeypatch):
    """CS_DEBUG_VALIDATE=1: an unsorted or out-of-range sel_idx is rejected with
    CS_ERR_INVALID_ARGUMENT before any other work is enqueued (the caches stay
    untouched), and a valid one gives the result of the unchecked call."""
    w = ragged(n_layers=2, chunk_lens=(100, 130, 103, 167))
    log("case debug validation of sel_idx")
    d = oracle.inputs.build(w)
    b = B()
    geo = b.Geo.from_workload(w)
    rng = np.random.default_rng(4)
    good = np.sort(rng.choice(np.arange(w.cs1, w.n_tokens), 57, replace=False)).astype(np.int32)
    k = len(good)
    unsorted = good.copy()
    unsorted[[10, 11]] = unsorted[[11, 10]]
    outside = good.copy()
    outside[-1] = w.n_tokens
    ws = torch.empty(b.selective_attend_scatter_workspace(geo, k, w.n_layers), dtype=torch.uint8, device="cuda")
    Q, KF, VF = to_dev(d["q_fresh"], w.dtype), to_dev(d["k_fresh"], w.dtype), to_dev(d["v_fresh"], w.dtype)

    def call(sel):
        K, V = to_dev(d["k_stored"], w.dtype), to_dev(d["v_stored"], w.dtype)
        out = empty((w.n_layers, w.n_q_heads, k, w.head_dim), w.dtype)
        S = torch.from_numpy(sel).cuda()
        try:
            b.selective_attend_scatter(geo, K, V, 0, w.n_layers, S, k, Q, KF, VF, out, None, ws)
        finally:
            torch.cuda.synchronize()
        return K, V, out

    plain = call(good)
    monkeypatch.setenv("CS_DEBUG_VALIDATE", "1")
    for sel, msg in ((unsorted, "ascending"), (outside, "outside")):
        K, V = to_dev(d["k_stored"], w.dtype), to_dev(d["v_stored"], w.dtype)
        out = empty((w.n_layers, w.n_q_heads, k, w.head_dim), w.dtype)
        with pytest.raises(b.CsError) as err:
            b.selective_attend_scatter(geo, K, V, 0, w.n_layers, torch.from_numpy(sel).cuda(), k, Q, KF, VF, out,
                                       None, ws)
        torch.cuda.synchronize()
        assert err.value.code == b.CS_ERR_INVALID_ARGUMENT and msg in str(err.value)
        assert np.array_equal(to_host(K, w.dtype), d["k_stored"]) and np.array_equal(to_host(V, w.dtype), d["v_stored"])
    checked = call(good)
    for x, y in zip(plain, checked):
        assert np.array_equal(to_host(x, w.dtype), to_host(y, w.dtype))


def test_graph_capture_replays_the_composition():
    """The whole composition (re-basing, scoring and selection, one attention
    call per layer) captured into a HIP graph: the library enqueues only kernel
    launches, so the graph replays it.  Every replay, with the caches restored
    by eager copies in between, is bit-identical to the eager composition."""
    w = ragged(n_layers=3, chunk_lens=(256, 320, 384, 200), G=8, Hkv=2)
    log("case graph capture of the composition")
    d = oracle.inputs.build(w)
    b = B()
    geo = b.Geo.from_workload(w)
    K0, V0 = to_dev(d["k_stored"], w.dtype), to_dev(d["v_stored"], w.dtype)
    Q, KF, VF = to_dev(d["q_fresh"], w.dtype), to_dev(d["k_fresh"], w.dtype), to_dev(d["v_fresh"], w.dtype)
    K, V = K0.clone(), V0.clone()
    n, rho = w.n_candidates, 0.3
    k = oracle.select.n_select(rho, n)
    scores = torch.empty(n, dtype=torch.float32, device="cuda")
    sel = torch.empty(n, dtype=torch.int32, device="cuda")
    out = empty((w.n_layers, w.n_q_heads, k, w.head_dim), w.dtype)
    lse = torch.empty((w.n_layers, w.n_q_heads, k), dtype=torch.float32, device="cuda")
    ws = torch.empty(b.selective_attend_scatter_workspace(geo, k, 1), dtype=torch.uint8, device="cuda")
    off = d["chunk_offsets"]

    def compose():
        b.compose_rebase_k(geo, K, off)
        assert b.score_deviation_topk(geo, K, w.score_layer, KF[w.score_layer], rho, scores, sel) == k
        for layer in range(w.n_layers):
            b.selective_attend_scatter(geo, K, V, layer, layer + 1, sel, k, Q, KF, VF, out, lse, ws)

    compose()
    torch.cuda.synchronize()
    ref = [t.clone() for t in (K, V, out, lse, sel)]
    K.copy_(K0)
    V.copy_(V0)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        compose()
    torch.cuda.synchronize()
    for rep in range(3):
        K.copy_(K0)
        V.copy_(V0)
        out.zero_()
        lse.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for got, want in zip((K, V, out, lse, sel), ref):
            assert torch.equal(got, want), f"replay {rep}"


def test_workspace_reuse_and_garbage_workspace():
    """Partial results of cut row tiles live in the caller's workspace: a workspace full of
    garbage must work, and repeated calls on one workspace must give
    bit-identical results."""
    w = ragged(chunk_lens=(1000, 1500, 1700, 800))
    d = oracle.inputs.build(w)
    th, sg = theta_sigma(w)
    k_reb = oracle.rebase.rebase_stored(d["k_stored"], w.dtype, d["chunk_start"], d["chunk_offsets"], th, sg)
    sc = oracle.score.deviation_f32(dec(k_reb[w.score_layer], w.dtype), dec(d["k_fresh"][w.score_layer], w.dtype), w.cs1)
    sel = oracle.select.select_top(sc, oracle.select.n_select(0.05, w.n_candidates), w.cs1)
    b = B()
    geo = b.Geo.from_workload(w)
    nbytes = b.selective_attend_scatter_workspace(geo, len(sel), 1)
    assert nbytes > 0   # this geometry cuts its long row tiles into key pieces
    ws = torch.full((nbytes,), 0xA5, dtype=torch.uint8, device="cuda")
    Q, KF, VF = to_dev(d["q_fresh"], w.dtype), to_dev(d["k_fresh"], w.dtype), to_dev(d["v_fresh"], w.dtype)
    S = torch.from_numpy(sel.astype(np.int32)).cuda()
    outs = []
    for rep in range(3):
        K, V = to_dev(k_reb, w.dtype), to_dev(d["v_stored"], w.dtype)
        out = empty((w.n_layers, w.n_q_heads, len(sel), w.head_dim), w.dtype)
        for layer in range(w.n_layers):
            b.selective_attend_scatter(geo, K, V, layer, layer + 1, S, len(sel), Q, KF, VF, out, None, ws)
        torch.cuda.synchronize()
        outs.append(to_host(out, w.dtype))
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])
    kp = oracle.attention.scatter_rows(k_reb[0], d["k_fresh"][0], sel, w.cs1)
    vp = oracle.attention.scatter_rows(d["v_stored"][0], d["v_fresh"][0], sel, w.cs1)
    o_ref, _ = oracle_attend_layer(w, d, kp, vp, sel, 0)
    assert rel_l2(dec(outs[0][0], w.dtype), o_ref) <= 1e-2


# ======================================================================== full size, sampled
def _sample_slots(k, rt, n_random, seed):
    """Slots at both ends, around row-tile boundaries and at random."""
    pick = {0, 1, k - 2, k - 1}
    for b in (rt, 2 * rt, k // 2, k - rt):
        pick.update({b - 1, b})
    rng = np.random.default_rng(seed)
    pick.update(rng.choice(k, size=min(n_random, k), replace=False).tolist())
    return np.array(sorted(x for x in pick if 0 <= x < k), dtype=np.int64)


def _isolated_full_size(w, rhos, n_random, check_rebase):
    """Stage-isolated checks at full size: every stage's GPU result from the
    oracle's own inputs.  Rebase: every element; scores: bit-exact on the
    oracle's rebased keys; selection: exact; scatter: exact; attention: the
    sampled slots of every layer and head (one call per layer, as timed)."""
    d = oracle.inputs.build(w, q_layers=[0])
    th, sg = theta_sigma(w)
    k_reb = oracle.rebase.rebase_stored(d["k_stored"], w.dtype, d["chunk_start"], d["chunk_offsets"], th, sg)
    b = B()
    geo = b.Geo.from_workload(w)
    if check_rebase:
        K = to_dev(d["k_stored"], w.dtype)
        b.compose_rebase_k(geo, K, d["chunk_offsets"])
        assert_rebase_close(w, to_host(K, w.dtype), k_reb, d["k_stored"])
        del K
    n = w.n_candidates
    ref_scores = oracle.score.deviation_f32(dec(k_reb[w.score_layer], w.dtype),
                                            dec(d["k_fresh"][w.score_layer], w.dtype), w.cs1)
    K = to_dev(k_reb, w.dtype)
    KF = to_dev(d["k_fresh"][w.score_layer], w.dtype)
    for rho in rhos:
        scores = torch.empty(n, dtype=torch.float32, device="cuda")
        sel = torch.empty(n, dtype=torch.int32, device="cuda")
        k = b.score_deviation_topk(geo, K, w.score_layer, KF, rho, scores, sel)
        torch.cuda.synchronize()
        assert k == oracle.select.n_select(rho, n)
        check_scores_and_selection(scores.cpu().numpy(), ref_scores, sel.cpu().numpy(), k, w.cs1,
                                   oracle.select.select_top)
        ref_sel = sel[:k].cpu().numpy().astype(np.int64)  # (equal to the oracle's, or within its tie window)
        kp, vp, out, lse = gpu_attend(w, k_reb, d["v_stored"], d, ref_sel)
        rt = 8 * (32 // (w.n_q_heads // w.n_kv_heads))
        slots = _sample_slots(k, rt, n_random, seed=int(rho * 1000) + 1)
        for layer in range(w.n_layers):
            kpo = oracle.attention.scatter_rows(k_reb[layer], d["k_fresh"][layer], ref_sel, w.cs1)
            vpo = oracle.attention.scatter_rows(d["v_stored"][layer], d["v_fresh"][layer], ref_sel, w.cs1)
            assert np.array_equal(kp[layer], kpo) and np.array_equal(vp[layer], vpo)
            o_ref, lse_ref = oracle_attend_layer(w, d, kpo, vpo, ref_sel, layer, rows=ref_sel[slots])
            check_attention(w, out[layer][:, slots], lse[layer][:, slots], o_ref, lse_ref,
                            f"{w.name} rho={rho} layer {layer}, {len(slots)} sampled slots of {k}")


def test_long65k_per_layer_sampled():
    """The timed configuration: 65536 tokens in 32 chunks of 2048, 16 Q / 2 KV
    heads, head_dim 128, bf16, one call per layer; its first two layers (the
    layers are independent and identically shaped), at rho = 0.1 and 1."""
    w = dataclasses.replace(synth.WORKLOADS["long65k"], n_layers=2)
    log(f"case long65k first two layers, T={w.n_tokens}")
    _isolated_full_size(w, rhos=(0.1, 1.0), n_random=48, check_rebase=True)


def test_attn32k_sampled():
    """The attention sweep's cache: 32,768 tokens in 16 chunks of 2048, its first
    two layers, at three of the swept rho, one call per layer."""
    w = dataclasses.replace(synth.WORKLOADS["attn32k"], n_layers=2)
    log(f"case attn32k first two layers, T={w.n_tokens}")
    _isolated_full_size(w, rhos=(0.05, 0.2, 0.5), n_random=32, check_rebase=False)


def test_rebase262k_full_size_sampled():
    """The rebase sweep's largest cache: 262,144 tokens in 128 chunks of 2048,
    36 layers x 2 KV heads (4.8 GB of keys: byte offsets past 2^32), every chunk
    moved on all three axes.  Sampled rows (each chunk's first and last token,
    the last plane, random rows) against the oracle's Eq. 3 per row."""
    w = synth.WORKLOADS["rebase262k"]
    P, T, D = w.n_layers * w.n_kv_heads, w.n_tokens, w.head_dim
    log(f"case rebase262k full size, {P} planes x {T} tokens")
    gen = torch.Generator(device="cuda")
    gen.manual_seed(262)
    K = torch.randn((P, T, D), generator=gen, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    rng = np.random.default_rng(262)
    cs = w.chunk_start
    nc = len(cs) - 1
    toks = np.concatenate([cs[:-1], cs[1:] - 1, rng.integers(0, T, 4096), T - 1 - np.arange(64)])
    planes = np.concatenate([rng.integers(0, P, 2 * nc), rng.integers(0, P, 4096), np.full(64, P - 1)])
    pi, ti = torch.from_numpy(planes).cuda(), torch.from_numpy(toks).cuda()
    before = to_host(K[pi, ti], "bf16")
    b = B()
    off = synth.chunk_offsets(w)
    b.compose_rebase_k(b.Geo.from_workload(w), K.view(w.n_layers, w.n_kv_heads, T, D), off)
    after = to_host(K[pi, ti], "bf16")
    th, sg = theta_sigma(w)
    chunk = np.searchsorted(cs, toks, side="right") - 1
    want = oracle.rebase.rebase_tokens_stored(before[None], "bf16", off[chunk], th, sg)[0]
    g_, o_ = dec(after, "bf16"), dec(want, "bf16")
    assert np.all(np.abs(g_ - o_) <= ulp(o_, "bf16") + 2.0 ** -20 * pair_norm(o_))
    assert not np.array_equal(after, before)


def test_more_than_1024_row_tiles():
    """G = 32 puts 8 selected rows in a row tile: 9000 selected rows make 1125
    row tiles, more than the planning workgroup's 1024 threads, with cut row
    tiles of up to three pieces."""
    w = ragged(n_layers=1, G=32, Hkv=1, chunk_lens=(64, 9000))
    log(f"case ragged G=32 Hkv=1 lens=(64, 9000) rho=1")
    _isolated_full_size(w, rhos=(1.0,), n_random=64, check_rebase=False)


def test_more_than_4096_row_tiles():
    """34,000 selected rows at G = 32 make 4,250 row tiles: more than the
    planning workgroup keeps in LDS, so the plan reads its arrays back from
    global memory (with this many row tiles the even schedule cuts none)."""
    w = ragged(n_layers=1, G=32, Hkv=1, chunk_lens=(64, 34000))
    log(f"case ragged G=32 Hkv=1 lens=(64, 34000) rho=1")
    _isolated_full_size(w, rhos=(1.0,), n_random=48, check_rebase=False)


# ======================================================================== per-token rebase (Section 3 policies)
def _gpu_rebase_tokens(w, k_stored, toff):
    b = B()
    geo = b.Geo.from_workload(w)
    K = to_dev(k_stored, w.dtype)
    O = torch.from_numpy(np.ascontiguousarray(toff, dtype=np.int32)).cuda()
    b.compose_rebase_k_tokens(geo, K, O)
    torch.cuda.synchronize()
    return to_host(K, w.dtype)


@pytest.mark.parametrize("name", ["qwen8k", "tiny", "bf16_d32"])
def test_rebase_tokens_policies(name, request):
    """Every policy's per-token offsets, GPU against the oracle's Eq. 3 per token;
    the three-axis offsets give exactly the per-chunk kernel's bits; the layer-0
    fidelity of the GPU's keys keeps Table 1's ordering."""
    if name == "bf16_d32":   # the generic kernel in bf16
        w = dataclasses.replace(synth.WORKLOADS["tiny"], name="bf16_d32", dtype="bf16", head_dim=32,
                                sections=(4, 6, 6), n_layers=2, score_layer=1)
    else:
        w = synth.WORKLOADS[name]
    log(f"case rebase_tokens {name}")
    d = request.getfixturevalue("qwen8k")[1] if name == "qwen8k" else oracle.inputs.build(w)
    th, sg = theta_sigma(w)
    loc, cs, off = d["local_coords"], d["chunk_start"], d["chunk_offsets"]
    out = {}
    for p in oracle.policies.POLICIES:
        toff = oracle.policies.token_offsets(p, loc, cs, off)
        got = _gpu_rebase_tokens(w, d["k_stored"], toff)
        want = oracle.rebase.rebase_tokens_stored(d["k_stored"], w.dtype, toff, th, sg)
        g, o = dec(got, w.dtype), dec(want, w.dtype)
        tol = ulp(o, w.dtype) + 2.0 ** -20 * pair_norm(o)
        assert np.all(np.abs(g - o) <= tol), p
        still = ~np.any(toff != 0, axis=1)
        assert np.array_equal(got[:, :, still], d["k_stored"][:, :, still])
        out[p] = got
    b = B()
    K = to_dev(d["k_stored"], w.dtype)
    b.compose_rebase_k(b.Geo.from_workload(w), K, off)
    assert np.array_equal(to_host(K, w.dtype), out["three_axis"])
    if w.n_tokens >= 1024:
        # layer 0 of Table 1 on the GPU's keys: joint keys from the oracle's own Eq. 2
        joint = oracle.rebase.rebase_tokens_f64(dec(d["k_stored"][0], w.dtype),
                                                oracle.policies.token_offsets("three_axis", loc, cs, off), th, sg)
        fid = {p: oracle.policies.fidelity(dec(out[p][0], w.dtype), joint) for p in out}
        log(f"  layer-0 fidelity {name}: " + ", ".join(f"{p} cos {c:.4f} relMSE {r:.2e}" for p, (c, r) in fid.items()))
        assert fid["three_axis"][1] < 1e-4 and fid["naive"][1] > 1e-2 and fid["scalar1d"][1] > fid["naive"][1]


def test_rebase_tokens_long65k_scalar1d():
    """Scalar re-basing of the timed cache geometry (65,536 tokens; every token
    moves on all three axes), first two layers, every element against the oracle."""
    w = dataclasses.replace(synth.WORKLOADS["long65k"], n_layers=2)
    log("case rebase_tokens long65k scalar1d")
    d = oracle.inputs.build(w, q_layers=[0])
    th, sg = theta_sigma(w)
    toff = oracle.policies.token_offsets("scalar1d", d["local_coords"], d["chunk_start"], d["chunk_offsets"])
    got = _gpu_rebase_tokens(w, d["k_stored"], toff)
    want = oracle.rebase.rebase_tokens_stored(d["k_stored"], w.dtype, toff, th, sg)
    g, o = dec(got, w.dtype), dec(want, w.dtype)
    assert np.all(np.abs(g - o) <= ulp(o, w.dtype) + 2.0 ** -20 * pair_norm(o))


# ======================================================================== fused rotary embedding of fresh rows (f2)
def _prerotary_fresh(w, d, layers):
    """Pre-rotary fresh queries and keys in the storage dtype (the generator's draws; the fresh key is
    the stored key's pre-rotary vector plus the token's noise, as in the oracle's input recipe)."""
    s = synth.draw_token_scale(w)[None, :, None]
    enc = (lambda x: obf.encode(x)) if w.dtype == "bf16" else (lambda x: x.astype(np.float32))
    qs, ks = [], []
    for layer in layers:
        t = synth.draw_layer(w, layer, ("k_pre", "zk", "q_pre"))
        qs.append(enc(t["q_pre"]))
        ks.append(enc(t["k_pre"][:, w.cs1:, :] + s * t["zk"]))
    return np.stack(qs), np.stack(ks)


@pytest.mark.parametrize("G,Hkv,lens,rho,dtype", [
    (8, 2, (300, 400, 333), 0.2, "bf16"),
    (2, 8, (100, 300, 200), 0.3, "bf16"),
    (8, 2, (1000, 1500, 1700, 800), 0.05, "bf16"),    # cut row tiles
    (2, 2, (32, 32), 0.25, "f32"),                    # generic kernels
])
def test_fused_rope_equals_prerotated(G, Hkv, lens, rho, dtype):
    """GPU fused path against the oracle's own rotation of the same pre-rotary rows
    followed by the oracle's scatter and attention."""
    w = ragged(G=G, Hkv=Hkv, chunk_lens=lens)
    if dtype == "f32":
        w = dataclasses.replace(w, dtype="f32", head_dim=16, sections=(2, 3, 3))
    log(f"case fused rope G={G} Hkv={Hkv} lens={lens} rho={rho} {dtype}")
    d = oracle.inputs.build(w)
    th, sg = theta_sigma(w)
    glob = d["global_coords"]
    k_reb = oracle.rebase.rebase_stored(d["k_stored"], w.dtype, d["chunk_start"], d["chunk_offsets"], th, sg)
    sc = oracle.score.deviation_f32(dec(k_reb[w.score_layer], w.dtype), dec(d["k_fresh"][w.score_layer], w.dtype),
                                    w.cs1)
    sel = oracle.select.select_top(sc, oracle.select.n_select(rho, w.n_candidates), w.cs1)
    q_pre, k_pre = _prerotary_fresh(w, d, range(w.n_layers))
    enc = (lambda x: obf.encode(x)) if w.dtype == "bf16" else (lambda x: x.astype(np.float32))
    q_rot = enc(oracle.rope.apply_mrope(dec(q_pre, w.dtype), glob[w.cs1:], th, sg))
    k_rot = enc(oracle.rope.apply_mrope(dec(k_pre, w.dtype), glob[w.cs1:], th, sg))
    b = B()
    geo = b.Geo.from_workload(w)
    K, V = to_dev(k_reb, w.dtype), to_dev(d["v_stored"], w.dtype)
    Q, KP, VF = to_dev(q_pre, w.dtype), to_dev(k_pre, w.dtype), to_dev(d["v_fresh"], w.dtype)
    C = torch.from_numpy(np.ascontiguousarray(glob, dtype=np.int32)).cuda()
    S = torch.from_numpy(sel.astype(np.int32)).cuda()
    k = len(sel)
    out = empty((w.n_layers, w.n_q_heads, k, w.head_dim), w.dtype)
    lse = torch.empty((w.n_layers, w.n_q_heads, k), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(b.selective_attend_scatter_rope_workspace(geo, k, 1), 1), dtype=torch.uint8, device="cuda")
    for layer in range(w.n_layers):
        b.selective_attend_scatter_rope(geo, K, V, layer, layer + 1, S, k, Q, KP, VF, C, out, lse, ws)
    torch.cuda.synchronize()
    kp, vp, o, ls = to_host(K, w.dtype), to_host(V, w.dtype), to_host(out, w.dtype), lse.cpu().numpy()
    for layer in range(w.n_layers):
        kpo = oracle.attention.scatter_rows(k_reb[layer], k_rot[layer], sel, w.cs1)
        vpo = oracle.attention.scatter_rows(d["v_stored"][layer], d["v_fresh"][layer], sel, w.cs1)
        assert np.array_equal(vp[layer], vpo)
        g_, o_ = dec(kp[layer], w.dtype), dec(kpo, w.dtype)
        assert np.all(np.abs(g_ - o_) <= ulp(o_, w.dtype) + 2.0 ** -20 * pair_norm(o_))
        other = np.ones(w.n_tokens, bool)
        other[sel] = False
        assert np.array_equal(kp[layer][:, other], k_reb[layer][:, other])
        o_ref, lse_ref = oracle.attention.attend_rows(dec(q_rot[layer], w.dtype), o_, dec(vpo, w.dtype), sel, w.cs1)
        check_attention(w, o[layer], ls[layer], o_ref, lse_ref, f"fused rope layer {layer}")
