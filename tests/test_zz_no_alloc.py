"""selective_attend_scatter_noalloc, the attention call that allocates nothing
(its plan and partials live in the library's per-GPU scratch array), against
selective_attend_scatter with a caller workspace on the same inputs.

Two calls in a row on one GPU, the second on a smaller cache: the first
(65,536 tokens, rho = 0.1) needs more partials than the scratch array holds,
so its key pieces are longer and its outputs differ from the workspace call's
by rounding only (attention bars: rel-L2 <= 1e-2 per layer, lse within 1e-2);
the second (8,192 tokens) fits and must be bit-identical.  The scattered K/V
rows are bit-identical in both."""
import numpy as np
import pytest

from tests.gpu_util import log, rel_l2

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

SCRATCH = 64 << 20


@pytest.fixture(scope="module", autouse=True)
def _gpu(built_lib):
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")


def _case(n_chunks, layers, rho, seed):
    from paper_2607_19547_amd import binding as b
    Hkv, G, D = 2, 8, 128
    cs = np.arange(n_chunks + 1, dtype=np.int64) * 2048
    T, cs1 = int(cs[-1]), int(cs[1])
    n = T - cs1
    geo = b.Geo(layers, Hkv * G, Hkv, D, (16, 24, 24), "bf16", cs)
    gen = torch.Generator(device="cuda").manual_seed(seed)

    def rnd(*shape):
        return torch.randn(*shape, device="cuda", generator=gen).to(torch.bfloat16)

    K, V = rnd(layers, Hkv, T, D), rnd(layers, Hkv, T, D)
    Q, KF, VF = rnd(layers, Hkv * G, n, D), rnd(layers, Hkv, n, D), rnd(layers, Hkv, n, D)
    k = int(np.ceil(rho * n - 1e-9))
    sel = (torch.randperm(n, device="cuda", generator=gen)[:k].sort().values + cs1).to(torch.int32)
    return geo, K, V, Q, KF, VF, sel, k


def _run(fn_noalloc, geo, K, V, Q, KF, VF, sel, k, layers, ranges):
    from paper_2607_19547_amd import binding as b
    Kc, Vc = K.clone(), V.clone()
    out = torch.empty((layers, Q.shape[1], k, 128), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((layers, Q.shape[1], k), dtype=torch.float32, device="cuda")
    if fn_noalloc:
        for lb, le in ranges:
            b.selective_attend_scatter_noalloc(geo, Kc, Vc, lb, le, sel, k, Q, KF, VF, out, lse)
    else:
        ws = torch.empty(max(1, b.selective_attend_scatter_workspace(geo, k, ranges[0][1] - ranges[0][0])),
                         dtype=torch.uint8, device="cuda")
        for lb, le in ranges:
            b.selective_attend_scatter(geo, Kc, Vc, lb, le, sel, k, Q, KF, VF, out, lse, ws)
    torch.cuda.synchronize()
    return Kc, Vc, out, lse


def test_noalloc_matches_workspace_call_twice():
    from paper_2607_19547_amd import binding as b
    for tag, n_chunks, layers, rho, ranges in (("65k tokens, per-layer calls", 32, 2, 0.1, [(0, 1), (1, 2)]),
                                               ("8k tokens, one 2-layer call", 4, 2, 0.1, [(0, 2)])):
        log(f"noalloc case: {tag}")
        geo, K, V, Q, KF, VF, sel, k = _case(n_chunks, layers, rho, seed=n_chunks)
        need = b.selective_attend_scatter_workspace(geo, k, ranges[0][1] - ranges[0][0])
        Kw, Vw, ow, lw = _run(False, geo, K, V, Q, KF, VF, sel, k, layers, ranges)
        Kn, Vn, on, ln = _run(True, geo, K, V, Q, KF, VF, sel, k, layers, ranges)
        assert torch.equal(Kn, Kw) and torch.equal(Vn, Vw), "scattered caches differ"
        if need <= SCRATCH:
            assert torch.equal(on, ow) and torch.equal(ln, lw), "within the scratch limit the outputs are identical"
            log(f"  workspace {need} bytes fits: bit-identical")
        else:
            for l in range(layers):
                err = rel_l2(on[l].float().cpu().numpy(), ow[l].float().cpu().numpy())
                lerr = float((ln[l] - lw[l]).abs().max())
                log(f"  workspace {need} bytes > scratch: layer {l} rel-L2 {err:.2e}, lse max abs {lerr:.2e}")
                assert err <= 1e-2 and lerr <= 1e-2
        del K, V, Q, KF, VF, Kw, Vw, Kn, Vn
        torch.cuda.empty_cache()
