"""The library's kernel trace (a measurement aid): per kernel name, the
launches and their total duration from events the dispatches stamp; with a
name filter only the kernels named are traced, and nothing while it is off."""
import numpy as np
import pytest

from tests.gpu_util import log

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu(built_lib):
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")


def test_trace_counts_and_filter():
    from paper_2607_19547_amd import binding as b
    T, k, L, hq, hkv = 20000, 2500, 2, 16, 2
    log(f"case kernel trace T={T} n_sel={k} layers={L}")
    cs1 = T // 8
    geo = b.Geo(L, hq, hkv, 128, (16, 24, 24), "bf16", np.array([0, cs1, T], dtype=np.int64))
    g = torch.Generator(device="cpu").manual_seed(5)
    r = lambda *s: torch.randn(*s, generator=g).to(torch.bfloat16).cuda()
    K, V = r(L, hkv, T, 128), r(L, hkv, T, 128)
    Q, KF, VF = r(L, hq, T - cs1, 128), r(L, hkv, T - cs1, 128), r(L, hkv, T - cs1, 128)
    rng = np.random.default_rng(5)
    sel = torch.from_numpy(np.sort(rng.choice(np.arange(cs1, T), size=k, replace=False)).astype(np.int32)).cuda()
    out = torch.empty((L, hq, k, 128), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(b.selective_attend_scatter_workspace(geo, k, 1), dtype=torch.uint8, device="cuda")

    def calls():
        for layer in range(L):
            b.selective_attend_scatter(geo, K, V, layer, layer + 1, sel, k, Q, KF, VF, out, None, ws)
        torch.cuda.synchronize()

    calls()  # (warm)
    for names, want in ((None, {"plan_scatter", "sel_attn_mfma", "sel_attn_combine"}),
                        (["sel_attn_mfma"], {"sel_attn_mfma"}),
                        (["sel_attn_combine", "plan_scatter"], {"sel_attn_combine", "plan_scatter"})):
        b.cs_trace_reset()
        b.cs_trace_only(names)
        b.cs_trace_enable(True)
        calls()
        b.cs_trace_enable(False)
        tr = b.cs_trace_collect()
        assert set(tr) == want, (names, tr)
        for name, (n, ms) in tr.items():
            assert n == L and ms > 0.0, (name, n, ms)
    b.cs_trace_only(None)
    b.cs_trace_reset()
    calls()  # tracing off: nothing collected
    assert b.cs_trace_collect() == {}
