"""compose_load_rebase_k_paged: the chunks copied from page-locked host
memory, their keys re-based while the values are in transfer, give exactly
the cache that copying them and then calling compose_rebase_k_paged gives,
with the copies on a stream of their own beside the compute stream (which
they wait for) and with one stream for everything; the values arrive
unchanged."""
import numpy as np
import pytest

from tests.gpu_util import log

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu(built_lib):
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")


@pytest.mark.parametrize("two_streams", [True, False])
def test_load_rebase_matches_copy_then_rebase(two_streams):
    from paper_2607_19547_amd import binding as b
    L, hq, hkv, D = 3, 16, 2, 128
    cs = np.array([0, 512, 896, 1408, 2048, 2100], dtype=np.int64)  # (the last chunk ragged)
    n_chunks = len(cs) - 1
    log(f"case load + re-base, {n_chunks} chunks, two streams={two_streams}")
    geo = b.Geo(L, hq, hkv, D, (16, 24, 24), "bf16", cs)
    g = torch.Generator(device="cpu").manual_seed(23)
    lens = [int(cs[c + 1] - cs[c]) for c in range(n_chunks)]
    kh = [torch.randn(L, hkv, n, D, generator=g).to(torch.bfloat16).pin_memory() for n in lens]
    vh = [torch.randn(L, hkv, n, D, generator=g).to(torch.bfloat16).pin_memory() for n in lens]
    rng = np.random.default_rng(23)
    off = np.stack([rng.integers(0, 100000, n_chunks), rng.integers(-16, 17, n_chunks),
                    rng.integers(-16, 17, n_chunks)], axis=1).astype(np.int32)
    off[1] = 0  # a chunk that is only copied
    kd = [torch.full((L, hkv, n, D), 7.0, dtype=torch.bfloat16, device="cuda") for n in lens]
    vd = [torch.full((L, hkv, n, D), 7.0, dtype=torch.bfloat16, device="cuda") for n in lens]
    copy = torch.cuda.Stream() if two_streams else None
    # work enqueued on the compute stream before the call (a spin, then writes to the destination
    # buffers) comes first: the copies on the other stream wait for it
    torch.cuda._sleep(2_000_000)
    for x in kd + vd:
        x.fill_(-3.0)
    b.compose_load_rebase_k_paged(geo, kd, vd, kh, vh, off, copy_stream=None if copy is None else copy.cuda_stream)
    torch.cuda.synchronize()
    ref = [h.cuda() for h in kh]
    b.compose_rebase_k_paged(geo, ref, off)
    torch.cuda.synchronize()
    for c in range(n_chunks):
        assert torch.equal(kd[c], ref[c]), f"chunk {c} keys"
        assert torch.equal(vd[c].cpu(), vh[c]), f"chunk {c} values"
    assert torch.equal(kd[1].cpu(), kh[1]), "a zero-offset chunk is copied unchanged"
