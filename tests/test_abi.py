"""The C-ABI library loads on a host without a GPU, exports every function the
header declares, and rejects invalid arguments with the documented status
before touching the device (no GPU needed: validation runs before any HIP call)."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2607_19547_amd import binding as b

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "chronostitch.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\**\s+\**(\w+)\s*\(", src, flags=re.M)))


def test_header_declares_the_three_entry_points():
    names = declared_functions()
    for n in ("compose_rebase_k", "score_deviation_topk", "selective_attend_scatter", "cs_last_error"):
        assert n in names


def test_library_exports_every_declared_symbol(built_lib):
    out = subprocess.run(["nm", "-D", "--defined-only", built_lib], capture_output=True, text=True).stdout
    exported = set(line.split()[-1] for line in out.splitlines() if line.strip())
    missing = [n for n in declared_functions() if n not in exported]
    assert not missing, missing
    L = b.lib()
    for n in declared_functions():
        assert hasattr(L, n)


def _geo(**kw):
    d = dict(n_layers=2, n_q_heads=4, n_kv_heads=2, head_dim=16, sections=(2, 3, 3), dtype="f32",
             chunk_start=[0, 32, 64])
    d.update(kw)
    return b.Geo(**d)


def _code(fn, *a, **kw):
    with pytest.raises(b.CsError) as e:
        fn(*a, **kw)
    return e.value.code, str(e.value)


FAKE = type("FakeTensor", (), {"data_ptr": lambda self: 0x1000, "numel": lambda self: 1 << 20,
                              "element_size": lambda self: 1})()


@pytest.mark.parametrize("kw,msg", [
    (dict(n_kv_heads=3), "multiple"),
    (dict(head_dim=15, sections=(2, 3, 2)), "even"),
    (dict(sections=(2, 3, 4)), "sum"),
    (dict(chunk_start=[0, 40, 30]), "increasing"),
    (dict(chunk_start=[1, 32, 64]), "chunk_start[0]"),
    (dict(dtype=7), "dtype"),
    (dict(n_layers=0), "n_layers"),
])
def test_bad_geometry_rejected(built_lib, kw, msg):
    code, text = _code(b.compose_rebase_k, _geo(**kw), FAKE, np.zeros((2, 3)), stream=0)
    assert code == b.CS_ERR_INVALID_ARGUMENT and msg in text


def test_rebase_argument_errors(built_lib):
    g = _geo()
    assert _code(b.compose_rebase_k, g, None, np.zeros((2, 3)), stream=0)[0] == b.CS_ERR_INVALID_ARGUMENT
    bad_base = b.Geo(2, 4, 2, 16, (2, 3, 3), "f32", [0, 32, 64], rope_base=float("nan"))
    assert _code(b.compose_rebase_k, bad_base, FAKE, np.zeros((2, 3)), stream=0)[0] == b.CS_ERR_INVALID_ARGUMENT


def test_rebase_tokens_argument_errors(built_lib):
    g = _geo()
    assert _code(b.compose_rebase_k_tokens, g, None, FAKE, stream=0)[0] == b.CS_ERR_INVALID_ARGUMENT
    assert _code(b.compose_rebase_k_tokens, g, FAKE, None, stream=0)[0] == b.CS_ERR_INVALID_ARGUMENT
    code, text = _code(b.compose_rebase_k_tokens, _geo(sections=(2, 3, 4)), FAKE, FAKE, stream=0)
    assert code == b.CS_ERR_INVALID_ARGUMENT and "sum" in text


def test_host_coordinate_shift_without_device_work(built_lib):
    """global = local + offset of the token's chunk; a geometry with every
    offset zero enqueues no kernel, so this runs on a CPU-only host."""
    g = _geo()
    loc = np.arange(64 * 3, dtype=np.int32).reshape(64, 3)
    glob = b.compose_rebase_k(g, FAKE, np.zeros((2, 3)), loc, want_global=True, stream=0)
    assert np.array_equal(glob, loc)


@pytest.mark.parametrize("rho", [-0.1, 1.01, float("nan")])
def test_score_rejects_bad_rho(built_lib, rho):
    code, _ = _code(b.score_deviation_topk, _geo(), FAKE, 0, FAKE, rho, FAKE, FAKE, stream=0)
    assert code == b.CS_ERR_INVALID_ARGUMENT


def test_score_rejects_bad_layer_and_small_workspace(built_lib):
    g = _geo()
    assert _code(b.score_deviation_topk, g, FAKE, 2, FAKE, 0.5, FAKE, FAKE, stream=0)[0] == b.CS_ERR_INVALID_ARGUMENT
    small = type("W", (), {"data_ptr": lambda self: 0x1000, "numel": lambda self: 8,
                           "element_size": lambda self: 1})()
    code, _ = _code(b.score_deviation_topk, g, FAKE, 0, FAKE, 0.5, None, FAKE, workspace=small, stream=0)
    assert code == b.CS_ERR_WORKSPACE_TOO_SMALL
    assert b.score_deviation_topk_workspace(g) >= 32 * 4


def test_score_rho_zero_selects_nothing_on_host(built_lib):
    """k is computed on the host; a single-chunk cache has no candidates and enqueues nothing."""
    g = _geo(chunk_start=[0, 64])
    assert b.score_deviation_topk(g, FAKE, 0, FAKE, 0.5, None, None, stream=0) == 0


def test_attention_argument_errors(built_lib):
    g = _geo()
    assert _code(b.selective_attend_scatter, g, FAKE, FAKE, 1, 3, FAKE, 4, FAKE, FAKE, FAKE, FAKE,
                 stream=0)[0] == b.CS_ERR_INVALID_ARGUMENT
    assert _code(b.selective_attend_scatter, g, FAKE, FAKE, 0, 1, FAKE, 33, FAKE, FAKE, FAKE, FAKE,
                 stream=0)[0] == b.CS_ERR_INVALID_ARGUMENT
    assert _code(b.selective_attend_scatter, g, None, FAKE, 0, 1, FAKE, 4, FAKE, FAKE, FAKE, FAKE,
                 stream=0)[0] == b.CS_ERR_INVALID_ARGUMENT
    # nothing to do: returns OK without touching the device
    b.selective_attend_scatter(g, None, None, 0, 1, None, 0, None, None, None, None, stream=0)


def test_attention_workspace_sizing(built_lib):
    q = b.Geo(36, 16, 2, 128, (16, 24, 24), "bf16", np.arange(33) * 2048)
    one = b.selective_attend_scatter_workspace(q, 6349, 1)
    # a workspace sized for n layers per call serves every call over fewer layers
    sizes = [b.selective_attend_scatter_workspace(q, 6349, n) for n in range(1, 37)]
    assert sizes[0] == one > 0
    assert all(x <= y for x, y in zip(sizes, sizes[1:]))
    assert b.selective_attend_scatter_workspace(q, 0, 1) == 0
    g = q
    small = type("W", (), {"data_ptr": lambda self: 0x1000, "numel": lambda self: 16,
                           "element_size": lambda self: 1})()
    if one:
        code, _ = _code(b.selective_attend_scatter, g, FAKE, FAKE, 0, 1, FAKE, 6349, FAKE, FAKE, FAKE,
                        FAKE, workspace=small, stream=0)
        assert code == b.CS_ERR_WORKSPACE_TOO_SMALL
    # the fp32 path needs no workspace
    assert b.selective_attend_scatter_workspace(_geo(), 8, 1) == 0


def test_fused_rope_argument_errors_and_workspace(built_lib):
    g = _geo()
    args = (g, FAKE, FAKE, 0, 1, FAKE, 4, FAKE, FAKE, FAKE, None, FAKE)
    assert _code(b.selective_attend_scatter_rope, *args, stream=0)[0] == b.CS_ERR_INVALID_ARGUMENT  # NULL coords
    assert _code(b.selective_attend_scatter_rope, g, FAKE, FAKE, 0, 1, FAKE, 33, FAKE, FAKE, FAKE, FAKE, FAKE,
                 stream=0)[0] == b.CS_ERR_INVALID_ARGUMENT                                          # n_sel > n
    # the fp32 path still needs room for the rotated queries: n_layers x H_q x n_sel x D x 4 bytes
    assert b.selective_attend_scatter_rope_workspace(g, 8, 1) == 1 * 4 * 8 * 16 * 4
    small = type("W", (), {"data_ptr": lambda self: 0x1000, "numel": lambda self: 16,
                           "element_size": lambda self: 1})()
    code, _ = _code(b.selective_attend_scatter_rope, g, FAKE, FAKE, 0, 1, FAKE, 8, FAKE, FAKE, FAKE, FAKE, FAKE,
                    workspace=small, stream=0)
    assert code == b.CS_ERR_WORKSPACE_TOO_SMALL
    q = b.Geo(36, 16, 2, 128, (16, 24, 24), "bf16", np.arange(33) * 2048)
    # bf16 / head_dim 128: the attention's workspace plus a cos/sin table of the selected tokens (64 pairs x 8 B),
    # the same for any number of layers per call
    assert (b.selective_attend_scatter_rope_workspace(q, 6349, 1)
            >= b.selective_attend_scatter_workspace(q, 6349, 1) + 6349 * 64 * 8)
    assert (b.selective_attend_scatter_rope_workspace(q, 6349, 1)
            < b.selective_attend_scatter_workspace(q, 6349, 1) + 6349 * 64 * 8 + 512)
    b.selective_attend_scatter_rope(g, None, None, 0, 1, None, 0, None, None, None, None, None, stream=0)  # nothing to do


def test_paged_argument_errors(built_lib):
    g = _geo()
    chunks = [FAKE, FAKE]
    assert _code(b.compose_rebase_k_paged, g, None, np.zeros((2, 3)), stream=0)[0] == b.CS_ERR_INVALID_ARGUMENT
    code, text = _code(b.compose_rebase_k_paged, g, [FAKE, None], np.zeros((2, 3)), stream=0)
    assert code == b.CS_ERR_INVALID_ARGUMENT and "chunk 1" in text
    assert _code(b.compose_rebase_k_tokens_paged, g, chunks, None, stream=0)[0] == b.CS_ERR_INVALID_ARGUMENT
    assert _code(b.score_deviation_topk_paged, g, chunks, 0, FAKE, 1.5, FAKE, FAKE,
                 stream=0)[0] == b.CS_ERR_INVALID_ARGUMENT
    # values are required by the attention calls
    assert _code(b.selective_attend_scatter_paged, g, chunks, None, 0, 1, FAKE, 4, FAKE, FAKE, FAKE, FAKE,
                 stream=0)[0] == b.CS_ERR_INVALID_ARGUMENT
    assert _code(b.selective_attend_scatter_rope_paged, g, chunks, [FAKE, None], 0, 1, FAKE, 4, FAKE, FAKE, FAKE,
                 FAKE, FAKE, stream=0)[0] == b.CS_ERR_INVALID_ARGUMENT
    # nothing to do: OK without looking at the chunk arrays
    b.selective_attend_scatter_paged(g, None, None, 0, 1, None, 0, None, None, None, None, stream=0)
    # load and re-base: device and host chunk arrays, each with every chunk
    off = np.zeros((2, 3))
    assert _code(b.compose_load_rebase_k_paged, g, chunks, None, chunks, chunks, off,
                 stream=0)[0] == b.CS_ERR_INVALID_ARGUMENT
    code, text = _code(b.compose_load_rebase_k_paged, g, chunks, chunks, [FAKE, None], chunks, off, stream=0)
    assert code == b.CS_ERR_INVALID_ARGUMENT and "host chunk 1" in text
    assert _code(b.compose_load_rebase_k_paged, g, chunks, chunks, chunks, None, off,
                 stream=0)[0] == b.CS_ERR_INVALID_ARGUMENT


def test_paged_limits(built_lib):
    # more chunks than the chunk table holds
    many = _geo(chunk_start=np.arange(66) * 2)            # 65 chunks, float32 / D = 16: at most 64
    code, text = _code(b.compose_rebase_k_paged, many, [FAKE] * 65, np.zeros((65, 3)), stream=0)
    assert code == b.CS_ERR_UNSUPPORTED and "64" in text
    q = b.Geo(1, 16, 2, 128, (16, 24, 24), "bf16", np.arange(130) * 64)   # 129 chunks: at most 128
    code, text = _code(b.score_deviation_topk_paged, q, [FAKE] * 129, 0, FAKE, 0.5, FAKE, FAKE, stream=0)
    assert code == b.CS_ERR_UNSUPPORTED and "128" in text
    # the MFMA attention reads whole 64-key tiles from one chunk
    q = b.Geo(1, 16, 2, 128, (16, 24, 24), "bf16", [0, 100, 200])
    assert b.selective_attend_scatter_workspace(q, 4, 1) <= FAKE.numel()
    code, text = _code(b.selective_attend_scatter_paged, q, [FAKE] * 2, [FAKE] * 2, 0, 1, FAKE, 4, FAKE, FAKE, FAKE,
                       FAKE, workspace=FAKE, stream=0)
    assert code == b.CS_ERR_UNSUPPORTED and "64" in text
    code, _ = _code(b.selective_attend_scatter_rope_paged, q, [FAKE] * 2, [FAKE] * 2, 0, 1, FAKE, 4, FAKE, FAKE, FAKE,
                    FAKE, FAKE, workspace=FAKE, stream=0)
    assert code == b.CS_ERR_UNSUPPORTED


def test_launch_sizes_beyond_the_grid_limits_are_rejected(built_lib):
    """A cache too large for one launch is refused with CS_ERR_UNSUPPORTED before
    anything is enqueued (every launch of a call is sized first)."""
    T = (1 << 31) - 128
    huge = b.Geo(36, 16, 2, 128, (16, 24, 24), "bf16", [0, 64, T])
    code, text = _code(b.compose_rebase_k, huge, FAKE, np.array([[0, 0, 0], [5, 0, 0]]), stream=0)
    assert code == b.CS_ERR_UNSUPPORTED and "too large" in text
    code, text = _code(b.score_deviation_topk, huge, FAKE, 0, FAKE, 0.5, FAKE, FAKE, stream=0)
    assert code == b.CS_ERR_UNSUPPORTED and "too large" in text
    big = (1 << 27)
    code, text = _code(b.selective_attend_scatter, huge, FAKE, FAKE, 0, 1, FAKE, big, FAKE, FAKE, FAKE, FAKE,
                       stream=0)
    assert code == b.CS_ERR_UNSUPPORTED and "too large" in text


def test_noalloc_attention_argument_errors(built_lib):
    """The no-workspace attention call rejects what selective_attend_scatter rejects, before any HIP call."""
    g = _geo()
    f = b.selective_attend_scatter_noalloc
    assert _code(f, g, FAKE, FAKE, 1, 3, FAKE, 4, FAKE, FAKE, FAKE, FAKE, stream=0)[0] == b.CS_ERR_INVALID_ARGUMENT
    assert _code(f, g, FAKE, FAKE, 0, 1, FAKE, 33, FAKE, FAKE, FAKE, FAKE, stream=0)[0] == b.CS_ERR_INVALID_ARGUMENT
    assert _code(f, g, None, FAKE, 0, 1, FAKE, 4, FAKE, FAKE, FAKE, FAKE, stream=0)[0] == b.CS_ERR_INVALID_ARGUMENT
    assert _code(f, g, FAKE, FAKE, 0, 1, FAKE, 4, None, FAKE, FAKE, FAKE, stream=0)[0] == b.CS_ERR_INVALID_ARGUMENT
    code, text = _code(f, _geo(sections=(2, 3, 4)), FAKE, FAKE, 0, 1, FAKE, 4, FAKE, FAKE, FAKE, FAKE, stream=0)
    assert code == b.CS_ERR_INVALID_ARGUMENT and "sum" in text
    f(g, None, None, 0, 1, None, 0, None, None, None, None, stream=0)  # nothing to do: OK, no device work
    T = (1 << 31) - 128
    huge = b.Geo(36, 16, 2, 128, (16, 24, 24), "bf16", [0, 64, T])
    code, text = _code(f, huge, FAKE, FAKE, 0, 1, FAKE, 1 << 27, FAKE, FAKE, FAKE, FAKE, stream=0)
    assert code == b.CS_ERR_UNSUPPORTED and "too large" in text


def test_trace_filter_without_a_gpu(built_lib):
    """cs_trace_only only records the names (no device call): it works on a host without a GPU."""
    from paper_2607_19547_amd import binding as b
    b.cs_trace_only(["sel_attn_mfma", "rebase_bf16_d128"])
    b.cs_trace_only([])
    b.cs_trace_only(None)
    assert b.cs_trace_collect() == {}
