"""Pins for scatter + causal GQA attention (Eq. 1 and the repair step).

Anchors: torch's scaled_dot_product_attention (float64, CPU) with an explicit
causal mask and K/V repeated over the query group, and closed-form special
cases (constant values, identical keys, zero query)."""
import numpy as np
import pytest
import torch

from oracle import attention, compose
from paper_2607_19547_amd import synth


def _sdpa_rows(q_all, k, v, rows):
    """Causal GQA SDPA over the full sequence; returns the given rows. q_all [Hq,T,D]."""
    Hq, T, D = q_all.shape
    G = Hq // k.shape[0]
    kk = torch.from_numpy(k).repeat_interleave(G, dim=0)
    vv = torch.from_numpy(v).repeat_interleave(G, dim=0)
    mask = torch.tril(torch.ones(T, T, dtype=torch.bool))
    o = torch.nn.functional.scaled_dot_product_attention(torch.from_numpy(q_all), kk, vv, attn_mask=mask)
    return o.numpy()[:, rows, :]


@pytest.mark.parametrize("G", [1, 2, 8])
def test_full_selection_equals_causal_sdpa(G):
    """P8: with every later token selected, selective attention is rows
    [cs1, T) of standard causal GQA attention over the post-scatter cache."""
    rng = np.random.default_rng(G)
    Hkv, T, D, cs1 = 2, 96, 32, 40
    Hq, n = Hkv * G, T - cs1
    k, v = rng.standard_normal((2, Hkv, T, D))
    kf, vf = rng.standard_normal((2, Hkv, n, D))
    qf = rng.standard_normal((Hq, n, D))
    sel = np.arange(cs1, T)
    kp = attention.scatter_rows(k, kf, sel, cs1)
    vp = attention.scatter_rows(v, vf, sel, cs1)
    o, lse = attention.attend_rows(qf, kp, vp, sel, cs1, block=7)
    q_all = np.zeros((Hq, T, D)); q_all[:, cs1:] = qf
    ref = _sdpa_rows(q_all, kp, vp, sel)
    assert np.allclose(o, ref, rtol=1e-10, atol=1e-12)
    # lse: log-sum-exp of the visible scaled scores, via scipy-free direct sum
    t = int(sel[3]); h = 1 % Hq
    s = (kp[h // G, :t + 1] @ qf[h, t - cs1]) / np.sqrt(D)
    assert lse[h, 3] == pytest.approx(np.log(np.sum(np.exp(s))), rel=1e-12)


def test_partial_selection_sees_fresh_and_stale_rows():
    """Rows attend over the post-scatter cache: selected rows carry fresh K/V,
    unselected rows keep the stored ones (I8), and the output of each selected
    row is the SDPA row of that mixed cache."""
    rng = np.random.default_rng(3)
    Hkv, T, D, cs1, G = 2, 64, 16, 32, 2
    n = T - cs1
    k, v = rng.standard_normal((2, Hkv, T, D))
    kf, vf = rng.standard_normal((2, Hkv, n, D))
    qf = rng.standard_normal((Hkv * G, n, D))
    sel = np.array([33, 35, 36, 50, 63])
    kp = attention.scatter_rows(k, kf, sel, cs1)
    assert np.array_equal(kp[:, sel], kf[:, sel - cs1])
    rest = np.setdiff1d(np.arange(T), sel)
    assert np.array_equal(kp[:, rest], k[:, rest])
    vp = attention.scatter_rows(v, vf, sel, cs1)
    o, _ = attention.attend_rows(qf, kp, vp, sel, cs1)
    q_all = np.zeros((Hkv * G, T, D)); q_all[:, cs1:] = qf
    assert np.allclose(o, _sdpa_rows(q_all, kp, vp, sel), rtol=1e-10, atol=1e-12)


def test_special_cases():
    """P9: constant V gives that vector; identical keys or a zero query give
    the mean of the visible values."""
    rng = np.random.default_rng(4)
    Hkv, T, D, cs1 = 1, 50, 8, 20
    sel = np.array([20, 31, 49])
    qf = rng.standard_normal((2, T - cs1, D))
    u = rng.standard_normal(D)
    v_const = np.broadcast_to(u, (Hkv, T, D)).copy()
    k = rng.standard_normal((Hkv, T, D))
    o, _ = attention.attend_rows(qf, k, v_const, sel, cs1)
    assert np.allclose(o, u[None, None, :], atol=1e-12)
    v = rng.standard_normal((Hkv, T, D))
    k_same = np.broadcast_to(rng.standard_normal(D), (Hkv, T, D)).copy()
    o, lse = attention.attend_rows(qf, k_same, v, sel, cs1)
    for m, t in enumerate(sel):
        assert np.allclose(o[:, m], v[0, :t + 1].mean(axis=0), atol=1e-12)
    o, lse = attention.attend_rows(np.zeros_like(qf), k, v, sel, cs1)
    for m, t in enumerate(sel):
        assert np.allclose(o[:, m], v[0, :t + 1].mean(axis=0), atol=1e-12)
        assert lse[0, m] == pytest.approx(np.log(t + 1), rel=1e-12)


def test_compose_chain_tiny_full_rho_zero_offsets_is_sdpa():
    """The chained oracle at rho = 1 with no re-basing is causal SDPA over the
    post-scatter cache (P8 through compose)."""
    w = synth.WORKLOADS["tiny"]
    from oracle import inputs
    d = inputs.build(w)
    zero = np.zeros_like(d["chunk_offsets"])
    r = compose.compose(w.dtype, w.head_dim, w.sections, w.base, d["chunk_start"], zero,
                        d["k_stored"], d["v_stored"], d["q_fresh"], d["k_fresh"], d["v_fresh"],
                        1.0, 0)
    cs1 = w.cs1
    assert r["sel"].tolist() == list(range(cs1, w.n_tokens))
    kp = r["k_post"][0].astype(np.float64); vp = r["v_post"][0].astype(np.float64)
    q_all = np.zeros((w.n_q_heads, w.n_tokens, w.head_dim))
    q_all[:, cs1:] = d["q_fresh"][0]
    ref = _sdpa_rows(q_all, kp, vp, r["sel"])
    assert np.allclose(r["attn"][0][0], ref, rtol=1e-10, atol=1e-12)
