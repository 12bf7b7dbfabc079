"""Host mirror of the attention plan's placement arithmetic (the planning
workgroup of plan_scatter / plan_items): for ascending selections and for
lists that break the ascending precondition (unsorted, reversed, repeated,
out-of-range values), every queue position receives exactly one item
descriptor, the pieces of a row tile partition its key tiles, and every
partial slot stays below the per-layer slot count.  This mirrors the kernel's
integer formulas one to one (no GPU is used: an out-of-contract selection is
never run on the device)."""
import math

import numpy as np
import pytest

KT, CUS, ITEMS_PER_CU, MIN_PIECE, MAX_PIECES, XCDS = 64, 256, 6, 16, 2048, 8


def n_queues(hkv):
    return XCDS if hkv % XCDS == 0 else (hkv if XCDS % hkv == 0 else 1)


def part_cap_of(n_tiles, T, hkv, cap=2560):
    max_pieces = min(MAX_PIECES, ((T + KT - 1) // KT + MIN_PIECE - 1) // MIN_PIECE)
    pc = min(cap, n_tiles * hkv * (max_pieces if max_pieces > 1 else 0))
    return 0 if pc < 2 * hkv else pc


def plan(sel, n_sel, RT, T, hkv, part_cap):
    n_tiles = -(-n_sel // RT)
    # key tiles of row tile t from its last row, as a running maximum over t
    nu_t = []
    run = 0
    for t in range(n_tiles):
        ml = min((t + 1) * RT, n_sel) - 1
        g = min(int(sel[ml]), T - 1)
        v = 1 if g < 0 else (g + KT) // KT
        run = max(run, v)
        nu_t.append(run)
    nu = nu_t[::-1]                     # longest-first order i = n_tiles - 1 - t
    W1, nmax = sum(nu), max(nu)
    per = CUS * ITEMS_PER_CU
    S0 = max(MIN_PIECE, -(-nmax // MAX_PIECES), -(-(W1 * hkv) // per))
    S = nmax
    if S0 < nmax:
        step = max(1, S0 // 8)
        for k in range(64):
            Sk = S0 + k * step
            if Sk >= nmax:
                break
            loc = sum(-(-v // Sk) for v in nu if v > Sk)
            if loc * hkv <= part_cap:
                S = Sk
                break
    nsp = [(-(-v // S) if v > S else 1) for v in nu]
    ppre = [0]
    for np_ in nsp:
        ppre.append(ppre[-1] + (np_ * hkv if np_ > 1 else 0))
    n_cut = sum(1 for x in nsp if x > 1)
    np_max = max(nsp)
    nq = n_queues(hkv)
    kvq = hkv // nq
    nj = np_max if np_max > 1 else 0
    pj = [0]
    for j in range(nj):
        need = max(j, 1)
        lo, up = 0, n_tiles             # bisection: first index with nsp <= need
        while lo < up:
            mid = (lo + up) >> 1
            if nsp[mid] > need:
                lo = mid + 1
            else:
                up = mid
        pj.append(pj[-1] + lo * kvq)
    p_end = pj[nj]
    nun = n_tiles - n_cut
    per_q = p_end + nun * kvq
    desc = {}
    for i in range(n_tiles):
        v, np_ = nu[i], nsp[i]
        if np_ > 1:
            for j in range(np_):
                cnt = (pj[j + 1] - pj[j]) // kvq
                b, e = j * S, min((j + 1) * S, v)
                for kvl in range(kvq):
                    pos = pj[j] + kvl * cnt + i
                    assert pos not in desc, f"position {pos} written twice"
                    desc[pos] = (i, kvl, j, b, e)
        else:
            for kvl in range(kvq):
                pos = p_end + kvl * nun + (i - n_cut)
                assert pos not in desc, f"position {pos} written twice"
                desc[pos] = (i, kvl, 0, 0, v)
    return dict(n_tiles=n_tiles, nu=nu, nsp=nsp, ppre=ppre, per_q=per_q, desc=desc, nq=nq, S=S)


def check(sel, n_sel, G, T, hkv, part_cap=None):
    RT = 8 * (32 // G)
    n_tiles = -(-n_sel // RT)
    if part_cap is None:
        part_cap = part_cap_of(n_tiles, T, hkv)
    p = plan(sel, n_sel, RT, T, hkv, part_cap)
    nq = p["nq"]
    per_q_bound = (n_tiles * hkv + part_cap + nq - 1) // nq     # the descriptor array's capacity
    assert sorted(p["desc"]) == list(range(p["per_q"])), "every queue position is written once"
    assert p["per_q"] <= per_q_bound
    assert p["ppre"][-1] <= part_cap, "partial slots within the per-layer count"
    assert all(a >= b for a, b in zip(p["nsp"], p["nsp"][1:])), "pieces non-increasing (cut row tiles lead)"
    assert max(p["nsp"]) <= MAX_PIECES, "the planning workgroup keeps at most MAX_PIECES sections"
    pieces = {}
    for (i, kvl, j, b, e) in p["desc"].values():
        assert 0 <= i < n_tiles and 0 <= kvl < hkv // nq and 0 <= j < p["nsp"][i]
        pieces.setdefault((i, kvl), []).append((j, b, e))
        if p["nsp"][i] > 1:
            for kv in range(hkv):
                slot = p["ppre"][i] + kv * p["nsp"][i] + j
                assert slot < p["ppre"][i + 1] <= part_cap
    for (i, kvl), ps in pieces.items():
        ps.sort()
        assert [x[0] for x in ps] == list(range(p["nsp"][i]))
        assert ps[0][1] == 0 and ps[-1][2] == p["nu"][i]
        assert all(ps[k][2] == ps[k + 1][1] for k in range(len(ps) - 1)), "pieces partition the key tiles"
    return p


GEOS = [(8, 2, 65536, 6349), (8, 2, 8192, 615), (1, 1, 30000, 4000), (4, 8, 4096, 900), (32, 16, 9000, 333),
        (2, 3, 20000, 2500), (16, 4, 65536, 61000), (32, 1, 301056, 40)]


@pytest.mark.parametrize("G,hkv,T,k", GEOS)
def test_plan_ascending(G, hkv, T, k):
    rng = np.random.default_rng(T + k)
    cs1 = T // 16
    sel = np.sort(rng.choice(np.arange(cs1, T), size=k, replace=False))
    p = check(sel, k, G, T, hkv)
    # ascending input: the running maximum is the row tiles' own last-token count
    RT = 8 * (32 // G)
    own = [(int(sel[min((t + 1) * RT, k) - 1]) + KT) // KT for t in range(p["n_tiles"])]
    assert p["nu"] == own[::-1]


@pytest.mark.parametrize("G,hkv,T,k", GEOS)
@pytest.mark.parametrize("kind", ["shuffled", "reversed", "repeated", "out_of_range"])
def test_plan_out_of_contract_selection(G, hkv, T, k, kind):
    rng = np.random.default_rng(7 * T + k)
    cs1 = T // 16
    sel = np.sort(rng.choice(np.arange(cs1, T), size=k, replace=False))
    if kind == "shuffled":
        sel = rng.permutation(sel)
    elif kind == "reversed":
        sel = sel[::-1].copy()
    elif kind == "repeated":
        sel = rng.choice(sel[: max(1, k // 10)], size=k)
    else:
        sel = rng.integers(-2 ** 31, 2 ** 31 - 1, size=k)
    check(sel, k, G, T, hkv)


def test_plan_advisor_example():
    """Hand case: last-row token counts [1, 1, 200] over three row tiles (longest-first [200, 1, 1] becomes
    the running maximum [200, 200, 200]): the uncut tiles never land at position -1 and no position repeats."""
    RT = 32
    sel = np.zeros(3 * RT, np.int64)
    sel[RT - 1], sel[2 * RT - 1], sel[3 * RT - 1] = 0, 0, 200 * KT - 1
    for hkv in (1, 2, 8):
        check(sel, 3 * RT, 8, 200 * KT, hkv, part_cap=8 * hkv)


def test_plan_capped_slots():
    """The scratch-bounded variant's smaller slot counts (down to none) still give a valid plan."""
    rng = np.random.default_rng(3)
    sel = np.sort(rng.choice(np.arange(2048, 65536), size=6349, replace=False))
    for cap in (0, 4, 100, 963, 2560):
        p = check(sel, 6349, 8, 65536, 2, part_cap=cap)
        if cap == 0:
            assert all(x == 1 for x in p["nsp"])
