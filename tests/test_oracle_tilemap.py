"""Pins of the oracle's elastic-grid, elastic-block and design-space functions.

Each check is a worked value from the paper's equations, a closed form, an
exhaustive invariant, or a comparison with an independent derivation (inverse
maps, Python's ``sorted``), never a retyping of the oracle's own loop.
"""
import itertools
import math

import pytest


# ---------------------------------------------------------------- Eq. (1)
@pytest.mark.parametrize("M,expected", [
    (12, [3, 6, 12]),
    (64, [1, 2, 4, 8, 16, 32, 64]),
    (49, [49]),
    (1568, [49, 98, 196, 392, 784, 1568]),
    (1, [1]),
    (6272, [49, 98, 196, 392, 784, 1568, 3136, 6272]),
])
def test_dichotomy_worked_values(orc, M, expected):
    # Eq. (1), §6.2: widths M/2^n .. M with n the 2-adic valuation of M
    assert orc.dichotomy(M) == expected


def test_dichotomy_closed_form(orc):
    for M in range(1, 600):
        w = orc.dichotomy(M)
        v2 = (M & -M).bit_length() - 1  # 2-adic valuation by bit trick
        assert len(w) == v2 + 1
        assert w[-1] == M and w[0] * (1 << v2) == M
        assert all(b == 2 * a for a, b in zip(w, w[1:]))


# ------------------------------------------------------------ slicing plans
@pytest.mark.parametrize("T", list(range(1, 70)) + [196, 3136, 6272])
def test_balanced_split_is_partition(orc, T):
    for n in range(1, min(T, 17) + 1):
        plan = orc.balanced_split(T, n)
        assert len(plan) == n
        assert plan[0][0] == 0
        assert all(b + l == nb for (b, l), (nb, _) in zip(plan, plan[1:]))
        assert plan[-1][0] + plan[-1][1] == T
        lens = [l for _, l in plan]
        assert max(lens) - min(lens) <= 1 and min(lens) >= 1


def test_balanced_split_matches_eq1_when_power_of_two(orc):
    # when 2^k divides T, n = 2^k shards all have the Eq. (1) width T/2^k
    for T in [12, 64, 1568, 6272, 96]:
        widths = orc.dichotomy(T)
        for k, wdt in enumerate(reversed(widths)):
            n = 1 << k
            plan = orc.balanced_split(T, n)
            assert all(l == wdt for _, l in plan)


def test_balanced_split_rejects(orc):
    with pytest.raises(ValueError):
        orc.balanced_split(4, 5)
    with pytest.raises(ValueError):
        orc.balanced_split(0, 1)


# ------------------------------------------------------ workgroup rank map
@pytest.mark.parametrize("G", list(range(1, 41)) + [255, 256, 257, 1000])
def test_wg_rank_bijection_and_die_locality(orc, G):
    X = 8
    ranks = [orc.wg_rank(g, G, X) for g in range(G)]
    assert sorted(ranks) == list(range(G))
    # all workgroups of one die (g mod X equal) hold one contiguous run of ranks,
    # in increasing g order
    for x in range(min(X, G)):
        rs = [ranks[g] for g in range(x, G, X)]
        assert rs == list(range(rs[0], rs[0] + len(rs)))
    # X = 1 is the identity
    assert [orc.wg_rank(g, G, 1) for g in range(G)] == list(range(G))


# -------------------------------------------------------------- owner map
def _inverse_rank(G, X, orc):
    inv = {}
    for g in range(G):
        inv[orc.wg_rank(g, G, X)] = g
    return inv


@pytest.mark.parametrize("T", [1, 2, 3, 7, 8, 13, 49, 64, 98, 196])
def test_owner_map_exact_once_and_closed_form(orc, T):
    for n in sorted({1, 2, 3, 4, 8, min(T, 16)}):
        if n > T:
            continue
        plan = orc.balanced_split(T, n)
        for G in [1, 2, 3, 5, 8, 16, 33, 256]:
            grids = [G] * n
            sh, wg, it, cnt = orc.owner_map(T, plan, grids)
            assert (cnt == 1).all()
            inv = _inverse_rank(G, 8, orc)
            # closed form: tile t of shard j sits at offset o = t - b_j;
            # it is run by the workgroup of rank o mod G in iteration o div G
            for j, (b, l) in enumerate(plan):
                for t in range(b, b + l):
                    o = t - b
                    assert sh[t] == j
                    assert it[t] == o // G
                    assert wg[t] == inv[o % G]


def test_owner_map_shard_order_irrelevant(orc):
    T = 49
    plan = orc.balanced_split(T, 4)
    grids = [3, 7, 1, 12]
    a = orc.owner_map(T, plan, grids)
    perm = [2, 0, 3, 1]
    b = orc.owner_map(T, [plan[i] for i in perm], [grids[i] for i in perm])
    # same (wg, iter, count) per tile; shard ids follow the permutation
    assert (a[1] == b[1]).all() and (a[2] == b[2]).all() and (a[3] == b[3]).all()
    assert ([perm[s] for s in b[0]] == a[0]).all()


def test_owner_map_detects_overlap_and_gap(orc):
    # overlapping shards count twice; a gap leaves count 0
    sh, wg, it, cnt = orc.owner_map(10, [(0, 6), (4, 6)], [2, 2])
    assert list(cnt) == [1, 1, 1, 1, 2, 2, 1, 1, 1, 1]
    sh, wg, it, cnt = orc.owner_map(10, [(0, 4), (6, 4)], [1, 1])
    assert list(cnt) == [1, 1, 1, 1, 0, 0, 1, 1, 1, 1]


def test_owner_map_rejects_bad_shards(orc):
    with pytest.raises(ValueError):
        orc.owner_map(10, [(8, 5)], [1])
    with pytest.raises(ValueError):
        orc.owner_map(10, [(0, 10)], [0])


# ------------------------------------------------------------- wave map
@pytest.mark.parametrize("P", [1, 2, 4])
def test_wave_map_is_bijection(orc, P):
    L = 4
    pairs = [orc.wave_map(L, P, lam) for lam in range(L)]
    assert sorted(pairs) == sorted(itertools.product(range(P), range(L // P)))
    # one round when the physical block is the logical block
    if P == L:
        assert pairs == [(lam, 0) for lam in range(L)]


def test_wave_map_hand_table(orc):
    # N:1 map of a 4-wave logical block onto P physical waves, written out by hand:
    # logical wave lam runs on physical wave lam mod P as that wave's (lam div P)-th logical wave
    table = {
        1: [(0, 0), (0, 1), (0, 2), (0, 3)],
        2: [(0, 0), (1, 0), (0, 1), (1, 1)],
        4: [(0, 0), (1, 0), (2, 0), (3, 0)],
    }
    for P, want in table.items():
        assert [orc.wave_map(4, P, lam) for lam in range(4)] == want, P


@pytest.mark.parametrize("P", [1, 2, 4])
def test_wave_map_from_logical_thread_loop(orc, P):
    # brute force over threads: a physical block of 64 P threads runs the 256 logical threads
    # of the logical block in rounds, physical thread tid taking logical thread i * 64 P + tid in
    # round i; every thread of a logical wave must land on one physical wave in one round, the
    # pair the oracle gives
    B = 64 * P
    where = {}
    for i in range(256 // B):
        for tid in range(B):
            tau = i * B + tid
            where.setdefault(tau // 64, set()).add((tid // 64, i))
    for lam in range(4):
        assert len(where[lam]) == 1
        assert orc.wave_map(4, P, lam) == next(iter(where[lam]))


def test_wave_map_rejects(orc):
    with pytest.raises(ValueError):
        orc.wave_map(4, 3, 0)


# ------------------------------------------------------------ tile coords
def test_tile_coords_roundtrip(orc):
    for (M, N, TM, TN) in [(3136, 64, 64, 64), (49, 512, 32, 64), (100, 70, 32, 32), (1, 1, 16, 16)]:
        mT, nT = math.ceil(M / TM), math.ceil(N / TN)
        seen = set()
        for t in range(3 * mT * nT):
            bi, mt, nt = orc.tile_coords(t, M, N, TM, TN)
            assert 0 <= mt < mT and 0 <= nt < nT
            assert (bi * mT + mt) * nT + nt == t
            seen.add((bi, mt, nt))
        assert len(seen) == 3 * mT * nT


# ----------------------------------------------------------- Eq. (2) / (4)
def test_eq2_hand_cases(orc):
    assert orc.eq2_grid_limit(256, 300) == 212
    assert orc.eq2_grid_limit(256, 49) == 207
    assert orc.eq2_grid_limit(256, 256) == 256
    assert orc.eq2_grid_limit(30, 45) == 15
    assert orc.eq2_block_limit(2048, 256) == 1792
    assert orc.eq2_feasible(256, 2048, 300, 256, 212, 1792)
    assert not orc.eq2_feasible(256, 2048, 300, 256, 213, 64)
    assert not orc.eq2_feasible(256, 2048, 300, 256, 10, 1793)


def test_wiscore_hand_value(orc):
    # ((10 mod 8) + 4) / 8 * (256 + 256) / 2048 = 0.75 * 0.25
    assert orc.wiscore(8, 2048, 10, 256, 4, 256) == pytest.approx(0.1875, abs=0)


def test_wiscore_in_unit_interval_on_feasible_set(orc):
    # the paper states WIScore lies in [0, 1]; under Eq. (2) both factors are <= 1
    for n_sm in [8, 30, 256]:
        for n_rt in [0, 1, 7, 49, 255, 256, 300, 1000]:
            for s_rt in [64, 256, 1024]:
                lim_g = orc.eq2_grid_limit(n_sm, n_rt)
                lim_b = orc.eq2_block_limit(2048, s_rt)
                for n_be in sorted({1, lim_g // 2 or 1, lim_g}):
                    for s_be in [64, 128, 256, lim_b]:
                        if not orc.eq2_feasible(n_sm, 2048, n_rt, s_rt, n_be, s_be):
                            continue
                        w = orc.wiscore(n_sm, 2048, n_rt, s_rt, n_be, s_be)
                        assert 0.0 <= w <= 1.0
    # the maximum 1 is reached exactly when the leftover SMs and threads are filled
    assert orc.wiscore(256, 2048, 300, 256, 212, 1792) == 1.0


# ------------------------------------------------------------------- Eq. (5)
def test_oscore_hand_cases(orc):
    assert orc.oscore([1, 2], [0.5, 0.5], 4.0, 2.0) == 1
    assert orc.oscore([1, 3], [0.5, 0.5], 4.0, 2.0) == 0   # sum 4 is not < 4
    assert orc.oscore([1, 2], [1.0, 1.5], 4.0, 2.0) == 0   # persistent-thread bar
    assert orc.oscore([], [], 0.1, 0.1) == 1


# ----------------------------------------------------------------- top 20 %
def test_top_fraction_against_sorted(orc):
    import random
    rnd = random.Random(5)
    for n in [1, 2, 4, 5, 9, 10, 11, 37, 100]:
        sc = [rnd.choice([0.0, 0.25, 0.5, 0.75, 1.0]) for _ in range(n)]
        gr = [rnd.choice([8, 16, 64, 256]) for _ in range(n)]
        bl = [rnd.choice([64, 128, 256]) for _ in range(n)]
        keep = orc.top_fraction(sc, gr, bl, 0.2)
        k = max(1, math.ceil(0.2 * n - 1e-12))
        assert len(keep) == k
        order = sorted(range(n), key=lambda i: (-sc[i], -gr[i], -bl[i], i))
        assert keep == order[:k]


# ----------------------------------------------------- shaded binary tree (§7)
def _all_nodes(b, e, depth=0):
    yield (b, e, depth)
    if e - b >= 2:
        m = (b + e) // 2
        yield from _all_nodes(b, m, depth + 1)
        yield from _all_nodes(m, e, depth + 1)


@pytest.mark.parametrize("T", [1, 2, 3, 5, 7, 8, 12, 49, 64, 100])
def test_tree_head_matches_recursive_enumeration(orc, T):
    nodes = list(_all_nodes(0, T))
    for L in [1, 2, 3, 5, 8, 13, T]:
        cursor = 0
        shards = []
        while cursor < T:
            ln, depth = orc.tree_head(T, cursor, L)
            cands = [(e - b, d) for (b, e, d) in nodes if b == cursor and e - b <= L]
            best_len = max(c[0] for c in cands)
            best_depth = min(d for ln2, d in cands if ln2 == best_len)
            assert (ln, depth) == (best_len, best_depth)
            shards.append((cursor, ln))
            cursor += ln
        # the shards partition [0, T) and each respects the length bound
        assert sum(l for _, l in shards) == T
        assert all(l <= L for _, l in shards)
        if L >= T:
            assert shards == [(0, T)]


def test_tree_head_power_of_two_gives_eq1_widths(orc):
    # T = 64: with max length 2^j every shard has width 2^j, an Eq. (1) width
    for j in range(7):
        cursor, lens = 0, []
        while cursor < 64:
            ln, _ = orc.tree_head(64, cursor, 1 << j)
            lens.append(ln)
            cursor += ln
        assert set(lens) == {1 << j}
