"""Pins of the oracle's step after acceptance: the Sec. 3.1 reuse criterion /
next-window selection and the App. E fallback statistics (CPU only)."""
import itertools

import numpy as np
import pytest

import oracle as orc


def random_tree(rng, n_nodes, vocab):
    parent = [-1]
    for i in range(1, n_nodes):
        parent.append(-1 if rng.random() < 0.25 else int(rng.integers(0, i)))
    tokens = rng.integers(0, vocab, size=n_nodes).tolist()
    return parent, tokens


def paths_by_dfs(parent, tokens):
    """Every root-to-node token path with its end node, by depth-first search
    from the roots over child lists (independent of the parent walk)."""
    children = {i: [] for i in range(len(parent))}
    roots = []
    for i, p in enumerate(parent):
        (roots if p == -1 else children[p]).append(i)
    out = []
    stack = [(r, (tokens[r],)) for r in roots]
    while stack:
        v, seq = stack.pop()
        out.append((seq, v))
        stack.extend((c, seq + (tokens[c],)) for c in children[v])
    return out


def test_reuse_matches_path_enumeration():
    rng = np.random.default_rng(1)
    for _ in range(300):
        parent, tokens = random_tree(rng, int(rng.integers(1, 14)), 4)
        paths = paths_by_dfs(parent, tokens)
        for _ in range(6):
            if rng.random() < 0.5:
                seq = list(paths[int(rng.integers(0, len(paths)))][0])
            else:
                seq = rng.integers(0, 4, size=int(rng.integers(1, 5))).tolist()
            acc, c = seq[:-1], seq[-1]
            hits = sorted(v for p, v in paths if list(p) == seq)
            case, node = orc.reuse_select(parent, tokens, acc, c)
            if hits:
                assert node == hits[0]
                assert case == (orc.NEXT_BRANCH if not acc else orc.NEXT_CONTINUE)
            else:
                assert (case, node) == (orc.NEXT_FRESH, -1)


def test_selection_cases_by_hand():
    # two roots (tokens 5 and 9); 5 -> 6 -> 7 and 9 -> 6
    parent, tokens = [-1, 0, 1, -1, 3], [5, 6, 7, 9, 6]
    assert orc.reuse_select(parent, tokens, [], 9) == (orc.NEXT_BRANCH, 3)
    assert orc.reuse_select(parent, tokens, [], 5) == (orc.NEXT_BRANCH, 0)
    assert orc.reuse_select(parent, tokens, [5, 6], 7) == (orc.NEXT_CONTINUE, 2)
    assert orc.reuse_select(parent, tokens, [9], 6) == (orc.NEXT_CONTINUE, 4)
    assert orc.reuse_select(parent, tokens, [5], 7) == (orc.NEXT_FRESH, -1)   # 7 sits at depth 3
    assert orc.reuse_select(parent, tokens, [], 6) == (orc.NEXT_FRESH, -1)    # 6 is never a root


def _topk(p, k):
    return sorted(range(len(p)), key=lambda y: (-p[y], y))[:k]


def _tree_from_roots(roots, depth, vocab):
    """Hypothesis tree: one chain of `depth` nodes under each root; a root's
    chain depends only on its own token, so trees grow by inclusion in kappa."""
    parent, tokens = [], []
    for r in roots:
        crng = np.random.default_rng(1000 + r)
        prev = -1
        for d in range(depth):
            parent.append(prev)
            tokens.append(r if d == 0 else int(crng.integers(0, vocab)))
            prev = len(parent) - 1
    return parent, tokens


def test_prop1_fallback_nonincreasing_in_kappa():
    """App. E Prop. 1: with roots = Top-kappa of the early-exit law, every
    event that reuses at kappa1 reuses at any kappa2 >= kappa1; at kappa = |V|
    no tau = 1 event falls back."""
    V, depth = 12, 3
    rng = np.random.default_rng(2)
    for _ in range(20):
        p_ee = rng.dirichlet(np.full(V, 0.3))
        trees = {k: _tree_from_roots(_topk(p_ee, k), depth, V) for k in range(1, V + 1)}
        events = [([], y) for y in range(V)]
        for k in (1, 3, 6):
            par, tok = trees[k]
            for v in range(len(par)):
                path = orc.tree_path(par, tok, v)
                events.append((path[:-1], int(rng.integers(0, V))))
                events.append((path[:-1], path[-1]))
        for acc, c in events:
            f = [orc.reuse_select(*trees[k], acc, c)[0] == orc.NEXT_FRESH for k in range(1, V + 1)]
            assert all(a >= b for a, b in zip(f, f[1:])), (acc, c, f)
        for y in range(V):
            assert orc.reuse_select(*trees[V], [], y)[0] == orc.NEXT_BRANCH


@pytest.mark.parametrize("kappa", [1, 2, 4, 8])
def test_tau1_fallback_probability_is_one_minus_omega(kappa):
    """App. E: when the first draft token is rejected, reuse succeeds iff the
    correction y ~ q lies in Top-kappa of the early-exit law, so
    P(F = 1 | A = 0) = 1 - Omega_kappa exactly (enumerated over y)."""
    V = 16
    rng = np.random.default_rng(3 + kappa)
    for _ in range(10):
        q = rng.dirichlet(np.full(V, 0.5))
        p_ee = rng.dirichlet(np.full(V, 0.5))
        roots = _topk(p_ee, kappa)
        par, tok = _tree_from_roots(roots, 2, V)
        ff = sum(q[y] for y in range(V) if orc.reuse_select(par, tok, [], y)[0] == orc.NEXT_FRESH)
        omega = orc.overlap_mass(np.log(q), roots)
        assert abs(ff - (1.0 - omega)) < 1e-12


def test_overlap_mass_closed_forms():
    z = np.array([1.0, 2.0, 3.0, 4.0])
    e = np.exp(z) / np.exp(z).sum()
    assert abs(orc.overlap_mass(z, [3]) - e[3]) < 1e-15
    assert abs(orc.overlap_mass(z, [0, 1, 2, 3]) - 1.0) < 1e-15
    assert abs(orc.overlap_mass(z + 1000.0, [2, 3]) - (e[2] + e[3])) < 1e-12  # shift-invariant
    for k in range(1, 5):  # nondecreasing in kappa along a fixed ranking
        assert orc.overlap_mass(z, [3, 2, 1, 0][:k]) >= orc.overlap_mass(z, [3, 2, 1, 0][:k - 1] or [3]) - 1e-15
