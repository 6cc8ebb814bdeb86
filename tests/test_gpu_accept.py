"""Acceptance (App. B operator, Sec. 2 greedy rule, Sec. 3.1 tree walk) and
KV commit (Sec. 2) through the C ABI, on planted inputs, against the oracle.

msd_accept reads only the block, the logits / argmax and the sampling inputs,
and msd_kv_commit only the cache, so both are driven directly with host-built
inputs whose decisions are planted: drafts that the target accepts to a chosen
depth, on a chosen branch, in every mode. Both sides get the same fp32 logits;
the oracle decides the expected outcome (and the tests assert that the planted
outcome is what it decided, so a case can never pass empty).
"""
import numpy as np
import pytest

import oracle as orc
from paper_2510_13161_amd import synth
from tests import harness as H

pytestmark = pytest.mark.gpu

TOL = H.TOL_LOGIT


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _model(vocab: int, n_layers: int = 1, n_kv_heads: int = 1, head_dim: int = 64):
    """A small model whose vocabulary (acceptance) or cache geometry (commit)
    is what matters."""
    from paper_2510_13161_amd import msd
    heads = max(n_kv_heads, 1)
    shape = synth.ModelShape(f"acc-v{vocab}", n_layers, 64 * max(1, heads * head_dim // 64), heads,
                             n_kv_heads, head_dim, 64, vocab)
    return msd.Model(shape, synth.device_weights(shape, 3), max_positions=256), shape


@pytest.fixture(scope="module", params=[4096, 5008, 152064], ids=["V4096", "V5008", "V152064"])
def vmodel(request):
    _torch()
    m, shape = _model(request.param)
    yield m, shape.vocab
    m.close()


def _dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _branch_tree(branches: int, gamma: int) -> np.ndarray:
    w = synth.Workload("t", synth.TINY, 1, (0, 0), "tree", gamma, branches=branches)
    return synth.topology(w)


def _children(parent):
    n = len(parent)
    return [[c for c in range(n) if parent[c] == s] for s in range(n)]


def _run_accept(model, parent, tokens, logits, mode="greedy", temperature=1.0, cand=None, q=None,
                ua=None, us=None, tol=TOL, chain=False, ws=False):
    """GPU acceptance of a batch through the C ABI; returns host arrays. ws:
    pass a workspace of MSD_ACCEPT_WS_PER_ROW bytes a row (the vocabulary
    statistics kernel and the chunked draws), else none (the walk's own
    passes)."""
    torch = _torch()
    from paper_2510_13161_amd import msd
    B, n = tokens.shape
    blk = msd.make_block(_dev(tokens.astype(np.int32)), None if chain else parent)
    lg = _dev(logits.reshape(B * n, -1).astype(np.float32))
    am = _dev(np.argmax(logits.reshape(B * n, -1), -1).astype(np.int32))
    keep = []
    if mode == "greedy":
        smp = msd.Sampling(msd.MSD_GREEDY, 1.0, 0, None, None, None, None, tol)
    else:
        dc, dq, da, du = _dev(cand), _dev(q), _dev(ua), _dev(us)
        keep += [dc, dq, da, du]
        smp = msd.Sampling(msd.MODES[mode], float(temperature), cand.shape[-1], dc.data_ptr(),
                           dq.data_ptr(), da.data_ptr(), du.data_ptr(), tol)
    acc = torch.full((B,), -9, dtype=torch.int32, device="cuda")
    nxt = torch.full((B,), -9, dtype=torch.int32, device="cuda")
    path = torch.full((B, n), -9, dtype=torch.int32, device="cuda")
    tie = torch.full((B,), 7, dtype=torch.uint8, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    wsb = torch.empty(B * n * msd.MSD_ACCEPT_WS_PER_ROW, dtype=torch.uint8, device="cuda") if ws else None
    msd.accept(model.handle, blk, lg, am, smp, acc, nxt, path, status, ws=wsb, near_tie=tie)
    torch.cuda.synchronize()
    return (acc.cpu().numpy(), nxt.cpu().numpy(), path.cpu().numpy(), tie.cpu().numpy(),
            int(status.item()))


def _oracle_accept(parent, tokens, logits, mode="greedy", temperature=1.0, cand=None, q=None, ua=None,
                   us=None, tol=TOL):
    out = []
    for b in range(tokens.shape[0]):
        kw = {}
        if mode != "greedy":
            kw = dict(cand_ids=cand[b], cand_q=q[b], u_accept=ua[b], u_sample=us[b])
        out.append(orc.Oracle.accept(parent, tokens[b], logits[b].astype(np.float64), mode, temperature,
                                     tol_logit=tol, return_tie=True, **kw))
    return out


def _assert_same(gpu, want, planted_A=None):
    """Exact comparison: A, next token, path (padded with -1) and the near-tie
    flag (set iff the oracle flagged any decision)."""
    acc, nxt, path, tie, status = gpu
    assert status == 0
    for b, (A, y, p, td, tn) in enumerate(want):
        if planted_A is not None:
            assert A == planted_A[b], f"seq {b}: the oracle accepted {A}, planted {planted_A[b]}"
        assert acc[b] == A, f"seq {b}: A {acc[b]} != {A}"
        assert nxt[b] == y, f"seq {b}: next {nxt[b]} != {y}"
        assert np.array_equal(path[b, :A + 1], p), f"seq {b}: path {path[b]} vs {p}"
        assert np.all(path[b, A + 1:] == -1)
        assert tie[b] == int(td >= 0 or tn), f"seq {b}: near_tie {tie[b]} vs oracle ({td}, {tn})"


def _base_logits(g, B, n, V):
    return g.normal(0.0, 1.0, size=(B, n, V)).astype(np.float32)


def _plant_top(z, tok, gap):
    """Make tok the row's argmax by `gap` (fp32)."""
    others = np.delete(z, tok)
    z[tok] = np.float32(others.max() + gap)


# ---------------------------------------------------------------------------
# GREEDY
# ---------------------------------------------------------------------------
def test_greedy_chain_every_accepted_length(vmodel):
    """A chain of gamma = 8 drafts, one sequence per A = 0..8: the drafts equal
    the target's argmax up to a planted mismatch (A = 8: all accepted, the
    bonus token is the last row's argmax). Decisive margins: no flags."""
    model, V = vmodel
    g = np.random.default_rng(100 + V)
    n, B = 9, 9
    parent = np.arange(-1, n - 1)
    z = _base_logits(g, B, n, V)
    tok = g.integers(0, V, size=(B, n)).astype(np.int32)
    for b in range(B):
        a = g.integers(0, V, size=n)
        for s in range(n):
            _plant_top(z[b, s], a[s], 1.0)
        for s in range(b):
            tok[b, s + 1] = a[s]
        if b + 1 < n:
            tok[b, b + 1] = (a[b] + 1 + g.integers(0, V - 1)) % V
            if tok[b, b + 1] == a[b]:
                tok[b, b + 1] = (a[b] + 1) % V
    want = _oracle_accept(parent, tok, z)
    _assert_same(_run_accept(model, parent, tok, z, chain=True), want, planted_A=list(range(B)))
    # the same block given as an explicit parent array
    _assert_same(_run_accept(model, parent, tok, z), want)


def test_greedy_tree_accepts_on_a_later_branch(vmodel):
    """Branch-complete tree of 4 branches x 6 (Sec. 3.1 T_t, 25 slots): the
    accepted path runs down branch b at depth A for (b, A) over every branch
    and A = 0..6; depth-1 tokens are distinct, so only branch b matches. One
    more sequence repeats branch 3's first token on branch 1: the walk takes
    the first child in slot order."""
    model, V = vmodel
    g = np.random.default_rng(200 + V)
    K, gam = 4, 6
    parent = _branch_tree(K, gam)
    n = len(parent)
    plan = [(1, 0), (1, 3), (2, 6), (3, 1), (3, 5), (0, 2), (2, 4), (1, 6), (3, 6)]
    B = len(plan) + 1
    z = _base_logits(g, B, n, V)
    tok = np.zeros((B, n), np.int32)
    slot = lambda br, r: 1 + br * gam + r - 1
    for b in range(B):
        first = g.choice(V, size=K, replace=False)
        for br in range(K):
            tok[b, slot(br, 1)] = first[br]
            for r in range(2, gam + 1):
                tok[b, slot(br, r)] = g.integers(0, V)
        tok[b, 0] = g.integers(0, V)
        br, A = plan[b] if b < len(plan) else (3, 4)
        if b == len(plan):
            tok[b, slot(1, 1)] = tok[b, slot(3, 1)]   # a repeated sibling token
        nodes = [0] + [slot(br, r) for r in range(1, gam + 1)]
        for s in range(n):
            _plant_top(z[b, s], g.integers(0, V), 1.0)
        for d in range(A):                         # node at depth d predicts depth d + 1
            _plant_top(z[b, nodes[d]], tok[b, nodes[d + 1]], 1.0)
        if A < gam:                                # mismatch at depth A: a token no child carries
            kids = {int(tok[b, c]) for c in _children(parent)[nodes[A]]}
            y = int(g.integers(0, V))
            while y in kids:
                y = int(g.integers(0, V))
            _plant_top(z[b, nodes[A]], y, 1.0)
    want = _oracle_accept(parent, tok, z)
    planted = [A for _, A in plan] + [None]
    for b, (br, A) in enumerate(plan):
        assert want[b][0] == A and (A == 0 or want[b][2][1] == slot(br, 1))
    assert want[-1][2][1] == slot(1, 1)            # first child in slot order
    assert sum(w[0] >= 1 and w[2][1] != 1 for w in want) >= 6
    _assert_same(_run_accept(model, parent, tok, z), want, planted_A=planted[:-1] + [want[-1][0]])


def test_greedy_random_forest_topologies(vmodel):
    """General trees (random parent arrays, 40 slots): the argmax is planted
    along a random root-to-leaf path, so the walk goes down to that leaf and
    returns its argmax as the bonus."""
    model, V = vmodel
    g = np.random.default_rng(300 + V)
    n, B = 40, 6
    parent = np.array([-1] + [int(g.integers(0, i)) for i in range(1, n)])
    kids = _children(parent)
    z = _base_logits(g, B, n, V)
    tok = g.integers(0, V, size=(B, n)).astype(np.int32)
    planted = []
    for b in range(B):
        s, depth = 0, 0
        while kids[s]:
            c = kids[s][int(g.integers(0, len(kids[s])))]
            for o in kids[s]:                      # siblings carry other tokens
                if o != c and tok[b, o] == tok[b, c]:
                    tok[b, o] = (tok[b, c] + 1) % V
            _plant_top(z[b, s], tok[b, c], 1.0)
            s, depth = c, depth + 1
        _plant_top(z[b, s], g.integers(0, V), 1.0)
        planted.append(depth)
    assert max(planted) >= 4
    want = _oracle_accept(parent, tok, z)
    _assert_same(_run_accept(model, parent, tok, z), want, planted_A=planted)


def test_greedy_near_tie_flags(vmodel):
    """A decision row whose top-1 minus top-2 logit lies inside the 2 tol band
    sets near_tie; one just outside it does not. Decisions stay exact (both
    sides see the same logits)."""
    model, V = vmodel
    g = np.random.default_rng(400 + V)
    n, B = 5, 6
    parent = np.arange(-1, n - 1)
    z = _base_logits(g, B, n, V)
    tok = g.integers(0, V, size=(B, n)).astype(np.int32)
    gaps = [0.5 * TOL, 1.5 * TOL, 1.9 * TOL, 2.5 * TOL, 4.0 * TOL, 0.0]
    for b in range(B):
        for s in range(n):
            _plant_top(z[b, s], g.integers(0, V), 1.0)
        for s in range(2):
            tok[b, s + 1] = int(np.argmax(z[b, s]))
        top = int(np.argmax(z[b, 2]))
        runner = (top + 17) % V
        z[b, 2, runner] = np.float32(z[b, 2, top] - np.float32(gaps[b]))
    want = _oracle_accept(parent, tok, z)
    flags = [int(w[3] >= 0 or w[4]) for w in want]
    assert flags == [1, 1, 1, 0, 0, 1]
    _assert_same(_run_accept(model, parent, tok, z, chain=True), want)


# ---------------------------------------------------------------------------
# stochastic rules
# ---------------------------------------------------------------------------
def _stochastic_case(g, parent, B, V, plan, mode, temperature, n_cand=32):
    """Planted inputs for REJECTION / MATCH.

    plan[b] = (slots of the path to accept, final token y*). At a node on the
    path, the accepted child's token dominates the node's law (boost of 14 in
    z / T): REJECTION gives it a draft mass of 0.02, below its target mass,
    so alpha = 1 (after any rejections too); MATCH's draw with u = 0.5 lands
    in its bin. Children tested before it carry a draft mass of 0.15 and
    almost no target mass: rejected. At the last node y* (no child's token)
    dominates: every child is rejected and y* is the correction, or, at a
    leaf, the bonus.
    """
    n = len(parent)
    kids = _children(parent)
    z = _base_logits(g, B, n, V)
    tok = np.zeros((B, n), np.int32)
    cand = np.zeros((B, n, n_cand), np.int32)
    q = np.zeros((B, n, n_cand), np.float32)
    for b in range(B):
        path, ystar = plan[b]
        tok[b, 0] = g.integers(0, V)
        for s in range(n):
            cand[b, s] = g.choice(V, size=n_cand, replace=False)
            for j, c in enumerate(kids[s]):
                tok[b, c] = cand[b, s, j]
        for s in range(n):
            on = path[path.index(s) + 1] if s in path[:-1] else None
            qq = synth.dirichlet_rows(g, 0.5, (n_cand,)).astype(np.float64)
            fixed = {}
            for j, c in enumerate(kids[s]):
                if c == on:
                    fixed[j] = 0.02
                    break
                fixed[j] = 0.15
            free = [j for j in range(n_cand) if j not in fixed]
            qq[free] *= (1.0 - sum(fixed.values())) / qq[free].sum()
            for j, m in fixed.items():
                qq[j] = m
            q[b, s] = (qq / qq.sum()).astype(np.float32)
            if on is not None:
                tgt = int(tok[b, on])
            else:
                tgt = int(ystar)
                while tgt in {int(tok[b, c]) for c in kids[s]}:
                    tgt = (tgt + 1) % V
                plan[b] = (path, tgt)
            zt = z[b, s] / np.float32(temperature)
            others = np.delete(zt, tgt)
            z[b, s, tgt] = np.float32((others.max() + 14.0) * temperature)
    ua = synth.uniforms01(g, (B, n)) * np.float32(0.8) + np.float32(0.1)
    us = np.full((B, n), 0.5, np.float32)
    return tok, z, cand, q, ua, us


def _chain_plan(n, A, ystar):
    return list(range(A + 1)), ystar


def _tree_plan(gam, br, A, ystar):
    return [0] + [1 + br * gam + r - 1 for r in range(1, A + 1)], ystar


@pytest.mark.parametrize("ws", [False, True], ids=["own", "stats"])
@pytest.mark.parametrize("mode,temperature", [("rejection", 1.0), ("rejection", 0.7), ("match", 1.0)])
def test_stochastic_chain_every_accepted_length(vmodel, mode, temperature, ws):
    """Chain of 8 drafts, A = 0..8 planted; REJECTION accepts a child whose
    draft mass is below its target mass (alpha = 1) and descends; MATCH
    descends when the draw lands on the child. A = 8 ends in the leaf bonus."""
    model, V = vmodel
    g = np.random.default_rng(500 + V + int(10 * temperature) + (mode == "match"))
    n, B = 9, 9
    parent = np.arange(-1, n - 1)
    plan = [_chain_plan(n, A, int(g.integers(0, V))) for A in range(B)]
    tok, z, cand, q, ua, us = _stochastic_case(g, parent, B, V, plan, mode, temperature)
    want = _oracle_accept(parent, tok, z, mode, temperature, cand, q, ua, us)
    for b in range(B):
        assert want[b][0] == b and want[b][1] == plan[b][1], (b, want[b][:2])
    _assert_same(_run_accept(model, parent, tok, z, mode, temperature, cand, q, ua, us, chain=True, ws=ws), want)


@pytest.mark.parametrize("ws", [False, True], ids=["own", "stats"])
@pytest.mark.parametrize("mode", ["rejection", "match"])
def test_stochastic_tree_descends_a_later_branch(vmodel, mode, ws):
    """Tree of 4 x 6: the accepted branch is 1, 2 or 3 (REJECTION rejects the
    siblings tried before it, in slot order, recursively without replacement),
    A up to 6 with the leaf bonus."""
    model, V = vmodel
    g = np.random.default_rng(600 + V + (mode == "match"))
    K, gam = 4, 6
    parent = _branch_tree(K, gam)
    combos = [(1, 2), (2, 6), (3, 4), (0, 3), (3, 6), (2, 1), (1, 0)]
    plan = [_tree_plan(gam, br, A, int(g.integers(0, V))) for br, A in combos]
    B = len(plan)
    tok, z, cand, q, ua, us = _stochastic_case(g, parent, B, V, plan, mode, 1.0)
    want = _oracle_accept(parent, tok, z, mode, 1.0, cand, q, ua, us)
    for b, (br, A) in enumerate(combos):
        assert want[b][0] == A and list(want[b][2]) == plan[b][0], (b, want[b])
        assert want[b][1] == plan[b][1]
    assert sum(w[0] >= 2 for w in want) >= 4
    _assert_same(_run_accept(model, parent, tok, z, mode, 1.0, cand, q, ua, us, ws=ws), want)


@pytest.mark.parametrize("ws", [False, True], ids=["own", "stats"])
@pytest.mark.parametrize("mode", ["rejection", "match"])
def test_stochastic_seeded_workload_inputs(vmodel, mode, ws):
    """The seeded tree workload's own inputs (Dirichlet(0.1) draft laws over 32
    candidates, children drawn from them, seeded uniforms) with random logits:
    whatever the oracle decides, the GPU decides the same, flags included."""
    model, V = vmodel
    shape = synth.ModelShape(f"v{V}", 1, 64, 1, 1, 64, 64, V)
    w = synth.WORKLOADS["14b_tree"].with_model(shape, batch=12, mode=mode, seed=61 + (mode == "match"))
    si = synth.step_inputs(w)
    g = np.random.default_rng(62)
    z = _base_logits(g, w.batch, w.n_slots, V) * np.float32(3.0)
    want = _oracle_accept(si.parent, si.tokens, z, mode, 1.0, si.cand_ids, si.cand_q, si.u_accept,
                          si.u_sample)
    _assert_same(_run_accept(model, si.parent, si.tokens, z, mode, 1.0, si.cand_ids, si.cand_q,
                             si.u_accept, si.u_sample, ws=ws), want)


def test_rejection_child_outside_candidates_sets_status(vmodel):
    """A REJECTION child whose token has no draft mass at its parent is a
    device-detected error (the oracle refuses it too)."""
    model, V = vmodel
    g = np.random.default_rng(700)
    parent = np.arange(-1, 2)
    plan = [_chain_plan(3, 2, 5)]
    tok, z, cand, q, ua, us = _stochastic_case(g, parent, 1, V, plan, "rejection", 1.0)
    tok[0, 1] = int(np.setdiff1d(np.arange(64), cand[0, 0])[0])
    with pytest.raises(ValueError):
        _oracle_accept(parent, tok, z, "rejection", 1.0, cand, q, ua, us)
    gpu = _run_accept(model, parent, tok, z, "rejection", 1.0, cand, q, ua, us)
    from paper_2510_13161_amd import msd
    assert gpu[4] & msd.MSD_DEV_CANDIDATE
    assert gpu[1][0] == -1 and gpu[3][0] == 1


# ---------------------------------------------------------------------------
# KV commit / rollback
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("head_dim,n_kv", [(64, 4), (128, 2)])
def test_kv_commit_tree_paths_bit_exact(head_dim, n_kv):
    """Cache rows len + path[r] move to len + r for r = 1..A in every layer and
    kv head, len advances by 1 + A (Sec. 2 commit; Sec. 3.1: the node at depth
    r lands at position t + r). The whole cache after the call equals the
    oracle's commit of the same cache, bit for bit, for paths down later
    branches (path[r] > r), A = 0 and full depth; a sequence whose block
    overflows the capacity is left untouched (device error path)."""
    torch = _torch()
    from paper_2510_13161_amd import msd
    model, shape = _model(1024, n_layers=3, n_kv_heads=n_kv, head_dim=head_dim)
    K, gam = 3, 5
    parent = _branch_tree(K, gam)
    n = len(parent)
    slot = lambda br, r: 1 + br * gam + r - 1
    combos = [(0, 0), (1, 3), (2, 5), (1, 1), (2, 2), (0, 5), (2, 4)]
    B, cap = len(combos) + 1, 96
    lens = np.array([0, 7, 33, 60, 80, 12, 41, 90], np.int32)    # the last overflows: 90 + 16 > 96
    acc = np.array([A for _, A in combos] + [2], np.int32)
    path = np.full((B, n), -1, np.int32)
    for b, (br, A) in enumerate(combos + [(1, 2)]):
        path[b, :A + 1] = [0] + [slot(br, r) for r in range(1, A + 1)]
    L, Hk, hd = shape.n_layers, shape.n_kv_heads, shape.head_dim
    gen = torch.Generator(device="cuda").manual_seed(5)
    k = torch.randint(-32768, 32767, (L, B, Hk, cap, hd), dtype=torch.int16, device="cuda", generator=gen)
    v = torch.randint(-32768, 32767, (L, B, Hk, cap, hd), dtype=torch.int16, device="cuda", generator=gen)
    k_host = k.cpu().numpy().view(np.uint16).copy()
    v_host = v.cpu().numpy().view(np.uint16).copy()
    ln = _dev(lens)
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    kv = msd.KVCache(k.data_ptr(), v.data_ptr(), ln.data_ptr(), status.data_ptr(), B, cap)
    blk = msd.make_block(_dev(np.zeros((B, n), np.int32)), parent)
    msd.kv_commit(model.handle, kv, blk, _dev(acc), _dev(path))
    torch.cuda.synchronize()
    want_len = lens.copy()
    for b in range(B - 1):
        kb = np.ascontiguousarray(k_host[:, b])
        vb = np.ascontiguousarray(v_host[:, b])
        want_len[b] = orc.Oracle.kv_commit(kb, vb, int(lens[b]), int(acc[b]), path[b, :acc[b] + 1])
        k_host[:, b] = kb
        v_host[:, b] = vb
    assert np.array_equal(ln.cpu().numpy(), want_len)
    assert want_len[-1] == lens[-1]
    assert np.array_equal(k.cpu().numpy().view(np.uint16), k_host)
    assert np.array_equal(v.cpu().numpy().view(np.uint16), v_host)
    assert sum(int(path[b, r] != r) for b in range(B - 1) for r in range(1, acc[b] + 1)) >= 10
    model.close()


def test_kv_commit_chain_advances_len_only():
    """On a chain the accepted rows already sit at len + r: the cache is
    unchanged and len advances by 1 + A."""
    torch = _torch()
    from paper_2510_13161_amd import msd
    model, shape = _model(1024, n_layers=2, n_kv_heads=2, head_dim=128)
    n, B, cap = 9, 5, 64
    lens = np.array([0, 10, 20, 30, 40], np.int32)
    acc = np.array([0, 3, 8, 1, 5], np.int32)
    path = np.full((B, n), -1, np.int32)
    for b in range(B):
        path[b, :acc[b] + 1] = np.arange(acc[b] + 1)
    k = torch.randint(-32768, 32767, (2, B, 2, cap, 128), dtype=torch.int16, device="cuda")
    v = torch.randint(-32768, 32767, (2, B, 2, cap, 128), dtype=torch.int16, device="cuda")
    k0, v0 = k.clone(), v.clone()
    ln = _dev(lens)
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    kv = msd.KVCache(k.data_ptr(), v.data_ptr(), ln.data_ptr(), status.data_ptr(), B, cap)
    msd.kv_commit(model.handle, kv, msd.make_block(_dev(np.zeros((B, n), np.int32))), _dev(acc), _dev(path))
    torch.cuda.synchronize()
    assert np.array_equal(ln.cpu().numpy(), lens + 1 + acc)
    assert torch.equal(k, k0) and torch.equal(v, v0)
    model.close()
