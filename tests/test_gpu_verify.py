"""Parity of the HIP verification step (through the C ABI) against the oracle."""
import numpy as np
import pytest

from paper_2510_13161_amd import synth
from tests import harness as H

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def check_ee_message(ids, logp, z, kappa, tol=H.TOL_LOGIT, report=None):
    """Complete validity check of the early-exit message M_t = Top-kappa(p^(l_e))
    (Sec. 3.1) on every row, against the oracle's early-exit logits z [n, V]:
    kappa distinct ids in the vocabulary; each id's oracle logit at least the
    oracle's kappa-th best minus 2 tol; the order non-increasing in oracle
    logit within 2 tol; each log-probability within tol of the oracle's
    log-softmax at that id. Where the oracle's kappa + 1 best logits are all
    more than 2 tol apart, the ids must equal the oracle's exactly."""
    n, V = z.shape
    assert ids.shape == (n, kappa) and logp.shape == (n, kappa)
    mx = z.max(-1, keepdims=True)
    lse = (np.log(np.exp(z - mx).sum(-1, keepdims=True)) + mx)[:, 0]
    srt = -np.sort(-z, axis=-1)
    firm = H.margins(z, kappa) >= H.TIE_MARGIN
    want_ids = np.argsort(-z, axis=-1, kind="stable")[:, :kappa]
    for i in range(n):
        r = ids[i].astype(np.int64)
        assert np.all((r >= 0) & (r < V)) and len(set(r.tolist())) == kappa, f"row {i}: ids {r}"
        zo = z[i, r]
        assert np.all(zo >= srt[i, kappa - 1] - 2 * tol), f"row {i}: an id outside the top-{kappa}"
        assert np.all(zo[:-1] >= zo[1:] - 2 * tol), f"row {i}: order"
        err = np.abs(logp[i] - (zo - lse[i]))
        assert err.max() <= tol, f"row {i}: early-exit logp {err.max():.3e}"
        if firm[i]:
            assert np.array_equal(r, want_ids[i]), f"row {i}: firm ids differ"
    if report is not None:
        report["ee_rows"] = report.get("ee_rows", 0) + n
        report["ee_firm_rows"] = report.get("ee_firm_rows", 0) + int(firm.sum())
    return n


def _compare(case, gr, seqs, check_ee=True, tol=H.TOL_LOGIT, min_decisions=1):
    """Element-wise comparison of one GPU step with the oracle's sequences.

    Decisions (A, path, next token) are exact except at the oracle's near-tie
    flags: a path decision in a band leaves only the path down to that node
    to compare; a next-token decision in a band leaves the token out. K/V
    rows (after verify, and the committed rows after the commit) are
    compared on every sequence whatever its decisions."""
    w, si = case.w, case.si
    n, V = w.n_slots, case.shape.vocab
    report = {"max_abs": 0.0, "flagged_rows": 0, "flagged_seqs": 0, "decisions": 0, "argmax_rows": 0}
    for b, o in seqs.items():
        rows = slice(b * n, (b + 1) * n)
        if gr.logits is not None:
            err = np.abs(gr.logits[rows] - o.logits)
            report["max_abs"] = max(report["max_abs"], float(err.max()))
            assert err.max() <= tol, f"seq {b}: logits max abs {err.max():.3e} > {tol}"
        lse_ref = np.log(np.exp(o.logits - o.logits.max(-1, keepdims=True)).sum(-1)) + o.logits.max(-1)
        assert np.max(np.abs(gr.lse[rows] - lse_ref)) <= tol
        top1 = np.argmax(o.logits, -1)
        tie = H.margins(o.logits, 1) < H.TIE_MARGIN
        report["flagged_rows"] += int(tie.sum())
        report["argmax_rows"] += int((~tie).sum())
        assert np.array_equal(gr.argmax[rows][~tie], top1[~tie]), f"seq {b}: argmax differs"
        if check_ee and o.ee_ids is not None:
            check_ee_message(gr.ee_ids[rows], gr.ee_logp[rows], o.ee_logits, w.kappa, tol, report)
        # decisions, exact outside the oracle's near-tie bands
        A = int(gr.acc_len[b])
        if o.tie_depth < 0:
            assert A == o.acc, f"seq {b}: accepted length {A} != {o.acc}"
            assert np.array_equal(gr.path[b][:o.acc + 1], o.path), f"seq {b}: path"
            if not o.tie_next:
                assert gr.next_tok[b] == o.nxt, f"seq {b}: next token {gr.next_tok[b]} != {o.nxt}"
            report["decisions"] += o.acc + 1
        else:
            report["flagged_seqs"] += 1
            d = min(o.tie_depth, o.acc)
            assert A >= d and np.array_equal(gr.path[b][:d + 1], o.path[:d + 1]), f"seq {b}: path prefix"
            report["decisions"] += d
        assert np.all(gr.path[b][A + 1:] == -1)
        assert gr.len_after[b] == si.ctx_len[b] + 1 + A
        if gr.near_tie is not None and o.tie_depth < 0 and not o.tie_next:
            assert gr.near_tie[b] == 0, f"seq {b}: GPU flags a near tie the oracle does not"
        # K/V rows the verify pass wrote at len + slot, and the committed rows
        # len + r <- len + path[r] (the GPU's own path)
        gpath = gr.path[b][:A + 1]
        for l in range(case.shape.n_layers):
            ko = np.transpose(o.blk_k[l], (1, 0, 2))     # [Hkv][n][hd]
            vo = np.transpose(o.blk_v[l], (1, 0, 2))
            sk = max(1.0, float(np.abs(ko).max()))
            sv = max(1.0, float(np.abs(vo).max()))
            kg = synth.bf16_bits_to_f32(gr.k_rows[l][b]).astype(np.float64)
            vg = synth.bf16_bits_to_f32(gr.v_rows[l][b]).astype(np.float64)
            assert np.max(np.abs(kg - ko)) <= tol * sk, f"layer {l} k rows"
            assert np.max(np.abs(vg - vo)) <= tol * sv, f"layer {l} v rows"
            if gr.k_commit is not None:
                kc = synth.bf16_bits_to_f32(gr.k_commit[l][b][:, :A + 1]).astype(np.float64)
                vc = synth.bf16_bits_to_f32(gr.v_commit[l][b][:, :A + 1]).astype(np.float64)
                assert np.max(np.abs(kc - ko[:, gpath])) <= tol * sk, f"layer {l} committed k rows"
                assert np.max(np.abs(vc - vo[:, gpath])) <= tol * sv, f"layer {l} committed v rows"
                # the committed rows are the verify pass's rows moved bit for bit
                assert np.array_equal(gr.k_commit[l][b][:, :A + 1], gr.k_rows[l][b][:, gpath])
                assert np.array_equal(gr.v_commit[l][b][:, :A + 1], gr.v_rows[l][b][:, gpath])
    assert gr.status == 0
    assert report["decisions"] + report["argmax_rows"] >= min_decisions, report
    return report


def test_device_generator_matches_host():
    torch = _torch()
    m = synth.TINY
    dev = synth.device_weights(m, 0)
    host = synth.host_weights(m, 0)
    for name, t in dev.items():
        d = t.view(torch.int16).cpu().numpy().view(np.uint16)
        assert np.array_equal(d, host[name]), name
    k = torch.zeros((1, 2, 4, 160, 64), dtype=torch.bfloat16, device="cuda")
    v = torch.zeros_like(k)
    lens = torch.tensor([100, 37], dtype=torch.int32, device="cuda")
    synth.device_fill_ctx(m, 3, k, v, lens)
    for b, L in enumerate([100, 37]):
        got = k[0, b, :, :L].view(torch.int16).cpu().numpy().view(np.uint16)
        assert np.array_equal(got, synth.host_ctx(m, 3, 0, "k", b, L))


@pytest.fixture(scope="module")
def tiny_case():
    _torch()
    return H.GpuCase(synth.WORKLOADS["tiny_chain"])


def test_tiny_chain_step(tiny_case):
    case = tiny_case
    case.reset_len()
    gr = case.run()
    o = H.oracle_sequence(case.shape, case.w, case.si, 0)
    rep = _compare(case, gr, {0: o})
    print("tiny chain:", rep)


PLANTED = {"tiny_chain": (synth.WORKLOADS["tiny_chain"], None, 4),
           "14b_chain_l2": (synth.WORKLOADS["14b_chain"], 2, 6)}


def _planted_root(name):
    import json
    import os
    with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "planted_roots.json")) as f:
        return json.load(f)[name]


def _check_planted_step(case, gr, A, want_next, slots, zs, ks, vs, tag):
    """One planted step: decisions exact (A, path, next token, no near tie),
    the decision rows' logits and K/V rows equal the oracle's greedy decoding
    rows, and the committed rows len + r are those rows moved into place."""
    L = int(case.si.ctx_len[0])
    assert gr.status == 0, tag
    assert gr.acc_len[0] == A, f"{tag}: A {gr.acc_len[0]} != {A}"
    assert gr.next_tok[0] == want_next, f"{tag}: next {gr.next_tok[0]} != {want_next}"
    assert list(gr.path[0][:A + 1]) == slots[:A + 1] and np.all(gr.path[0][A + 1:] == -1), tag
    assert gr.near_tie[0] == 0, tag
    assert gr.len_after[0] == L + 1 + A, tag
    err = np.abs(gr.logits[slots[:A + 1]] - zs[:A + 1]).max()
    assert err <= H.TOL_LOGIT, f"{tag}: decision-row logits {err:.3e}"
    for l in range(case.shape.n_layers):
        ko = np.transpose(ks[l][:A + 1], (1, 0, 2))
        vo = np.transpose(vs[l][:A + 1], (1, 0, 2))
        tk = H.TOL_LOGIT * max(1.0, float(np.abs(ko).max()))
        tv = H.TOL_LOGIT * max(1.0, float(np.abs(vo).max()))
        kr = synth.bf16_bits_to_f32(gr.k_rows[l][0][:, slots[:A + 1]]).astype(np.float64)
        kc = synth.bf16_bits_to_f32(gr.k_commit[l][0][:, :A + 1]).astype(np.float64)
        vc = synth.bf16_bits_to_f32(gr.v_commit[l][0][:, :A + 1]).astype(np.float64)
        assert np.abs(kr - ko).max() <= tk, f"{tag}: layer {l} k rows"
        assert np.abs(kc - ko).max() <= tk, f"{tag}: layer {l} committed k rows"
        assert np.abs(vc - vo).max() <= tv, f"{tag}: layer {l} committed v rows"


@pytest.mark.parametrize("name", ["tiny_chain", "14b_chain_l2"])
def test_planted_greedy_verify_accept_commit(name):
    """Drafts taken from the oracle's token-by-token greedy decoding (Sec. 2)
    from a root whose every step has a decisive top-1/top-2 margin (chosen by
    tests/golden/make_planted_roots.py), with a planted mismatch, verified,
    accepted and committed through the C ABI:
    * a chain with every accepted length A = 0..gamma (A = gamma takes the
      bonus token);
    * the branch-complete tree (Sec. 3.1 T_t, 4 branches) accepting down
      branch 2 at every depth, and down branches 1 and 3: the accepted nodes
      sit at slots past their depth, so the commit moves their K/V rows.
    The GPU's A, path and next token must be the oracle's exactly, the
    decision rows' logits and K/V rows within tolerance, and the committed
    cache rows len..len + A the accepted nodes' rows."""
    torch = _torch()
    import oracle as orc
    w, layers, tree_gamma = PLANTED[name]
    pr = _planted_root(name)
    case = H.GpuCase(w, n_layers=layers)
    shape = case.shape
    assert shape.n_layers == pr["layers"]
    L = int(w.ctx[0])
    o = orc.Oracle(shape, synth.host_weights(shape, w.seed))
    cc = {l: (synth.host_ctx(shape, w.seed, l, "k", 0, L), synth.host_ctx(shape, w.seed, l, "v", 0, L))
          for l in range(shape.n_layers)}
    root = pr["root"]
    y, zs, ks, vs = o.decode_greedy(root, L, pr["steps"], lambda l: cc[l], L, return_kv=True)
    assert [int(t) for t in y] == pr["tokens"]
    assert H.margins(zs, 1).min() >= H.TIE_MARGIN
    V = shape.vocab
    g = np.random.default_rng(77)
    steps = 0
    # chain, A = 0..gamma
    gam = w.gamma
    for A in range(gam + 1):
        tok = np.concatenate([[root], y[:A], g.integers(0, V, size=gam - A)]).astype(np.int32)
        if A < gam:
            tok[A + 1] = (y[A] + 1) % V
        case.si = synth.StepInputs(parent=np.arange(-1, gam, dtype=np.int32), tokens=tok[None],
                                   ctx_len=np.array([L], np.int32))
        case.reset_len()
        gr = case.run(ee=False)
        _check_planted_step(case, gr, A, int(y[A]), list(range(gam + 1)), zs, ks, vs, f"chain A={A}")
        steps += 1
    # tree of 4 branches x tree_gamma
    K = 4
    tw = w.with_model(shape, topology="tree", gamma=tree_gamma, branches=K)
    case.w = tw
    parent = synth.topology(tw)
    slot = lambda br, r: 1 + br * tree_gamma + r - 1
    plan = [(2, A) for A in range(tree_gamma + 1)] + [(1, 1), (3, tree_gamma)]
    moved = 0
    for br, A in plan:
        tok = g.integers(0, V, size=tw.n_slots).astype(np.int32)
        tok[0] = root
        for b2 in range(K):
            if tok[slot(b2, 1)] == y[0]:
                tok[slot(b2, 1)] = (y[0] + 3) % V
        for r in range(1, A + 1):
            tok[slot(br, r)] = y[r - 1]
        if A < tree_gamma:
            tok[slot(br, A + 1)] = (y[A] + 1) % V
        case.si = synth.StepInputs(parent=parent, tokens=tok[None], ctx_len=np.array([L], np.int32))
        case.reset_len()
        gr = case.run(ee=False)
        slots = [0] + [slot(br, r) for r in range(1, tree_gamma + 1)]
        _check_planted_step(case, gr, A, int(y[A]), slots, zs, ks, vs, f"tree branch {br} A={A}")
        moved += sum(slots[r] != r for r in range(1, A + 1))
        steps += 1
    assert steps == gam + 1 + len(plan) and moved >= 10
    print(f"{name}: {steps} planted steps, {moved} committed rows moved")


def planted_rejection_inputs(g, parent, slots, A, root, y, p, V, C=32):
    """REJECTION inputs that accept the path `slots` down to depth A: at the
    node at depth d < A the child on the path carries y[d] with a draft mass
    of p[d, y[d]] / 4 (a quarter of its target mass under the oracle's law at
    that row, so alpha = 1 even after rejections); the children tested before
    it carry other tokens with a draft mass of 0.5 / (children) and almost no
    target mass (rejected); at depth A every child is rejected the same way.
    Returns tokens [n], cand_ids [n][C], cand_q [n][C]."""
    n = len(parent)
    kids = [[c for c in range(n) if parent[c] == s] for s in range(n)]
    tok = g.integers(0, V, size=n).astype(np.int32)
    tok[0] = root
    cand = np.zeros((n, C), np.int32)
    q = np.zeros((n, C), np.float32)
    for s in range(n):
        d = slots.index(s) if s in slots[:A + 1] else None
        on = slots[d + 1] if d is not None and d < A else None
        fixed = []                                   # (token, draft mass), tested children in slot order
        for c in kids[s]:
            if c == on:
                tok[c] = y[d]
                fixed.append((int(tok[c]), p[d, y[d]] / 4))
                break
            while (d is not None and tok[c] == y[d]) or int(tok[c]) in [t for t, _ in fixed]:
                tok[c] = (tok[c] + 1) % V
            fixed.append((int(tok[c]), 0.5 / len(kids[s])))
        ids = [t for t, _ in fixed]
        for t in g.choice(V, size=2 * C, replace=False):
            if len(ids) == C:
                break
            if int(t) not in ids:
                ids.append(int(t))
        free = synth.dirichlet_rows(g, 0.5, (C - len(fixed),)).astype(np.float64)
        vals = [m for _, m in fixed] + list(free * (1.0 - sum(m for _, m in fixed)))
        cand[s] = ids
        q[s] = np.array(vals, np.float32) / np.float32(np.sum(vals, dtype=np.float32))
    return tok, cand, q


def test_tiny_planted_rejection_descends():
    """REJECTION through the whole step on the tiny model (planted_rejection_inputs):
    a chain accepting 0, 2 and 4 drafts (4: the leaf bonus) and the 4 x 4
    tree descending branch 2 after rejecting branches 0 and 1. A and the path
    are exact; the next token is compared unless the oracle flags its
    inverse-CDF draw."""
    _torch()
    import oracle as orc
    import scipy.special
    w = synth.WORKLOADS["tiny_chain"]
    pr = _planted_root("tiny_chain")
    case = H.GpuCase(w)
    shape = case.shape
    L = int(w.ctx[0])
    weights = synth.host_weights(shape, w.seed)
    o = orc.Oracle(shape, weights)
    cc = {l: (synth.host_ctx(shape, w.seed, l, "k", 0, L), synth.host_ctx(shape, w.seed, l, "v", 0, L))
          for l in range(shape.n_layers)}
    root = pr["root"]
    y, zs = o.decode_greedy(root, L, pr["steps"], lambda l: cc[l], L)
    p = scipy.special.softmax(zs, axis=-1)
    g = np.random.default_rng(78)
    gam = w.gamma
    compared = 0
    for topo, br, A in [("chain", 0, 0), ("chain", 0, 2), ("chain", 0, 4), ("tree", 2, 3), ("tree", 2, 0)]:
        tw = w.with_model(shape, topology=topo, gamma=gam, branches=4 if topo == "tree" else 1,
                          mode="rejection")
        case.w = tw
        parent = synth.topology(tw)
        slots = [0] + (list(range(1, gam + 1)) if topo == "chain" else
                       [1 + br * gam + r - 1 for r in range(1, gam + 1)])
        tok, cand, q = planted_rejection_inputs(g, parent, slots, A, root, y, p, shape.vocab)
        n = tw.n_slots
        case.si = synth.StepInputs(parent=parent, tokens=tok[None], ctx_len=np.array([L], np.int32),
                                   cand_ids=cand[None], cand_q=q[None],
                                   u_accept=np.full((1, n), 0.5, np.float32),
                                   u_sample=synth.uniforms01(g, (1, n)))
        case.reset_len()
        gr = case.run(ee=False)
        oseq = H.oracle_sequence(shape, tw, case.si, 0, ee=False, weights=weights)
        assert oseq.acc == A and list(oseq.path) == slots[:A + 1], (topo, A, oseq.acc, oseq.path)
        rep = _compare(case, gr, {0: oseq}, check_ee=False)
        assert rep["flagged_seqs"] == 0
        compared += 1 + (not oseq.tie_next)
    assert compared >= 5


def test_tiny_tree_rejection_and_match():
    _torch()
    w = synth.WORKLOADS["14b_tree"].with_model(synth.TINY, ee_layer=1, kappa=4, seed=7, ctx=(96, 96))
    case = H.GpuCase(w)
    for mode in ("rejection", "match", "greedy"):
        case.reset_len()
        gr = case.run(mode=mode)
        o = H.oracle_sequence(case.shape, w, case.si, 0, mode=mode)
        _compare(case, gr, {0: o})


@pytest.mark.parametrize("kappa", [16, 32])
def test_tiny_wide_early_exit_message(kappa):
    """The early-exit message at kappa above 8 (wider merge lists)."""
    _torch()
    w = synth.WORKLOADS["tiny_chain"].with_model(synth.TINY, ee_layer=1, kappa=kappa, seed=11)
    case = H.GpuCase(w)
    case.reset_len()
    gr = case.run()
    o = H.oracle_sequence(case.shape, w, case.si, 0)
    _compare(case, gr, {0: o})
    assert gr.ee_ids.shape[-1] == kappa


@pytest.mark.parametrize("which,M,kappa", [("tiny", 9, 8), ("tiny", 144, 4), ("14b", 9, 8),
                                             ("14b", 144, 4), ("14b", 9, 32), ("14b", 144, 13),
                                             ("14b", 9, 1)])
def test_early_exit_topk_entry_point(which, M, kappa):
    """msd_early_exit_topk on its own (the Sec. 3.1 token channel from a
    residual): seeded fp32 residual rows, final norm, LM head and top-kappa
    with log-probabilities, at one row tile (M = 9) and at the batch-16 block
    size (M = 144, nine row tiles), checked row by row against the oracle's
    head on the same rows (check_ee_message); every merge width (kappa 1, up
    to 8, up to 32) over the 14B vocabulary's 5 or 10 merge parts."""
    torch = _torch()
    import oracle as orc
    from paper_2510_13161_amd import msd
    shape = synth.TINY if which == "tiny" else synth.QWEN14B.with_layers(1)
    seed = 31
    model = msd.Model(shape, synth.device_weights(shape, seed), max_positions=64)
    g = np.random.default_rng(32 + M)
    x = g.normal(0.0, 1.0, size=(M, shape.d_model)).astype(np.float32)
    x[0] *= np.float32(50.0)        # the norm is scale-free: a large row and a small one
    x[-1] *= np.float32(0.01)
    hidden = torch.from_numpy(x).cuda()
    ids = torch.full((M, kappa), -1, dtype=torch.int32, device="cuda")
    logp = torch.zeros((M, kappa), dtype=torch.float32, device="cuda")
    ws = torch.empty(msd.workspace_bytes(model.handle, 1, M, kappa, 1), dtype=torch.uint8, device="cuda")
    msd.early_exit_topk(model.handle, hidden, kappa, ids, logp, ws)
    torch.cuda.synchronize()
    o = orc.Oracle(shape, synth.host_weights(shape, seed, layers=[], with_globals=True))
    z = o.head(x.astype(np.float64))
    rep = {}
    assert check_ee_message(ids.cpu().numpy(), logp.cpu().numpy(), z, kappa, report=rep) == M
    print(which, M, rep)
    model.close()


def test_tiny_reuse_selection_and_fallback_statistics():
    """Sec. 3.1 reuse criterion and next-window selection with the App. E
    fallback statistics, through the C ABI, against the oracle. Accept
    outcomes are planted (A cycles through 0..gamma along the chain block,
    corrections drawn), the hypothesis tree (4 chains of gamma + 1 nodes,
    shared topology, per-sequence tokens) holds the corrected prefix on two
    sequences in three; Omega is taken at the root row over the oracle's
    early-exit ids. Two calls accumulate the statistics."""
    torch = _torch()
    import oracle as orc
    from paper_2510_13161_amd import msd
    w = synth.WORKLOADS["14b_batch16"].with_model(synth.TINY, ee_layer=1, kappa=4, seed=5, ctx=(64, 96))
    case = H.GpuCase(w)
    case.reset_len()
    gr = case.run(commit=False)
    B, n, V, kap = w.batch, w.n_slots, case.shape.vocab, w.kappa
    rng = np.random.default_rng(9)
    acc = np.array([b % n for b in range(B)], np.int32)
    nxt = rng.integers(0, V, size=B).astype(np.int32)
    path = np.full((B, n), -1, np.int32)
    for b in range(B):
        path[b, :acc[b] + 1] = np.arange(acc[b] + 1)
    parent = []
    for r in range(4):
        for d in range(n):
            parent.append(-1 if d == 0 else len(parent) - 1)
    ttok = rng.integers(0, V, size=(B, len(parent))).astype(np.int32)
    for b in range(B):
        if b % 3 != 2:
            pi = [int(t) for t in case.si.tokens[b, 1:acc[b] + 1]] + [int(nxt[b])]
            ttok[b, (b % 4) * n:(b % 4) * n + len(pi)] = pi
    ee_ids = np.zeros((B * n, kap), np.int32)
    want_case, want_node, want_omega = [], [], []
    weights = synth.host_weights(case.shape, w.seed)
    for b in range(B):
        o = H.oracle_sequence(case.shape, w, case.si, b, weights=weights)
        c_, v_ = orc.reuse_select(parent, ttok[b], case.si.tokens[b, 1:acc[b] + 1], int(nxt[b]))
        want_case.append(c_)
        want_node.append(v_)
        want_omega.append(orc.overlap_mass(o.logits[0], o.ee_ids[0]))
        ee_ids[b * n] = o.ee_ids[0]
    assert {orc.NEXT_BRANCH, orc.NEXT_CONTINUE, orc.NEXT_FRESH} <= set(want_case)

    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    tok_dev = dev(case.si.tokens)
    blk = msd.make_block(tok_dev, None)
    tree = msd.hyp_tree(parent, dev(ttok))
    out_case = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    out_node = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    omega = torch.zeros(B, dtype=torch.float32, device="cuda")
    stats = torch.zeros(64, dtype=torch.uint8, device="cuda")
    logits, lse = dev(gr.logits), dev(gr.lse)
    a_acc, a_nxt, a_path, a_ids = dev(acc), dev(nxt), dev(path), dev(ee_ids)
    for _ in range(2):
        msd.reuse_select(case.model.handle, blk, a_acc, a_nxt, a_path, tree, out_case, out_node,
                         logits, lse, a_ids, kap, omega, stats)
    torch.cuda.synchronize()
    assert out_case.cpu().numpy().tolist() == want_case
    assert out_node.cpu().numpy().tolist() == want_node
    om = omega.cpu().numpy().astype(np.float64)
    assert np.max(np.abs(om - np.array(want_omega))) <= 1e-3
    st = msd.read_reuse_stats(stats)
    fresh = [c == orc.NEXT_FRESH for c in want_case]
    assert st["trials"] == 2 * B and st["omega_trials"] == 2 * B
    assert st["fallbacks"] == 2 * sum(fresh)
    assert st["fallbacks_tau1"] == 2 * sum(f and a == 0 for f, a in zip(fresh, acc))
    assert abs(st["omega_sum"] - 2 * sum(want_omega)) <= 2e-3 * B
    # without Omega inputs: the same selection, statistics without Omega
    stats.zero_()
    msd.reuse_select(case.model.handle, blk, a_acc, a_nxt, a_path, tree, out_case, out_node, stats=stats)
    torch.cuda.synchronize()
    assert out_case.cpu().numpy().tolist() == want_case
    st = msd.read_reuse_stats(stats)
    assert st["trials"] == B and st["omega_trials"] == 0 and st["omega_sum"] == 0.0


@pytest.mark.parametrize("name,ctx,topo,gamma,branches", [
    ("root_only", 96, "chain", 0, 1),        # n_slots = 1: no draft token, A = 0
    ("empty_context", 0, "chain", 4, 1),     # L = 0: the block attends only to itself
    ("one_chunk", 251, "chain", 4, 1),       # L + n_slots = 256 keys: one attention chunk
    ("chunk_plus_one", 252, "chain", 4, 1),  # 257 keys: a second chunk holding one key
    ("max_tree", 40, "tree", 9, 7),          # 1 + 7 x 9 = 64 slots (ancestor bit 63, M = 64)
])
def test_tiny_degenerate_blocks(name, ctx, topo, gamma, branches):
    """The method's degenerate and boundary blocks, element by element against the oracle."""
    _torch()
    w = synth.WORKLOADS["tiny_chain"].with_model(synth.TINY, ctx=(ctx, ctx), topology=topo, gamma=gamma,
                                                 branches=branches, ee_layer=1, kappa=4, seed=21)
    assert w.n_slots <= 64
    case = H.GpuCase(w)
    case.reset_len()
    gr = case.run()
    o = H.oracle_sequence(case.shape, w, case.si, 0)
    rep = _compare(case, gr, {0: o})
    print(name, rep)


@pytest.mark.parametrize("mode,seed", [("greedy", k) for k in range(6)] + [("rejection", k) for k in range(4)]
                         + [("match", k) for k in range(2)])
def test_tiny_random_tree_blocks(mode, seed):
    """Random trees (each slot's parent drawn among the earlier slots, 2 to 64
    slots, so depths and ancestor sets of every shape a forest in slot order
    allows) over random contexts and batch sizes: the attention's ancestor
    masks, the rotary positions and cache rows at each node's depth, and the
    acceptance walk over a general tree (greedy, and the stochastic rules
    with each child's token drawn from its parent's candidates), element by
    element against the oracle."""
    _torch()
    g = np.random.default_rng(1000 + seed + (0 if mode == "greedy" else 100 * len(mode)))
    n = int(g.integers(2, 65))
    B = int(g.integers(1, min(4, 144 // n) + 1))
    lo = int(g.integers(0, 600))
    hi = lo + int(g.integers(0, 500))
    parent = tuple([-1] + [int(g.integers(0, i)) for i in range(1, n)])
    w = synth.WORKLOADS["tiny_chain"].with_model(synth.TINY, batch=B, ctx=(lo, hi), topology="forest", gamma=0,
                                                 parents=parent, ee_layer=1, kappa=4, mode=mode,
                                                 temperature=1.0, seed=70 + seed)
    assert w.n_slots == n
    case = H.GpuCase(w)
    case.reset_len()
    gr = case.run()
    weights = synth.host_weights(case.shape, w.seed)
    seqs = {b: H.oracle_sequence(case.shape, w, case.si, b, weights=weights) for b in range(B)}
    par = np.asarray(parent)
    depth = np.zeros(n, dtype=np.int32)
    for i in range(1, n):
        depth[i] = depth[par[i]] + 1
    leaves = n - len(set(par[1:].tolist()))
    print("random tree", mode, seed, "slots", n, "batch", B, "ctx", case.si.ctx_len.tolist(), "max depth",
          int(depth.max()), "leaves", leaves, "accepted", gr.acc_len.tolist(), _compare(case, gr, seqs))


def test_tiny_ragged_batch():
    """Sequences of different context lengths in one block batch (1 to 2 chunks)."""
    _torch()
    w = synth.WORKLOADS["14b_batch16"].with_model(synth.TINY, batch=5, ctx=(1, 400), ee_layer=1, kappa=4,
                                                  seed=23)
    case = H.GpuCase(w)
    case.reset_len()
    gr = case.run()
    weights = synth.host_weights(case.shape, w.seed)
    seqs = {b: H.oracle_sequence(case.shape, w, case.si, b, weights=weights) for b in range(w.batch)}
    assert len(set(case.si.ctx_len.tolist())) > 1
    print("ragged:", _compare(case, gr, seqs))


def test_device_errors_are_flagged():
    """Device-detected errors set the caller's status word: a block that does
    not fit the cache (len + n_slots > capacity) and a token outside the
    vocabulary; the cache rows past len are left as they were."""
    torch = _torch()
    from paper_2510_13161_amd import msd
    w = synth.WORKLOADS["tiny_chain"].with_model(synth.TINY, ctx=(62, 62), seed=25)
    case = H.GpuCase(w, capacity=64)     # 62 + 5 slots > 64
    case.reset_len()
    k_before = case.cache.k.clone()
    gr = case.run(commit=False)
    assert gr.status & msd.MSD_DEV_CAPACITY
    assert torch.equal(case.cache.k, k_before)
    w2 = synth.WORKLOADS["tiny_chain"].with_model(synth.TINY, seed=26)
    si = synth.step_inputs(w2)
    si.tokens[0, 2] = w2.model.vocab + 5
    case2 = H.GpuCase(w2, inputs=si)
    case2.reset_len()
    gr2 = case2.run(commit=False)
    assert gr2.status & msd.MSD_DEV_TOKEN


# LayerNorm, ReLU, learned positions, biases and a tied head (the 66B
# shape's features) at tiny widths: 4 MHA heads of 64
TINY_LN = synth.ModelShape("tiny_ln", 2, 256, 4, 4, 64, 1024, 4096, norm="layer", act="relu", pos="learned",
                           bias=True, tied_head=True, norm_eps=1.0e-5, max_positions=1024)


@pytest.mark.parametrize("which", ["tiny", "14b", "tiny_ln"])
@pytest.mark.parametrize("jt", [2, 4])
def test_qkv_tile_widths_at_one_row_tile(monkeypatch, which, jt):
    """The QKV projection at one row tile in 32-column whole-K tiles (the
    default where they fit the compute units) and in 64-column tiles with
    splits of K (MSD_QKV_JT=4): RoPE pairs split across the tile's halves,
    the KV append and the query image (tiny and 14B widths, 2 layers of the
    latter), and the q/k/v biases without a rotary table (tiny LayerNorm
    model with learned positions)."""
    _torch()
    monkeypatch.setenv("MSD_QKV_JT", str(jt))
    if which == "14b":
        w = synth.WORKLOADS["14b_chain"].with_model(synth.QWEN14B)
    else:
        w = synth.WORKLOADS["tiny_chain"].with_model(synth.TINY if which == "tiny" else TINY_LN, seed=43)
    case = H.GpuCase(w, n_layers=2 if which == "14b" else None)
    case.reset_len()
    gr = case.run()
    o = H.oracle_sequence(case.shape, w, case.si, 0)
    print("qkv tiles", which, jt, _compare(case, gr, {0: o}))


def test_depth_reduced_14b_chain():
    """14B widths (d 5120, GQA 40/8, FFN 13824, vocab 152064) with 2 layers."""
    _torch()
    w = synth.WORKLOADS["14b_chain"].with_model(synth.QWEN14B)
    case = H.GpuCase(w, n_layers=2)
    gr = case.run()
    o = H.oracle_sequence(case.shape, w, case.si, 0)
    rep = _compare(case, gr, {0: o})
    print("14b L2 chain:", rep)


@pytest.mark.parametrize("mode,seed,batch", [("greedy", 0, 1), ("rejection", 1, 1), ("greedy", 2, 3)])
def test_depth_reduced_14b_random_tree(mode, seed, batch):
    """Random trees at 14B widths with 2 layers: 20 to 64 slots whose parents
    are drawn among the earlier slots, contexts of 600 to 3000 keys (the
    ring-fed attention with the tree's ancestor masks; the multi-row-tile
    GEMMs from 3 row tiles on), greedy and REJECTION acceptance."""
    _torch()
    g = np.random.default_rng(2000 + seed)
    n = int(g.integers(20, 65))
    n = min(n, 144 // batch)
    parent = tuple([-1] + [int(g.integers(0, i)) for i in range(1, n)])
    w = synth.WORKLOADS["14b_tree"].with_model(synth.QWEN14B, batch=batch, ctx=(600, 3000), topology="forest",
                                               gamma=0, parents=parent, mode=mode, seed=80 + seed)
    case = H.GpuCase(w, n_layers=2)
    case.reset_len()
    gr = case.run()
    seqs = {b: H.oracle_sequence(case.shape, w, case.si, b) for b in range(batch)}
    print("14b L2 random tree", mode, seed, "slots", n, "batch", batch, "ctx", case.si.ctx_len.tolist(),
          _compare(case, gr, seqs))


@pytest.mark.parametrize("gamma", [0, 8])
def test_draft_shape(gamma):
    """The 0.6B-shaped draft decoder that the latency-law measurement runs (d
    1024, GQA 16/8 x 128, SwiGLU 3072, tied head over the target's 152064
    vocabulary), 4 layers, kappa = 8 sequences after a 1024-key context: one
    slot each (one greedy draft decode step of the kappa branches, 8 rows)
    and gamma + 1 = 9 slots each (the Speculative Streaming pass: per branch
    the main stream and gamma lookahead streams form a chain; 72 rows, five
    row tiles)."""
    _torch()
    w = synth.Workload("draft_shape", synth.DRAFT06B, 8, (1024, 1024), "chain", gamma, ee_layer=2,
                       kappa=4, seed=5)
    case = H.GpuCase(w, n_layers=4)
    gr = case.run()
    weights = synth.host_weights(case.shape, w.seed)
    seqs = {b: H.oracle_sequence(case.shape, w, case.si, b, weights=weights) for b in (0, 3, 7)}
    print("draft shape, gamma", gamma, _compare(case, gr, seqs))


def _gqa64_tree():
    shape = synth.ModelShape("gqa64", 2, 1024, 16, 4, 64, 2048, 4096, rope_theta=1.0e4)
    return synth.Workload("gqa64_tree", shape, 4, (4600, 4800), "tree", 6, branches=4, ee_layer=1,
                          kappa=4, seed=11)


def test_attention_query_tile_groups(monkeypatch):
    """Attention workgroups that take several query tiles in turn (the
    one-span kernel, forced): GQA 16/4 with head_dim 64 and a 25-slot tree
    (7 query tiles of the 100 queries per kv head), 4 sequences with contexts
    up to 4800 (19 key chunks merged across workgroups): 19 x 4 x 4 x 7
    workgroups exceed the grouping threshold, so the tiles go 2 per
    workgroup with a ragged last group."""
    _torch()
    monkeypatch.setenv("MSD_ATTN_SPANS", "1")
    w = _gqa64_tree()
    case = H.GpuCase(w)
    gr = case.run()
    seqs = {b: H.oracle_sequence(case.shape, w, case.si, b) for b in (0, 3)}
    rep = _compare(case, gr, seqs)
    print("query tile groups:", rep)


def test_attention_streaming_chosen():
    """The same workload with the launch shape the library picks: the
    streaming kernel (19 one-span chunks x 4 kv heads x 4 sequences x 3 tile
    groups exceed one workgroup per compute unit, so a workgroup walks 4
    spans with an online softmax), 3 query tiles a workgroup with a ragged
    last group of 1, head_dim 64, the tree mask in the last span."""
    _torch()
    w = _gqa64_tree()
    case = H.GpuCase(w)
    gr = case.run()
    seqs = {b: H.oracle_sequence(case.shape, w, case.si, b) for b in (0, 3)}
    rep = _compare(case, gr, seqs)
    print("streaming attention:", rep)


@pytest.mark.parametrize("spans", [2, 3])
def test_attention_streaming_ragged_batch(monkeypatch, spans):
    """Streaming kernel forced on a ragged batch (contexts 1 to 1000, one
    query tile): sequences whose keys fit one chunk of `spans` spans write
    their output directly, longer ones merge two chunks; waves whose blocks
    lie past the last key contribute nothing."""
    _torch()
    monkeypatch.setenv("MSD_ATTN_SPANS", str(spans))
    w = synth.WORKLOADS["14b_batch16"].with_model(synth.TINY, batch=6, ctx=(1, 1000), ee_layer=1, kappa=4,
                                                  seed=27)
    case = H.GpuCase(w)
    case.reset_len()
    gr = case.run()
    weights = synth.host_weights(case.shape, w.seed)
    seqs = {b: H.oracle_sequence(case.shape, w, case.si, b, weights=weights) for b in range(w.batch)}
    lens = case.si.ctx_len + w.n_slots
    assert lens.min() <= 256 * spans < lens.max()
    print("streaming ragged:", _compare(case, gr, seqs))


# widths whose tile counts are not multiples of 4: 15 q/k/v tiles, 5 output
# and down tiles, 34 SwiGLU up tiles, 63 LM-head tiles (the last half padding)
ROWS_RAGGED = synth.ModelShape("rows_ragged", 2, 320, 5, 5, 64, 1088, 4000, rope_theta=1.0e4)


@pytest.mark.parametrize("shape,batch,splits", [("tiny", 16, 1), ("tiny", 16, 4), ("tiny", 6, 2),
                                                ("ragged", 16, 2), ("tiny", 4, 2), ("ragged", 2, 4)])
def test_rows_kernel_every_gemm(monkeypatch, shape, batch, splits):
    """The GEMM kernel that shares the activation through LDS (4 tiles a
    workgroup, a loader wave) forced on every GEMM of 64-column tiles: nine
    row tiles (batch 16 x 9 slots), five (batch 6: 54 rows, padding rows in
    the last tile), three (batch 4) and two (batch 2; the SwiGLU up
    projection keeps its 128-column tiles below four row tiles), whole-K and
    split-K (the FFN down projection, 32 k-steps, takes the splits); and
    widths whose last workgroup has waves past the matrix."""
    _torch()
    monkeypatch.setenv("MSD_ROWS_MIN_MT", "2")
    monkeypatch.setenv("MSD_ROWS_MIN_TILES", "1")
    monkeypatch.setenv("MSD_ROWS_MAX_SPLITS", str(splits))
    model = synth.TINY if shape == "tiny" else ROWS_RAGGED
    w = synth.WORKLOADS["14b_batch16"].with_model(model, batch=batch, ctx=(1, 600), ee_layer=1, kappa=4,
                                                  seed=31 + batch + splits)
    case = H.GpuCase(w)
    case.reset_len()
    gr = case.run(ee=True)
    weights = synth.host_weights(case.shape, w.seed)
    seqs = {b: H.oracle_sequence(case.shape, w, case.si, b, weights=weights) for b in range(w.batch)}
    print("rows kernel", shape, batch, splits, _compare(case, gr, seqs))


@pytest.mark.parametrize("shape,batch", [("tiny", 16), ("tiny", 6), ("ragged", 16), ("tiny", 4)])
def test_rows_narrow_deferred_epilogue(monkeypatch, shape, batch):
    """Narrow GEMMs at 3, 5 and 9 row tiles in the LDS-shared kernel with their
    split sum and epilogue in a kernel of their own (MSD_ROWS_NARROW): the
    FFN down projection (32 k-steps) takes 4 splits, summed and finished one
    wave per row tile; widths of 5 and 15 tiles leave idle waves."""
    _torch()
    monkeypatch.setenv("MSD_ROWS_NARROW", "2")
    model = synth.TINY if shape == "tiny" else ROWS_RAGGED
    w = synth.WORKLOADS["14b_batch16"].with_model(model, batch=batch, ctx=(1, 600), ee_layer=1, kappa=4,
                                                  seed=41 + batch)
    case = H.GpuCase(w)
    case.reset_len()
    gr = case.run(ee=True)
    weights = synth.host_weights(case.shape, w.seed)
    seqs = {b: H.oracle_sequence(case.shape, w, case.si, b, weights=weights) for b in range(w.batch)}
    print("narrow deferred", shape, batch, _compare(case, gr, seqs))


@pytest.mark.parametrize("spans", [1, 2])
def test_attention_deferred_merge(monkeypatch, spans):
    """The attention's chunk merge in a kernel of its own, forced, under both
    attention kernels (one-span and streaming): a ragged batch (contexts 1
    to 1000) where some sequences fit one chunk (written by it, skipped by
    the merge kernel) and others merge up to 4."""
    _torch()
    monkeypatch.setenv("MSD_ATTN_DEFER", "1")
    monkeypatch.setenv("MSD_ATTN_SPANS", str(spans))
    w = synth.WORKLOADS["14b_batch16"].with_model(synth.TINY, batch=6, ctx=(1, 1000), ee_layer=1, kappa=4,
                                                  seed=20)
    case = H.GpuCase(w)
    case.reset_len()
    gr = case.run()
    weights = synth.host_weights(case.shape, w.seed)
    seqs = {b: H.oracle_sequence(case.shape, w, case.si, b, weights=weights) for b in range(w.batch)}
    lens = case.si.ctx_len + w.n_slots
    assert lens.min() <= 256 * spans < lens.max()
    print("deferred merge:", _compare(case, gr, seqs))


def test_attention_streaming_max_tree(monkeypatch):
    """Streaming kernel forced on the 64-slot tree (4 query tiles: a group of
    3 and a group of 1) after a 700-key context: the tree rows straddle two
    64-key blocks of the last span, so both take the masked path."""
    _torch()
    monkeypatch.setenv("MSD_ATTN_SPANS", "2")
    w = synth.WORKLOADS["tiny_chain"].with_model(synth.TINY, ctx=(700, 700), topology="tree", gamma=9,
                                                 branches=7, ee_layer=1, kappa=4, seed=29)
    assert w.n_slots == 64
    case = H.GpuCase(w)
    case.reset_len()
    gr = case.run()
    o = H.oracle_sequence(case.shape, w, case.si, 0)
    print("streaming max tree:", _compare(case, gr, {0: o}))


def test_attention_streaming_two_query_tiles(monkeypatch):
    """Streaming kernel forced with two query tiles a workgroup: the 25-slot
    tree (4 x 6) at one query head per kv head is 2 query tiles, after a
    900-key context (3 chunks of 2 spans; the tree rows in the last span,
    under the tree mask), in rejection mode."""
    _torch()
    monkeypatch.setenv("MSD_ATTN_SPANS", "2")
    w = synth.WORKLOADS["14b_tree"].with_model(synth.TINY, ee_layer=1, kappa=4, seed=37, ctx=(900, 900))
    assert (w.model.n_heads // w.model.n_kv_heads * w.n_slots + 15) // 16 == 2
    case = H.GpuCase(w)
    case.reset_len()
    gr = case.run()
    o = H.oracle_sequence(case.shape, w, case.si, 0)
    print("streaming two query tiles:", _compare(case, gr, {0: o}))


def test_attention_streaming_14b_widths(monkeypatch):
    """Streaming kernel forced at 14B widths (head_dim 128, GQA 40/8: 3 query
    tiles in one group), 2 layers, a 1024-key context in 3 chunks of 2 spans."""
    _torch()
    monkeypatch.setenv("MSD_ATTN_SPANS", "2")
    monkeypatch.setenv("MSD_ATTN_RING", "0")
    w = synth.WORKLOADS["14b_chain"].with_model(synth.QWEN14B)
    case = H.GpuCase(w, n_layers=2)
    gr = case.run()
    o = H.oracle_sequence(case.shape, w, case.si, 0)
    print("streaming 14b L2 chain:", _compare(case, gr, {0: o}))


def test_attention_ring_14b_widths(monkeypatch):
    """Ring-fed kernel (K and V blocks copied into an LDS ring by two loader
    waves, one compute wave per query tile) at 14B widths, 2 layers: a
    1033-key context in 3 chunks of 2 spans, the 3 query tiles of a kv head
    in one workgroup, chunks merged by the last to arrive."""
    _torch()
    monkeypatch.setenv("MSD_ATTN_SPANS", "2")
    w = synth.WORKLOADS["14b_chain"].with_model(synth.QWEN14B)
    case = H.GpuCase(w, n_layers=2)
    gr = case.run()
    o = H.oracle_sequence(case.shape, w, case.si, 0)
    print("ring 14b L2 chain:", _compare(case, gr, {0: o}))


@pytest.mark.parametrize("heads,defer", [(8, 0), (8, 1), (16, 0)])
def test_attention_ring_ragged_batch(monkeypatch, heads, defer):
    """Ring-fed kernel on a ragged batch (head dim 128, 2 kv heads, contexts
    1 to 1000, chunks of 2 spans): sequences of at most 512 keys are written
    by their only chunk, longer ones merge two (by the last to arrive, or by
    the merge kernel); blocks past a sequence's last key are masked. With 8
    query heads a kv head has 3 query tiles (one workgroup); with 16 it has 5
    (a group of 4 and a group of 1 whose other compute waves hold no tile)."""
    _torch()
    monkeypatch.setenv("MSD_ATTN_SPANS", "2")
    monkeypatch.setenv("MSD_ATTN_DEFER", str(defer))
    shape = synth.ModelShape(f"h128x{heads}", 2, 512, heads, 2, 128, 1024, 4096, rope_theta=1.0e4)
    w = synth.WORKLOADS["14b_batch16"].with_model(shape, batch=6, ctx=(1, 1000), ee_layer=1, kappa=4,
                                                  seed=32 + heads)
    case = H.GpuCase(w)
    case.reset_len()
    gr = case.run()
    weights = synth.host_weights(case.shape, w.seed)
    seqs = {b: H.oracle_sequence(case.shape, w, case.si, b, weights=weights) for b in range(w.batch)}
    lens = case.si.ctx_len + w.n_slots
    assert lens.min() <= 512 < lens.max()
    print("ring ragged", heads, defer, _compare(case, gr, seqs))


def test_attention_ring_max_tree(monkeypatch):
    """Ring-fed kernel (forced to chunks of 2 spans) on the 64-slot tree at
    head dim 128 with 4 query heads per kv head: 256 queries, 16 query tiles
    in 4 groups of 4 (all 8 compute waves hold a tile), after a 700-key
    context; the tree rows straddle two 64-key blocks of the last chunk, so
    the masked path runs in both halves of each."""
    _torch()
    monkeypatch.setenv("MSD_ATTN_SPANS", "2")
    shape = synth.ModelShape("h128x8t", 2, 512, 8, 2, 128, 1024, 4096, rope_theta=1.0e4)
    w = synth.WORKLOADS["tiny_chain"].with_model(shape, ctx=(700, 700), topology="tree", gamma=9,
                                                 branches=7, ee_layer=1, kappa=4, seed=29)
    assert w.n_slots == 64
    case = H.GpuCase(w)
    case.reset_len()
    gr = case.run()
    o = H.oracle_sequence(case.shape, w, case.si, 0)
    print("ring max tree:", _compare(case, gr, {0: o}))


@pytest.mark.parametrize("which,spans", [("tiny", None), ("tiny", 1), ("h128", None)])
def test_attention_at_maximum_capacity(monkeypatch, which, spans):
    """A chain block that fills the cache to its maximum capacity (32768
    positions: 32759 cached keys + 9 slots, 128 chunks of 256 keys per kv
    head): head dim 64 under the kernel chosen by size, the one-span kernel
    forced (128 chunks merged by the merge kernel), and head dim 128 (the
    ring-fed kernel)."""
    _torch()
    if spans is not None:
        monkeypatch.setenv("MSD_ATTN_SPANS", str(spans))
    shape = synth.TINY if which == "tiny" else synth.ModelShape("h128x8t", 2, 512, 8, 2, 128, 1024, 4096,
                                                              rope_theta=1.0e4)
    L = 32768 - 9
    w = synth.WORKLOADS["tiny_chain"].with_model(shape, ctx=(L, L), gamma=8, ee_layer=1, kappa=4, seed=37)
    assert w.n_slots == 9
    case = H.GpuCase(w, capacity=32768)
    case.reset_len()
    gr = case.run()
    o = H.oracle_sequence(case.shape, w, case.si, 0)
    print("maximum capacity", which, spans, _compare(case, gr, {0: o}))
    assert int(case.cache.len[0]) <= 32768


def test_streaming_attention_is_deterministic(monkeypatch):
    """Two steps over the same inputs through the streaming attention kernel
    (forced, 3 spans a chunk, ragged contexts: direct writes and two-chunk
    merges, the lazily moved softmax reference) give bit-identical outputs."""
    _torch()
    monkeypatch.setenv("MSD_ATTN_SPANS", "3")
    w = synth.WORKLOADS["14b_batch16"].with_model(synth.TINY, batch=6, ctx=(1, 1000), ee_layer=1, kappa=4,
                                                  seed=27)
    case = H.GpuCase(w)
    case.reset_len()
    a = case.run(commit=False)
    case.reset_len()
    b = case.run(commit=False)
    assert np.array_equal(a.logits, b.logits)
    assert np.array_equal(a.ee_logp, b.ee_logp) and np.array_equal(a.ee_ids, b.ee_ids)
    for l in range(case.shape.n_layers):
        assert np.array_equal(a.k_rows[l], b.k_rows[l]) and np.array_equal(a.v_rows[l], b.v_rows[l])


def test_depth_reduced_66b_tree():
    """66B widths (MHA 72 heads, LayerNorm, learned positions, ReLU, biases, tied head), 2 layers."""
    _torch()
    w = synth.WORKLOADS["66b_tree"]
    case = H.GpuCase(w, n_layers=2)
    gr = case.run()
    o = H.oracle_sequence(case.shape, w, case.si, 0)
    rep = _compare(case, gr, {0: o})
    print("66b L2 tree:", rep)


def test_depth_reduced_66b_chain():
    """66B widths on a 9-slot chain (one row tile), 2 layers: the QKV (432
    tiles) and ReLU up (576 tiles) projections run whole-K 4-wave
    workgroups, the narrow ones 8-wave split-K workgroups, the tied head
    4-wave workgroups over 786 tiles (the last one partial)."""
    _torch()
    w = synth.WORKLOADS["66b_tree"].with_model(synth.OPT66B, topology="chain", gamma=8, branches=1, seed=41)
    assert w.n_slots == 9
    case = H.GpuCase(w, n_layers=2)
    gr = case.run()
    o = H.oracle_sequence(case.shape, w, case.si, 0)
    print("66b L2 chain:", _compare(case, gr, {0: o}))


def test_step_is_deterministic(tiny_case):
    case = tiny_case
    case.si = synth.step_inputs(case.w)
    case.reset_len()
    a = case.run()
    case.reset_len()
    b = case.run()
    assert np.array_equal(a.logits, b.logits)
    assert np.array_equal(a.ee_logp, b.ee_logp)
    assert np.array_equal(a.k_rows[0], b.k_rows[0])


def test_step_replays_under_graph_capture():
    """verify + accept (rejection, a 16-slot tree) captured in one HIP graph:
    neither allocates, clears memory with a memset or waits on the host, so
    every replay, each after an eager step on outputs of its own and with the
    graph's outputs poisoned, matches the eager step bit for bit."""
    torch = _torch()
    from paper_2510_13161_amd import msd
    w = synth.WORKLOADS["tiny_chain"].with_model(synth.TINY, ctx=(300, 300), topology="tree", gamma=5,
                                                 branches=3, ee_layer=1, kappa=4, seed=43,
                                                 mode="rejection")
    case = H.GpuCase(w)
    case.reset_len()
    si, dev = case.si, "cuda"
    B, n, V, M = w.batch, w.n_slots, case.shape.vocab, w.batch * w.n_slots
    # a temporary tokens tensor: the block keeps it alive (the allocations
    # below would otherwise reuse its memory)
    blk = msd.make_block(torch.from_numpy(si.tokens).to(dev), si.parent)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    cid, cq, ua, us = t(si.cand_ids), t(si.cand_q), t(si.u_accept), t(si.u_sample)
    smp = msd.Sampling(msd.MODES["rejection"], float(w.temperature), si.cand_ids.shape[-1],
                       cid.data_ptr(), cq.data_ptr(), ua.data_ptr(), us.data_ptr())
    nb = msd.workspace_bytes(case.model.handle, B, n, w.kappa, case.capacity)
    ws = torch.empty(nb, dtype=torch.uint8, device=dev)

    def outputs():
        e = lambda shape, dt: torch.empty(shape, dtype=dt, device=dev)
        return dict(logits=e((M, V), torch.float32), argmax=e(M, torch.int32), lse=e(M, torch.float32),
                    ids=e((M, w.kappa), torch.int32), logp=e((M, w.kappa), torch.float32),
                    acc=e(B, torch.int32), nxt=e(B, torch.int32), path=e((B, n), torch.int32))

    def step(o):
        req = msd.EERequest(w.ee_layer, w.kappa, o["ids"].data_ptr(), o["logp"].data_ptr(), None)
        msd.verify_block(case.model.handle, case.cache.c, blk, req, o["logits"], o["argmax"], o["lse"], ws)
        msd.accept(case.model.handle, blk, o["logits"], o["argmax"], smp, o["acc"], o["nxt"], o["path"],
                   case.cache.status)

    ref = outputs()
    step(ref)
    cap = outputs()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step(cap)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(cap)
    torch.cuda.synchronize()
    for r in range(3):
        for v in cap.values():
            v.fill_(-7)
        eager = outputs()
        step(eager)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k in ref:
            assert torch.equal(eager[k], ref[k]), ("eager", r, k)
            assert torch.equal(cap[k], ref[k]), ("replay", r, k)
    assert int(case.cache.status.item()) == 0
    gr = case.run(commit=False)  # the harness's own step, tokens held by the harness
    assert np.array_equal(gr.logits, ref["logits"].cpu().numpy())
    print("graph replays bit-identical; A =", ref["acc"].tolist())


# ---------------------------------------------------------------------------
# full-depth workloads (the shapes the benchmark times)
# ---------------------------------------------------------------------------
def _free(case):
    import torch
    del case
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


# Logit tolerance against the oracle without the bf16 cache reading (its
# block K/V kept at fp64). The kernels store the block's keys and values in
# the cache's bf16 format before attending to them (the cache is bf16), so
# against that plain reading the gap is the cache rounding propagated through
# every layer, not arithmetic error; the tests print the oracle's own
# bf16-vs-plain gap beside the GPU's to show it. Measured at full depth (GPU /
# oracle's own gap): 14B chain 5.22e-2 / 5.23e-2, 14B tree 3.54e-2 /
# 3.54e-2, 14B batch-16 longest sequence 1.10e-2 / 1.11e-2, 66B branch
# 5.9e-3 / 6.8e-3; against the bf16-cache reading the GPU is within 1e-3 on
# all of them. Bounds: about twice the largest measured gap per shape.
PLAIN_TOL = {"14b": 1.0e-1, "66b": 1.5e-2}


def _plain_gap(gr, rows, runs, b, bound, tag, gpu_rows=None):
    """Max |GPU - plain oracle| over the rows' logits, and the oracle's own
    bf16-cache vs plain gap on the same rows."""
    plain, cached = runs[(b, False)], runs[(b, True)]
    g = gr.logits[rows] if gpu_rows is None else gr.logits[gpu_rows]
    gap = float(np.abs(g - plain.logits).max())
    own = float(np.abs(cached.logits - plain.logits).max())
    print(f"{tag}: GPU vs plain oracle {gap:.3e} (bound {bound}); oracle bf16-cache vs plain {own:.3e}")
    assert gap <= bound, f"{tag}: GPU vs plain oracle {gap:.3e} > {bound}"
    return gap, own


@pytest.mark.slow
def test_full_14b_chain_greedy():
    """14B-shaped, 48 layers, gamma = 8 chain, ctx 1024, early exit kappa 8 at
    layer 36: against the bf16-cache oracle at 2e-2 and the plain oracle."""
    _torch()
    w = synth.WORKLOADS["14b_chain"]
    case = H.GpuCase(w)
    gr = case.run()
    runs = H.oracle_runs(case.shape, w, case.si, [(0, True), (0, False)])
    rep = _compare(case, gr, {0: runs[(0, True)]}, min_decisions=5)
    rep["plain"] = _plain_gap(gr, slice(0, w.n_slots), runs, 0, PLAIN_TOL["14b"], "14b chain")
    print("14b full chain:", rep)
    _free(case)


@pytest.mark.slow
def test_full_14b_tree_rejection():
    """Branch-complete tree (4 x 6), ctx 4096, rejection sampling at T = 1,
    against both oracle readings."""
    _torch()
    w = synth.WORKLOADS["14b_tree"]
    case = H.GpuCase(w)
    gr = case.run()
    runs = H.oracle_runs(case.shape, w, case.si, [(0, True), (0, False)])
    rep = _compare(case, gr, {0: runs[(0, True)]}, min_decisions=5)
    rep["plain"] = _plain_gap(gr, slice(0, w.n_slots), runs, 0, PLAIN_TOL["14b"], "14b tree")
    print("14b full tree:", rep)
    _free(case)


def test_depth_reduced_14b_batch16_every_sequence():
    """14B widths, 2 layers, the batch-16 block (M = 144, nine row tiles,
    contexts in [512, 8192]): every sequence element by element."""
    _torch()
    w = synth.WORKLOADS["14b_batch16"]
    case = H.GpuCase(w, n_layers=2)
    gr = case.run(ee=True)
    runs = H.oracle_runs(case.shape, w, case.si, [(b, True) for b in range(w.batch)])
    rep = _compare(case, gr, {b: runs[(b, True)] for b in range(w.batch)}, min_decisions=100)
    print("14b L2 batch16:", rep)
    _free(case)


@pytest.mark.slow
def test_full_14b_batch16_sampled_sequences():
    """16 sequences with contexts in [512, 8192] (M = 144), 48 layers: four
    sequences (the first, the shortest and longest contexts, one more) element
    by element; the longest also against the plain oracle; every sequence's
    commit and status are checked."""
    _torch()
    w = synth.WORKLOADS["14b_batch16"]
    case = H.GpuCase(w)
    gr = case.run(ee=True)
    lens = case.si.ctx_len
    picks = sorted({0, int(np.argmax(lens)), int(np.argmin(lens)), 9})
    longest = int(np.argmax(lens))
    runs = H.oracle_runs(case.shape, w, case.si, [(b, True) for b in picks] + [(longest, False)])
    rep = _compare(case, gr, {b: runs[(b, True)] for b in picks}, min_decisions=30)
    n = w.n_slots
    rep["plain"] = _plain_gap(gr, slice(longest * n, (longest + 1) * n), runs, longest, PLAIN_TOL["14b"],
                              "14b batch16 longest")
    print("14b batch16:", rep)
    # every sequence: the commit advanced len by 1 + A, paths are valid chains
    assert np.array_equal(gr.len_after, case.si.ctx_len + 1 + gr.acc_len)
    for b in range(w.batch):
        A = gr.acc_len[b]
        assert np.array_equal(gr.path[b][:A + 1], np.arange(A + 1))
    _free(case)


@pytest.mark.slow
def test_full_66b_tree():
    """66B-shaped, 64 layers (LayerNorm, learned positions, ReLU, biases, tied
    head), tree 4 x 8, ctx 2048: all 33 rows, the early-exit message, the
    acceptance walk and the K/V rows against the bf16-cache oracle; branch 0
    (a depth-r node holds the token at position t + r, so the branch scored as
    a chain gives the same rows) against the plain oracle."""
    _torch()
    w = synth.WORKLOADS["66b_tree"]
    case = H.GpuCase(w)
    gr = case.run(ee=True)
    runs = H.oracle_runs(case.shape, w, case.si, [(0, True)])
    rep = _compare(case, gr, {0: runs[(0, True)]}, min_decisions=20)
    branch = [0] + list(range(1, 1 + w.gamma))
    ci = H.chain_inputs(case.si, 0, branch)
    cw = w.with_model(w.model, topology="chain", branches=1)
    chain_runs = H.oracle_runs(case.shape, cw, ci, [(0, False), (0, True)], ee=False)
    rep["plain"] = _plain_gap(gr, None, chain_runs, 0, PLAIN_TOL["66b"], "66b branch 0", gpu_rows=branch)
    tree_vs_chain = float(np.abs(runs[(0, True)].logits[branch] - chain_runs[(0, True)].logits).max())
    assert tree_vs_chain < 1e-9, tree_vs_chain
    print("66b full tree:", rep)
    _free(case)
