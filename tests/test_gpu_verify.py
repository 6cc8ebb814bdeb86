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


def _compare(case, gr, seqs, check_ee=True, tol=H.TOL_LOGIT):
    """Element-wise comparison of one GPU step with the oracle's sequences."""
    w, si = case.w, case.si
    n, V = w.n_slots, case.shape.vocab
    report = {"max_abs": 0.0, "flagged_rows": 0, "flagged_seqs": 0}
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
        assert np.array_equal(gr.argmax[rows][~tie], top1[~tie]), f"seq {b}: argmax differs"
        if check_ee and o.ee_ids is not None:
            # rows whose kappa+1 best early-exit logits are closer than the margin are flagged
            firm = o.ee_margin >= H.TIE_MARGIN
            report["ee_flagged_rows"] = report.get("ee_flagged_rows", 0) + int((~firm).sum())
            assert np.array_equal(gr.ee_ids[rows][firm], o.ee_ids[firm]), f"seq {b}: early-exit ids"
            same = np.all(gr.ee_ids[rows] == o.ee_ids, axis=-1)
            err = np.abs(gr.ee_logp[rows] - o.ee_logp)[same]
            assert err.max(initial=0.0) <= tol, f"seq {b}: early-exit logp {err.max():.3e}"
        # decisions: exact unless the oracle's walk passed a flagged node
        visited_tie = any(tie[s] for s in o.path)
        if visited_tie and w.mode == "greedy":
            report["flagged_seqs"] += 1
            continue
        assert gr.acc_len[b] == o.acc, f"seq {b}: accepted length {gr.acc_len[b]} != {o.acc}"
        assert gr.next_tok[b] == o.nxt, f"seq {b}: next token {gr.next_tok[b]} != {o.nxt}"
        assert np.array_equal(gr.path[b][:o.acc + 1], o.path)
        assert np.all(gr.path[b][o.acc + 1:] == -1)
        assert gr.len_after[b] == si.ctx_len[b] + 1 + o.acc
        # K/V rows the verify pass wrote at len + slot
        for l in range(case.shape.n_layers):
            kg = synth.bf16_bits_to_f32(gr.k_rows[l][b]).astype(np.float64)   # [Hkv][n][hd]
            vg = synth.bf16_bits_to_f32(gr.v_rows[l][b]).astype(np.float64)
            ko = np.transpose(o.blk_k[l], (1, 0, 2))
            vo = np.transpose(o.blk_v[l], (1, 0, 2))
            scale = max(1.0, float(np.abs(ko).max()))
            assert np.max(np.abs(kg - ko)) <= tol * scale, f"layer {l} k rows"
            assert np.max(np.abs(vg - vo)) <= tol * max(1.0, float(np.abs(vo).max())), f"layer {l} v rows"
    assert gr.status == 0
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


def test_tiny_planted_acceptance(tiny_case):
    """Drafts equal to the oracle's greedy continuation up to a planted mismatch:
    the GPU accepts exactly the prefix token-by-token argmax decoding gives."""
    import oracle as orc
    case = tiny_case
    w = case.w
    o = orc.Oracle(case.shape, synth.host_weights(case.shape, w.seed))
    L = int(case.si.ctx_len[0])
    ctx = lambda l: (synth.host_ctx(case.shape, w.seed, l, "k", 0, L),
                     synth.host_ctx(case.shape, w.seed, l, "v", 0, L))
    root = int(case.si.tokens[0, 0])
    y, zs = o.decode_greedy(root, L, w.gamma + 1, ctx, L)
    for mism in range(1, w.gamma + 2):
        drafts = y[:w.gamma].copy()
        if mism <= w.gamma:
            drafts[mism - 1] = (drafts[mism - 1] + 1) % case.shape.vocab
        si = synth.StepInputs(parent=case.si.parent, tokens=np.concatenate([[root], drafts])[None].astype(np.int32),
                              ctx_len=case.si.ctx_len)
        case.si = si
        case.reset_len()
        gr = case.run(ee=False)
        want = min(mism - 1, w.gamma)
        margin = np.min([np.sort(z)[-1] - np.sort(z)[-2] for z in zs[:want + 1]])
        if margin < H.TIE_MARGIN:
            continue
        assert gr.acc_len[0] == want
        assert gr.next_tok[0] == y[want]
        assert gr.len_after[0] == L + 1 + want


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


def test_tiny_reuse_selection_and_fallback_statistics():
    """Sec. 3.1 reuse criterion and next-window selection with the App. C
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


def test_depth_reduced_14b_chain():
    """14B widths (d 5120, GQA 40/8, FFN 13824, vocab 152064) with 2 layers."""
    _torch()
    w = synth.WORKLOADS["14b_chain"].with_model(synth.QWEN14B)
    case = H.GpuCase(w, n_layers=2)
    gr = case.run()
    o = H.oracle_sequence(case.shape, w, case.si, 0)
    rep = _compare(case, gr, {0: o})
    print("14b L2 chain:", rep)


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
    w = synth.WORKLOADS["14b_chain"].with_model(synth.QWEN14B)
    case = H.GpuCase(w, n_layers=2)
    gr = case.run()
    o = H.oracle_sequence(case.shape, w, case.si, 0)
    print("streaming 14b L2 chain:", _compare(case, gr, {0: o}))


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


@pytest.mark.slow
def test_full_14b_chain_greedy():
    """14B-shaped, 48 layers, gamma = 8 chain, ctx 1024, early exit kappa 8 at layer 36."""
    _torch()
    w = synth.WORKLOADS["14b_chain"]
    case = H.GpuCase(w)
    gr = case.run()
    o = H.oracle_sequence(case.shape, w, case.si, 0, oracle_obj=H.streaming_oracle(case.shape, w.seed))
    rep = _compare(case, gr, {0: o})
    print("14b full chain:", rep)
    _free(case)


@pytest.mark.slow
def test_full_14b_tree_rejection():
    """Branch-complete tree (4 x 6), ctx 4096, rejection sampling at T = 1."""
    _torch()
    w = synth.WORKLOADS["14b_tree"]
    case = H.GpuCase(w)
    gr = case.run()
    o = H.oracle_sequence(case.shape, w, case.si, 0, oracle_obj=H.streaming_oracle(case.shape, w.seed))
    rep = _compare(case, gr, {0: o})
    print("14b full tree:", rep)
    _free(case)


@pytest.mark.slow
def test_full_14b_batch16_sampled_sequences():
    """16 sequences with contexts in [512, 8192] (M = 144): sequences 0 and the
    longest are recomputed by the oracle one by one; every sequence's commit
    and status are checked."""
    _torch()
    w = synth.WORKLOADS["14b_batch16"]
    case = H.GpuCase(w)
    gr = case.run(ee=True)
    orc_obj = H.streaming_oracle(case.shape, w.seed)
    picks = sorted({0, int(np.argmax(case.si.ctx_len))})
    seqs = {b: H.oracle_sequence(case.shape, w, case.si, b, oracle_obj=orc_obj) for b in picks}
    rep = _compare(case, gr, seqs)
    print("14b batch16:", rep)
    # every sequence: the commit advanced len by 1 + A, paths are valid chains
    assert np.array_equal(gr.len_after, case.si.ctx_len + 1 + gr.acc_len)
    for b in range(w.batch):
        A = gr.acc_len[b]
        assert np.array_equal(gr.path[b][:A + 1], np.arange(A + 1))
    _free(case)


@pytest.mark.slow
def test_full_66b_tree_branch():
    """66B-shaped, 64 layers (LayerNorm, learned positions, ReLU, biases, tied
    head), tree 4 x 8, ctx 2048. The oracle scores branch 0 as a chain: a
    depth-r node holds the token at position t + r (tree node == its chain)."""
    _torch()
    w = synth.WORKLOADS["66b_tree"]
    case = H.GpuCase(w)
    gr = case.run(ee=True)
    branch = [0] + list(range(1, 1 + w.gamma))
    ci = H.chain_inputs(case.si, 0, branch)
    cw = w.with_model(w.model, topology="chain", branches=1)
    o = H.oracle_sequence(case.shape, cw, ci, 0, oracle_obj=H.streaming_oracle(case.shape, w.seed))
    err = np.abs(gr.logits[branch] - o.logits).max()
    print("66b full branch: max abs", err)
    assert err <= H.TOL_LOGIT
    tie = H.margins(o.logits, 1) < H.TIE_MARGIN
    assert np.array_equal(gr.argmax[branch][~tie], np.argmax(o.logits, -1)[~tie])
    firm = o.ee_margin >= H.TIE_MARGIN
    assert np.array_equal(gr.ee_ids[branch][firm], o.ee_ids[firm])
    assert gr.status == 0
    _free(case)
