"""Pins of the fp64 oracle against what the paper and mathematics fix.

Each test checks the oracle against something other than itself: closed
forms of special weight settings (evaluated with torch/scipy library
routines), invariants of the method (block verification == token-by-token
decoding; a tree node == its root-to-node chain; RoPE relative-position
invariance), brute-force autoregressive decoding, and the sampling law of the
stochastic acceptance rules.
"""
import dataclasses

import numpy as np
import pytest
import scipy.special
import scipy.stats
import torch
import torch.nn.functional as F

import oracle as orc
from paper_2510_13161_amd import synth

TINY = synth.TINY
TINY1 = TINY.with_layers(1)
TINY_GQA = synth.ModelShape("tiny-gqa", 1, 256, 4, 2, 64, 1024, 4096)
TINY_OPT = synth.ModelShape("tiny-opt", 1, 256, 4, 4, 64, 1024, 4096, norm="layer", act="relu",
                            pos="learned", bias=True, tied_head=True, norm_eps=1e-5,
                            max_positions=256)


def b16(a):
    return synth.f32_to_bf16_bits(np.asarray(a, dtype=np.float32))


def f64(bits):
    return synth.bf16_bits_to_f32(bits).astype(np.float64)


def eye(rows, cols):
    return b16(np.eye(rows, cols, dtype=np.float32))


def zeros(rows, cols):
    return np.zeros((rows, cols), dtype=np.uint16)


def ctx_fn(m, seed, n_ctx):
    cache = {l: (synth.host_ctx(m, seed, l, "k", 0, n_ctx), synth.host_ctx(m, seed, l, "v", 0, n_ctx))
             for l in range(m.n_layers)}
    return lambda l: cache[l]


def rms(x, eps=1e-6):
    t = torch.from_numpy(np.asarray(x, dtype=np.float64))
    return F.rms_norm(t, (t.shape[-1],), eps=eps).numpy()


@pytest.fixture(scope="module")
def tiny():
    w = synth.host_weights(TINY, 0)
    return orc.Oracle(TINY, w), w


# ---------------------------------------------------------------------------
# closed forms of special weight settings
# ---------------------------------------------------------------------------
def test_head_closed_form_rmsnorm_and_lm_head():
    """Sec. 2: next-token logits = W h_t with h_t the final-normed residual.
    With W_o = W_down = 0 every block is the identity, so logits = W_LM rms(E[tok])."""
    w = synth.host_weights(TINY1, 1)
    w["l0.wo"] = zeros(256, 256)
    w["l0.w_down"] = zeros(256, 1024)
    o = orc.Oracle(TINY1, w, kv_cache_bf16=False)
    tok = np.array([3, 4000, 17])
    r = o.forward(tok, np.array([0, 1, 2]), np.array([-1, 0, 1]))
    e = f64(w["embed"])[tok]
    ref = rms(e) @ f64(w["lm_head"]).T
    assert np.allclose(r.x_final, e, rtol=0, atol=0)
    assert np.max(np.abs(r.logits - ref)) < 1e-12


def test_single_row_over_empty_cache_returns_its_value():
    """Softmax over a single key is 1: with W_v = W_o = I, x' = x + rms(x)."""
    w = synth.host_weights(TINY1, 2)
    w["l0.wv"] = eye(256, 256)
    w["l0.wo"] = eye(256, 256)
    w["l0.w_down"] = zeros(256, 1024)
    o = orc.Oracle(TINY1, w, kv_cache_bf16=False)
    r = o.forward(np.array([99]), np.array([7]), np.array([-1]))
    e = f64(w["embed"])[[99]]
    assert np.max(np.abs(r.x_final - (e + rms(e)))) < 1e-14


def test_block_keys_values_are_stored_in_the_cache_format():
    """With the cache-format reading the single row's value is the bf16
    rounding (nearest 8-bit significand, ties to even) of W_v h."""
    w = synth.host_weights(TINY1, 2)
    w["l0.wv"] = eye(256, 256)
    w["l0.wo"] = eye(256, 256)
    w["l0.w_down"] = zeros(256, 1024)
    o = orc.Oracle(TINY1, w, kv_cache_bf16=True)
    r = o.forward(np.array([99]), np.array([7]), np.array([-1]))
    e = f64(w["embed"])[[99]]
    want = e + f64(b16(rms(e)))
    # one bf16 ulp of slack for a float32 tie met on the way to bf16
    assert np.all(np.abs(r.x_final - want) <= 2.0 ** -8 * np.abs(rms(e)))
    assert np.array_equal(r.blk_v[0].reshape(-1), f64(b16(rms(e))).reshape(-1)) or \
        np.max(np.abs(r.blk_v[0].reshape(-1) - rms(e).reshape(-1))) <= 2.0 ** -8 * np.abs(rms(e)).max()


def test_uniform_attention_pins_tree_mask_and_gqa_grouping():
    """W_q = 0 makes every score 0, so each query averages exactly the values it
    may see: the cache plus its ancestors-or-self (Sec. 3.1 tree, a depth-r node
    sits at t + r); query head h reads kv head h // (H / H_kv)."""
    m = TINY_GQA
    w = synth.host_weights(m, 3)
    w["l0.wq"] = zeros(256, 256)
    w["l0.wv"] = eye(128, 256)
    w["l0.wo"] = eye(256, 256)
    w["l0.w_down"] = zeros(256, 1024)
    o = orc.Oracle(m, w, kv_cache_bf16=False)
    n_ctx = 5
    ctx = ctx_fn(m, 3, n_ctx)
    parent = np.array([-1, 0, 1, 0, 3])          # two branches of depth 2
    tok = np.array([1, 2, 3, 4, 5])
    pos = n_ctx + np.array([0, 1, 2, 1, 2])
    r = o.forward(tok, pos, parent, ctx, n_ctx)
    e = f64(w["embed"])[tok]
    v_blk = rms(e)[:, :128].reshape(5, 2, 64)
    v_ctx = f64(ctx(0)[1])                        # [2][n_ctx][64]
    anc = {0: [0], 1: [0, 1], 2: [0, 1, 2], 3: [0, 3], 4: [0, 3, 4]}
    for i in range(5):
        for h in range(4):
            kh = h // 2
            vals = list(v_ctx[kh]) + [v_blk[a, kh] for a in anc[i]]
            want = np.mean(vals, axis=0)
            got = r.x_final[i, h * 64:(h + 1) * 64] - e[i, h * 64:(h + 1) * 64]
            assert np.max(np.abs(got - want)) < 1e-13, (i, h)


def _rope_complex(u, pos, theta):
    """Rotary embedding as complex multiplication (Su et al. 2021): pairs
    (j, j + hd/2) form z_j = u_j + i u_{j+hd/2}, rotated by exp(i pos theta^(-2j/hd))."""
    hd = u.shape[-1]
    half = hd // 2
    j = np.arange(half)
    z = u[..., :half] + 1j * u[..., half:]
    z = z * np.exp(1j * pos[:, None] * theta ** (-2.0 * j / hd))
    return np.concatenate([z.real, z.imag], axis=-1)


def test_rotary_causal_attention_matches_library_sdpa():
    """Chain block over an empty cache with W_q = W_k = W_v = W_o = I: the layer's
    attention output equals torch's causal scaled-dot-product attention on
    complex-rotated q, k (scale 1/sqrt(hd))."""
    w = synth.host_weights(TINY1, 4)
    for n in ("wq", "wk", "wv", "wo"):
        w["l0." + n] = eye(256, 256)
    w["l0.w_down"] = zeros(256, 1024)
    o = orc.Oracle(TINY1, w, kv_cache_bf16=False)
    tok = np.array([10, 20, 30, 40])
    pos = np.array([5, 6, 7, 8])
    r = o.forward(tok, pos, np.array([-1, 0, 1, 2]))
    e = f64(w["embed"])[tok]
    h = rms(e).reshape(4, 4, 64)                  # [row][head][hd]
    qk = np.stack([_rope_complex(h[:, hh], pos.astype(np.float64), TINY.rope_theta)
                   for hh in range(4)])           # [head][row][hd]
    v = np.transpose(h, (1, 0, 2))
    att = F.scaled_dot_product_attention(torch.from_numpy(qk)[None], torch.from_numpy(qk)[None],
                                         torch.from_numpy(np.ascontiguousarray(v))[None],
                                         is_causal=True).numpy()[0]
    want = np.transpose(att, (1, 0, 2)).reshape(4, 256)
    assert np.max(np.abs((r.x_final - e) - want)) < 1e-12


def test_swiglu_closed_form():
    """FFN(h) = W_down (silu(W_gate h) * W_up h) with selecting weights gives
    x' = x + silu(h) h, h = rms(x)."""
    w = synth.host_weights(TINY1, 5)
    w["l0.wo"] = zeros(256, 256)
    w["l0.w_gate"] = eye(1024, 256)
    w["l0.w_up"] = eye(1024, 256)
    w["l0.w_down"] = eye(256, 1024)
    o = orc.Oracle(TINY1, w, kv_cache_bf16=False)
    r = o.forward(np.array([8, 9]), np.array([0, 1]), np.array([-1, 0]))
    e = f64(w["embed"])[[8, 9]]
    h = torch.from_numpy(rms(e))
    want = e + (F.silu(h) * h).numpy()
    assert np.max(np.abs(r.x_final - want)) < 1e-13


def test_layernorm_learned_positions_relu_biases_tied_head():
    """66B-style block (pre-LayerNorm, learned positions, ReLU FFN, biases, head
    tied to the embedding) against torch layer_norm/relu in a special setting."""
    m = TINY_OPT
    w = synth.host_weights(m, 6)
    g = np.random.default_rng(0)
    for n in ("l0.mlp_norm.g", "l0.mlp_norm.b", "final_norm.g", "final_norm.b"):
        w[n] = b16(g.normal(0.5, 0.3, 256))
    w["l0.wo"] = zeros(256, 256)
    w["l0.w_up"] = eye(1024, 256)
    w["l0.w_down"] = eye(256, 1024)
    o = orc.Oracle(m, w, kv_cache_bf16=False)
    tok, pos = np.array([5, 6, 7]), np.array([30, 31, 32])
    r = o.forward(tok, pos, np.array([-1, 0, 1]))
    x1 = f64(w["embed"])[tok] + f64(w["pos_embed"])[pos] + f64(w["l0.bo"])

    def ln(x, gn, bn):
        t = torch.from_numpy(x)
        return F.layer_norm(t, (256,), torch.from_numpy(f64(w[gn])), torch.from_numpy(f64(w[bn])),
                            eps=1e-5).numpy()

    hid = ln(x1, "l0.mlp_norm.g", "l0.mlp_norm.b")
    want = x1 + np.maximum(hid + f64(w["l0.b_up"])[:256], 0) + f64(w["l0.b_down"])
    assert np.max(np.abs(r.x_final - want)) < 1e-13
    logits = ln(r.x_final, "final_norm.g", "final_norm.b") @ f64(w["embed"]).T
    assert np.max(np.abs(r.logits - logits)) < 1e-12


def test_value_bias_closed_form():
    """Projection biases of the attention block (66B-style shape): with
    W_v = 0 every block value row is b_v, so over an empty cache each row's
    attention output is b_v whatever its scores; with W_o = I, W_down = 0
    the block gives x' = x + b_v + b_o + b_down."""
    m = TINY_OPT
    w = synth.host_weights(m, 7)
    g = np.random.default_rng(1)
    for n in ("l0.bv", "l0.bo", "l0.b_down"):
        w[n] = b16(g.normal(0.0, 1.0, 256))
    w["l0.wv"] = zeros(256, 256)
    w["l0.wo"] = eye(256, 256)
    w["l0.w_down"] = zeros(256, 1024)
    o = orc.Oracle(m, w, kv_cache_bf16=False)
    tok, pos = np.array([11, 12, 13, 14]), np.array([3, 4, 4, 5])
    r = o.forward(tok, pos, np.array([-1, 0, 0, 2]))
    want = (f64(w["embed"])[tok] + f64(w["pos_embed"])[pos] + f64(w["l0.bv"]) + f64(w["l0.bo"])
            + f64(w["l0.b_down"]))
    assert np.max(np.abs(r.x_final - want)) < 1e-12


@pytest.mark.parametrize("rotary", [False, True])
def test_query_key_bias_closed_form(rotary):
    """Query and key biases: with W_q = W_k = W_v = 0 a row's query is b_q and
    every block key b_k (rotated to the row's position when the model uses
    rotary positions, bias first); the scores against the cached keys and the
    visible block keys, softmax (scipy) and the value average (block values
    b_v) give the attention output exactly. A dropped or misplaced b_q or b_k
    changes every score."""
    m = TINY_OPT if not rotary else dataclasses.replace(TINY1, name="tiny-bias", bias=True)
    seed = 8
    w = synth.host_weights(m, seed)
    g = np.random.default_rng(2)
    for n in ("l0.bq", "l0.bk", "l0.bv"):
        w[n] = b16(g.normal(0.0, 1.0, 256))
    for n in ("l0.wq", "l0.wk", "l0.wv"):
        w[n] = zeros(256, 256)
    w["l0.wo"] = eye(256, 256)
    w["l0.w_down"] = zeros(256, 1024)
    if m.bias:
        w["l0.bo"] = np.zeros(256, np.uint16)
        w["l0.b_down"] = np.zeros(256, np.uint16)
    o = orc.Oracle(m, w, kv_cache_bf16=False)
    n_ctx = 6
    ctx = ctx_fn(m, seed, n_ctx)
    parent = np.array([-1, 0, 1, 0])
    tok = np.array([21, 22, 23, 24])
    pos = n_ctx + orc.depths(parent)
    r = o.forward(tok, pos, parent, ctx, n_ctx)
    hd, H = m.head_dim, m.n_heads
    bq = f64(w["l0.bq"]).reshape(H, hd)
    bk = f64(w["l0.bk"]).reshape(H, hd)
    bv = f64(w["l0.bv"]).reshape(H, hd)
    kc, vc = (f64(a) for a in ctx(0))            # [H][n_ctx][hd]
    anc = {0: [0], 1: [0, 1], 2: [0, 1, 2], 3: [0, 3]}
    e = f64(w["embed"])[tok]
    if m.pos == "learned":
        e = e + f64(w["pos_embed"])[pos]
    for i in range(4):
        for h in range(H):
            q = bq[h][None]
            kb = np.repeat(bk[h][None], 4, 0)
            if rotary:
                q = _rope_complex(q, np.array([pos[i]], np.float64), m.rope_theta)
                kb = _rope_complex(kb, pos.astype(np.float64), m.rope_theta)
            keys = np.concatenate([kc[h, :n_ctx], kb[anc[i]]])
            vals = np.concatenate([vc[h, :n_ctx], np.repeat(bv[h][None], len(anc[i]), 0)])
            p = scipy.special.softmax(keys @ q[0] / np.sqrt(hd))
            got = r.x_final[i, h * hd:(h + 1) * hd] - e[i, h * hd:(h + 1) * hd]
            assert np.max(np.abs(got - p @ vals)) < 1e-12, (i, h)


# ---------------------------------------------------------------------------
# invariants of the method
# ---------------------------------------------------------------------------
def test_block_verification_equals_token_by_token_forward(tiny):
    """Sec. 2: the verifier's one pass over the window is the teacher-forced
    roll-forward; each row must equal the sequential one-token forward, bitwise."""
    o, _ = tiny
    n_ctx = 16
    ctx = ctx_fn(TINY, 0, n_ctx)
    tok = np.array([5, 77, 901, 4095, 0, 1234])
    pos = n_ctx + np.arange(6)
    blk = o.forward(tok, pos, np.arange(-1, 5), ctx, n_ctx)
    ek = [[] for _ in range(TINY.n_layers)]
    ev = [[] for _ in range(TINY.n_layers)]
    for s in range(6):
        extra = None if s == 0 else [(np.concatenate(ek[l]), np.concatenate(ev[l]))
                                     for l in range(TINY.n_layers)]
        one = o.forward(tok[s:s + 1], pos[s:s + 1], np.array([-1]), ctx, n_ctx, extra)
        assert np.array_equal(one.logits[0], blk.logits[s])
        for l in range(TINY.n_layers):
            assert np.array_equal(one.blk_k[l][0], blk.blk_k[l][s])
            ek[l].append(one.blk_k[l])
            ev[l].append(one.blk_v[l])


def test_tree_node_equals_its_root_to_node_chain(tiny):
    """Sec. 3.1: a node at depth r of the hypothesis tree holds the token at
    position t + r; scoring the tree under its mask equals scoring each
    root-to-node path as a chain, bitwise."""
    o, _ = tiny
    n_ctx = 9
    ctx = ctx_fn(TINY, 0, n_ctx)
    w = synth.Workload("t", TINY, 1, (n_ctx, n_ctx), "tree", 3, branches=3)
    parent = synth.topology(w)
    tok = np.random.default_rng(1).integers(0, TINY.vocab, w.n_slots)
    depth = orc.depths(parent)
    tree = o.forward(tok, n_ctx + depth, parent, ctx, n_ctx)
    for i in range(w.n_slots):
        path = []
        a = i
        while a >= 0:
            path.append(a)
            a = parent[a]
        path = path[::-1]
        chain = o.forward(tok[path], n_ctx + np.arange(len(path)), np.arange(-1, len(path) - 1),
                          ctx, n_ctx)
        assert np.array_equal(chain.logits[-1], tree.logits[i]), i


def test_rope_relative_position_invariance(tiny):
    """Rotary positions encode offsets only: shifting a block over an empty cache
    leaves its logits unchanged up to fp64 rounding (keys kept at fp64: bf16
    storage of a rotated key depends on its absolute angle)."""
    o = orc.Oracle(TINY, tiny[1], kv_cache_bf16=False)
    tok = np.array([11, 22, 33, 44, 55])
    par = np.arange(-1, 4)
    a = o.forward(tok, np.arange(5), par)
    b = o.forward(tok, 1000 + np.arange(5), par)
    assert np.max(np.abs(a.logits - b.logits)) < 1e-9
    c = o.forward(tok, np.array([0, 1, 2, 3, 5]), par)   # broken offset changes them
    assert np.max(np.abs(a.logits[-1] - c.logits[-1])) > 1e-6


def test_rope_at_position_zero_is_the_identity(tiny):
    o, w = tiny
    shape = dataclasses.replace(TINY, pos="learned", max_positions=4)
    w2 = dict(w)
    w2["pos_embed"] = np.zeros((4, 256), dtype=np.uint16)
    o2 = orc.Oracle(shape, w2)
    a = o.forward(np.array([123]), np.array([0]), np.array([-1]))
    b = o2.forward(np.array([123]), np.array([0]), np.array([-1]))
    assert np.array_equal(a.logits, b.logits)


# ---------------------------------------------------------------------------
# early-exit top-kappa
# ---------------------------------------------------------------------------
def test_topk_equals_full_sort_and_logsumexp():
    g = np.random.default_rng(2)
    z = np.round(g.normal(0, 2, (6, 500)), 1)        # many exact ties
    ids, logp, lse = orc.Oracle.topk(z, 8)
    for i in range(6):
        order = np.lexsort((np.arange(500), -z[i]))    # logit desc, then id asc
        assert np.array_equal(ids[i], order[:8])
        l = scipy.special.logsumexp(z[i])
        assert abs(lse[i] - l) < 1e-12
        assert np.max(np.abs(logp[i] - (z[i, order[:8]] - l))) < 1e-12


def test_early_exit_applies_head_to_intermediate_residual(tiny):
    """Sec. 3.1: p^(l_e) = Softmax(W_LM h^(l_e)) with the final norm (reading:
    the same head the last layer uses); equals the last-layer head of a model
    truncated after l_e layers."""
    o, w = tiny
    tok, pos, par = np.array([1, 2, 3]), np.array([0, 1, 2]), np.array([-1, 0, 1])
    r = o.forward(tok, pos, par, ee_layer=1)
    ids, logp, _ = o.early_exit(r.x_ee, 4)
    trunc = orc.Oracle(TINY1, w).forward(tok, pos, par)
    ids2, logp2, _ = orc.Oracle.topk(trunc.logits, 4)
    assert np.array_equal(ids, ids2) and np.array_equal(logp, logp2)


# ---------------------------------------------------------------------------
# acceptance
# ---------------------------------------------------------------------------
def test_greedy_acceptance_equals_autoregressive_decoding(tiny):
    """Sec. 2 / App. B: A_t is the longest prefix of the window equal to the
    target's argmax tokens; the next token is the target's token after it."""
    o, _ = tiny
    n_ctx = 16
    ctx = ctx_fn(TINY, 0, n_ctx)
    root = 321
    y, _ = o.decode_greedy(root, n_ctx, 5, ctx, n_ctx)
    gamma = 4
    par = np.arange(-1, gamma)
    for mism in range(1, gamma + 2):            # gamma + 1: no mismatch
        drafts = y[:gamma].copy()
        if mism <= gamma:
            drafts[mism - 1] = (drafts[mism - 1] + 1) % TINY.vocab
        tok = np.concatenate([[root], drafts])
        r = o.forward(tok, n_ctx + np.arange(gamma + 1), par, ctx, n_ctx)
        A, nxt, path = o.accept(par, tok, r.logits)
        want_A = min(mism - 1, gamma)
        assert A == want_A
        assert nxt == y[want_A]
        assert np.array_equal(path, np.arange(want_A + 1))


def test_greedy_acceptance_on_a_tree_takes_the_matching_branch(tiny):
    o, _ = tiny
    n_ctx = 16
    ctx = ctx_fn(TINY, 0, n_ctx)
    root = 77
    y, _ = o.decode_greedy(root, n_ctx, 4, ctx, n_ctx)
    w = synth.Workload("t", TINY, 1, (n_ctx, n_ctx), "tree", 3, branches=3)
    par = synth.topology(w)
    tok = np.random.default_rng(3).integers(0, TINY.vocab, w.n_slots)
    tok[0] = root
    # branch 2 (slots 7, 8, 9) follows the target for two steps, then deviates
    tok[7], tok[8], tok[9] = y[0], y[1], (y[2] + 5) % TINY.vocab
    for s in (1, 4):                              # other branches must not start with y[0]
        if tok[s] == y[0]:
            tok[s] = (tok[s] + 1) % TINY.vocab
    r = o.forward(tok, n_ctx + orc.depths(par), par, ctx, n_ctx)
    A, nxt, path = o.accept(par, tok, r.logits)
    assert (A, nxt) == (2, y[2])
    assert np.array_equal(path, [0, 7, 8])


def test_greedy_ties_go_to_the_smaller_id():
    z = np.zeros((2, 10))
    z[0, 3] = z[0, 7] = 5.0
    A, nxt, _ = orc.Oracle.accept(np.array([-1, 0]), np.array([0, 7]), z)
    assert (A, nxt) == (0, 3)


def test_near_tie_bands_closed_forms():
    """Near-tie bands of the acceptance decisions, each on a hand-computed case
    (tol 0.02). Argmax: top-1 minus top-2 of 0.03 lies in the 2 tol band, 0.05
    does not. Inverse CDF on p = (0.7, 0.3): id 0's bin is [0, 0.7], so
    u = 0.69 lies within 4 tol min(c, 1 - c) = 0.024 of its upper edge, u =
    0.5 does not. Accept test with p(x) = 0.3, q(x) = 0.6 (alpha = 0.5): u =
    0.51 lies within 2 tol alpha / T = 0.02, u = 0.9 does not."""
    tol = 0.02
    par2 = np.array([-1, 0])
    # greedy: the flag sits at the depth of the row, and covers the next token
    for gap, flagged in ((0.03, True), (0.05, False)):
        z = np.zeros((2, 6))
        z[0, 2] = 1.0
        z[1, 4] = 1.0
        z[1, 1] = 1.0 - gap
        A, nxt, path, td, tn = orc.Oracle.accept(par2, np.array([9, 2]), z, tol_logit=tol, return_tie=True)
        assert (A, nxt, list(path)) == (1, 4, [0, 1])
        assert (td, tn) == ((1, True) if flagged else (-1, False))
    # MATCH draw on (0.7, 0.3): id 0 drawn, no child carries it
    zr = np.log(np.array([[0.7, 0.3], [0.5, 0.5]]))
    for u, flagged in ((0.69, True), (0.5, False)):
        A, nxt, _, td, tn = orc.Oracle.accept(par2, np.array([0, 1]), zr, "match", 1.0,
                                              u_sample=np.array([u, 0.5], np.float32),
                                              tol_logit=tol, return_tie=True)
        assert (A, nxt) == (0, 0)
        assert (td, tn) == ((0, True) if flagged else (-1, False))
    # REJECTION accept test of child x = 1: p(1) = 0.3, q(1) = 0.6, alpha = 0.5
    cid = np.array([[1, 0], [1, 0]], np.int32)
    cq = np.array([[0.6, 0.4], [0.6, 0.4]], np.float32)
    for u, flagged, acc in ((0.51, True, 0), (0.49, True, 1), (0.9, False, 0)):
        A, nxt, _, td, tn = orc.Oracle.accept(par2, np.array([0, 1]), zr, "rejection", 1.0, cid, cq,
                                              np.array([0.0, u], np.float32),
                                              np.array([0.5, 0.5], np.float32),
                                              tol_logit=tol, return_tie=True)
        assert A == acc
        assert td == (0 if flagged else -1)
        if acc == 0:
            # rejected: r = normalise((p - q)^+) = (1, 0), so id 0 whatever u
            assert nxt == 0
    # no tolerance: nothing is flagged, not even an exact tie (the smaller id wins)
    z = np.zeros((2, 6))
    z[0, 2] = z[0, 3] = 1.0
    assert orc.Oracle.accept(par2, np.array([9, 2]), z, tol_logit=0.0, return_tie=True)[3:] == (-1, False)
    assert orc.Oracle.accept(par2, np.array([9, 2]), z, tol_logit=1e-9, return_tie=True)[3:] == (0, True)


def _first_token_law(p_root, q, cands, n_children, mode, n_samples, seed, V):
    """Empirical law of the first committed token: the accepted child's token,
    else the next token. Children are drawn from q without replacement."""
    g = np.random.default_rng(seed)
    n = 1 + n_children
    parent = np.array([-1] + [0] * n_children)
    C = len(cands)
    cand_ids = np.tile(cands, (n, 1)).astype(np.int32)
    cand_q = np.tile(q, (n, 1)).astype(np.float32)
    logits = np.tile(np.log(p_root), (n, 1))
    counts = np.zeros(V)
    acc = 0
    qd = q.astype(np.float64) / q.sum(dtype=np.float64)
    for _ in range(n_samples):
        pick = g.choice(C, size=n_children, replace=False, p=qd)
        tok = np.concatenate([[0], cands[pick]]).astype(np.int32)
        ua = synth.uniforms01(g, n)
        us = synth.uniforms01(g, n)
        A, nxt, path = orc.Oracle.accept(parent, tok, logits, mode, 1.0, cand_ids, cand_q, ua, us)
        first = tok[path[1]] if A >= 1 else nxt
        counts[first] += 1
        acc += A >= 1
    return counts, acc / n_samples


@pytest.mark.parametrize("n_children", [1, 2, 3])
def test_rejection_sampling_reproduces_the_target_law(n_children):
    """Lossless stochastic verification (Leviathan et al. 2023, Thm. 1; several
    children drawn without replacement: recursive rejection, Jeon et al. 2024):
    the first committed token is distributed as p = Softmax(z / T)."""
    V = 10
    g = np.random.default_rng(10 + n_children)
    p = g.dirichlet(np.ones(V))
    cands = np.array([1, 4, 5, 8])
    q = synth.dirichlet_rows(g, 0.5, (len(cands),))
    N = 30000
    counts, acc = _first_token_law(p, q, cands, n_children, "rejection", N, 99, V)
    chi = scipy.stats.chisquare(counts, p * N)
    assert chi.pvalue > 1e-4, (counts / N, p)
    if n_children == 1:
        # acceptance probability of a single draft: sum_x min(p(x), q(x))
        closed = sum(min(p[c], float(qq)) for c, qq in zip(cands, q))
        assert abs(acc - closed) < 4 * np.sqrt(closed * (1 - closed) / N)


def _threshold(decide, lo=0.0, hi=1.0, iters=32):
    """The point t in [lo, hi] where a monotone yes-below / no-above decision
    of the oracle flips (decide(u) is True for u < t). The uniforms are fp32
    inputs, so t is resolved to their spacing (2^-24 near 1)."""
    if not decide(lo):
        return lo
    if decide(hi):
        return hi
    for _ in range(iters):
        mid = 0.5 * (lo + hi)
        if decide(mid):
            lo = mid
        else:
            hi = mid
    return 0.5 * (lo + hi)


def _bins(draw, V, lo=0.0, hi=1.0 - 2.0 ** -24, iters=32):
    """Measure of {u in [0, 1): draw(u) = y} for every y, for a nondecreasing
    step function draw (inverse-CDF sampling over ascending ids), by
    bisection for its breakpoints."""
    mass = np.zeros(V)

    def rec(a, b, ya, yb):
        if ya == yb:
            mass[ya] += b - a
            return
        if b - a < 2.0 ** -iters:
            mass[ya] += (b - a) / 2
            mass[yb] += (b - a) / 2
            return
        m = 0.5 * (a + b)
        ym = draw(m)
        rec(a, m, ya, ym)
        rec(m, b, ym, yb)

    rec(lo, hi, draw(lo), draw(hi))
    mass[draw(hi)] += 1.0 - hi
    return mass


@pytest.mark.parametrize("n_children", [1, 2, 3])
def test_rejection_output_law_exact_enumeration(n_children):
    """Losslessness of REJECTION by exact enumeration (Leviathan et al. 2023,
    Thm. 1; several children drawn without replacement: recursive rejection,
    Jeon et al. 2024), with the oracle as a black box: every ordered draw of
    the children from q is enumerated with its probability; each accept
    test's outcome is a threshold in its uniform, found by bisection on the
    oracle's decision; the final draw's bins in u_sample likewise. The law of
    the first committed token must equal p = Softmax(z) to 1e-6 (the
    uniforms are fp32: each threshold is resolved to 2^-24)."""
    import itertools
    V = 10
    g = np.random.default_rng(40 + n_children)
    p = g.dirichlet(np.ones(V))
    cands = np.array([1, 4, 5, 8])
    q = synth.dirichlet_rows(g, 0.5, (len(cands),))
    qd = q.astype(np.float64)
    n = 1 + n_children
    parent = np.array([-1] + [0] * n_children)
    cand_ids = np.tile(cands, (n, 1)).astype(np.int32)
    cand_q = np.tile(q, (n, 1)).astype(np.float32)
    logits = np.tile(np.log(p), (n, 1))
    law = np.zeros(V)
    for order in itertools.permutations(range(len(cands)), n_children):
        w, left = 1.0, 1.0
        for j in order:
            w *= qd[j] / left
            left -= qd[j]
        tok = np.concatenate([[0], cands[list(order)]]).astype(np.int32)
        u_acc = np.full(n, 0.5, np.float32)

        def run(ua, us0=0.5):
            us = np.full(n, us0, np.float32)
            return orc.Oracle.accept(parent, tok, logits, "rejection", 1.0, cand_ids, cand_q,
                                     ua.astype(np.float32), us)

        reach = w                                   # probability of testing child c
        for c in range(1, n):
            def accepted(u, c=c):
                ua = u_acc.copy()
                ua[c] = u
                A, _, path = run(ua)
                return A >= 1 and path[1] == c
            alpha = _threshold(accepted)
            law[tok[c]] += reach * alpha
            reach *= 1.0 - alpha
            u_acc[c] = np.float32(min(alpha + (1.0 - alpha) / 2, 1.0 - 2.0 ** -24))
        if reach > 0:                               # every child rejected: the residual draw
            law += reach * _bins(lambda u: run(u_acc, u)[1], V)
    assert abs(law.sum() - 1.0) < 1e-6
    assert np.max(np.abs(law - p)) < 1e-6, (law, p)


def test_match_output_law_exact_enumeration():
    """MATCH (the paper's sample-and-compare): the first committed token is
    the draw y = Sample(p, u); its bins in u, found by bisection on the
    oracle, have the masses p exactly."""
    V = 10
    p = np.random.default_rng(50).dirichlet(np.ones(V))
    parent = np.array([-1, 0, 0])
    tok = np.array([0, 3, 7], np.int32)
    logits = np.tile(np.log(p), (3, 1))

    def first(u):
        A, nxt, path = orc.Oracle.accept(parent, tok, logits, "match", 1.0,
                                         u_sample=np.array([u, 0.5, 0.5], np.float32))
        return int(tok[path[1]]) if A >= 1 else nxt

    law = _bins(first, V)
    assert np.max(np.abs(law - p)) < 1e-6


def test_match_rule_reproduces_the_target_law():
    """The paper's sample-and-compare operator: y ~ p, matched against the draft."""
    V = 10
    g = np.random.default_rng(21)
    p = g.dirichlet(np.ones(V))
    cands = np.array([0, 2, 3, 9])
    q = synth.dirichlet_rows(g, 0.5, (4,))
    N = 20000
    counts, _ = _first_token_law(p, q, cands, 2, "match", N, 5, V)
    assert scipy.stats.chisquare(counts, p * N).pvalue > 1e-4


def test_rejection_flags_a_child_outside_the_candidate_set():
    z = np.zeros((2, 8))
    with pytest.raises(ValueError):
        orc.Oracle.accept(np.array([-1, 0]), np.array([0, 6]), z, "rejection", 1.0,
                          np.array([[1, 2], [1, 2]]), np.array([[0.5, 0.5], [0.5, 0.5]],
                                                               dtype=np.float32),
                          np.zeros(2, np.float32), np.zeros(2, np.float32))


# ---------------------------------------------------------------------------
# commit
# ---------------------------------------------------------------------------
def test_kv_commit_equals_a_fresh_forward_of_the_accepted_path(tiny):
    """After committing the accepted root-to-node path, the cache rows equal those
    a plain chain forward of the committed tokens writes."""
    o, _ = tiny
    L, Hk, hd = TINY.n_layers, TINY.n_kv_heads, TINY.head_dim
    n_ctx, cap = 16, 40
    kc = np.zeros((L, Hk, cap, hd), np.uint16)
    vc = np.zeros_like(kc)
    for l in range(L):
        kc[l, :, :n_ctx] = synth.host_ctx(TINY, 0, l, "k", 0, n_ctx)
        vc[l, :, :n_ctx] = synth.host_ctx(TINY, 0, l, "v", 0, n_ctx)
    ctx = lambda l: (kc[l], vc[l])
    root = 5
    y, _ = o.decode_greedy(root, n_ctx, 3, ctx, n_ctx)
    w = synth.Workload("t", TINY, 1, (n_ctx, n_ctx), "tree", 3, branches=2)
    par = synth.topology(w)
    tok = np.array([root, (y[0] + 1) % TINY.vocab, 1, 2, y[0], y[1], (y[2] + 1) % TINY.vocab])
    r = o.forward(tok, n_ctx + orc.depths(par), par, ctx, n_ctx)
    for l in range(L):                 # verify writes every block row after the context
        kc[l, :, n_ctx:n_ctx + 7] = b16(np.transpose(r.blk_k[l], (1, 0, 2)))
        vc[l, :, n_ctx:n_ctx + 7] = b16(np.transpose(r.blk_v[l], (1, 0, 2)))
    A, nxt, path = o.accept(par, tok, r.logits)
    assert A == 2 and list(path) == [0, 4, 5]
    new_len = o.kv_commit(kc, vc, n_ctx, A, path)
    assert new_len == n_ctx + 1 + A
    fresh = o.forward(np.array([root, y[0], y[1]]), n_ctx + np.arange(3), np.array([-1, 0, 1]),
                      ctx, n_ctx)
    for l in range(L):
        assert np.array_equal(kc[l, :, n_ctx:new_len], b16(np.transpose(fresh.blk_k[l], (1, 0, 2))))
        assert np.array_equal(vc[l, :, n_ctx:new_len], b16(np.transpose(fresh.blk_v[l], (1, 0, 2))))
