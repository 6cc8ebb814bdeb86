"""The shared seeded input generator: determinism and its own two implementations."""
import numpy as np
import pytest

from paper_2510_13161_amd import synth


def test_host_generator_matches_numpy_reference():
    spec = synth.TensorSpec("l3.w_up", (37, 129), "normal", 0.02)
    a = synth.host_tensor(11, spec)
    b = synth.np_values(synth.tensor_key(11, spec.name), np.arange(37 * 129), 0.02)
    assert np.array_equal(a.reshape(-1), b)


def test_ctx_generator_matches_numpy_reference_and_is_layout_free():
    m = synth.TINY
    a = synth.host_ctx(m, 5, 1, "v", 2, 33)
    b = synth.np_ctx(m, 5, 1, "v", 2, 33)
    assert np.array_equal(a, b)
    # a longer fill reproduces the shorter one as a prefix
    c = synth.host_ctx(m, 5, 1, "v", 2, 50)
    assert np.array_equal(c[:, :33], a)


def test_generator_is_deterministic_and_seed_dependent():
    spec = synth.TensorSpec("embed", (64, 256), "normal", 0.02)
    assert np.array_equal(synth.host_tensor(0, spec), synth.host_tensor(0, spec))
    assert not np.array_equal(synth.host_tensor(0, spec), synth.host_tensor(1, spec))


def test_generator_moments():
    spec = synth.TensorSpec("x", (1 << 20,), "normal", 0.02)
    x = synth.bf16_bits_to_f32(synth.host_tensor(3, spec)).astype(np.float64)
    assert abs(x.mean()) < 1e-4
    assert abs(x.std() - 0.02) < 2e-4
    # Irwin-Hall(8): excess kurtosis -6/(5*8) = -0.15
    k = ((x - x.mean()) ** 4).mean() / x.var() ** 2 - 3.0
    assert abs(k + 0.15) < 0.02


def test_small_inputs_are_valid():
    w = synth.WORKLOADS["14b_tree"].with_model(synth.TINY)
    si = synth.step_inputs(w)
    par = si.parent
    assert par[0] == -1 and all(par[i] < i for i in range(1, len(par)))
    # children tokens lie in their parent's candidate set, siblings distinct
    for s in range(w.n_slots):
        kids = [c for c in range(w.n_slots) if par[c] == s]
        toks = [si.tokens[0, c] for c in kids]
        assert len(set(toks)) == len(toks)
        assert all(t in set(si.cand_ids[0, s].tolist()) for t in toks)
    assert np.all(si.cand_q > 0)
    assert np.all(np.abs(si.cand_q.sum(-1, dtype=np.float64) - 1) < 1e-6)
    assert np.all((si.u_accept >= 0) & (si.u_accept < 1))
    b = synth.WORKLOADS["14b_batch16"]
    lens = synth.ctx_lens(b)
    assert lens.shape == (16,) and lens.min() >= 512 and lens.max() <= 8192
    assert np.array_equal(lens, synth.ctx_lens(b))


def test_workload_shapes():
    W = synth.WORKLOADS
    assert W["14b_chain"].rows == 9 and W["14b_chain"].draft_tokens == 8
    assert W["14b_tree"].rows == 25 and W["14b_tree"].draft_tokens == 24
    assert W["14b_batch16"].rows == 144 and W["14b_batch16"].draft_tokens == 128
    assert W["66b_tree"].rows == 33
    # 14B-shaped weights: ~29.5 GB of bf16 with an untied head
    gb = synth.QWEN14B.weight_bytes() / 1e9
    assert 29.0 < gb < 30.0


def test_forest_topology_inputs():
    """An explicit parent array ("forest") is returned as given, bad ones are
    refused, and stochastic inputs follow it: each child's token lies in its
    parent's candidate set."""
    parents = (-1, 0, 0, 1, 3, 2, 0, 4)
    w = synth.WORKLOADS["tiny_chain"].with_model(synth.TINY, topology="forest", parents=parents, gamma=0,
                                                 mode="rejection", batch=2)
    assert w.n_slots == 8 and w.rows == 16
    assert synth.topology(w).tolist() == list(parents)
    si = synth.step_inputs(w)
    for b in range(2):
        for c in range(1, 8):
            assert si.tokens[b, c] in set(si.cand_ids[b, parents[c]].tolist())
    for bad in [(0, 0), (-1, 1), (-1, 0, 2), (-1, -1)]:
        wb = synth.WORKLOADS["tiny_chain"].with_model(synth.TINY, topology="forest", parents=bad, gamma=0)
        with pytest.raises(ValueError):
            synth.topology(wb)
