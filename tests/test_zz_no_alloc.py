"""msd_verify_block_static (no workspace: the library's static scratch)
against msd_verify_block with a caller workspace, through the C ABI.

Both run the same kernels, so every output (logits, argmax, lse, the
early-exit message, the block's K/V rows) must be bit-identical. Two calls in
a row on the static scratch, the second with a smaller block, check that what
one call leaves in the scratch does not reach the next.
"""
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


def _verify(case, static: bool):
    """One verify pass of the case's block (no accept/commit); host copies."""
    torch = _torch()
    from paper_2510_13161_amd import msd
    w, si = case.w, case.si
    B, n, V = w.batch, w.n_slots, case.shape.vocab
    M = B * n
    case.reset_len()
    blk = msd.make_block(torch.from_numpy(si.tokens).cuda(), None if w.topology == "chain" else si.parent)
    out = dict(logits=torch.full((M, V), -7.0, device="cuda"),
               argmax=torch.full((M,), -7, dtype=torch.int32, device="cuda"),
               lse=torch.full((M,), -7.0, device="cuda"),
               ids=torch.full((M, w.kappa), -7, dtype=torch.int32, device="cuda"),
               logp=torch.full((M, w.kappa), -7.0, device="cuda"))
    ee = msd.EERequest(min(w.ee_layer, case.shape.n_layers - 1), w.kappa, out["ids"].data_ptr(),
                       out["logp"].data_ptr(), None)
    if static:
        msd.verify_block_static(case.model.handle, case.cache.c, blk, ee, out["logits"], out["argmax"],
                                out["lse"])
    else:
        ws = torch.empty(msd.workspace_bytes(case.model.handle, B, n, w.kappa, case.capacity),
                         dtype=torch.uint8, device="cuda")
        msd.verify_block(case.model.handle, case.cache.c, blk, ee, out["logits"], out["argmax"],
                         out["lse"], ws)
    torch.cuda.synchronize()
    res = {k: v.cpu().numpy() for k, v in out.items()}
    res["k"], res["v"] = case._rows(si.ctx_len, np.full(B, n))
    res["status"] = int(case.cache.status.item())
    return res


def _same(a, b, tag):
    for k in ("logits", "argmax", "lse", "ids", "logp"):
        assert np.array_equal(a[k], b[k]), f"{tag}: {k}"
    for l in range(len(a["k"])):
        assert np.array_equal(a["k"][l], b["k"][l]) and np.array_equal(a["v"][l], b["v"][l]), f"{tag}: kv {l}"
    assert a["status"] == b["status"] == 0


def test_static_scratch_matches_workspace_two_calls():
    """Static-scratch verify == workspace verify, bit for bit, on two calls
    in a row: a ragged batch of 4 tree blocks (M = 68, 2 attention chunks),
    then a smaller block (the tiny chain, M = 5); then the 14B-width chain
    (2 layers, M = 9) and the first block again."""
    _torch()
    big = H.GpuCase(synth.WORKLOADS["14b_batch16"].with_model(
        synth.TINY, batch=4, ctx=(40, 400), topology="tree", gamma=4, branches=4, ee_layer=1, kappa=4,
        seed=51))
    small = H.GpuCase(synth.WORKLOADS["tiny_chain"])
    s1 = _verify(big, True)
    s2 = _verify(small, True)
    _same(s1, _verify(big, False), "first call, M = 68")
    _same(s2, _verify(small, False), "second call, M = 5")
    assert np.isfinite(s1["logits"]).all() and np.isfinite(s2["logits"]).all()
    wide = H.GpuCase(synth.WORKLOADS["14b_chain"].with_model(synth.QWEN14B), n_layers=2)
    _same(_verify(wide, True), _verify(wide, False), "14B widths, M = 9")
    _same(_verify(big, True), s1, "first block again")


def test_static_scratch_rejects_blocks_beyond_its_size():
    """A block whose workspace exceeds the static scratch (a batch of 16
    long-context GQA blocks: 128 key chunks of partial attention outputs) is
    refused on the host with MSD_ERR_WORKSPACE; nothing is enqueued."""
    torch = _torch()
    from paper_2510_13161_amd import msd
    shape = synth.ModelShape("gqa64", 2, 1024, 16, 4, 64, 2048, 4096)
    B, n, cap = 16, 9, 32768
    model = msd.Model(shape, synth.device_weights(shape, 3), max_positions=cap)
    need = msd.workspace_bytes(model.handle, B, n, 4, cap)
    assert need > msd.MSD_STATIC_SCRATCH_BYTES
    cache = msd.Cache(shape, B, cap)            # a real cache of that capacity: nothing would be out of bounds
    tokens = torch.zeros((B, n), dtype=torch.int32, device="cuda")
    blk = msd.make_block(tokens)
    logits = torch.full((B * n, shape.vocab), -7.0, device="cuda")
    argmax = torch.full((B * n,), -7, dtype=torch.int32, device="cuda")
    with pytest.raises(msd.MsdError) as e:
        msd.verify_block_static(model.handle, cache.c, blk, None, logits, argmax, None)
    assert e.value.status == msd.MSD_ERR_WORKSPACE and "static scratch" in str(e.value)
    torch.cuda.synchronize()
    assert bool((argmax == -7).all()) and int(cache.status.item()) == 0
    model.close()
