#!/usr/bin/env python3
"""Throughput of the Mirror-SD verification step on one MI355X.

One step = the target's whole verification of one draft block (every row of
the hot path): embedding, N decoder layers over the block against the KV
cache, the early-exit top-kappa message after layer l_e, the final head,
acceptance and the KV commit/rollback. Inputs are seeded and synthetic
(random-init weights of the named shape, random cached K/V and draft
tokens), resident in HBM before the timed region.

Prints ONE JSON line: verified draft tokens/s (the metric), ms per step, the
roofline of the dominant kernel (the FFN up-projection GEMM, timed with HIP
events that the library records on its own stream around its launches in
every sixth layer inside the timed region), the time from the start of a step to the
early-exit message, and the fp64 oracle's throughput on the host cores over
one whole step of sequence 0.

``--copy-calibration BYTES`` instead times a plain device-to-device copy of
BYTES bytes (the reference kernel that scales the HBM traffic counters).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
MFMA_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
PROFILE_STRIDE = 6     # layers between timed FFN up-projection launches
METRIC = "verified tokens/sec per verify step + % HBM roofline, 14B-shaped γ=8"


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="14b_chain")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-kernel-events", action="store_true",
                    help="time the steps without the per-launch HIP events")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES")
    ap.add_argument("--latency-law", action="store_true",
                    help="measure the Sec. 3.4 latency law with a synthetic draft on a second stream")
    return ap.parse_args()


def step_bytes(shape, w, ctx_mean: float) -> dict:
    """Algorithmic HBM bytes of one step: every weight once, the LM head twice
    (early exit + final), cached K/V read once, block K/V written, logits out."""
    import re
    import numpy as np
    from paper_2510_13161_amd import synth
    specs = synth.tensor_specs(shape)
    layer_w = sum(2 * int(np.prod(s.shape)) for s in specs if re.match(r"l\d+\.", s.name))
    head = 2 * shape.vocab * shape.d_model
    M = w.rows
    kv_read = shape.n_layers * 2 * shape.n_kv_heads * shape.head_dim * 2 * (ctx_mean + w.n_slots) * w.batch
    kv_write = shape.n_layers * 2 * shape.n_kv_heads * shape.head_dim * 2 * M
    logits = M * shape.vocab * 4
    return {"weights": layer_w, "heads": 2 * head, "kv": kv_read + kv_write, "logits": logits,
            "total": layer_w + 2 * head + kv_read + kv_write + logits}


def step_gemm_flops(shape, w) -> float:
    """Algorithmic GEMM flops of one step: 2·M per weight of every
    projection matrix, the LM head twice (attention's score and value
    products, a few per cent at these shapes, are not counted)."""
    import re
    import numpy as np
    from paper_2510_13161_amd import synth
    mats = sum(int(np.prod(s.shape)) for s in synth.tensor_specs(shape)
               if re.match(r"l\d+\.", s.name) and len(s.shape) == 2)
    return 2.0 * w.rows * (mats + 2 * shape.vocab * shape.d_model)


def ffn_up_bytes(shape, M: int) -> int:
    """Algorithmic bytes of one FFN up-projection launch: its weights (gate and
    up for SwiGLU) once, the normed rows in, the activation rows out."""
    n_mats = 2 if shape.act == "swiglu" else 1
    return n_mats * shape.d_ffn * shape.d_model * 2 + M * shape.d_model * 2 + M * shape.d_ffn * 2


def measured_traffic():
    """HBM bytes per launch of the dominant kernel from the committed
    rocprofv3 FETCH_SIZE / WRITE_SIZE summary, or None once the GEMM source
    has changed since those counters were taken."""
    import hashlib
    import re
    root = os.path.dirname(os.path.abspath(__file__))
    prof = os.path.join(root, "profiles", "ffn_up_gemm_14b_chain_traffic.md")
    src = os.path.join(root, "paper_2510_13161_amd", "csrc", "gemm.hip")
    try:
        text = open(prof).read()
        sha = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
    except OSError:
        return None
    m = re.search(r"gemm_source_sha256_16: ([0-9a-f]{16}); traffic_bytes_per_launch: (\d+)", text)
    if not m or m.group(1) != sha:
        return None
    return int(m.group(2))


def cpu_baseline(shape, w, reps: int = 4) -> dict:
    """The fp64 oracle on the host over one whole verification step of
    sequence 0: embed, every decoder layer, the early-exit and final heads,
    top-kappa and acceptance, each oracle call run `reps` times on the same
    input (a bounded sample of about ten to fifteen seconds). Layer weights are generated
    just before their layer runs and dropped after it (only the oracle calls
    are timed)."""
    import numpy as np
    import oracle as orc
    from paper_2510_13161_amd import synth
    if not os.path.exists(orc.LIB_PATH):
        orc.build()
    si = synth.step_inputs(w)
    L = int(si.ctx_len[0])
    glob = synth.host_weights(shape, w.seed, layers=[], with_globals=True)
    o = orc.Oracle(shape, glob)
    pos = L + orc.depths(si.parent)
    timed = 0.0
    t0 = time.perf_counter()
    for _ in range(reps):
        x = o.embed(si.tokens[0], pos)
    timed += time.perf_counter() - t0
    for l in range(shape.n_layers):
        lw = synth.host_weights(shape, w.seed, layers=[l], with_globals=False)
        ck = synth.host_ctx(shape, w.seed, l, "k", 0, L)
        cv = synth.host_ctx(shape, w.seed, l, "v", 0, L)
        o.layer_source = lambda _l, lw=lw: lw
        x_in = x.copy()
        t0 = time.perf_counter()
        for _ in range(reps):
            x = x_in.copy()
            o.layer(l, x, pos, si.parent, ck, cv, L)
            if l + 1 == w.ee_layer:
                orc.Oracle.topk(o.head(x), w.kappa)
        timed += time.perf_counter() - t0
        del lw
    t0 = time.perf_counter()
    for _ in range(reps):
        z = o.head(x)
        o.accept(si.parent, si.tokens[0], z)
    timed += time.perf_counter() - t0
    timed /= reps
    threads = orc.omp_threads()
    per_seq_tokens = w.n_slots - 1
    single = tiny_single_thread(orc, synth)
    return {"value": round(per_seq_tokens / timed, 4), "unit": "verified tokens/s", "cores": threads,
            "kind": "oracle", "cpu": cpu_model(), "host_cpus": os.cpu_count(),
            "tiny_single_thread": single,
            "sample": (f"one whole step of sequence 0 of {w.name} ({per_seq_tokens} draft tokens): "
                       f"embed, {shape.n_layers} decoder layers, early-exit and final heads, "
                       f"top-{w.kappa}, acceptance; fp64 C oracle, OpenMP over {threads} threads; "
                       f"each call run {reps} times, {timed * reps:.1f} s of oracle time in all, "
                       f"{timed:.2f} s per step (weight generation untimed)")}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def tiny_single_thread(orc, synth, seconds: float = 1.0) -> dict:
    """The oracle on one thread over whole steps of the tiny chain workload
    (2 layers, d 256, 4 drafts), repeated for about `seconds`."""
    w = synth.WORKLOADS["tiny_chain"]
    shape = w.model
    si = synth.step_inputs(w)
    L = int(si.ctx_len[0])
    o = orc.Oracle(shape, synth.host_weights(shape, w.seed))
    cc = {l: (synth.host_ctx(shape, w.seed, l, "k", 0, L), synth.host_ctx(shape, w.seed, l, "v", 0, L))
          for l in range(shape.n_layers)}
    pos = L + orc.depths(si.parent)
    before = orc.omp_threads()
    orc.set_omp_threads(1)
    try:
        n, t0 = 0, time.perf_counter()
        while True:
            r = o.forward(si.tokens[0], pos, si.parent, lambda l: cc[l], L, ee_layer=w.ee_layer)
            orc.Oracle.topk(o.head(r.x_ee), w.kappa)
            o.accept(si.parent, si.tokens[0], r.logits)
            n += 1
            el = time.perf_counter() - t0
            if el >= seconds:
                break
    finally:
        orc.set_omp_threads(before)
    return {"value": round((w.n_slots - 1) * n / el, 2), "unit": "verified tokens/s", "cores": 1,
            "steps": n, "workload": w.name}


def copy_rate(nbytes: int, reps: int = 1) -> dict:
    """A plain device-to-device copy of nbytes: (read + write bytes) / time,
    the best of reps timed copies after 3 untimed ones."""
    import torch
    n = nbytes // 4
    a = torch.empty(n, dtype=torch.float32, device="cuda").fill_(1.0)
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    best = None
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        b.copy_(a)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        best = ms if best is None else min(best, ms)
    del a, b
    return {"copy_bytes": 4 * n, "ms": round(best, 4), "read_plus_write_gbs": round(8 * n / (best * 1e-3) / 1e9, 1)}


def copy_calibration(nbytes: int) -> None:
    """A plain HBM copy of known size: its FETCH_SIZE / WRITE_SIZE counters
    against nbytes give the factor that turns those counters into bytes."""
    print(json.dumps(copy_rate(nbytes)), flush=True)


def after_accept(msd, torch, np, model, blk, acc, nxt, path, logits, lse, ids, w, vocab, reps=50):
    """The step after acceptance (Sec. 3.1 reuse criterion and next-window
    selection, App. E statistics) on the last timed step's outputs, timed on
    its own: the hypothesis tree has kappa chains of gamma + 1 nodes (the
    window's depth; fewer if kappa chains would exceed the tree's node limit)
    rooted at each sequence's early-exit top-kappa (root row), continuation
    tokens drawn. Returns its mean launch time, the fallback frequency and the
    mean overlap mass of the tree it decided on."""
    B, n, kap = w.batch, w.n_slots, w.kappa
    nc_len = min(w.gamma + 1, msd.MSD_MAX_TREE_NODES // kap)
    parent = [(-1 if d == 0 else r * nc_len + d - 1) for r in range(kap) for d in range(nc_len)]
    roots = ids.view(B, n, kap)[:, 0, :].cpu().numpy()
    rng = np.random.default_rng(w.seed + 100)
    ttok = rng.integers(0, vocab, size=(B, kap * nc_len)).astype(np.int32)
    for r in range(kap):
        ttok[:, r * nc_len] = roots[:, r]
    tree = msd.hyp_tree(parent, torch.from_numpy(ttok).cuda())
    nc = torch.empty(B, dtype=torch.int32, device="cuda")
    nn_ = torch.empty(B, dtype=torch.int32, device="cuda")
    om = torch.empty(B, dtype=torch.float32, device="cuda")
    stats = torch.zeros(64, dtype=torch.uint8, device="cuda")
    call = lambda st: msd.reuse_select(model.handle, blk, acc, nxt, path, tree, nc, nn_, logits, lse,
                                       ids, kap, om, st)
    call(stats)
    torch.cuda.synchronize()
    r = msd.read_reuse_stats(stats)
    for _ in range(3):
        call(None)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(reps):
        call(None)
    e1.record()
    torch.cuda.synchronize()
    return {"reuse_select_us": round(e0.elapsed_time(e1) * 1e3 / reps, 2),
            "fallback_frequency": r["fallbacks"] / max(r["trials"], 1),
            "mean_omega": round(r["omega_sum"] / max(r["omega_trials"], 1), 6),
            "tree": f"{kap} chains x {nc_len} nodes on the early-exit top-{kap}"}


def latency_law(args) -> dict:
    """Sec. 3.4 latency law on one GPU: the 14B chain target step, and a
    synthetic 0.6B-shaped draft that generates gamma tokens over the kappa
    early-exit branches (kappa sequences decoded greedily in lockstep, the
    roots taken from the early-exit top-kappa, each step's argmax feeding the
    next) on a second stream that waits for the early-exit message's ready
    event. Measures T_target, T^{1:l_e} (step start to the message), the
    overlap budget Delta = T_target - T^{1:l_e}, T_draft alone, the overlapped
    step, the law's prediction T^{1:l_e} + max(Delta, T_draft) and the
    sequential (vanilla SD) T_target + T_draft. Both models share one GPU's
    HBM, which two devices would not."""
    import numpy as np
    import torch
    from paper_2510_13161_amd import msd, synth
    w = synth.WORKLOADS["14b_chain"]
    shape, dshape = w.model, synth.DRAFT06B
    si = synth.step_inputs(w)
    B, n, kap, gam = w.batch, w.n_slots, w.kappa, w.gamma
    M = B * n
    cap = int(-(-(int(si.ctx_len.max()) + n + 8) // 64) * 64)
    model = msd.Model(shape, synth.device_weights(shape, w.seed), max_positions=cap)
    cache = msd.Cache(shape, B, cap)
    len0 = torch.from_numpy(si.ctx_len).cuda()
    cache.len.copy_(len0)
    synth.device_fill_ctx(shape, w.seed, cache.k, cache.v, cache.len)
    tokens = torch.from_numpy(si.tokens).cuda()
    blk = msd.make_block(tokens, None)
    logits = torch.empty((M, shape.vocab), dtype=torch.float32, device="cuda")
    argmax = torch.empty(M, dtype=torch.int32, device="cuda")
    lse = torch.empty(M, dtype=torch.float32, device="cuda")
    ids = torch.empty((M, kap), dtype=torch.int32, device="cuda")
    logp = torch.empty((M, kap), dtype=torch.float32, device="cuda")
    ws = torch.empty(msd.workspace_bytes(model.handle, B, n, kap, cap), dtype=torch.uint8, device="cuda")
    acc = torch.empty(B, dtype=torch.int32, device="cuda")
    nxt = torch.empty(B, dtype=torch.int32, device="cuda")
    path = torch.empty((B, n), dtype=torch.int32, device="cuda")
    ee = msd.EERequest(w.ee_layer, kap, ids.data_ptr(), logp.data_ptr(), None)

    # draft: kappa sequences with the target's context length, one slot per step
    dcap = int(-(-(int(si.ctx_len.max()) + gam + 8) // 64) * 64)
    dmodel = msd.Model(dshape, synth.device_weights(dshape, w.seed + 50), max_positions=dcap)
    dcache = msd.Cache(dshape, kap, dcap)
    dlen0 = torch.full((kap,), int(si.ctx_len[0]), dtype=torch.int32, device="cuda")
    dcache.len.copy_(dlen0)
    synth.device_fill_ctx(dshape, w.seed + 50, dcache.k, dcache.v, dcache.len)
    dargmax = [torch.empty(kap, dtype=torch.int32, device="cuda") for _ in range(gam)]
    droots = ids[0].view(kap, 1)  # the early-exit top-kappa of the root row
    dblks = [msd.make_block(droots if i == 0 else dargmax[i - 1].view(kap, 1), None) for i in range(gam)]
    dws = torch.empty(msd.workspace_bytes(dmodel.handle, kap, 1, 1, dcap), dtype=torch.uint8, device="cuda")
    dzero = torch.zeros(kap, dtype=torch.int32, device="cuda")
    dpath = torch.zeros((kap, 1), dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()

    def target_step():
        msd.verify_block(model.handle, cache.c, blk, ee, logits, argmax, lse, ws)
        msd.accept(model.handle, blk, logits, argmax, None, acc, nxt, path, cache.status)
        msd.kv_commit(model.handle, cache.c, blk, acc, path)
        cache.len.copy_(len0)  # every step sees the same context

    def draft_gen():
        for i in range(gam):
            msd.verify_block(dmodel.handle, dcache.c, dblks[i], None, None, dargmax[i], None, dws)
            msd.kv_commit(dmodel.handle, dcache.c, dblks[i], dzero, dpath)
        dcache.len.copy_(dlen0)

    def timed(fn, steps):
        for _ in range(2):
            fn(0)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for k in range(steps):
            fn(k)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    steps = args.steps
    ready = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    for e in ready + starts:  # torch only times events it has seen recorded once
        e.record()
    torch.cuda.synchronize()

    def target_only(k):
        target_step()

    def target_with_ready(k):
        ee.ready = ready[k].cuda_event
        starts[k].record()
        target_step()

    t_target = timed(target_only, steps)
    timed(target_with_ready, steps)
    t_prefix = float(np.median([a.elapsed_time(b) for a, b in zip(starts, ready)]))
    t_draft = timed(lambda k: draft_gen(), steps)

    side = torch.cuda.Stream()
    done = [torch.cuda.Event() for _ in range(steps)]

    def overlapped(k):
        ee.ready = ready[k].cuda_event
        starts[k].record()
        target_step()  # records ready[k] right after the early-exit message
        side.wait_event(ready[k])
        with torch.cuda.stream(side):
            draft_gen()
            done[k].record()
        torch.cuda.current_stream().wait_event(done[k])

    def sequential(k):
        target_step()
        draft_gen()

    t_overlap = timed(overlapped, steps)
    t_seq = timed(sequential, steps)

    # the same with the CUs split between two masked streams (224 for the
    # target, 32 for the draft): two "devices" that still share HBM
    part = None
    masked = cu_masked_streams(torch, [(0, 224), (224, 256)])
    if masked is not None:
        ts, ds = masked

        def target_masked(k):
            with torch.cuda.stream(ts):
                target_step()

        def draft_masked(k):
            with torch.cuda.stream(ds):
                draft_gen()

        def overlapped_masked(k):
            with torch.cuda.stream(ts):
                ee.ready = ready[k].cuda_event
                starts[k].record()
                target_step()
            ds.wait_event(ready[k])
            with torch.cuda.stream(ds):
                draft_gen()
                done[k].record()
            ts.wait_event(done[k])
            torch.cuda.current_stream().wait_stream(ts)

        ee.ready = None
        pt = timed(target_masked, steps)
        pd = timed(draft_masked, steps)
        po = timed(overlapped_masked, steps)
        pp = float(np.median([a.elapsed_time(b) for a, b in zip(starts, ready)]))
        part = {"cus": [224, 32], "t_target_ms": round(pt, 4), "t_prefix_ms": round(pp, 4),
                "t_draft_ms": round(pd, 4), "t_overlap_ms": round(po, 4),
                "t_law_ms": round(pp + max(pt - pp, pd), 4)}
    ee.ready = None
    delta = t_target - t_prefix

    # Speculative Streaming draft (Sec. 3.2, timing only): one draft forward
    # carries, for each of the kappa branches, the main stream (the branch
    # root) and gamma lookahead streams, stream j attending to the verified
    # prefix and to streams 1..j: a chain of gamma + 1 slots per branch, i.e.
    # a batch-kappa chain block, with the shared LM head over every stream.
    # Trained stream embeddings would replace the token embeddings of the
    # lookahead slots at the same cost. J = ceil(gamma / eta) such steps give
    # gamma tokens when a step emits eta on average.
    ss_n = gam + 1
    ss_tok = torch.cat([droots, droots.expand(kap, gam)], dim=1).contiguous()
    ss_blk = msd.make_block(ss_tok, None)
    ss_arg = torch.empty(kap * ss_n, dtype=torch.int32, device="cuda")
    ss_ws = torch.empty(msd.workspace_bytes(dmodel.handle, kap, ss_n, 1, dcap), dtype=torch.uint8, device="cuda")
    ss_path = torch.zeros((kap, ss_n), dtype=torch.int32, device="cuda")

    def ss_step():
        msd.verify_block(dmodel.handle, dcache.c, ss_blk, None, None, ss_arg, None, ss_ws)
        msd.kv_commit(dmodel.handle, dcache.c, ss_blk, dzero, ss_path)
        dcache.len.copy_(dlen0)

    t_ss = timed(lambda k: ss_step(), steps)
    ss_laws = []
    for eta in (1, 2, 4, gam):
        J = -(-gam // eta)

        def ss_gen(J=J):
            for _ in range(J):
                ss_step()

        def ss_overlapped(k, J=J):
            ee.ready = ready[k].cuda_event
            starts[k].record()
            target_step()
            side.wait_event(ready[k])
            with torch.cuda.stream(side):
                ss_gen()
                done[k].record()
            torch.cuda.current_stream().wait_event(done[k])

        t_ov = timed(ss_overlapped, steps)
        ss_laws.append({"eta": eta, "J": J, "t_draft_ms": round(J * t_ss, 4),
                        "t_law_ms": round(t_prefix + max(delta, J * t_ss), 4),
                        "t_overlap_ms": round(t_ov, 4)})
    ee.ready = None
    ss = {"rows": kap * ss_n, "block": f"{kap} branches x (main + {gam} lookahead streams)",
          "t_step_ms": round(t_ss, 4), "by_tokens_per_step": ss_laws}
    return {"mode": "latency_law", "workload": w.name,
            "draft": f"{dshape.n_layers}L d{dshape.d_model} {dshape.n_heads}/{dshape.n_kv_heads}x{dshape.head_dim} "
                     f"F{dshape.d_ffn} V{dshape.vocab} tied; {kap} branches x {gam} greedy steps",
            "steps": steps, "t_target_ms": round(t_target, 4), "t_prefix_ms": round(t_prefix, 4),
            "delta_ms": round(delta, 4), "t_draft_ms": round(t_draft, 4),
            "t_overlap_ms": round(t_overlap, 4), "t_law_ms": round(t_prefix + max(delta, t_draft), 4),
            "t_sequential_ms": round(t_seq, 4), "cu_partition": part, "ss_draft": ss,
            "note": "one GPU: the draft and the target suffix share HBM (and, unpartitioned, CUs)"}


def cu_masked_streams(torch, ranges):
    """Streams restricted to CU index ranges [lo, hi) (hipExtStreamCreateWithCUMask),
    as torch external streams; None if the runtime refuses."""
    import ctypes
    try:
        hip = ctypes.CDLL("libamdhip64.so")
    except OSError:
        return None
    fn = hip.hipExtStreamCreateWithCUMask
    fn.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint32, ctypes.POINTER(ctypes.c_uint32)]
    fn.restype = ctypes.c_int
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    out = []
    for lo, hi in ranges:
        if hi > n_cu:
            return None
        words = (n_cu + 31) // 32
        mask = (ctypes.c_uint32 * words)()
        for c in range(lo, hi):
            mask[c // 32] |= 1 << (c % 32)
        h = ctypes.c_void_p()
        if fn(ctypes.byref(h), words, mask) != 0:
            return None
        out.append(torch.cuda.ExternalStream(h.value))
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: the library runs the verify step on exactly one GPU; --gpus {args.gpus} is not "
              "supported (sharding over several GPUs is described, not implemented)", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch
    from paper_2510_13161_amd import msd, synth

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.latency_law:
        print(json.dumps(latency_law(args)), flush=True)
        return
    w = synth.WORKLOADS[args.workload]
    shape = w.model
    si = synth.step_inputs(w)
    dev = "cuda"
    total_steps = args.warmup + args.steps
    capacity = int(-(-(int(si.ctx_len.max()) + w.n_slots + total_steps + 8) // 64) * 64)

    t0 = time.perf_counter()
    weights = synth.device_weights(shape, w.seed, dev)
    maxpos = capacity if shape.pos == "rope" else shape.max_positions
    model = msd.Model(shape, weights, max_positions=maxpos)
    cache = msd.Cache(shape, w.batch, capacity, dev)
    len0 = torch.from_numpy(si.ctx_len).to(dev)
    cache.len.copy_(len0)
    synth.device_fill_ctx(shape, w.seed, cache.k, cache.v, cache.len)
    torch.cuda.synchronize()
    t_setup = time.perf_counter() - t0

    B, n = w.batch, w.n_slots
    M = B * n
    tokens = torch.from_numpy(si.tokens).to(dev)
    blk = msd.make_block(tokens, None if w.topology == "chain" else si.parent)
    logits = torch.empty((M, shape.vocab), dtype=torch.float32, device=dev)
    argmax = torch.empty(M, dtype=torch.int32, device=dev)
    lse = torch.empty(M, dtype=torch.float32, device=dev)
    ids = torch.empty((M, w.kappa), dtype=torch.int32, device=dev)
    logp = torch.empty((M, w.kappa), dtype=torch.float32, device=dev)
    ee_ready = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ee = msd.EERequest(w.ee_layer, w.kappa, ids.data_ptr(), logp.data_ptr(), None)
    # one workspace for the verify pass and then the acceptance's vocabulary statistics
    ws = torch.empty(max(msd.workspace_bytes(model.handle, B, n, w.kappa, capacity),
                         M * msd.MSD_ACCEPT_WS_PER_ROW), dtype=torch.uint8, device=dev)
    acc = torch.empty(B, dtype=torch.int32, device=dev)
    nxt = torch.empty(B, dtype=torch.int32, device=dev)
    path = torch.empty((B, n), dtype=torch.int32, device=dev)
    smp = None
    keep = []
    if w.mode != "greedy":
        t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
        keep = [t(si.cand_ids), t(si.cand_q), t(si.u_accept), t(si.u_sample)]
        smp = msd.Sampling(msd.MODES[w.mode], float(w.temperature), si.cand_ids.shape[-1],
                           *[k.data_ptr() for k in keep])

    def step():
        msd.verify_block(model.handle, cache.c, blk, ee, logits, argmax, lse, ws)
        msd.accept(model.handle, blk, logits, argmax, smp, acc, nxt, path, cache.status, ws=ws)
        msd.kv_commit(model.handle, cache.c, blk, acc, path)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # HIP events: the library records begin/end around the FFN up-projection
    # launch of every PROFILE_STRIDE-th layer on the stream it launches on
    # (a sample of the launches, so that the events' own pipeline bubbles
    # stay small), and the early-exit message's ready event; the step starts
    # are recorded on the same (current) stream.
    L = shape.n_layers
    sampled = list(range(0, L, PROFILE_STRIDE))
    events = not args.no_kernel_events
    if events:
        evb = [[torch.cuda.Event(enable_timing=True) for _ in sampled] for _ in range(args.steps)]
        eve = [[torch.cuda.Event(enable_timing=True) for _ in sampled] for _ in range(args.steps)]
        starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
        for e in [x for r in evb + eve for x in r] + starts + ee_ready:
            e.record()
        torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for k in range(args.steps):
        if events:
            pb, pe = [None] * L, [None] * L
            for i, l in enumerate(sampled):
                pb[l], pe[l] = evb[k][i].cuda_event, eve[k][i].cuda_event
            msd.set_profile(model.handle, msd.MSD_K_FFN_UP, pb, pe)
            ee.ready = ee_ready[k].cuda_event
            starts[k].record()
        step()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    msd.set_profile(model.handle, msd.MSD_K_FFN_UP, [], [])
    ee.ready = None
    status = int(cache.status.item())
    if status != 0:
        print(f"bench.py: device status {status}", file=sys.stderr)
        sys.exit(1)

    post = after_accept(msd, torch, np, model, blk, acc, nxt, path, logits, lse, ids, w, shape.vocab)

    roof, t_ee = None, None
    if events:
        dur = [b.elapsed_time(e) for rb, re_ in zip(evb, eve) for b, e in zip(rb, re_)]
        avg_ms = float(np.mean(dur))
        per_launch = ffn_up_bytes(shape, M)
        achieved = per_launch / (avg_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": measured_traffic(),
                "kernel": "gemm_kernel<EPI_SWIGLU> (FFN gate+up projection)",
                "bytes_per_launch": per_launch, "avg_launch_us": round(avg_ms * 1e3, 2),
                "launches": len(dur)}
        t_ee = float(np.median([s_.elapsed_time(r) for s_, r in zip(starts, ee_ready)]))

    # a streaming ceiling measured on this device (outside the timed region):
    # a plain 1 GiB device copy, read + write bytes per second
    ceiling = copy_rate(1 << 30, reps=5)

    ctx_mean = float(si.ctx_len.mean()) + (args.warmup + args.steps)  # len grows by 1 per step
    sb = step_bytes(shape, w, ctx_mean)
    fl = step_gemm_flops(shape, w)
    step_gbs = sb["total"] / (ms * 1e-3) / 1e9
    value = w.draft_tokens / (ms * 1e-3)
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "verified tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded random-init weights, random cached K/V and draft tokens)",
        "config": {"workload": w.name,
                   "shape": (f"{shape.n_layers}L d{shape.d_model} {shape.n_heads}/{shape.n_kv_heads}"
                             f"x{shape.head_dim} F{shape.d_ffn} V{shape.vocab}"),
                   "batch": w.batch, "n_slots": n,
                   "topology": w.topology, "ctx": list(w.ctx), "ee_layer": w.ee_layer,
                   "kappa": w.kappa, "acceptance": w.mode},
        "step_bytes": sb["total"], "step_hbm_gbs": round(step_gbs, 1),
        "step_hbm_frac": round(step_gbs / HBM_PEAK_GBS, 4),
        "roofline": roof,
        # MFMA work: each GEMM runs two bf16 products per weight (the
        # activation's hi and lo parts), so the issued work is twice the
        # algorithmic flops; against the dense bf16 MFMA peak
        "mfma": {"gemm_tflop_per_step": round(fl / 1e12, 4), "issued_tflop_per_step": round(2 * fl / 1e12, 4),
                 "achieved_tflops": round(2 * fl / (ms * 1e-3) / 1e12, 1), "peak_tflops": MFMA_PEAK_TFLOPS,
                 "frac": round(2 * fl / (ms * 1e-3) / 1e12 / MFMA_PEAK_TFLOPS, 4)},
        "ms_to_early_exit": None if t_ee is None else round(t_ee, 4),
        # the overlap budget of the Sec. 3.4 latency law: the target's time
        # from the early-exit message to the end of the step
        "overlap_budget_ms": None if t_ee is None else round(ms - t_ee, 4),
        "hbm_ceiling": {"probe": "device-to-device copy of 1 GiB, best of 5",
                        "read_plus_write_gbs": ceiling["read_plus_write_gbs"],
                        "step_frac_of_ceiling": round(step_gbs / ceiling["read_plus_write_gbs"], 4)},
        "after_accept": post,
        "setup_s": round(t_setup, 2),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(shape, w)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
