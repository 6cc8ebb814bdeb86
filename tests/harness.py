"""Test-side driver: one seeded workload through the HIP library and the oracle.

Only the shared input generator feeds both sides; the oracle never sees a
byte that the HIP path produced.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np

import oracle as orc
from paper_2510_13161_amd import synth

TOL_LOGIT = 2e-2          # max |logit_gpu - logit_oracle| (bf16 operands, fp32 accumulation)
TIE_MARGIN = 2 * TOL_LOGIT  # decisions closer than this in the oracle are flagged


def round_up(x: int, m: int) -> int:
    return (x + m - 1) // m * m


@dataclasses.dataclass
class GpuResult:
    logits: Optional[np.ndarray]   # [M, V] fp32
    argmax: np.ndarray             # [M]
    lse: np.ndarray                # [M]
    ee_ids: Optional[np.ndarray]   # [M, kappa]
    ee_logp: Optional[np.ndarray]
    acc_len: np.ndarray            # [B]
    next_tok: np.ndarray           # [B]
    path: np.ndarray               # [B, n_slots]
    len_after: np.ndarray          # [B]
    status: int
    k_rows: List[np.ndarray]       # per layer [B][Hkv][n_slots][hd] bf16 bits (after verify)
    v_rows: List[np.ndarray]
    near_tie: Optional[np.ndarray] = None   # [B] flags of msd_accept
    k_commit: Optional[List[np.ndarray]] = None  # per layer [B][Hkv][n_slots][hd] rows at
    v_commit: Optional[List[np.ndarray]] = None  # len_before + r after the commit (first 1 + A valid)


class GpuCase:
    """A workload (optionally depth-reduced) resident on the GPU."""

    def __init__(self, w: synth.Workload, n_layers: Optional[int] = None,
                 capacity: Optional[int] = None, inputs: Optional[synth.StepInputs] = None):
        import torch
        from paper_2510_13161_amd import msd
        self.torch, self.msd = torch, msd
        self.w = w
        self.shape = w.model if n_layers is None else w.model.with_layers(n_layers)
        self.si = inputs if inputs is not None else synth.step_inputs(w)
        lens = self.si.ctx_len
        self.capacity = capacity or round_up(int(lens.max()) + w.n_slots, 64)
        self.dev = synth.device_weights(self.shape, w.seed)
        maxpos = self.capacity if self.shape.pos == "rope" else self.shape.max_positions
        self.model = msd.Model(self.shape, self.dev, max_positions=maxpos)
        self.cache = msd.Cache(self.shape, w.batch, self.capacity)
        self.cache.len.copy_(torch.from_numpy(lens))
        synth.device_fill_ctx(self.shape, w.seed, self.cache.k, self.cache.v, self.cache.len)
        torch.cuda.synchronize()

    def reset_len(self):
        self.cache.len.copy_(self.torch.from_numpy(self.si.ctx_len))
        self.cache.status.zero_()

    def _rows(self, start: np.ndarray, count: np.ndarray):
        """Cache rows [start_b, start_b + count_b) of every layer (bf16 bits,
        zero past count_b), per layer [B][Hkv][n_slots][hd]."""
        torch = self.torch
        B, n = self.w.batch, self.w.n_slots
        ks, vs = [], []
        for l in range(self.shape.n_layers):
            kr = np.zeros((B, self.shape.n_kv_heads, n, self.shape.head_dim), np.uint16)
            vr = np.zeros_like(kr)
            for b in range(B):
                L = int(start[b])
                hi = min(L + int(count[b]), self.capacity)  # a block that overflows the cache has no rows there
                if hi <= L:
                    continue
                kr[b, :, :hi - L] = self.cache.k[l, b, :, L:hi].view(torch.int16).cpu().numpy().view(np.uint16)
                vr[b, :, :hi - L] = self.cache.v[l, b, :, L:hi].view(torch.int16).cpu().numpy().view(np.uint16)
            ks.append(kr)
            vs.append(vr)
        return ks, vs

    def run(self, ee: bool = True, want_logits: bool = True, commit: bool = True,
            mode: Optional[str] = None) -> GpuResult:
        torch, msd = self.torch, self.msd
        w, si = self.w, self.si
        dev = "cuda"
        B, n = w.batch, w.n_slots
        M = B * n
        V = self.shape.vocab
        mode = mode or w.mode
        tokens = torch.from_numpy(si.tokens).to(dev)
        parent = None if w.topology == "chain" else si.parent
        blk = msd.make_block(tokens, parent)
        logits = torch.empty((M, V), dtype=torch.float32, device=dev) if want_logits else None
        argmax = torch.empty(M, dtype=torch.int32, device=dev)
        lse = torch.empty(M, dtype=torch.float32, device=dev)
        req = None
        if ee:
            ids = torch.empty((M, w.kappa), dtype=torch.int32, device=dev)
            logp = torch.empty((M, w.kappa), dtype=torch.float32, device=dev)
            req = msd.EERequest(min(w.ee_layer, self.shape.n_layers - 1), w.kappa, ids.data_ptr(),
                                logp.data_ptr(), None)
        nb = msd.workspace_bytes(self.model.handle, B, n, w.kappa if ee else 1, self.capacity)
        # one workspace for both calls (stream-ordered): the verify pass, then
        # the acceptance's vocabulary statistics
        ws = torch.empty(max(nb, M * msd.MSD_ACCEPT_WS_PER_ROW), dtype=torch.uint8, device=dev)
        msd.verify_block(self.model.handle, self.cache.c, blk, req, logits, argmax, lse, ws)
        # block rows written by the verify pass
        k_rows, v_rows = self._rows(si.ctx_len, np.full(B, n))
        acc = torch.empty(B, dtype=torch.int32, device=dev)
        nxt = torch.empty(B, dtype=torch.int32, device=dev)
        path = torch.empty((B, n), dtype=torch.int32, device=dev)
        smp = None
        keep = []
        if mode != "greedy":
            t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
            cid, cq = t(si.cand_ids), t(si.cand_q)
            ua, us = t(si.u_accept), t(si.u_sample)
            keep += [cid, cq, ua, us]
            smp = msd.Sampling(msd.MODES[mode], float(w.temperature), si.cand_ids.shape[-1],
                               cid.data_ptr(), cq.data_ptr(), ua.data_ptr(), us.data_ptr(), TOL_LOGIT)
        else:
            smp = msd.Sampling(msd.MSD_GREEDY, 1.0, 0, None, None, None, None, TOL_LOGIT)
        tie = torch.empty(B, dtype=torch.uint8, device=dev) if want_logits else None
        msd.accept(self.model.handle, blk, logits, argmax, smp, acc, nxt, path, self.cache.status,
                   ws=ws, near_tie=tie)
        k_com = v_com = None
        if commit:
            msd.kv_commit(self.model.handle, self.cache.c, blk, acc, path)
            torch.cuda.synchronize()
            k_com, v_com = self._rows(si.ctx_len, 1 + acc.cpu().numpy())
        torch.cuda.synchronize()
        return GpuResult(
            logits=logits.cpu().numpy() if logits is not None else None,
            argmax=argmax.cpu().numpy(), lse=lse.cpu().numpy(),
            ee_ids=ids.cpu().numpy() if ee else None, ee_logp=logp.cpu().numpy() if ee else None,
            acc_len=acc.cpu().numpy(), next_tok=nxt.cpu().numpy(), path=path.cpu().numpy(),
            len_after=self.cache.len.cpu().numpy(), status=int(self.cache.status.item()),
            k_rows=k_rows, v_rows=v_rows, near_tie=tie.cpu().numpy() if tie is not None else None,
            k_commit=k_com, v_commit=v_com)


@dataclasses.dataclass
class OracleSeq:
    logits: np.ndarray
    ee_ids: Optional[np.ndarray]
    ee_logp: Optional[np.ndarray]
    ee_margin: Optional[np.ndarray]
    blk_k: List[np.ndarray]
    blk_v: List[np.ndarray]
    acc: int
    nxt: int
    path: np.ndarray
    tie_depth: int = -1            # first depth with a path decision in a near-tie band
    tie_next: bool = False         # the next-token decision is in a band
    ee_logits: Optional[np.ndarray] = None  # [n, V] early-exit head logits


def oracle_sequence(shape, w: synth.Workload, si: synth.StepInputs, b: int, ee: bool = True,
                    weights: Optional[Dict[str, np.ndarray]] = None, mode: Optional[str] = None,
                    oracle_obj: Optional[orc.Oracle] = None) -> OracleSeq:
    """The oracle's verification step for sequence b of the workload."""
    o = oracle_obj or orc.Oracle(shape, weights if weights is not None else synth.host_weights(shape, w.seed))
    L = int(si.ctx_len[b])
    cache = {}

    def ctx(l):
        if l not in cache:
            cache.clear()
            cache[l] = (synth.host_ctx(shape, w.seed, l, "k", b, L), synth.host_ctx(shape, w.seed, l, "v", b, L))
        return cache[l]

    pos = L + orc.depths(si.parent)
    ee_layer = min(w.ee_layer, shape.n_layers - 1) if ee else None
    r = o.forward(si.tokens[b], pos, si.parent, ctx, L, ee_layer=ee_layer)
    ids = logp = marg = z_ee = None
    if ee:
        z_ee = o.head(r.x_ee)
        ids, logp, _ = orc.Oracle.topk(z_ee, w.kappa)
        marg = margins(z_ee, w.kappa)
    mode = mode or w.mode
    kw = {}
    if mode != "greedy":
        kw = dict(cand_ids=si.cand_ids[b], cand_q=si.cand_q[b], u_accept=si.u_accept[b],
                  u_sample=si.u_sample[b])
    A, nxt, path, td, tn = o.accept(si.parent, si.tokens[b], r.logits, mode, w.temperature,
                                    tol_logit=TOL_LOGIT, return_tie=True, **kw)
    return OracleSeq(r.logits, ids, logp, marg, r.blk_k, r.blk_v, A, nxt, path, td, tn, z_ee)


def margins(z: np.ndarray, k: int) -> np.ndarray:
    """Smallest gap among the k+1 largest logits of each row."""
    part = -np.sort(-z, axis=-1)[..., :k + 1]
    return np.min(part[..., :-1] - part[..., 1:], axis=-1)


def streaming_oracle(shape, seed: int, kv_cache_bf16: bool = True) -> orc.Oracle:
    """Oracle whose layer weights are regenerated on the host layer by layer."""
    glob = synth.host_weights(shape, seed, layers=[], with_globals=True)
    src = lambda l: synth.host_weights(shape, seed, layers=[l], with_globals=False)
    return orc.Oracle(shape, glob, layer_source=src, kv_cache_bf16=kv_cache_bf16)


def chain_inputs(si: synth.StepInputs, b: int, slots) -> synth.StepInputs:
    """The root-to-node chain through `slots` of sequence b as its own block."""
    slots = list(slots)
    toks = si.tokens[b, slots][None].astype(np.int32)
    par = np.arange(-1, len(slots) - 1, dtype=np.int32)
    return synth.StepInputs(parent=par, tokens=toks, ctx_len=si.ctx_len[b:b + 1].copy())


def oracle_runs(shape, w: synth.Workload, si: synth.StepInputs, specs, ee: bool = True,
                mode: Optional[str] = None) -> Dict[tuple, OracleSeq]:
    """Oracle steps for several (sequence b, kv_cache_bf16) pairs in lockstep
    over the layers, so each layer's weights are generated on the host once
    for all of them (full-depth workloads). Returns {(b, kv_cache_bf16): OracleSeq}."""
    glob = synth.host_weights(shape, w.seed, layers=[], with_globals=True)
    memo: Dict[int, Dict[str, np.ndarray]] = {}

    def src(l):
        if l not in memo:
            memo.clear()
            memo[l] = synth.host_weights(shape, w.seed, layers=[l], with_globals=False)
        return memo[l]

    oracles = {m: orc.Oracle(shape, glob, layer_source=src, kv_cache_bf16=m) for m in {m for _, m in specs}}
    ee_layer = min(w.ee_layer, shape.n_layers - 1) if ee else None
    state = {}
    for b, m in specs:
        pos = int(si.ctx_len[b]) + orc.depths(si.parent)
        state[(b, m)] = dict(x=oracles[m].embed(si.tokens[b], pos), pos=pos, k=[], v=[], x_ee=None)
    for l in range(shape.n_layers):
        for b in sorted({b for b, _ in specs}):
            L = int(si.ctx_len[b])
            ck = synth.host_ctx(shape, w.seed, l, "k", b, L) if L > 0 else None
            cv = synth.host_ctx(shape, w.seed, l, "v", b, L) if L > 0 else None
            for m in sorted({m for bb, m in specs if bb == b}):
                st = state[(b, m)]
                k, v = oracles[m].layer(l, st["x"], st["pos"], si.parent, ck, cv, L)
                st["k"].append(k)
                st["v"].append(v)
                if ee_layer is not None and l + 1 == ee_layer:
                    st["x_ee"] = st["x"].copy()
    mode = mode or w.mode
    out = {}
    for (b, m), st in state.items():
        o = oracles[m]
        logits = o.head(st["x"])
        ids = logp = marg = z_ee = None
        if ee:
            z_ee = o.head(st["x_ee"])
            ids, logp, _ = orc.Oracle.topk(z_ee, w.kappa)
            marg = margins(z_ee, w.kappa)
        kw = {}
        if mode != "greedy":
            kw = dict(cand_ids=si.cand_ids[b], cand_q=si.cand_q[b], u_accept=si.u_accept[b],
                      u_sample=si.u_sample[b])
        A, nxt, path, td, tn = o.accept(si.parent, si.tokens[b], logits, mode, w.temperature,
                                        tol_logit=TOL_LOGIT, return_tie=True, **kw)
        out[(b, m)] = OracleSeq(logits, ids, logp, marg, st["k"], st["v"], A, nxt, path, td, tn, z_ee)
    return out
