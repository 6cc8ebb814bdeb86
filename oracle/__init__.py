"""Python face of the msdo oracle (fp64 C, ``oracle/msdo.c``).

TEST INFRASTRUCTURE ONLY: the test suite, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg use it; the product path never does.

The functions here only marshal arrays into the C oracle and sequence its
per-layer calls; every number of the verification pass comes from
``msdo.c``. The step after acceptance (the Sec. 3.1 reuse criterion over the
draft's hypothesis tree, the App. E overlap mass) is written at the end of
this file in plain Python and NumPy fp64. The model description and weights
come from the shared input generator (``synth``), which holds none of the
method's arithmetic.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass
from typing import Callable, Dict, List, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmsdo.so")

GREEDY, REJECTION, MATCH = 0, 1, 2
MODES = {"greedy": GREEDY, "rejection": REJECTION, "match": MATCH}


def build(verbose: bool = False) -> str:
    """Compile msdo.c into libmsdo.so (gcc, OpenMP, no FP contraction)."""
    cmd = ["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off", "-std=c11",
           "-Wall", "-Wextra", "-o", LIB_PATH, os.path.join(_HERE, "msdo.c"), "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    return LIB_PATH


class _Cfg(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("n_layers", "d_model", "n_heads", "n_kv_heads", "head_dim", "d_ffn", "vocab",
                 "layer_norm", "relu_ffn", "learned_pos", "has_bias")] + \
               [("rope_theta", ctypes.c_double), ("norm_eps", ctypes.c_double)]


_U16P = ctypes.POINTER(ctypes.c_uint16)


class _LayerW(ctypes.Structure):
    _fields_ = [(n, _U16P) for n in
                ("attn_g", "attn_b", "wq", "wk", "wv", "bq", "bk", "bv", "wo", "bo",
                 "mlp_g", "mlp_b", "w_gate", "w_up", "b_up", "w_down", "b_down")]


class _GlobalW(ctypes.Structure):
    _fields_ = [(n, _U16P) for n in ("embed", "pos_embed", "final_g", "final_b", "lm_head")]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run oracle.build()")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        i32 = ctypes.c_int32
        L.msdo_embed.argtypes = [P, P, i32, P, P, P]
        L.msdo_layer.argtypes = [P, P, i32, P, P, P, i32, i32, P, P, i32, P, P, P, P, i32]
        L.msdo_head.argtypes = [P, P, i32, P, P]
        L.msdo_topk.argtypes = [i32, i32, P, i32, P, P, P]
        L.msdo_accept.argtypes = [i32, P, P, i32, P, i32, ctypes.c_double, i32, P, P, P, P,
                                  ctypes.c_double, P, P, P, P, P]
        L.msdo_accept.restype = i32
        L.msdo_kv_commit.argtypes = [i32, i32, i32, i32, P, P, i32, i32, P]
        L.msdo_kv_commit.restype = i32
        for f in (L.msdo_embed, L.msdo_layer, L.msdo_head, L.msdo_topk):
            f.restype = None
        _lib = L
    return _lib


def _gomp():
    lib()  # the oracle's OpenMP runtime is the one it was linked with
    g = ctypes.CDLL("libgomp.so.1")
    g.omp_get_max_threads.restype = ctypes.c_int
    g.omp_set_num_threads.argtypes = [ctypes.c_int]
    return g


def omp_threads() -> int:
    """Threads the oracle's parallel loops use."""
    return int(_gomp().omp_get_max_threads())


def set_omp_threads(n: int) -> None:
    _gomp().omp_set_num_threads(int(n))


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


def _u16(a):
    if a is None:
        return None
    a = np.ascontiguousarray(a, dtype=np.uint16)
    return a


@dataclass
class ForwardResult:
    logits: Optional[np.ndarray]        # [n, V] float64
    x_ee: Optional[np.ndarray]          # [n, d] residual after the early-exit layer
    x_final: np.ndarray                 # [n, d]
    blk_k: List[np.ndarray]             # per layer [n, Hkv, hd] float64
    blk_v: List[np.ndarray]


class Oracle:
    """fp64 reference of the target model's verification pass.

    shape    a ``synth.ModelShape`` (sizes, norm/activation/position kinds)
    weights  dict name -> uint16 bf16 bits for global tensors, and either the
             layer tensors too or ``layer_source(l) -> dict`` to stream them.
    kv_cache_bf16  the block's keys/values are stored in the KV cache's bf16
             format before they are attended to (the cache holds the given
             context in that format); False keeps them at fp64.
    """

    def __init__(self, shape, weights: Dict[str, np.ndarray],
                 layer_source: Optional[Callable[[int], Dict[str, np.ndarray]]] = None,
                 kv_cache_bf16: bool = True):
        self.m = shape
        self.kv_cache_bf16 = int(kv_cache_bf16)
        self.cfg = _Cfg(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads,
                        shape.head_dim, shape.d_ffn, shape.vocab,
                        int(shape.norm == "layer"), int(shape.act == "relu"),
                        int(shape.pos == "learned"), int(shape.bias),
                        float(shape.rope_theta), float(shape.norm_eps))
        self.w = weights
        self.layer_source = layer_source
        self._keep = []
        g = _GlobalW()
        for field, name in (("embed", "embed"), ("pos_embed", "pos_embed"),
                            ("final_g", "final_norm.g"), ("final_b", "final_norm.b")):
            setattr(g, field, self._ptr(weights.get(name)))
        head = weights.get("lm_head", weights["embed"]) if shape.tied_head else weights["lm_head"]
        g.lm_head = self._ptr(head)
        self.gw = g

    def _ptr(self, a):
        if a is None:
            return None
        a = _u16(a)
        self._keep.append(a)
        return ctypes.cast(a.ctypes.data, _U16P)

    def _layer_struct(self, l: int) -> Tuple[_LayerW, list]:
        src = self.layer_source(l) if self.layer_source else self.w
        p = f"l{l}."
        keep = []

        def ptr(name):
            a = src.get(p + name)
            if a is None:
                return None
            a = _u16(a)
            keep.append(a)
            return ctypes.cast(a.ctypes.data, _U16P)

        w = _LayerW()
        for field, name in (("attn_g", "attn_norm.g"), ("attn_b", "attn_norm.b"), ("wq", "wq"),
                            ("wk", "wk"), ("wv", "wv"), ("bq", "bq"), ("bk", "bk"), ("bv", "bv"),
                            ("wo", "wo"), ("bo", "bo"), ("mlp_g", "mlp_norm.g"),
                            ("mlp_b", "mlp_norm.b"), ("w_gate", "w_gate"), ("w_up", "w_up"),
                            ("b_up", "b_up"), ("w_down", "w_down"), ("b_down", "b_down")):
            setattr(w, field, ptr(name))
        return w, keep

    # -- primitives ---------------------------------------------------------
    def embed(self, tokens: np.ndarray, pos: np.ndarray) -> np.ndarray:
        tokens = np.ascontiguousarray(tokens, dtype=np.int32)
        pos = np.ascontiguousarray(pos, dtype=np.int32)
        x = np.zeros((len(tokens), self.m.d_model), dtype=np.float64)
        lib().msdo_embed(ctypes.byref(self.cfg), ctypes.byref(self.gw), len(tokens),
                         _p(tokens), _p(pos), _p(x))
        return x

    def layer(self, l: int, x: np.ndarray, pos, parent, ctx_k=None, ctx_v=None, n_ctx: int = 0,
              extra_k=None, extra_v=None) -> Tuple[np.ndarray, np.ndarray]:
        """One layer in place on x; returns the block's (k, v) rows."""
        m = self.m
        n = x.shape[0]
        pos = np.ascontiguousarray(pos, dtype=np.int32)
        parent = np.ascontiguousarray(parent, dtype=np.int32)
        blk_k = np.zeros((n, m.n_kv_heads, m.head_dim), dtype=np.float64)
        blk_v = np.zeros_like(blk_k)
        if n_ctx > 0:
            ctx_k = _u16(ctx_k)
            ctx_v = _u16(ctx_v)
            assert ctx_k.shape[0] == m.n_kv_heads and ctx_k.shape[2] == m.head_dim
            assert ctx_k.shape[1] >= n_ctx and ctx_v.shape == ctx_k.shape
            stride = ctx_k.shape[1]
        else:
            ctx_k = ctx_v = None
            stride = 0
        n_extra = 0 if extra_k is None else extra_k.shape[0]
        if n_extra:
            extra_k = np.ascontiguousarray(extra_k, dtype=np.float64)
            extra_v = np.ascontiguousarray(extra_v, dtype=np.float64)
        w, keep = self._layer_struct(l)
        lib().msdo_layer(ctypes.byref(self.cfg), ctypes.byref(w), n, _p(x), _p(pos), _p(parent),
                         n_ctx, stride, _p(ctx_k), _p(ctx_v), n_extra,
                         _p(extra_k) if n_extra else None, _p(extra_v) if n_extra else None,
                         _p(blk_k), _p(blk_v), self.kv_cache_bf16)
        del keep
        return blk_k, blk_v

    def head(self, x: np.ndarray) -> np.ndarray:
        x = np.ascontiguousarray(x, dtype=np.float64)
        logits = np.zeros((x.shape[0], self.m.vocab), dtype=np.float64)
        lib().msdo_head(ctypes.byref(self.cfg), ctypes.byref(self.gw), x.shape[0], _p(x),
                        _p(logits))
        return logits

    # -- composed pass --------------------------------------------------------
    def forward(self, tokens, pos, parent, ctx: Optional[Callable[[int], Tuple[np.ndarray, np.ndarray]]] = None,
                n_ctx: int = 0, extra: Optional[Sequence[Tuple[np.ndarray, np.ndarray]]] = None,
                ee_layer: Optional[int] = None, want_logits: bool = True) -> ForwardResult:
        """Embed -> layers 1..N -> final head, for one sequence's block.

        ctx(l) returns (k, v) uint16 [Hkv][stride][hd] of the cached context of
        layer l; extra[l] = (k, v) fp64 [n_extra][Hkv][hd] rows after it.
        ee_layer (1-indexed) records the residual after that layer.
        """
        x = self.embed(tokens, pos)
        blk_k, blk_v = [], []
        x_ee = None
        for l in range(self.m.n_layers):
            ck, cv = ctx(l) if (ctx is not None and n_ctx > 0) else (None, None)
            ek, ev = extra[l] if extra is not None else (None, None)
            k, v = self.layer(l, x, pos, parent, ck, cv, n_ctx, ek, ev)
            blk_k.append(k)
            blk_v.append(v)
            if ee_layer is not None and l + 1 == ee_layer:
                x_ee = x.copy()
        logits = self.head(x) if want_logits else None
        return ForwardResult(logits, x_ee, x.copy(), blk_k, blk_v)

    # -- token-level operations -------------------------------------------------
    @staticmethod
    def topk(logits: np.ndarray, kappa: int):
        logits = np.ascontiguousarray(logits, dtype=np.float64)
        n, V = logits.shape
        ids = np.zeros((n, kappa), dtype=np.int32)
        logp = np.zeros((n, kappa), dtype=np.float64)
        lse = np.zeros(n, dtype=np.float64)
        lib().msdo_topk(n, V, _p(logits), kappa, _p(ids), _p(logp), _p(lse))
        return ids, logp, lse

    def early_exit(self, x_ee: np.ndarray, kappa: int):
        """Sec. 3.1 token channel: Top-kappa of Softmax(W_LM norm_f(h^(l_e)))."""
        return self.topk(self.head(x_ee), kappa)

    @staticmethod
    def accept(parent, tokens, logits, mode="greedy", temperature=1.0, cand_ids=None,
               cand_q=None, u_accept=None, u_sample=None, tol_logit: float = 0.0,
               return_tie: bool = False):
        """App. B acceptance over one sequence's block: (A, next token, path).
        With return_tie, also (tie_depth, tie_next): the depth of the first
        node where a decision choosing the way down lies in a near-tie band
        of tol_logit (-1 if none), and whether the decision that produced the
        next token does (bands in msdo.c)."""
        parent = np.ascontiguousarray(parent, dtype=np.int32)
        tokens = np.ascontiguousarray(tokens, dtype=np.int32)
        logits = np.ascontiguousarray(logits, dtype=np.float64)
        n, V = logits.shape
        md = MODES[mode] if isinstance(mode, str) else int(mode)
        n_cand = 0 if cand_ids is None else cand_ids.shape[-1]
        cand_ids = None if cand_ids is None else np.ascontiguousarray(cand_ids, dtype=np.int32)
        cand_q = None if cand_q is None else np.ascontiguousarray(cand_q, dtype=np.float32)
        u_accept = None if u_accept is None else np.ascontiguousarray(u_accept, dtype=np.float32)
        u_sample = None if u_sample is None else np.ascontiguousarray(u_sample, dtype=np.float32)
        A = np.zeros(1, dtype=np.int32)
        nxt = np.zeros(1, dtype=np.int32)
        tie = np.zeros(1, dtype=np.int32)
        tie_next = np.zeros(1, dtype=np.int32)
        path = np.zeros(n + 1, dtype=np.int32)
        rc = lib().msdo_accept(n, _p(parent), _p(tokens), V, _p(logits), md, float(temperature),
                               n_cand, _p(cand_ids), _p(cand_q), _p(u_accept), _p(u_sample),
                               float(tol_logit), _p(A), _p(nxt), _p(path), _p(tie),
                               _p(tie_next))
        if rc != 0:
            raise ValueError("draft token outside its parent's candidate set")
        a = int(A[0])
        if return_tie:
            return a, int(nxt[0]), path[:a + 1].copy(), int(tie[0]), bool(tie_next[0])
        return a, int(nxt[0]), path[:a + 1].copy()

    @staticmethod
    def kv_commit(k: np.ndarray, v: np.ndarray, length: int, acc_len: int, path) -> int:
        """In place on uint16 caches [L][Hkv][cap][hd] of one sequence."""
        assert k.dtype == np.uint16 and v.dtype == np.uint16
        assert k.flags.c_contiguous and v.flags.c_contiguous and k.shape == v.shape
        L, H, cap, hd = k.shape
        path = np.ascontiguousarray(path, dtype=np.int32)
        assert length + acc_len < cap
        return int(lib().msdo_kv_commit(L, H, cap, hd, _p(k), _p(v), length, acc_len, _p(path)))

    # -- brute force ----------------------------------------------------------------
    def decode_greedy(self, root_token: int, start_pos: int, steps: int,
                      ctx: Optional[Callable[[int], Tuple[np.ndarray, np.ndarray]]] = None,
                      n_ctx: int = 0, return_kv: bool = False):
        """Token-by-token argmax decoding (Sec. 2 AR factorisation) from a root.

        Returns the tokens y_1..y_steps and the per-step logits; every step is
        a one-row forward whose earlier rows are committed as extra cache rows.
        With return_kv, also the rows each step wrote: per layer fp64
        [steps][n_kv_heads][head_dim] keys and values (row s at start_pos + s).
        """
        L = self.m.n_layers
        extra_k: List[List[np.ndarray]] = [[] for _ in range(L)]
        extra_v: List[List[np.ndarray]] = [[] for _ in range(L)]
        tok = int(root_token)
        out, all_logits = [], []
        for s in range(steps):
            ex = None
            if s > 0:
                ex = [(np.concatenate(extra_k[l], 0), np.concatenate(extra_v[l], 0))
                      for l in range(L)]
            r = self.forward(np.array([tok]), np.array([start_pos + s]), np.array([-1]),
                             ctx, n_ctx, ex)
            for l in range(L):
                extra_k[l].append(r.blk_k[l])
                extra_v[l].append(r.blk_v[l])
            z = r.logits[0]
            tok = int(np.argmax(z))
            out.append(tok)
            all_logits.append(z)
        y, zs = np.array(out, dtype=np.int32), np.stack(all_logits)
        if return_kv:
            ks = [np.concatenate(extra_k[l], 0) for l in range(L)]
            vs = [np.concatenate(extra_v[l], 0) for l in range(L)]
            return y, zs, ks, vs
        return y, zs


def depths(parent: np.ndarray) -> np.ndarray:
    """depth[0] = 0, depth[i] = depth[parent[i]] + 1 (Sec. 3.1: depth r holds position t + r)."""
    d = np.zeros(len(parent), dtype=np.int32)
    for i in range(1, len(parent)):
        d[i] = d[parent[i]] + 1
    return d


# ---------------------------------------------------------------------------
# After acceptance: reuse criterion and next-window selection (Sec. 3.1),
# fallback statistics (App. E). Plain Python over the hypothesis tree (a few
# hundred nodes at most), NumPy fp64 for the overlap mass.
# ---------------------------------------------------------------------------
NEXT_BRANCH, NEXT_CONTINUE, NEXT_FRESH = 0, 1, 2


def tree_path(parent: Sequence[int], tokens: Sequence[int], v: int) -> List[int]:
    """Tokens on the root-to-node path of node v of a hypothesis tree, root
    first (the root at depth 1 holds the token for position t + 1)."""
    seq = []
    while v != -1:
        seq.append(int(tokens[v]))
        v = int(parent[v])
    return seq[::-1]


def reuse_select(parent: Sequence[int], tokens: Sequence[int], accepted: Sequence[int],
                 correction: int) -> Tuple[int, int]:
    """Sec. 3.1: with the accepted prefix Pi_t (A tokens) and the correction
    c at tau = A + 1, reuse happens iff Pi_t^+ = (Pi_t, c) is a root-to-depth-
    tau path of the hypothesis tree T_t. The next window is then the branch
    rooted at c (A = 0) or the precomputed continuation at depth tau along
    Pi_t (A >= 1); otherwise a fresh rollout. Returns (case, node): the case
    (NEXT_BRANCH / NEXT_CONTINUE / NEXT_FRESH) and the smallest node whose
    path is Pi_t^+, or -1."""
    target = [int(x) for x in accepted] + [int(correction)]
    for v in range(len(parent)):
        if tree_path(parent, tokens, v) == target:
            return (NEXT_BRANCH if len(accepted) == 0 else NEXT_CONTINUE), v
    return NEXT_FRESH, -1


def overlap_mass(logits_row: np.ndarray, ids: Sequence[int]) -> float:
    """Sec. 3.1 (sampling width at early exit), App. E: Omega_kappa = sum
    over the early-exit Top-kappa ids of
    q(y) = Softmax(logits)(y), the final head's next-token law, in fp64."""
    z = np.asarray(logits_row, dtype=np.float64)
    mx = z.max()
    lse = mx + np.log(np.exp(z - mx).sum())
    return float(sum(np.exp(z[int(y)] - lse) for y in ids))

