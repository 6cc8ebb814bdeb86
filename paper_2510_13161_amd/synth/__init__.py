"""Seeded synthetic inputs for the verification step.

This module owns every input both the HIP path and the oracle consume, and
none of the method's arithmetic:

* model shapes and workloads (the tiny parity model, the 14B-shaped chain,
  tree and batch-16 workloads, the 66B-shaped tree workload);
* big tensors (weights, KV context) from a counter-based generator whose host
  (``synth_host.c``) and device (``synth_dev.hip``) implementations agree bit
  for bit, so any slice can be regenerated on the host for the oracle;
* small inputs (root and draft tokens, tree topology, draft candidates and
  their Dirichlet probabilities, uniforms, context lengths) from NumPy
  ``SeedSequence`` streams keyed by name.

Draft tokens are inputs: the draft model itself is outside the verification
step (the paper's draft runs on other devices, overlapped with the target).
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
HOST_LIB = os.path.join(_HERE, "libmsd_synth_host.so")
DEV_LIB = os.path.join(_HERE, "libmsd_synth_dev.so")

MASK64 = (1 << 64) - 1
GOLDEN = 0x9E3779B97F4A7C15
# Irwin-Hall sum of 8 discrete uniforms on [0, 65535]: 2S - 524280 has
# standard deviation 2 * sqrt(8 * (65536**2 - 1) / 12).
_SIGMA_2S = 2.0 * math.sqrt(8.0 * (65536.0 ** 2 - 1.0) / 12.0)
CTX_POS_BITS = 20  # positions per (sequence, head) in the context index space


# ----------------------------------------------------------------------------
# shapes and workloads
# ----------------------------------------------------------------------------
@dataclass(frozen=True)
class ModelShape:
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ffn: int
    vocab: int
    norm: str = "rms"          # "rms" | "layer"
    act: str = "swiglu"        # "swiglu" | "relu"
    pos: str = "rope"          # "rope" | "learned"
    bias: bool = False
    tied_head: bool = False
    rope_theta: float = 1.0e4
    norm_eps: float = 1.0e-6
    max_positions: int = 0     # rows of the learned position table
    init_std: float = 0.02

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    def with_layers(self, n_layers: int) -> "ModelShape":
        d = dict(self.__dict__)
        d["n_layers"] = n_layers
        d["name"] = f"{self.name}-L{n_layers}"
        return ModelShape(**d)

    def weight_bytes(self) -> int:
        return sum(int(np.prod(s.shape)) * 2 for s in tensor_specs(self))


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelShape
    batch: int
    ctx: Tuple[int, int]        # (lo, hi) inclusive range of committed context lengths
    topology: str               # "chain" | "tree" | "forest" (the explicit parents below)
    gamma: int                  # chain length, or tree depth
    branches: int = 1           # tree: number of branches at the root
    ee_layer: int = 1           # early exit after this layer (1-indexed)
    kappa: int = 4              # early-exit top-kappa
    mode: str = "greedy"        # "greedy" | "rejection" | "match"
    temperature: float = 1.0
    n_cand: int = 32
    seed: int = 0
    parents: Optional[Tuple[int, ...]] = None  # "forest": parent[i] < i, parent[0] = -1

    @property
    def n_slots(self) -> int:
        if self.topology == "forest":
            return len(self.parents)
        if self.topology == "chain":
            return self.gamma + 1
        return 1 + self.branches * self.gamma

    @property
    def rows(self) -> int:
        return self.batch * self.n_slots

    @property
    def draft_tokens(self) -> int:
        return self.batch * (self.n_slots - 1)

    def with_model(self, model: ModelShape, **kw) -> "Workload":
        d = dict(self.__dict__)
        d["model"] = model
        d.update(kw)
        return Workload(**d)


TINY = ModelShape("tiny", 2, 256, 4, 4, 64, 1024, 4096, rope_theta=1.0e4)
QWEN14B = ModelShape("14b", 48, 5120, 40, 8, 128, 13824, 152064, rope_theta=1.0e6)
OPT66B = ModelShape("66b", 64, 9216, 72, 72, 128, 36864, 50272, norm="layer", act="relu",
                    pos="learned", bias=True, tied_head=True, norm_eps=1.0e-5,
                    max_positions=4096)
# a 0.6B-shaped draft decoder on the 14B target's vocabulary (tied head)
DRAFT06B = ModelShape("0.6b", 28, 1024, 16, 8, 128, 3072, 152064, tied_head=True,
                      rope_theta=1.0e6)

WORKLOADS: Dict[str, Workload] = {
    "tiny_chain": Workload("tiny_chain", TINY, 1, (128, 128), "chain", 4, ee_layer=1, kappa=4,
                           seed=0),
    "14b_chain": Workload("14b_chain", QWEN14B, 1, (1024, 1024), "chain", 8, ee_layer=36,
                          kappa=8, seed=1),
    "14b_tree": Workload("14b_tree", QWEN14B, 1, (4096, 4096), "tree", 6, branches=4,
                         ee_layer=36, kappa=4, mode="rejection", temperature=1.0, seed=2),
    "14b_batch16": Workload("14b_batch16", QWEN14B, 16, (512, 8192), "chain", 8, ee_layer=36,
                            kappa=4, seed=3),
    "66b_tree": Workload("66b_tree", OPT66B, 1, (2048, 2048), "tree", 8, branches=4,
                         ee_layer=48, kappa=8, seed=4),
}


# ----------------------------------------------------------------------------
# tensor inventory
# ----------------------------------------------------------------------------
@dataclass(frozen=True)
class TensorSpec:
    name: str
    shape: Tuple[int, ...]
    init: str          # "normal" | "ones" | "zeros"
    std: float = 0.0


def layer_tensor_specs(m: ModelShape, l: int) -> List[TensorSpec]:
    d, F = m.d_model, m.d_ffn
    s = m.init_std
    p = f"l{l}."
    out = [TensorSpec(p + "attn_norm.g", (d,), "ones")]
    if m.norm == "layer":
        out.append(TensorSpec(p + "attn_norm.b", (d,), "zeros"))
    out += [TensorSpec(p + "wq", (m.q_dim, d), "normal", s),
            TensorSpec(p + "wk", (m.kv_dim, d), "normal", s),
            TensorSpec(p + "wv", (m.kv_dim, d), "normal", s)]
    if m.bias:
        out += [TensorSpec(p + "bq", (m.q_dim,), "normal", s),
                TensorSpec(p + "bk", (m.kv_dim,), "normal", s),
                TensorSpec(p + "bv", (m.kv_dim,), "normal", s)]
    out.append(TensorSpec(p + "wo", (d, m.q_dim), "normal", s))
    if m.bias:
        out.append(TensorSpec(p + "bo", (d,), "normal", s))
    out.append(TensorSpec(p + "mlp_norm.g", (d,), "ones"))
    if m.norm == "layer":
        out.append(TensorSpec(p + "mlp_norm.b", (d,), "zeros"))
    if m.act == "swiglu":
        out += [TensorSpec(p + "w_gate", (F, d), "normal", s),
                TensorSpec(p + "w_up", (F, d), "normal", s),
                TensorSpec(p + "w_down", (d, F), "normal", s)]
    else:
        out += [TensorSpec(p + "w_up", (F, d), "normal", s)]
        if m.bias:
            out.append(TensorSpec(p + "b_up", (F,), "normal", s))
        out.append(TensorSpec(p + "w_down", (d, F), "normal", s))
        if m.bias:
            out.append(TensorSpec(p + "b_down", (d,), "normal", s))
    return out


def global_tensor_specs(m: ModelShape) -> List[TensorSpec]:
    d, s = m.d_model, m.init_std
    out = [TensorSpec("embed", (m.vocab, d), "normal", s)]
    if m.pos == "learned":
        out.append(TensorSpec("pos_embed", (m.max_positions, d), "normal", s))
    out.append(TensorSpec("final_norm.g", (d,), "ones"))
    if m.norm == "layer":
        out.append(TensorSpec("final_norm.b", (d,), "zeros"))
    if not m.tied_head:
        out.append(TensorSpec("lm_head", (m.vocab, d), "normal", s))
    return out


def tensor_specs(m: ModelShape) -> List[TensorSpec]:
    out = global_tensor_specs(m)
    for l in range(m.n_layers):
        out += layer_tensor_specs(m, l)
    return out


def kv_std(m: ModelShape) -> float:
    """Scale of the synthetic cached K/V: that of a projection of a unit-RMS row."""
    return m.init_std * math.sqrt(m.d_model)


# ----------------------------------------------------------------------------
# counter-based generator: key derivation and a NumPy reference of it
# ----------------------------------------------------------------------------
def fnv1a64(text: str) -> int:
    """FNV-1a 64-bit hash (Fowler, Noll, Vo) of the UTF-8 bytes of `text`."""
    h = 0xCBF29CE484222325
    for b in text.encode("utf-8"):
        h ^= b
        h = (h * 0x100000001B3) & MASK64
    return h


def mix64(z: int) -> int:
    z &= MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def tensor_key(seed: int, name: str) -> int:
    return mix64(fnv1a64(name) ^ mix64(seed))


def scale_for(std: float) -> float:
    """fp32 multiplier turning the integer 2S - 524280 into N(0, std)."""
    return float(np.float32(std / _SIGMA_2S))


def _np_mix64(z: np.ndarray) -> np.ndarray:
    z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
    z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
    return z ^ (z >> np.uint64(31))


def np_values(key: int, idx: np.ndarray, std: float) -> np.ndarray:
    """Reference (NumPy) implementation of the generator: bf16 bits as uint16."""
    idx = idx.astype(np.uint64)
    with np.errstate(over="ignore"):
        g = np.uint64(GOLDEN)
        k = np.uint64(key)
        a = _np_mix64(k + (np.uint64(2) * idx + np.uint64(1)) * g)
        b = _np_mix64(k + (np.uint64(2) * idx + np.uint64(2)) * g)
    s = np.zeros(idx.shape, dtype=np.int64)
    for j in range(4):
        sh = np.uint64(16 * j)
        s += ((a >> sh) & np.uint64(0xFFFF)).astype(np.int64)
        s += ((b >> sh) & np.uint64(0xFFFF)).astype(np.int64)
    v = (2 * s - 524280).astype(np.float32) * np.float32(scale_for(std))
    u = v.view(np.uint32).astype(np.uint64)
    u = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return u.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return u.astype(np.uint16)


BF16_ONE = 0x3F80
BF16_ZERO = 0x0000


# ----------------------------------------------------------------------------
# host generation (C + OpenMP)
# ----------------------------------------------------------------------------
_host = None


def _host_lib():
    global _host
    if _host is None:
        if not os.path.exists(HOST_LIB):
            raise RuntimeError(f"{HOST_LIB} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(HOST_LIB)
        lib.sy_fill_linear.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint64,
                                       ctypes.c_int64, ctypes.c_float]
        lib.sy_fill_linear.restype = None
        lib.sy_fill_ctx.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int32,
                                    ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                    ctypes.c_float]
        lib.sy_fill_ctx.restype = None
        _host = lib
    return _host


def host_tensor(seed: int, spec: TensorSpec) -> np.ndarray:
    """bf16 bits (uint16) of one named tensor, generated on the host."""
    n = int(np.prod(spec.shape))
    if spec.init == "ones":
        return np.full(spec.shape, BF16_ONE, dtype=np.uint16)
    if spec.init == "zeros":
        return np.zeros(spec.shape, dtype=np.uint16)
    out = np.empty(n, dtype=np.uint16)
    _host_lib().sy_fill_linear(out.ctypes.data, tensor_key(seed, spec.name), 0, n,
                               scale_for(spec.std))
    return out.reshape(spec.shape)


def host_weights(m: ModelShape, seed: int, layers: Optional[Sequence[int]] = None,
                 with_globals: bool = True) -> Dict[str, np.ndarray]:
    out: Dict[str, np.ndarray] = {}
    if with_globals:
        for s in global_tensor_specs(m):
            out[s.name] = host_tensor(seed, s)
    for l in (range(m.n_layers) if layers is None else layers):
        for s in layer_tensor_specs(m, l):
            out[s.name] = host_tensor(seed, s)
    return out


def ctx_key(seed: int, layer: int, which: str) -> int:
    return tensor_key(seed, f"ctx_{which}/l{layer}")


def host_ctx(m: ModelShape, seed: int, layer: int, which: str, seq: int, n_pos: int) -> np.ndarray:
    """Synthetic cached K or V of one sequence and layer: uint16 [Hkv][n_pos][hd]."""
    out = np.empty((m.n_kv_heads, n_pos, m.head_dim), dtype=np.uint16)
    if n_pos > 0:
        _host_lib().sy_fill_ctx(out.ctypes.data, ctx_key(seed, layer, which), seq,
                                m.n_kv_heads, n_pos, m.head_dim, scale_for(kv_std(m)))
    return out


def np_ctx(m: ModelShape, seed: int, layer: int, which: str, seq: int, n_pos: int) -> np.ndarray:
    """NumPy reference of host_ctx (small sizes only)."""
    h = np.arange(m.n_kv_heads, dtype=np.uint64)[:, None, None]
    p = np.arange(n_pos, dtype=np.uint64)[None, :, None]
    j = np.arange(m.head_dim, dtype=np.uint64)[None, None, :]
    row = ((np.uint64(seq) * np.uint64(m.n_kv_heads) + h) << np.uint64(CTX_POS_BITS)) | p
    idx = row * np.uint64(m.head_dim) + j
    return np_values(ctx_key(seed, layer, which), idx, kv_std(m))


# ----------------------------------------------------------------------------
# small inputs (NumPy SeedSequence streams keyed by name)
# ----------------------------------------------------------------------------
def rng(seed: int, name: str) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, fnv1a64(name) & 0xFFFFFFFF,
                                                                       fnv1a64(name) >> 32])))


def topology(w: Workload) -> np.ndarray:
    """parent[] of the block (slot 0 = root, parent[0] = -1, parent[i] < i).

    Chain: parent[i] = i - 1. Tree: `branches` chains of depth `gamma` hang
    off the root, branch-major (slot 1 + b*gamma + r - 1 holds branch b at
    depth r), which is the branch-complete rollout shape of the paper's
    Eq. (branch-complete) seen from the verifier.
    """
    n = w.n_slots
    if w.topology == "forest":
        par = np.asarray(w.parents, dtype=np.int32)
        if par[0] != -1 or any(not 0 <= par[i] < i for i in range(1, n)):
            raise ValueError("parents must satisfy parent[0] = -1 and 0 <= parent[i] < i")
        return par
    par = np.empty(n, dtype=np.int32)
    par[0] = -1
    if w.topology == "chain":
        par[1:] = np.arange(n - 1, dtype=np.int32)
    else:
        for b in range(w.branches):
            for r in range(1, w.gamma + 1):
                s = 1 + b * w.gamma + (r - 1)
                par[s] = 0 if r == 1 else s - 1
    return par


def ctx_lens(w: Workload) -> np.ndarray:
    lo, hi = w.ctx
    if lo == hi:
        return np.full(w.batch, lo, dtype=np.int32)
    return rng(w.seed, "ctx_lens").integers(lo, hi + 1, size=w.batch).astype(np.int32)


@dataclass
class StepInputs:
    """Everything one verification step consumes besides weights and cache."""
    parent: np.ndarray            # int32 [n_slots]
    tokens: np.ndarray            # int32 [batch, n_slots] (slot 0 = root)
    ctx_len: np.ndarray           # int32 [batch]
    cand_ids: Optional[np.ndarray] = None   # int32 [batch, n_slots, n_cand]
    cand_q: Optional[np.ndarray] = None     # float32 [batch, n_slots, n_cand]
    u_accept: Optional[np.ndarray] = None   # float32 [batch, n_slots]
    u_sample: Optional[np.ndarray] = None   # float32 [batch, n_slots]


def uniforms01(g: np.random.Generator, shape) -> np.ndarray:
    """fp32 uniforms on [0, 1) drawn as 24-bit integers, so none rounds to 1.0."""
    return (g.integers(0, 1 << 24, size=shape, dtype=np.int64).astype(np.float32)
            * np.float32(1.0 / (1 << 24)))


def dirichlet_rows(g: np.random.Generator, alpha: float, shape) -> np.ndarray:
    """Dirichlet(alpha * 1) rows as fp32 summing to 1 with no zero entry."""
    q = g.dirichlet(np.full(shape[-1], alpha), size=shape[:-1]).astype(np.float64)
    q = np.maximum(q, np.finfo(np.float32).tiny)
    q = q / q.sum(axis=-1, keepdims=True)
    q32 = q.astype(np.float32)
    q32 = (q32 / q32.sum(axis=-1, keepdims=True, dtype=np.float64)).astype(np.float32)
    assert np.all(q32 > 0)
    assert np.all(np.abs(q32.sum(axis=-1, dtype=np.float64) - 1.0) < 1e-6)
    return q32


def step_inputs(w: Workload) -> StepInputs:
    V = w.model.vocab
    par = topology(w)
    B, n = w.batch, w.n_slots
    lens = ctx_lens(w)
    tokens = np.empty((B, n), dtype=np.int32)
    tokens[:, 0] = rng(w.seed, "root").integers(0, V, size=B)
    si = StepInputs(parent=par, tokens=tokens, ctx_len=lens)
    if w.mode == "greedy":
        tokens[:, 1:] = rng(w.seed, "drafts").integers(0, V, size=(B, n - 1))
        return si
    # stochastic modes: every node carries a sparse draft distribution over
    # n_cand distinct candidate ids; children are drawn from their parent's.
    gc = rng(w.seed, "cands")
    cand = np.empty((B, n, w.n_cand), dtype=np.int32)
    for b in range(B):
        for s in range(n):
            cand[b, s] = gc.choice(V, size=w.n_cand, replace=False)
    q = dirichlet_rows(rng(w.seed, "dirichlet"), 0.1, (B, n, w.n_cand))
    gd = rng(w.seed, "drafts")
    children = [[c for c in range(n) if par[c] == s] for s in range(n)]
    for b in range(B):
        for s in range(n):
            kids = children[s]
            if not kids:
                continue
            pick = gd.choice(w.n_cand, size=len(kids), replace=False,
                             p=q[b, s].astype(np.float64) / q[b, s].sum(dtype=np.float64))
            for c, j in zip(kids, pick):
                tokens[b, c] = cand[b, s, j]
    si.cand_ids, si.cand_q = cand, q
    si.u_accept = uniforms01(rng(w.seed, "u_accept"), (B, n))
    si.u_sample = uniforms01(rng(w.seed, "u_sample"), (B, n))
    return si


def prompt_tokens(w: Workload, seq: int = 0) -> np.ndarray:
    """Context tokens for workloads whose cache is built by a prefill (tiny model)."""
    return rng(w.seed, f"prompt/{seq}").integers(0, w.model.vocab, size=w.ctx[1]).astype(np.int32)


# ----------------------------------------------------------------------------
# device generation (HIP), through torch for memory and streams
# ----------------------------------------------------------------------------
_dev = None


def _dev_lib():
    global _dev
    if _dev is None:
        import torch  # noqa: F401  (the HIP runtime must come from torch's process)
        if not os.path.exists(DEV_LIB):
            raise RuntimeError(f"{DEV_LIB} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(DEV_LIB)
        lib.sy_dev_fill_linear.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint64,
                                           ctypes.c_int64, ctypes.c_float, ctypes.c_void_p]
        lib.sy_dev_fill_const.argtypes = [ctypes.c_void_p, ctypes.c_uint16, ctypes.c_int64,
                                          ctypes.c_void_p]
        lib.sy_dev_fill_ctx.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_void_p,
                                        ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                        ctypes.c_int32, ctypes.c_float, ctypes.c_void_p]
        for f in (lib.sy_dev_fill_linear, lib.sy_dev_fill_const, lib.sy_dev_fill_ctx):
            f.restype = ctypes.c_int
        _dev = lib
    return _dev


def _check(rc: int, what: str):
    if rc != 0:
        raise RuntimeError(f"{what} failed with hip error {rc}")


def device_tensor(seed: int, spec: TensorSpec, device="cuda"):
    import torch
    t = torch.empty(spec.shape, dtype=torch.bfloat16, device=device)
    stream = torch.cuda.current_stream(t.device).cuda_stream
    n = t.numel()
    lib = _dev_lib()
    if spec.init == "ones":
        _check(lib.sy_dev_fill_const(t.data_ptr(), BF16_ONE, n, stream), "fill_const")
    elif spec.init == "zeros":
        _check(lib.sy_dev_fill_const(t.data_ptr(), BF16_ZERO, n, stream), "fill_const")
    else:
        _check(lib.sy_dev_fill_linear(t.data_ptr(), tensor_key(seed, spec.name), 0, n,
                                      scale_for(spec.std), stream), "fill_linear")
    return t


def device_weights(m: ModelShape, seed: int, device="cuda") -> Dict[str, "object"]:
    return {s.name: device_tensor(seed, s, device) for s in tensor_specs(m)}


def device_fill_ctx(m: ModelShape, seed: int, k_cache, v_cache, ctx_len_dev) -> None:
    """Write the synthetic context into caches shaped [L][batch][Hkv][cap][hd]."""
    import torch
    L, B, H, cap, hd = k_cache.shape
    stream = torch.cuda.current_stream(k_cache.device).cuda_stream
    lib = _dev_lib()
    sc = scale_for(kv_std(m))
    for l in range(L):
        for which, cache in (("k", k_cache), ("v", v_cache)):
            _check(lib.sy_dev_fill_ctx(cache[l].data_ptr(), ctx_key(seed, l, which),
                                       ctx_len_dev.data_ptr(), B, H, cap, hd, sc, stream),
                   "fill_ctx")
