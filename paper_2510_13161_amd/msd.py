"""Python binding of libmsd.so (include/msd.h): argument marshalling only.

Every step of the verification pass runs in the library's HIP kernels; this
module converts torch tensors into pointers and checks status codes. PyTorch
provides device memory and streams. If the library is not built the import
of any entry point raises: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional, Sequence

import torch  # the HIP runtime libmsd.so binds to is the one torch loaded

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmsd.so")

# status codes / enums (msd.h)
MSD_OK = 0
MSD_ERR_INVALID_ARG, MSD_ERR_SHAPE, MSD_ERR_CAPACITY = -1, -2, -3
MSD_ERR_UNSUPPORTED, MSD_ERR_WORKSPACE, MSD_ERR_HIP = -4, -5, -6
MSD_DEV_CAPACITY, MSD_DEV_CANDIDATE, MSD_DEV_TOKEN = 1, 2, 4
MSD_NORM_RMS, MSD_NORM_LAYER = 0, 1
MSD_ACT_SWIGLU, MSD_ACT_RELU = 0, 1
MSD_POS_ROPE, MSD_POS_LEARNED = 0, 1
MSD_GREEDY, MSD_REJECTION, MSD_MATCH = 0, 1, 2
MODES = {"greedy": MSD_GREEDY, "rejection": MSD_REJECTION, "match": MSD_MATCH}

GLOBAL_SLOTS = ["embed", "pos_embed", "final_norm.g", "final_norm.b", "lm_head"]
LAYER_SLOTS = ["attn_norm.g", "attn_norm.b", "wq", "wk", "wv", "bq", "bk", "bv", "wo", "bo",
               "mlp_norm.g", "mlp_norm.b", "w_gate", "w_up", "b_up", "w_down", "b_down"]

EXPORTED = ["msd_last_error", "msd_model_create", "msd_model_destroy", "msd_workspace_bytes",
            "msd_verify_block", "msd_early_exit_topk", "msd_accept", "msd_kv_commit",
            "msd_reuse_select", "msd_set_profile", "msd_verify_block_static"]
MSD_STATIC_SCRATCH_BYTES = 64 << 20
MSD_ACCEPT_WS_PER_ROW = 1024  # bytes a row of the acceptance workspace (msd.h)
MSD_K_QKV, MSD_K_ATTN, MSD_K_OPROJ, MSD_K_FFN_UP, MSD_K_FFN_DOWN = 0, 1, 2, 3, 4
MSD_NEXT_BRANCH, MSD_NEXT_CONTINUE, MSD_NEXT_FRESH = 0, 1, 2
MSD_MAX_TREE_NODES = 256


class MsdError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"msd status {status}: {msg}")
        self.status = status


class ModelConfig(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("n_layers", "d_model", "n_heads", "n_kv_heads", "head_dim", "d_ffn", "vocab",
                 "norm", "act", "pos", "has_bias", "tied_head", "max_positions")] + \
               [("rope_theta", ctypes.c_float), ("norm_eps", ctypes.c_float)]


class KVCache(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("len", ctypes.c_void_p),
                ("status", ctypes.c_void_p), ("batch_cap", ctypes.c_int32),
                ("capacity", ctypes.c_int32)]


class Block(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_slots", ctypes.c_int32),
                ("tokens", ctypes.c_void_p), ("parent", ctypes.POINTER(ctypes.c_int32))]


class EERequest(ctypes.Structure):
    _fields_ = [("layer", ctypes.c_int32), ("kappa", ctypes.c_int32), ("ids", ctypes.c_void_p),
                ("logp", ctypes.c_void_p), ("ready", ctypes.c_void_p)]


class Sampling(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int32), ("temperature", ctypes.c_float),
                ("n_cand", ctypes.c_int32), ("cand_ids", ctypes.c_void_p),
                ("cand_q", ctypes.c_void_p), ("u_accept", ctypes.c_void_p),
                ("u_sample", ctypes.c_void_p), ("tol_logit", ctypes.c_float)]


class HypTree(ctypes.Structure):
    _fields_ = [("n_nodes", ctypes.c_int32), ("parent", ctypes.POINTER(ctypes.c_int32)),
                ("tokens", ctypes.c_void_p)]


class ReuseStats(ctypes.Structure):
    """Layout of msd_reuse_stats (40 bytes); keep it in a device tensor."""
    _fields_ = [("trials", ctypes.c_uint64), ("fallbacks", ctypes.c_uint64),
                ("fallbacks_tau1", ctypes.c_uint64), ("omega_trials", ctypes.c_uint64),
                ("omega_sum", ctypes.c_double)]


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build(); "
                               "there is no fallback path")
        L = ctypes.CDLL(LIB_PATH)
        P, i32 = ctypes.c_void_p, ctypes.c_int32
        L.msd_last_error.restype = ctypes.c_char_p
        L.msd_last_error.argtypes = []
        L.msd_model_create.argtypes = [P, P, i32, P]
        L.msd_model_destroy.argtypes = [P]
        L.msd_model_destroy.restype = None
        L.msd_workspace_bytes.argtypes = [P, i32, i32, i32, i32]
        L.msd_workspace_bytes.restype = ctypes.c_size_t
        L.msd_verify_block.argtypes = [P, P, P, P, P, P, P, P, ctypes.c_size_t, P]
        L.msd_verify_block_static.argtypes = [P, P, P, P, P, P, P, P]
        L.msd_early_exit_topk.argtypes = [P, P, i32, i32, P, P, P, ctypes.c_size_t, P]
        L.msd_accept.argtypes = [P, P, P, P, P, P, P, P, P, P, P, ctypes.c_size_t, P]
        L.msd_kv_commit.argtypes = [P, P, P, P, P, P]
        L.msd_set_profile.argtypes = [P, i32, P, P, i32]
        L.msd_reuse_select.argtypes = [P, P, P, P, P, P, P, P, P, i32, P, P, P, P, P]
        for f in ("msd_model_create", "msd_verify_block", "msd_verify_block_static",
                  "msd_early_exit_topk", "msd_accept",
                  "msd_kv_commit", "msd_reuse_select", "msd_set_profile"):
            getattr(L, f).restype = ctypes.c_int
        _lib = L
    return _lib


def last_error() -> str:
    return lib().msd_last_error().decode()


def _check(status: int):
    if status != MSD_OK:
        raise MsdError(status, last_error())


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    assert t.is_cuda and t.is_contiguous(), "device tensors must be contiguous CUDA tensors"
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


# ---------------------------------------------------------------------------
# entry points (same names as the C ABI)
# ---------------------------------------------------------------------------
def model_create(cfg: ModelConfig, tensor_ptrs: Sequence[int]) -> ctypes.c_void_p:
    arr = (ctypes.c_void_p * len(tensor_ptrs))(*[p or None for p in tensor_ptrs])
    out = ctypes.c_void_p()
    _check(lib().msd_model_create(ctypes.byref(cfg), arr, len(tensor_ptrs), ctypes.byref(out)))
    return out


def model_destroy(handle) -> None:
    lib().msd_model_destroy(handle)


def workspace_bytes(handle, batch: int, n_slots: int, kappa: int, capacity: int) -> int:
    return int(lib().msd_workspace_bytes(handle, batch, n_slots, kappa, capacity))


def verify_block(handle, kv: KVCache, block: Block, ee: Optional[EERequest], logits, argmax, lse,
                 ws: torch.Tensor, stream=None) -> None:
    _check(lib().msd_verify_block(handle, ctypes.byref(kv), ctypes.byref(block),
                                  ctypes.byref(ee) if ee is not None else None, _ptr(logits),
                                  _ptr(argmax), _ptr(lse), _ptr(ws), ws.numel(), _stream(stream)))


def verify_block_static(handle, kv: KVCache, block: Block, ee: Optional[EERequest], logits, argmax,
                        lse, stream=None) -> None:
    """msd_verify_block with the library's static scratch (no workspace)."""
    _check(lib().msd_verify_block_static(handle, ctypes.byref(kv), ctypes.byref(block),
                                         ctypes.byref(ee) if ee is not None else None, _ptr(logits),
                                         _ptr(argmax), _ptr(lse), _stream(stream)))


def early_exit_topk(handle, hidden: torch.Tensor, kappa: int, ids, logp, ws: torch.Tensor,
                    stream=None) -> None:
    _check(lib().msd_early_exit_topk(handle, _ptr(hidden), hidden.shape[0], kappa, _ptr(ids),
                                     _ptr(logp), _ptr(ws), ws.numel(), _stream(stream)))


def accept(handle, block: Block, logits, argmax, sampling: Optional[Sampling], acc_len, next_tok,
           path, status, ws: Optional[torch.Tensor] = None, stream=None, near_tie=None) -> None:
    """near_tie: optional device uint8 [batch] of near-tie flags (msd.h)."""
    _check(lib().msd_accept(handle, ctypes.byref(block), _ptr(logits), _ptr(argmax),
                            ctypes.byref(sampling) if sampling is not None else None,
                            _ptr(acc_len), _ptr(next_tok), _ptr(path), _ptr(near_tie),
                            _ptr(status), _ptr(ws), 0 if ws is None else ws.numel(),
                            _stream(stream)))


def kv_commit(handle, kv: KVCache, block: Block, acc_len, path, stream=None) -> None:
    _check(lib().msd_kv_commit(handle, ctypes.byref(kv), ctypes.byref(block), _ptr(acc_len),
                               _ptr(path), _stream(stream)))


def hyp_tree(parent, tokens) -> "HypTree":
    """msd_hyp_tree over a host parent list (-1 = root) and a device int32
    tensor of tokens [batch][n_nodes]; keeps the host array alive."""
    n = len(parent)
    P = (ctypes.c_int32 * n)(*parent)
    t = HypTree(n, ctypes.cast(P, ctypes.POINTER(ctypes.c_int32)), _ptr(tokens))
    t._keep = (P, tokens)
    return t


def reuse_select(handle, block: Block, acc_len, next_tok, path, tree: HypTree, next_case, next_node,
                 logits=None, lse=None, ee_ids=None, kappa: int = 0, omega=None, stats=None,
                 stream=None) -> None:
    """stats: a device tensor of at least 40 bytes holding msd_reuse_stats."""
    _check(lib().msd_reuse_select(handle, ctypes.byref(block), _ptr(acc_len), _ptr(next_tok),
                                  _ptr(path), ctypes.byref(tree), _ptr(logits), _ptr(lse),
                                  _ptr(ee_ids), int(kappa), _ptr(next_case), _ptr(next_node),
                                  _ptr(omega), _ptr(stats), _stream(stream)))


def read_reuse_stats(stats) -> dict:
    """Copies a device msd_reuse_stats to the host."""
    raw = bytes(stats.detach().cpu().contiguous().view(-1).numpy().tobytes()[:ctypes.sizeof(ReuseStats)])
    r = ReuseStats.from_buffer_copy(raw)
    return {f: getattr(r, f) for f, _ in ReuseStats._fields_}


def set_profile(handle, kclass: int, begin_events, end_events) -> None:
    """begin/end: sequences of raw hipEvent_t handles (ints), one per layer,
    None to skip a layer; [] turns it off."""
    n = len(begin_events)
    B = (ctypes.c_void_p * max(n, 1))(*begin_events)
    E = (ctypes.c_void_p * max(n, 1))(*end_events)
    _check(lib().msd_set_profile(handle, kclass, B if n else None, E if n else None, n))


# ---------------------------------------------------------------------------
# conveniences: still marshalling only
# ---------------------------------------------------------------------------
def config_of(shape) -> ModelConfig:
    """ModelConfig from a shape description with the synth.ModelShape fields."""
    return ModelConfig(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads,
                       shape.head_dim, shape.d_ffn, shape.vocab,
                       MSD_NORM_LAYER if shape.norm == "layer" else MSD_NORM_RMS,
                       MSD_ACT_RELU if shape.act == "relu" else MSD_ACT_SWIGLU,
                       MSD_POS_LEARNED if shape.pos == "learned" else MSD_POS_ROPE,
                       int(shape.bias), int(shape.tied_head),
                       int(getattr(shape, "max_positions_rt", 0) or shape.max_positions or 0),
                       float(shape.rope_theta), float(shape.norm_eps))


class Model:
    """Owns a msd_model handle built from named bf16 device tensors."""

    def __init__(self, shape, tensors: Dict[str, torch.Tensor], max_positions: int):
        cfg = config_of(shape)
        if shape.pos != "learned":
            cfg.max_positions = max_positions
        self.shape = shape
        self.cfg = cfg
        self.tensors = tensors  # keep alive
        ptrs: List[Optional[int]] = [None] * (len(GLOBAL_SLOTS) + len(LAYER_SLOTS) * shape.n_layers)
        for i, n in enumerate(GLOBAL_SLOTS):
            if n in tensors:
                ptrs[i] = _ptr(tensors[n])
        for l in range(shape.n_layers):
            for j, n in enumerate(LAYER_SLOTS):
                t = tensors.get(f"l{l}.{n}")
                if t is not None:
                    ptrs[len(GLOBAL_SLOTS) + l * len(LAYER_SLOTS) + j] = _ptr(t)
        self.handle = model_create(cfg, ptrs)

    def close(self):
        if getattr(self, "handle", None):
            model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Cache:
    """KV cache tensors [L][batch_cap][Hkv][capacity][hd] bf16, len, status."""

    def __init__(self, shape, batch_cap: int, capacity: int, device="cuda"):
        dims = (shape.n_layers, batch_cap, shape.n_kv_heads, capacity, shape.head_dim)
        self.k = torch.zeros(dims, dtype=torch.bfloat16, device=device)
        self.v = torch.zeros(dims, dtype=torch.bfloat16, device=device)
        self.len = torch.zeros(batch_cap, dtype=torch.int32, device=device)
        self.status = torch.zeros(1, dtype=torch.int32, device=device)
        self.c = KVCache(self.k.data_ptr(), self.v.data_ptr(), self.len.data_ptr(),
                         self.status.data_ptr(), batch_cap, capacity)


def make_block(tokens: torch.Tensor, parent=None) -> Block:
    """tokens: device int32 [batch][n_slots]; parent: host sequence or None (chain)."""
    assert tokens.dtype == torch.int32 and tokens.dim() == 2
    b = Block(tokens.shape[0], tokens.shape[1], _ptr(tokens), None)
    b._keep = (tokens,)  # the block holds only the address: keep the tensor alive with it
    if parent is not None:
        arr = (ctypes.c_int32 * len(parent))(*[int(p) for p in parent])
        b.parent = ctypes.cast(arr, ctypes.POINTER(ctypes.c_int32))
        b._keep = (tokens, arr)
    return b
