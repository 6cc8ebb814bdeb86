"""The C ABI library, without a GPU: it loads, exports every entry point the
header declares, and rejects host-checkable errors before touching HIP."""
import ctypes
import os
import re

import pytest

from paper_2510_13161_amd import msd, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    text = open(os.path.join(ROOT, "include", "msd.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(msd_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_entry_point():
    lib = msd.lib()
    names = header_functions()
    assert {"msd_verify_block", "msd_early_exit_topk", "msd_accept", "msd_kv_commit"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(msd.EXPORTED)


def test_binding_structs_match_header_sizes():
    # field counts of the ABI structs as declared
    assert ctypes.sizeof(msd.ModelConfig) == 13 * 4 + 2 * 4
    assert ctypes.sizeof(msd.KVCache) == 4 * 8 + 2 * 4
    assert ctypes.sizeof(msd.Block) == 2 * 4 + 2 * 8
    assert ctypes.sizeof(msd.Sampling) == 4 + 4 + 4 + 4 + 4 * 8 + 4 + 4


def test_accept_workspace_constant():
    """The acceptance workspace row size of msd.h (64 vocabulary chunks of an
    fp64 (max, sum) pair) is the binding's."""
    text = open(os.path.join(ROOT, "include", "msd.h")).read()
    assert "#define MSD_ACCEPT_WS_PER_ROW 1024" in text
    assert msd.MSD_ACCEPT_WS_PER_ROW == 64 * 16


def test_tensor_slot_layout():
    assert len(msd.GLOBAL_SLOTS) == 5 and len(msd.LAYER_SLOTS) == 17
    text = open(os.path.join(ROOT, "include", "msd.h")).read()
    assert "#define MSD_TENSOR_INDEX(layer, slot) (MSD_T_GLOBAL_COUNT + (layer) * MSD_L_COUNT + (slot))" in text


def _cfg(**kw):
    c = msd.config_of(synth.TINY)
    c.max_positions = 256
    for k, v in kw.items():
        setattr(c, k, v)
    return c


@pytest.mark.parametrize("field,value", [("head_dim", 96), ("n_kv_heads", 3), ("d_model", 200),
                                         ("vocab", 4100), ("norm", 7), ("norm_eps", 0.0),
                                         ("n_layers", 0)])
def test_model_create_rejects_bad_configs(field, value):
    lib = msd.lib()
    cfg = _cfg(**{field: value})
    n = 5 + 17 * max(cfg.n_layers, 1)
    arr = (ctypes.c_void_p * n)()
    out = ctypes.c_void_p()
    rc = lib.msd_model_create(ctypes.byref(cfg), arr, n, ctypes.byref(out))
    assert rc in (msd.MSD_ERR_SHAPE, msd.MSD_ERR_INVALID_ARG)
    assert out.value is None
    assert msd.last_error()


def test_model_create_rejects_missing_tensors_and_count():
    lib = msd.lib()
    cfg = _cfg()
    arr = (ctypes.c_void_p * (5 + 17 * 2))()
    out = ctypes.c_void_p()
    assert lib.msd_model_create(ctypes.byref(cfg), arr, 5 + 17 * 2, ctypes.byref(out)) == msd.MSD_ERR_INVALID_ARG
    assert "missing tensor" in msd.last_error()
    assert lib.msd_model_create(ctypes.byref(cfg), arr, 3, ctypes.byref(out)) == msd.MSD_ERR_SHAPE
    assert lib.msd_model_create(None, arr, 3, ctypes.byref(out)) == msd.MSD_ERR_INVALID_ARG


def test_entry_points_reject_null_model_and_bad_blocks():
    lib = msd.lib()
    blk = msd.Block(1, 9, None, None)
    kv = msd.KVCache()
    assert lib.msd_verify_block(None, ctypes.byref(kv), ctypes.byref(blk), None, None, None, None,
                                None, 0, None) == msd.MSD_ERR_INVALID_ARG
    assert lib.msd_accept(None, ctypes.byref(blk), None, None, None, None, None, None, None, None,
                          None, 0, None) == msd.MSD_ERR_INVALID_ARG
    assert lib.msd_kv_commit(None, ctypes.byref(kv), ctypes.byref(blk), None, None,
                             None) == msd.MSD_ERR_INVALID_ARG
    assert lib.msd_early_exit_topk(None, None, 9, 8, None, None, None, 0, None) == msd.MSD_ERR_INVALID_ARG
    assert lib.msd_workspace_bytes(None, 1, 9, 8, 1024) == 0
    assert lib.msd_set_profile(None, 3, None, None, 0) == msd.MSD_ERR_INVALID_ARG
