"""C-ABI contract checks that need no GPU: the library builds, loads, exports
every symbol include/pbd.h declares, sizes buffers, and rejects bad host-side
arguments before touching the device."""
import ctypes
import os
import re

import pytest

import synth
from paper_2607_12422_amd import binding as b

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pbd.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(b.LIB_PATH):
        from paper_2607_12422_amd import build
        build.build()
    return b.load_library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pbd_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert len(names) >= 12
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(b.EXPORTED) == names


def test_struct_layout_matches_header():
    # pbd_config: 18 four-byte fields; layer weights: 11 + 14 pointers.
    assert ctypes.sizeof(b.PbdConfig) == 18 * 4
    assert ctypes.sizeof(b.PbdLayerWeights) == 25 * ctypes.sizeof(ctypes.c_void_p)


def test_buffer_sizes(lib):
    cfg = b.make_config(synth.QWEN3_0_6B, 1, 1024)
    kv = lib.pbd_kv_bytes(ctypes.byref(cfg))
    # K and V, 28 layers, 8 KV heads, 1024 positions, head dim 128, bf16
    assert kv == 2 * 28 * 1 * 8 * 1024 * 128 * 2
    packed = lib.pbd_packed_weight_bytes(ctypes.byref(cfg))
    assert packed >= 596_049_920 * 2          # every backbone weight at least once
    assert lib.pbd_workspace_bytes(ctypes.byref(cfg)) > 0
    tiny = b.make_config(synth.TINY, 2, 256)
    assert lib.pbd_kv_bytes(ctypes.byref(tiny)) == 2 * 2 * 2 * 2 * 256 * 64 * 4


@pytest.mark.parametrize("field,value", [
    ("head_dim", 96), ("hidden", 100), ("vocab", 4095), ("block", -1), ("block", 40),
    ("lora_rank", 12), ("n_kv_heads", 3), ("mask_id", 4096), ("dtype", 7), ("max_seq", 5),
    ("prefill_chunk", -1), ("prefill_chunk", 1025), ("prefill_chunk", 4096),
])
def test_invalid_config_sizes_are_zero(lib, field, value):
    cfg = b.make_config(synth.TINY, 1, 256)
    setattr(cfg, field, value)
    assert lib.pbd_packed_weight_bytes(ctypes.byref(cfg)) == 0
    assert lib.pbd_workspace_bytes(ctypes.byref(cfg)) == 0


def test_init_rejects_bad_arguments_without_device(lib):
    cfg = b.make_config(synth.TINY, 1, 256)
    ctx = ctypes.c_void_p()
    rc = lib.pbd_init_weights(ctypes.byref(cfg), None, None, 0, None, 0, None, 0, None, ctypes.byref(ctx))
    assert rc == b.PBD_ERR_INVALID_ARG and ctx.value is None
    assert "weights" in b.pbd_last_error()
    cfg.head_dim = 96
    rc = lib.pbd_init_weights(ctypes.byref(cfg), None, None, 0, None, 0, None, 0, None, ctypes.byref(ctx))
    assert rc == b.PBD_ERR_SHAPE
    assert "head_dim" in b.pbd_last_error()


def test_calls_reject_null_context(lib):
    assert lib.pbd_draft_block(None, 1, None, None, 0, None, None, None) == b.PBD_ERR_INVALID_ARG
    assert lib.pbd_draft_block_layers(None, 1, None, None, 0, 1, None, None, None) == b.PBD_ERR_INVALID_ARG
    assert lib.pbd_draft_block_denoise(None, 1, None, None, 0, 1, None, None, None, None, None) == b.PBD_ERR_INVALID_ARG
    assert lib.pbd_verify_block(None, 1, None, None, None, 0, None, None, None) == b.PBD_ERR_INVALID_ARG
    assert lib.pbd_draft_block_unanchored(None, 1, None, None, 0, None, None, None, None) == b.PBD_ERR_INVALID_ARG
    assert lib.pbd_verify_block_unanchored(None, 1, None, None, 0, None, None, None) == b.PBD_ERR_INVALID_ARG
    assert lib.pbd_accept_commit(None, 1, None, None, None, None, None, None, None, None) == b.PBD_ERR_INVALID_ARG
    assert lib.pbd_prefill(None, 1, None, None, 1, None, None, None) == b.PBD_ERR_INVALID_ARG
    st = ctypes.c_int32()
    assert lib.pbd_sync_status(None, None, ctypes.byref(st)) == b.PBD_ERR_INVALID_ARG
    assert lib.pbd_set_attn_keys_per_split(None, 64) == b.PBD_ERR_INVALID_ARG
    assert lib.pbd_set_attn_query_split(None, 1) == b.PBD_ERR_INVALID_ARG
    lib.pbd_destroy(None)


def test_missing_library_fails_loudly(tmp_path):
    with pytest.raises(RuntimeError, match="not built"):
        b.load_library(str(tmp_path / "libpbd.so"))
