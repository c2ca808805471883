"""Thin ctypes binding of libpbd (include/pbd.h): argument marshalling only.

Every computation of the speculative step runs in the HIP library; PyTorch
provides device memory and the stream.  The functions below carry the C names
and take torch tensors (device int32 / float32) or raw pointers.  If the built
library is missing, loading fails loudly: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "lib", "libpbd.so")

PBD_OK = 0
PBD_ERR_INVALID_ARG = -1
PBD_ERR_SHAPE = -2
PBD_ERR_CAPACITY = -3
PBD_ERR_STATE = -4
PBD_ERR_HIP = -5
PBD_ERR_UNSUPPORTED = -6

PBD_DTYPE_F32 = 0
PBD_DTYPE_BF16 = 1

PBD_PASS_DEFAULT = 0
PBD_PASS_ADAPTER_ON = 1
PBD_PASS_ADAPTER_OFF = 2
PBD_PASS_MASK_BLOCK = 4
PBD_PASS_MASK_CAUSAL = 8

PBD_OPERANDS_BF16 = 0
PBD_OPERANDS_BF16X2 = 1

KCLASSES = ("gemm", "lmhead", "attn", "combine", "norm", "other", "fused")

PBD_STATUS_CAPACITY = 1
PBD_STATUS_TOKEN = 2
PBD_STATUS_FORCED_N = 4
PBD_STATUS_TIMEOUT = 8

EXPORTED = (
    "pbd_packed_weight_bytes", "pbd_kv_bytes", "pbd_workspace_bytes", "pbd_init_weights",
    "pbd_prefill", "pbd_draft_block", "pbd_draft_block_layers", "pbd_draft_block_denoise",
    "pbd_verify_block", "pbd_verify_block_noalloc", "pbd_draft_block_unanchored", "pbd_verify_block_unanchored", "pbd_accept_commit",
    "pbd_sync_status", "pbd_set_attn_keys_per_split", "pbd_set_attn_query_split", "pbd_set_operand_precision",
    "pbd_set_pass_mode", "pbd_set_wait_limit", "pbd_profile_enable", "pbd_profile_read", "pbd_profile_stage_times", "pbd_last_error", "pbd_destroy",
)


class PbdConfig(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32), ("hidden", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("ffn", ctypes.c_int32),
        ("vocab", ctypes.c_int32), ("lora_rank", ctypes.c_int32), ("lora_alpha", ctypes.c_float),
        ("block", ctypes.c_int32), ("mask_id", ctypes.c_int32), ("rms_eps", ctypes.c_float),
        ("rope_theta", ctypes.c_float), ("qk_norm", ctypes.c_int32), ("dtype", ctypes.c_int32),
        ("max_batch", ctypes.c_int32), ("max_seq", ctypes.c_int32), ("prefill_chunk", ctypes.c_int32),
    ]


class PbdLayerWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "attn_norm", "q", "k", "v", "o", "q_norm", "k_norm", "mlp_norm", "gate", "up", "down")] + [
        ("lora_a", ctypes.c_void_p * 7), ("lora_b", ctypes.c_void_p * 7)]


class PbdWeights(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("final_norm", ctypes.c_void_p),
                ("layers", ctypes.POINTER(PbdLayerWeights))]


_lib = None


def load_library(path: Optional[str] = None) -> ctypes.CDLL:
    """Load libpbd.so (built by paper_2607_12422_amd.build); raises if absent."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"PEFT-BD HIP library not built: {p} is missing "
                           "(run paper_2607_12422_amd.build.build())")
    lib = ctypes.CDLL(p)
    vp, i32, u32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint32, ctypes.c_size_t
    cfgp = ctypes.POINTER(PbdConfig)
    sig = {
        "pbd_packed_weight_bytes": (sz, [cfgp]),
        "pbd_kv_bytes": (sz, [cfgp]),
        "pbd_workspace_bytes": (sz, [cfgp]),
        "pbd_init_weights": (ctypes.c_int, [cfgp, ctypes.POINTER(PbdWeights), vp, sz, vp, sz, vp, sz, vp,
                                            ctypes.POINTER(vp)]),
        "pbd_prefill": (ctypes.c_int, [vp, i32, vp, vp, i32, vp, vp, vp]),
        "pbd_draft_block": (ctypes.c_int, [vp, i32, vp, vp, u32, vp, vp, vp]),
        "pbd_draft_block_layers": (ctypes.c_int, [vp, i32, vp, vp, u32, i32, vp, vp, vp]),
        "pbd_draft_block_denoise": (ctypes.c_int, [vp, i32, vp, vp, u32, i32, vp, vp, vp, vp, vp]),
        "pbd_draft_block_unanchored": (ctypes.c_int, [vp, i32, vp, vp, u32, vp, vp, vp, vp]),
        "pbd_verify_block_unanchored": (ctypes.c_int, [vp, i32, vp, vp, u32, vp, vp, vp]),
        "pbd_verify_block": (ctypes.c_int, [vp, i32, vp, vp, vp, u32, vp, vp, vp]),
        "pbd_verify_block_noalloc": (ctypes.c_int, [vp, i32, vp, vp, vp, u32, vp, vp, vp]),
        "pbd_accept_commit": (ctypes.c_int, [vp, i32, vp, vp, vp, vp, vp, vp, vp, vp]),
        "pbd_sync_status": (ctypes.c_int, [vp, vp, ctypes.POINTER(i32)]),
        "pbd_set_attn_keys_per_split": (ctypes.c_int, [vp, i32]),
        "pbd_set_attn_query_split": (ctypes.c_int, [vp, i32]),
        "pbd_set_operand_precision": (ctypes.c_int, [vp, i32]),
        "pbd_set_pass_mode": (ctypes.c_int, [vp, i32]),
        "pbd_set_wait_limit": (ctypes.c_int, [vp, i32]),
        "pbd_profile_enable": (ctypes.c_int, [vp, i32]),
        "pbd_profile_read": (ctypes.c_int, [vp, i32, ctypes.POINTER(ctypes.c_double),
                                            ctypes.POINTER(ctypes.c_int64)]),
        "pbd_profile_stage_times": (ctypes.c_int, [vp, ctypes.POINTER(ctypes.c_uint64), i32,
                                                    ctypes.POINTER(i32)]),
        "pbd_last_error": (ctypes.c_char_p, [vp]),
        "pbd_destroy": (None, [vp]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    if path is None:
        _lib = lib
    return lib


class PbdError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{msg} (status {code})")
        self.code = code


def make_config(cfg, max_batch: int, max_seq: int, prefill_chunk: int = 0) -> PbdConfig:
    """pbd_config from a model description with the attribute names of pbd_config."""
    return PbdConfig(
        n_layers=cfg.n_layers, hidden=cfg.hidden, n_q_heads=cfg.n_q_heads, n_kv_heads=cfg.n_kv_heads,
        head_dim=cfg.head_dim, ffn=cfg.ffn, vocab=cfg.vocab, lora_rank=cfg.lora_rank,
        lora_alpha=cfg.lora_alpha, block=cfg.block, mask_id=cfg.mask_id, rms_eps=cfg.rms_eps,
        rope_theta=cfg.rope_theta, qk_norm=1 if cfg.qk_norm else 0,
        dtype=PBD_DTYPE_BF16 if cfg.dtype == "bf16" else PBD_DTYPE_F32,
        max_batch=max_batch, max_seq=max_seq, prefill_chunk=prefill_chunk)


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else stream


def pbd_packed_weight_bytes(cfg: PbdConfig) -> int:
    return load_library().pbd_packed_weight_bytes(ctypes.byref(cfg))


def pbd_kv_bytes(cfg: PbdConfig) -> int:
    return load_library().pbd_kv_bytes(ctypes.byref(cfg))


def pbd_workspace_bytes(cfg: PbdConfig) -> int:
    return load_library().pbd_workspace_bytes(ctypes.byref(cfg))


def pbd_last_error(ctx=None) -> str:
    s = load_library().pbd_last_error(ctx)
    return s.decode() if s else ""


def _check(rc: int, ctx=None):
    if rc != PBD_OK:
        raise PbdError(rc, pbd_last_error(ctx))


class Engine:
    """Owns the device buffers (torch tensors) of one pbd context.

    ``weights`` is a mapping/object with the canonical weights already on the
    device (see ``upload_weights``).  Buffers are allocated with torch, so the
    library itself never allocates device memory.
    """

    def __init__(self, cfg, dev_weights, max_batch: int, max_seq: int, device="cuda:0", stream=None,
                 prefill_chunk: int = 0):
        import torch
        self.lib = load_library()
        self.cfg = cfg
        self.pcfg = make_config(cfg, max_batch, max_seq, prefill_chunk)
        self.device = torch.device(device)
        nb = self.lib.pbd_packed_weight_bytes(ctypes.byref(self.pcfg))
        if nb == 0:
            raise PbdError(PBD_ERR_SHAPE, "configuration rejected by pbd_packed_weight_bytes")
        nkv = self.lib.pbd_kv_bytes(ctypes.byref(self.pcfg))
        nws = self.lib.pbd_workspace_bytes(ctypes.byref(self.pcfg))
        self.packed = torch.empty(nb, dtype=torch.uint8, device=self.device)
        self.kv = torch.empty(nkv, dtype=torch.uint8, device=self.device)
        self.ws = torch.empty(nws, dtype=torch.uint8, device=self.device)
        self._w = dev_weights
        layers = (PbdLayerWeights * cfg.n_layers)()
        for i, lw in enumerate(dev_weights["layers"]):
            L = layers[i]
            for n in ("attn_norm", "q", "k", "v", "o", "q_norm", "k_norm", "mlp_norm", "gate", "up", "down"):
                setattr(L, n, _ptr(lw[n]))
            for j, n in enumerate(("q", "k", "v", "o", "gate", "up", "down")):
                A, B = lw["lora"][n] if cfg.lora_rank > 0 else (None, None)
                L.lora_a[j] = _ptr(A)
                L.lora_b[j] = _ptr(B)
        self._layers = layers
        pw = PbdWeights(embed=_ptr(dev_weights["embed"]), final_norm=_ptr(dev_weights["final_norm"]),
                        layers=ctypes.cast(layers, ctypes.POINTER(PbdLayerWeights)))
        ctx = ctypes.c_void_p()
        rc = self.lib.pbd_init_weights(ctypes.byref(self.pcfg), ctypes.byref(pw), _ptr(self.packed), nb,
                                       _ptr(self.kv), nkv, _ptr(self.ws), nws, _stream(stream),
                                       ctypes.byref(ctx))
        _check(rc, None)
        self.ctx = ctx.value

    # -- the C calls, same names ------------------------------------------------
    def pbd_prefill(self, tokens, lengths, max_len: int, seq_len, anchor, stream=None):
        rc = self.lib.pbd_prefill(self.ctx, int(lengths.shape[0]), _ptr(tokens), _ptr(lengths), int(max_len),
                                  _ptr(seq_len), _ptr(anchor), _stream(stream))
        _check(rc, self.ctx)

    def pbd_draft_block(self, seq_len, anchor, draft, logits=None, flags: int = PBD_PASS_DEFAULT,
                        batch: Optional[int] = None, stream=None):
        B = int(seq_len.shape[0]) if batch is None else batch
        rc = self.lib.pbd_draft_block(self.ctx, B, _ptr(seq_len), _ptr(anchor), flags, _ptr(draft),
                                      _ptr(logits), _stream(stream))
        _check(rc, self.ctx)

    def pbd_draft_block_layers(self, seq_len, anchor, draft, n_layers: int, logits=None,
                               flags: int = PBD_PASS_DEFAULT, batch: Optional[int] = None, stream=None):
        B = int(seq_len.shape[0]) if batch is None else batch
        rc = self.lib.pbd_draft_block_layers(self.ctx, B, _ptr(seq_len), _ptr(anchor), flags, int(n_layers),
                                             _ptr(draft), _ptr(logits), _stream(stream))
        _check(rc, self.ctx)

    def pbd_draft_block_denoise(self, seq_len, anchor, draft, n_steps: int, conf=None, fixed_at=None,
                                logits=None, flags: int = PBD_PASS_DEFAULT, batch: Optional[int] = None,
                                stream=None):
        B = int(seq_len.shape[0]) if batch is None else batch
        rc = self.lib.pbd_draft_block_denoise(self.ctx, B, _ptr(seq_len), _ptr(anchor), flags, int(n_steps),
                                              _ptr(draft), _ptr(conf), _ptr(fixed_at), _ptr(logits),
                                              _stream(stream))
        _check(rc, self.ctx)

    def pbd_verify_block(self, seq_len, anchor, draft, verify, logits=None, flags: int = PBD_PASS_DEFAULT,
                         batch: Optional[int] = None, stream=None):
        B = int(seq_len.shape[0]) if batch is None else batch
        rc = self.lib.pbd_verify_block(self.ctx, B, _ptr(seq_len), _ptr(anchor), _ptr(draft), flags,
                                       _ptr(verify), _ptr(logits), _stream(stream))
        _check(rc, self.ctx)

    def pbd_verify_block_noalloc(self, seq_len, anchor, draft, verify, logits=None,
                                 flags: int = PBD_PASS_DEFAULT, batch: Optional[int] = None, stream=None):
        B = int(seq_len.shape[0]) if batch is None else batch
        rc = self.lib.pbd_verify_block_noalloc(self.ctx, B, _ptr(seq_len), _ptr(anchor), _ptr(draft), flags,
                                               _ptr(verify), _ptr(logits), _stream(stream))
        _check(rc, self.ctx)

    def pbd_draft_block_unanchored(self, seq_len, anchor, draft, verify, logits=None,
                                   flags: int = PBD_PASS_DEFAULT, batch: Optional[int] = None, stream=None):
        B = int(seq_len.shape[0]) if batch is None else batch
        rc = self.lib.pbd_draft_block_unanchored(self.ctx, B, _ptr(seq_len), _ptr(anchor), flags, _ptr(draft),
                                                 _ptr(verify), _ptr(logits), _stream(stream))
        _check(rc, self.ctx)

    def pbd_verify_block_unanchored(self, seq_len, draft, verify, logits=None, flags: int = PBD_PASS_DEFAULT,
                                    batch: Optional[int] = None, stream=None):
        B = int(seq_len.shape[0]) if batch is None else batch
        rc = self.lib.pbd_verify_block_unanchored(self.ctx, B, _ptr(seq_len), _ptr(draft), flags, _ptr(verify),
                                                  _ptr(logits), _stream(stream))
        _check(rc, self.ctx)

    def pbd_accept_commit(self, draft, verify, seq_len, anchor, n_accepted, out_tokens, forced_n=None,
                          batch: Optional[int] = None, stream=None):
        B = int(seq_len.shape[0]) if batch is None else batch
        rc = self.lib.pbd_accept_commit(self.ctx, B, _ptr(draft), _ptr(verify), _ptr(forced_n), _ptr(seq_len),
                                        _ptr(anchor), _ptr(n_accepted), _ptr(out_tokens), _stream(stream))
        _check(rc, self.ctx)

    def pbd_sync_status(self, stream=None) -> int:
        st = ctypes.c_int32(0)
        rc = self.lib.pbd_sync_status(self.ctx, _stream(stream), ctypes.byref(st))
        _check(rc, self.ctx)
        return st.value

    def pbd_set_attn_keys_per_split(self, keys: int):
        _check(self.lib.pbd_set_attn_keys_per_split(self.ctx, int(keys)), self.ctx)

    def pbd_set_attn_query_split(self, mode: int):
        _check(self.lib.pbd_set_attn_query_split(self.ctx, int(mode)), self.ctx)

    def pbd_set_operand_precision(self, mode: int):
        _check(self.lib.pbd_set_operand_precision(self.ctx, int(mode)), self.ctx)

    def pbd_set_pass_mode(self, mode: int):
        _check(self.lib.pbd_set_pass_mode(self.ctx, int(mode)), self.ctx)

    def pbd_set_wait_limit(self, polls: int):
        _check(self.lib.pbd_set_wait_limit(self.ctx, int(polls)), self.ctx)

    def pbd_profile_enable(self, on: bool = True):
        _check(self.lib.pbd_profile_enable(self.ctx, 1 if on else 0), self.ctx)

    def pbd_profile_read(self, kclass: int):
        ms = ctypes.c_double(0.0)
        n = ctypes.c_int64(0)
        _check(self.lib.pbd_profile_read(self.ctx, int(kclass), ctypes.byref(ms), ctypes.byref(n)), self.ctx)
        return ms.value, n.value

    def pbd_profile_stage_times(self):
        """Stage timestamps of the last persistent pass: uint64 array [8][32][64][8][4]."""
        import numpy as np
        n = 8 * 32 * 64 * 8 * 4
        buf = (ctypes.c_uint64 * n)()
        got = ctypes.c_int32(0)
        _check(self.lib.pbd_profile_stage_times(self.ctx, buf, n, ctypes.byref(got)), self.ctx)
        return np.frombuffer(buf, dtype=np.uint64, count=got.value).reshape(8, 32, 64, 8, 4).copy()

    def close(self):
        if getattr(self, "ctx", None):
            self.lib.pbd_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def upload_weights(w, dtype: str, device="cuda:0"):
    """Copy host weights (objects with the canonical attribute names, float32
    NumPy arrays) to device tensors of the model dtype; returns the mapping the
    Engine reads.  Values are copied unchanged (bf16 inputs must already be
    bf16-representable)."""
    import torch
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32

    def dev(a):
        return torch.from_numpy(a).to(device=device).to(tdt).contiguous()

    layers = []
    for lw in w.layers:
        d = {n: dev(getattr(lw, n)) for n in
             ("attn_norm", "q", "k", "v", "o", "q_norm", "k_norm", "mlp_norm", "gate", "up", "down")}
        d["lora"] = {n: (dev(A), dev(B)) for n, (A, B) in lw.lora.items()}
        layers.append(d)
    return {"embed": dev(w.embed), "final_norm": dev(w.final_norm), "layers": layers}
