"""Thin ctypes binding of libw4layer.so (include/w4layer.h).

Argument marshalling only: every step of the layer runs in the HIP kernels of
the library.  Tensors are torch tensors on the GPU (PyTorch provides device
memory and streams); the functions keep the C names and return the C status
codes, and ``check`` turns a non-zero code into a ``W4Error``.

Importing this module loads the library and raises if it is missing: there is
no fallback path.
"""
from __future__ import annotations

import atexit
import ctypes
import os
import re
import sys
import weakref
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libw4layer.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "w4layer.h")

W4_OK, W4_EINVAL, W4_EUNSUPPORTED, W4_ECAPACITY, W4_EWORKSPACE, W4_EHIP = 0, -1, -2, -3, -4, -5
W4_FLAG_WAIT_TIMEOUT, W4_FLAG_F16_RANGE, W4_FLAG_TOKEN_ID = 1, 2, 4
W4_WEIGHTS_INT4, W4_WEIGHTS_INT8, W4_WEIGHTS_BF16 = 0, 1, 2
WEIGHT_FORMAT_CODE = {"int4": W4_WEIGHTS_INT4, "int8": W4_WEIGHTS_INT8, "bf16": W4_WEIGHTS_BF16}
STAGE_PREFILL, STAGE_PREFILL_KV, STAGE_DECODE = 0, 1, 2
LINEAR_INDEX = {"q": 0, "k": 1, "v": 2, "o": 3, "gate": 4, "up": 5, "down": 6}

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run python -m paper_2607_15865_amd.build "
                      "(the layer has no CPU fallback)")
# torch ships its own HIP runtime under the same soname (libamdhip64.so.7) as
# the system one the library links; whichever loads first serves the whole
# process.  Load torch's first so that torch and the library share it.
import torch  # noqa: E402,F401

_lib = ctypes.CDLL(LIB_PATH)


class W4Error(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"w4layer error {code}: {msg}")
        self.code = code


class layer_config(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("ffn", ctypes.c_int32), ("group_size", ctypes.c_int32),
                ("rms_eps", ctypes.c_float), ("rope_base", ctypes.c_float),
                ("max_seq", ctypes.c_int32), ("max_batch", ctypes.c_int32), ("weight_format", ctypes.c_int32)]


class qlinear_host(ctypes.Structure):
    _fields_ = [("qweight", ctypes.c_void_p), ("scales", ctypes.c_void_p), ("zeros", ctypes.c_void_p),
                ("q8", ctypes.c_void_p), ("w16", ctypes.c_void_p)]


class layer_weights_host(ctypes.Structure):
    _fields_ = [("attn_norm", ctypes.c_void_p), ("mlp_norm", ctypes.c_void_p)] + \
               [(n, qlinear_host) for n in ("q", "k", "v", "o", "gate", "up", "down")]


class lm_config(ctypes.Structure):
    _fields_ = [("vocab", ctypes.c_int32), ("hidden", ctypes.c_int32), ("group_size", ctypes.c_int32),
                ("rms_eps", ctypes.c_float), ("max_batch", ctypes.c_int32)]


class lm_weights_host(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("final_norm", ctypes.c_void_p), ("head", qlinear_host)]


class kv_desc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32), ("max_seq", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("stride_b", ctypes.c_int64), ("stride_h", ctypes.c_int64),
                ("stride_s", ctypes.c_int64), ("bytes", ctypes.c_size_t)]


_P = ctypes.c_void_p
_I = ctypes.c_int32
_SIG = {
    "layer_create": (ctypes.c_int, [ctypes.POINTER(layer_config), ctypes.POINTER(layer_weights_host), ctypes.POINTER(_P)]),
    "layer_destroy": (ctypes.c_int, [_P]),
    "kv_layout": (ctypes.c_int, [ctypes.POINTER(layer_config), _I, ctypes.POINTER(kv_desc)]),
    "layer_workspace_size": (ctypes.c_size_t, [_P, _I, _I, _I, _I]),
    "layer_prefill": (ctypes.c_int, [_P, _P, _P, _I, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "layer_prefill_kv": (ctypes.c_int, [_P, _P, _P, _I, _I, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "layer_prefill_chunked_workspace_size": (ctypes.c_size_t, [_P, _I, _I]),
    "layer_prefill_chunked": (ctypes.c_int, [_P, _P, _P, _I, _I, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "layer_decode": (ctypes.c_int, [_P, _P, _P, _P, _I, _P, _I, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "layer_decode_noalloc": (ctypes.c_int, [_P, _P, _P, _P, _I, _P, _I, _P, _P, _P, _P]),
    "layer_decode_noalloc_max_bytes": (ctypes.c_size_t, []),
    "kv_append": (ctypes.c_int, [ctypes.POINTER(kv_desc), _P, _P, _P, _P, _I, _I, _P, _P]),
    "layer_debug_dequant": (ctypes.c_int, [_P, _I, _P, _P]),
    "layer_set_decode_path": (ctypes.c_int, [_P, _I]),
    "layer_decode_phase_times": (ctypes.c_int, [_P, _P, _P]),
    "layer_debug_decode_stamps": (ctypes.c_int, [_P, _P, _I]),
    "layer_set_decode_trace": (ctypes.c_int, [_P, _I]),
    "layer_set_decode_spin_limit": (ctypes.c_int, [_P, _I]),
    "layer_profile_kernel": (ctypes.c_int, [_P, _I, _I]),
    "layer_profile_read": (ctypes.c_int, [_P, _I, ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_int32)]),
    "layer_last_error": (ctypes.c_char_p, []),
    "layer_error": (ctypes.c_int, [_P, ctypes.POINTER(ctypes.c_int32)]),
    "w4_ceiling_read": (ctypes.c_int, [_P, ctypes.c_size_t, _P, _I, _P]),
    "w4_ceiling_mfma": (ctypes.c_int, [_P, _I, _I, _I, ctypes.POINTER(ctypes.c_double), _P]),
    "stack_workspace_size": (ctypes.c_size_t, [_P, _I, _I, _I, _I, _I]),
    "stack_prefill": (ctypes.c_int, [_P, _I, _P, _P, _I, _I, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "stack_decode": (ctypes.c_int, [_P, _I, _P, _P, _P, _I, _P, _I, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "lm_create": (ctypes.c_int, [ctypes.POINTER(lm_config), ctypes.POINTER(lm_weights_host), ctypes.POINTER(_P)]),
    "lm_destroy": (ctypes.c_int, [_P]),
    "lm_embed": (ctypes.c_int, [_P, _P, _I, _P, _P]),
    "lm_head_workspace_size": (ctypes.c_size_t, [_P, _I]),
    "lm_head": (ctypes.c_int, [_P, _P, _I, _P, _P, _P, ctypes.c_size_t, _P]),
    "lm_error": (ctypes.c_int, [_P, ctypes.POINTER(ctypes.c_int32)]),
    "model_decode_workspace_size": (ctypes.c_size_t, [_P, _I, _P, _I, _I]),
    "model_decode_greedy": (ctypes.c_int, [_P, _I, _P, _P, _P, _P, _I, _I, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
}
for _name, (_res, _args) in _SIG.items():
    _f = getattr(_lib, _name)
    _f.restype = _res
    _f.argtypes = _args


def declared_functions() -> list:
    """Names of the functions include/w4layer.h declares."""
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w]+\s*\**\s+\**(\w+)\s*\(", text, flags=re.M)))


def exported(name: str) -> bool:
    try:
        getattr(_lib, name)
        return True
    except AttributeError:
        return False


def layer_last_error() -> str:
    return (_lib.layer_last_error() or b"").decode()


def check(rc: int) -> int:
    if rc != W4_OK:
        raise W4Error(rc, layer_last_error())
    return rc


def make_config(cfg, weight_format: int = W4_WEIGHTS_INT4) -> layer_config:
    """layer_config from any object with the LayerConfig attribute names."""
    return layer_config(cfg.hidden, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.ffn, cfg.group_size,
                        cfg.rms_eps, cfg.rope_base, cfg.max_seq, cfg.max_batch, weight_format)


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


# ------------------------------------------------------------ C-named calls

def layer_create(cfg, weights: dict):
    """weights: the host format of qlinear_host (numpy arrays): for each
    linear a dict with "format" ("int4" when absent, "int8" or "bf16"; all
    seven alike) and, for int4, qweight int32 [K/8][N], scales fp16
    [ceil(K/G)][N], optional zeros uint8; for int8, q8 [K][N] (int8 codes, or
    uint8 codes with per-column zeros uint8 [N]) and scales fp16 [N]; for
    bf16, w16 bf16 bit patterns [K][N]; attn_norm / mlp_norm bf16 bit
    patterns (uint16)."""
    keep = []

    def arr(a, dtype):
        a = np.ascontiguousarray(a)
        if a.dtype != dtype:
            a = a.view(dtype) if a.dtype.itemsize == np.dtype(dtype).itemsize else a.astype(dtype)
        keep.append(a)
        return a.ctypes.data

    wh = layer_weights_host()
    wh.attn_norm = arr(weights["attn_norm"], np.uint16)
    wh.mlp_norm = arr(weights["mlp_norm"], np.uint16)
    fmts = {weights[n].get("format", "int4") for n in ("q", "k", "v", "o", "gate", "up", "down")}
    if len(fmts) != 1:
        raise ValueError(f"the seven linears of a layer share one weight format, got {sorted(fmts)}")
    fmt = fmts.pop()
    for name in ("q", "k", "v", "o", "gate", "up", "down"):
        lin = weights[name]
        z = lin.get("zeros")
        zp = None if z is None else arr(z, np.uint8)
        if fmt == "int4":
            ql = qlinear_host(arr(lin["qweight"], np.int32), arr(lin["scales"], np.uint16), zp, None, None)
        elif fmt == "int8":
            ql = qlinear_host(None, arr(lin["scales"], np.uint16), zp, arr(lin["q8"], np.uint8), None)
        else:
            ql = qlinear_host(None, None, None, None, arr(lin["w16"], np.uint16))
        setattr(wh, name, ql)
    c = make_config(cfg, WEIGHT_FORMAT_CODE[fmt])
    h = _P()
    rc = _lib.layer_create(ctypes.byref(c), ctypes.byref(wh), ctypes.byref(h))
    return rc, h.value


def layer_destroy(handle) -> int:
    return _lib.layer_destroy(handle)


def kv_layout(cfg, batch: int):
    d = kv_desc()
    rc = _lib.kv_layout(ctypes.byref(make_config(cfg)), batch, ctypes.byref(d))
    return rc, d


def layer_workspace_size(handle, stage: int, batch: int, T: int, max_ctx: int) -> int:
    return _lib.layer_workspace_size(handle, stage, batch, T, max_ctx)


def layer_prefill(handle, x, pos, T, k_cache, v_cache, y, ws, ws_bytes, stream=None) -> int:
    return _lib.layer_prefill(handle, _ptr(x), _ptr(pos), T, _ptr(k_cache), _ptr(v_cache), _ptr(y), _ptr(ws),
                              ws_bytes, _stream(stream))


def layer_prefill_kv(handle, x, pos, T, hist_len, k_cache, v_cache, y, ws, ws_bytes, stream=None) -> int:
    return _lib.layer_prefill_kv(handle, _ptr(x), _ptr(pos), T, hist_len, _ptr(k_cache), _ptr(v_cache), _ptr(y),
                                 _ptr(ws), ws_bytes, _stream(stream))


def layer_prefill_chunked_workspace_size(handle, T, chunk) -> int:
    return _lib.layer_prefill_chunked_workspace_size(handle, T, chunk)


def layer_prefill_chunked(handle, x, pos, T, chunk, k_cache, v_cache, y, ws, ws_bytes, stream=None) -> int:
    return _lib.layer_prefill_chunked(handle, _ptr(x), _ptr(pos), T, chunk, _ptr(k_cache), _ptr(v_cache), _ptr(y),
                                      _ptr(ws), ws_bytes, _stream(stream))


def layer_decode(handle, x, pos, ctx_lens, max_ctx, attn_mask, B, k_cache, v_cache, y, ws, ws_bytes,
                 stream=None) -> int:
    return _lib.layer_decode(handle, _ptr(x), _ptr(pos), _ptr(ctx_lens), max_ctx, _ptr(attn_mask), B,
                             _ptr(k_cache), _ptr(v_cache), _ptr(y), _ptr(ws), ws_bytes, _stream(stream))


def layer_decode_noalloc(handle, x, pos, ctx_lens, max_ctx, attn_mask, B, k_cache, v_cache, y, stream=None) -> int:
    return _lib.layer_decode_noalloc(handle, _ptr(x), _ptr(pos), _ptr(ctx_lens), max_ctx, _ptr(attn_mask), B,
                                     _ptr(k_cache), _ptr(v_cache), _ptr(y), _stream(stream))


def layer_decode_noalloc_max_bytes() -> int:
    return _lib.layer_decode_noalloc_max_bytes()


def _ptr_array(handles):
    arr = (ctypes.c_void_p * len(handles))(*[_ptr(h) for h in handles])
    return arr


def stack_workspace_size(handles, stage: int, batch: int, T: int, max_ctx: int) -> int:
    return _lib.stack_workspace_size(_ptr_array(handles), len(handles), stage, batch, T, max_ctx)


def stack_prefill(handles, x, pos, T, hist_len, k_caches, v_caches, y, ws, ws_bytes, stream=None) -> int:
    return _lib.stack_prefill(_ptr_array(handles), len(handles), _ptr(x), _ptr(pos), T, hist_len,
                              _ptr_array(k_caches), _ptr_array(v_caches), _ptr(y), _ptr(ws), ws_bytes,
                              _stream(stream))


def stack_decode(handles, x, pos, ctx_lens, max_ctx, attn_mask, B, k_caches, v_caches, y, ws, ws_bytes,
                 stream=None) -> int:
    return _lib.stack_decode(_ptr_array(handles), len(handles), _ptr(x), _ptr(pos), _ptr(ctx_lens), max_ctx,
                             _ptr(attn_mask), B, _ptr_array(k_caches), _ptr_array(v_caches), _ptr(y), _ptr(ws),
                             ws_bytes, _stream(stream))


def kv_append(desc: kv_desc, k_cache, v_cache, k_new, v_new, B, T, slot_start, stream=None) -> int:
    ss = np.ascontiguousarray(np.asarray(slot_start, dtype=np.int32))
    return _lib.kv_append(ctypes.byref(desc), _ptr(k_cache), _ptr(v_cache), _ptr(k_new), _ptr(v_new), B, T,
                          ss.ctypes.data, _stream(stream))


def layer_debug_dequant(handle, which, out, stream=None) -> int:
    if isinstance(which, str):
        which = LINEAR_INDEX[which]
    return _lib.layer_debug_dequant(handle, which, _ptr(out), _stream(stream))


def w4_ceiling_read(buf, nbytes: int, sink, blocks: int, stream=None) -> int:
    return _lib.w4_ceiling_read(_ptr(buf), nbytes, _ptr(sink), blocks, _stream(stream))


def w4_ceiling_mfma(sink, blocks: int, iters: int, big: bool, stream=None):
    """Returns (rc, flop of the launch)."""
    f = ctypes.c_double()
    rc = _lib.w4_ceiling_mfma(_ptr(sink), blocks, iters, int(big), ctypes.byref(f), _stream(stream))
    return rc, f.value


def layer_error(handle):
    """(status, flag): the layer's W4_FLAG_* bits since the last call, cleared."""
    f = ctypes.c_int32(0)
    rc = _lib.layer_error(handle, ctypes.byref(f))
    return rc, f.value


def layer_decode_phase_times(handle):
    us = (ctypes.c_float * 5)()
    err = ctypes.c_int32()
    rc = _lib.layer_decode_phase_times(handle, ctypes.cast(us, ctypes.c_void_p), ctypes.cast(ctypes.pointer(err), ctypes.c_void_p))
    return rc, list(us), err.value


def layer_debug_decode_stamps(handle, n: int = 8 + 32 * 1024):
    out = np.zeros(n, dtype=np.uint64)
    rc = _lib.layer_debug_decode_stamps(handle, out.ctypes.data, n)
    return rc, out


def layer_set_decode_trace(handle, on: int) -> int:
    return _lib.layer_set_decode_trace(handle, int(on))


def layer_set_decode_spin_limit(handle, polls: int) -> int:
    return _lib.layer_set_decode_spin_limit(handle, polls)


def layer_set_decode_path(handle, path: int) -> int:
    return _lib.layer_set_decode_path(handle, path)


def layer_profile_kernel(handle, stage: int, kernel: int) -> int:
    return _lib.layer_profile_kernel(handle, stage, kernel)


def layer_profile_read(handle, stage: int):
    ms = ctypes.c_float()
    n = ctypes.c_int32()
    rc = _lib.layer_profile_read(handle, stage, ctypes.byref(ms), ctypes.byref(n))
    return rc, ms.value, n.value


# ------------------------------------------------------------ convenience

def lm_create(vocab: int, hidden: int, group_size: int, rms_eps: float, max_batch: int, lm: dict):
    """lm: the host format of synth.make_lm (embed bf16 bits [vocab][hidden],
    final_norm bf16 bits [hidden], head a linear dict hidden x vocab)."""
    keep = []

    def arr(a, dtype):
        a = np.ascontiguousarray(a)
        if a.dtype != dtype:
            a = a.view(dtype) if a.dtype.itemsize == np.dtype(dtype).itemsize else a.astype(dtype)
        keep.append(a)
        return a.ctypes.data

    head = lm["head"]
    z = head.get("zeros")
    wh = lm_weights_host(arr(lm["embed"], np.uint16), arr(lm["final_norm"], np.uint16),
                         qlinear_host(arr(head["qweight"], np.int32), arr(head["scales"], np.uint16),
                                      None if z is None else arr(z, np.uint8)))
    c = lm_config(vocab, hidden, group_size, rms_eps, max_batch)
    h = _P()
    rc = _lib.lm_create(ctypes.byref(c), ctypes.byref(wh), ctypes.byref(h))
    return rc, h.value


def lm_destroy(handle) -> int:
    return _lib.lm_destroy(handle)


def lm_embed(handle, tokens, B, x, stream=None) -> int:
    return _lib.lm_embed(handle, _ptr(tokens), B, _ptr(x), _stream(stream))


def lm_head_workspace_size(handle, B) -> int:
    return _lib.lm_head_workspace_size(handle, B)


def lm_head(handle, x, B, logits, next_tokens, ws, ws_bytes, stream=None) -> int:
    return _lib.lm_head(handle, _ptr(x), B, _ptr(logits), _ptr(next_tokens), _ptr(ws), ws_bytes, _stream(stream))


def lm_error(handle):
    f = ctypes.c_int32(0)
    rc = _lib.lm_error(handle, ctypes.byref(f))
    return rc, f.value


def model_decode_workspace_size(handles, lm_handle, B, max_ctx) -> int:
    return _lib.model_decode_workspace_size(_ptr_array(handles), len(handles), lm_handle, B, max_ctx)


def model_decode_greedy(handles, lm_handle, tokens, pos, ctx_lens, max_ctx, B, k_caches, v_caches, logits,
                        next_tokens, ws, ws_bytes, stream=None) -> int:
    return _lib.model_decode_greedy(_ptr_array(handles), len(handles), lm_handle, _ptr(tokens), _ptr(pos),
                                    _ptr(ctx_lens), max_ctx, B, _ptr_array(k_caches), _ptr_array(v_caches),
                                    _ptr(logits), _ptr(next_tokens), _ptr(ws), ws_bytes, _stream(stream))


# Handles still open when the interpreter exits are closed by an exit hook,
# which runs before the interpreter and the HIP runtime tear down; the
# finalisers of the owning objects make no library (HIP) call once the
# interpreter is finalising.
_live = weakref.WeakSet()


@atexit.register
def _close_all():
    for obj in list(_live):
        try:
            obj.close()
        except Exception:
            pass


class LM:
    """Owns a model-ends handle (embedding, LM head, greedy sampling) plus
    reusable workspace; methods raise W4Error."""

    def __init__(self, cfg, lm: dict, max_batch: int = 8):
        import torch
        self.cfg, self.vocab = cfg, lm["vocab"]
        rc, self.handle = lm_create(self.vocab, cfg.hidden, cfg.group_size, cfg.rms_eps, max_batch, lm)
        check(rc)
        _live.add(self)
        self._ws = torch.empty(0, dtype=torch.uint8, device="cuda")

    def close(self):
        if self.handle:
            lm_destroy(self.handle)
            self.handle = None

    def __del__(self):
        if sys is None or sys.is_finalizing():
            return
        try:
            self.close()
        except Exception:
            pass

    def embed(self, tokens, x, stream=None):
        check(lm_embed(self.handle, tokens, tokens.shape[0], x, stream))

    def head(self, x, logits, next_tokens=None, stream=None):
        import torch
        B = x.shape[0]
        n = lm_head_workspace_size(self.handle, B)
        if n == 0:
            raise W4Error(W4_EINVAL, "invalid workspace query")
        if self._ws.numel() < n:
            self._ws = torch.empty(n, dtype=torch.uint8, device="cuda")
        check(lm_head(self.handle, x, B, logits, next_tokens, self._ws, self._ws.numel(), stream))

    def error(self) -> int:
        rc, f = lm_error(self.handle)
        check(rc)
        return f


class Layer:
    """Owns a layer handle plus reusable workspace; methods raise W4Error."""

    def __init__(self, cfg, weights: dict):
        import torch
        self.cfg = cfg
        rc, self.handle = layer_create(cfg, weights)
        check(rc)
        _live.add(self)
        self._ws = torch.empty(0, dtype=torch.uint8, device="cuda")

    def close(self):
        if self.handle:
            layer_destroy(self.handle)
            self.handle = None

    def __del__(self):
        if sys is None or sys.is_finalizing():
            return
        try:
            self.close()
        except Exception:
            pass

    def error(self) -> int:
        """The layer's W4_FLAG_* bits since the last call (read and cleared)."""
        rc, f = layer_error(self.handle)
        check(rc)
        return f

    def workspace(self, stage, batch, T, max_ctx):
        import torch
        n = layer_workspace_size(self.handle, stage, batch, T, max_ctx)
        if n == 0:
            raise W4Error(W4_EINVAL, "invalid workspace query")
        if self._ws.numel() < n:
            self._ws = torch.empty(n, dtype=torch.uint8, device="cuda")
        return self._ws, self._ws.numel()

    def new_cache(self, batch: int, fill_bits: Optional[int] = None):
        """A K and a V cache in the kv_layout(cfg, batch) layout (uint16 bf16
        bit patterns), optionally filled with one bit pattern."""
        import torch
        rc, d = kv_layout(self.cfg, batch)
        check(rc)
        shape = (batch, d.n_kv_heads, d.max_seq, d.head_dim)
        k = torch.empty(shape, dtype=torch.int16, device="cuda")
        v = torch.empty(shape, dtype=torch.int16, device="cuda")
        if fill_bits is not None:
            val = int(np.array([fill_bits], dtype=np.uint16).view(np.int16)[0])
            k.fill_(val)
            v.fill_(val)
        return k, v

    def prefill(self, x, pos, k_cache, v_cache, y, stream=None):
        ws, n = self.workspace(STAGE_PREFILL, 1, x.shape[0], 0)
        check(layer_prefill(self.handle, x, pos, x.shape[0], k_cache, v_cache, y, ws, n, stream))

    def prefill_kv(self, x, pos, hist_len, k_cache, v_cache, y, stream=None):
        ws, n = self.workspace(STAGE_PREFILL_KV, 1, x.shape[0], hist_len)
        check(layer_prefill_kv(self.handle, x, pos, x.shape[0], hist_len, k_cache, v_cache, y, ws, n, stream))

    def prefill_chunked(self, x, pos, chunk, k_cache, v_cache, y, stream=None):
        import torch
        T = x.shape[0]
        n = layer_prefill_chunked_workspace_size(self.handle, T, chunk)
        if n == 0:
            raise W4Error(W4_EINVAL, "invalid workspace query")
        if self._ws.numel() < n:
            self._ws = torch.empty(n, dtype=torch.uint8, device="cuda")
        check(layer_prefill_chunked(self.handle, x, pos, T, chunk, k_cache, v_cache, y, self._ws, self._ws.numel(),
                                    stream))

    def decode(self, x, pos, ctx_lens, max_ctx, k_cache, v_cache, y, attn_mask=None, stream=None):
        B = x.shape[0]
        ws, n = self.workspace(STAGE_DECODE, B, 1, max_ctx)
        check(layer_decode(self.handle, x, pos, ctx_lens, max_ctx, attn_mask, B, k_cache, v_cache, y, ws, n, stream))

    def set_decode_path(self, path: int):
        """0 automatic, 1 separate kernels, 2 one persistent launch."""
        check(layer_set_decode_path(self.handle, path))

    def debug_dequant(self, which):
        import torch
        K, N = self.cfg.linear_shape(which)
        out = torch.empty((K, N), dtype=torch.float32, device="cuda")
        check(layer_debug_dequant(self.handle, which, out))
        return out


class Stack:
    """A list of Layer objects run back to back (stack_prefill / stack_decode),
    each with its own K and V cache, sharing one workspace."""

    def __init__(self, layers):
        import torch
        self.layers = list(layers)
        self.handles = [l.handle for l in self.layers]
        self._ws = torch.empty(0, dtype=torch.uint8, device="cuda")

    def workspace(self, stage, batch, T, max_ctx):
        import torch
        n = stack_workspace_size(self.handles, stage, batch, T, max_ctx)
        if n == 0:
            raise W4Error(W4_EINVAL, "invalid workspace query")
        if self._ws.numel() < n:
            self._ws = torch.empty(n, dtype=torch.uint8, device="cuda")
        return self._ws, self._ws.numel()

    def prefill(self, x, pos, hist_len, k_caches, v_caches, y, stream=None):
        stage = STAGE_PREFILL_KV if hist_len > 0 else STAGE_PREFILL
        ws, n = self.workspace(stage, 1, x.shape[0], hist_len)
        check(stack_prefill(self.handles, x, pos, x.shape[0], hist_len, k_caches, v_caches, y, ws, n, stream))

    def decode(self, x, pos, ctx_lens, max_ctx, k_caches, v_caches, y, attn_mask=None, stream=None):
        B = x.shape[0]
        ws, n = self.workspace(STAGE_DECODE, B, 1, max_ctx)
        check(stack_decode(self.handles, x, pos, ctx_lens, max_ctx, attn_mask, B, k_caches, v_caches, y, ws, n,
                           stream))
