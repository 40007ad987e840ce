"""The C ABI on the host, no GPU needed: the library loads and exports every
function include/w4layer.h declares, the KV layout arithmetic, and the
argument validation that happens before any HIP call."""
import os

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2607_15865_amd", "libw4layer.so")

if not os.path.exists(LIB):  # the driver builds first; build here if it has not
    from paper_2607_15865_amd import build as _b
    _b.build()

from paper_2607_15865_amd import binding as B  # noqa: E402
from paper_2607_15865_amd import synth  # noqa: E402
from conftest import read_golden  # noqa: E402


def test_every_declared_function_is_exported():
    names = B.declared_functions()
    assert {"layer_prefill", "layer_prefill_kv", "layer_decode", "kv_append", "kv_layout",
            "layer_create", "layer_destroy", "layer_workspace_size"} <= set(names)
    missing = [n for n in names if not B.exported(n)]
    assert not missing, missing


def test_kv_layout_strides():
    cfg = synth.CONFIGS["llama8b"]
    rc, d = B.kv_layout(cfg, 3)
    assert rc == 0
    assert (d.batch, d.n_kv_heads, d.max_seq, d.head_dim) == (3, 8, 4096, 128)
    assert d.stride_s == 128 and d.stride_h == 4096 * 128 and d.stride_b == 8 * 4096 * 128
    assert d.bytes == 3 * 8 * 4096 * 128 * 2
    assert B.kv_layout(cfg, 0)[0] == B.W4_EINVAL


def test_kv_bytes_of_the_paper_example():
    """The worked example of Sec. 2.3: 32 layers, 100 tokens, 2 kv heads,
    head_dim 128 -> K and V of 100 * 2 * 128 bf16 values per layer."""
    cfg = synth.replace(synth.CONFIGS["llama8b"], n_kv_heads=2, max_seq=100)
    rc, d = B.kv_layout(cfg, 1)
    assert rc == 0
    assert 32 * 2 * d.bytes == 32 * 2 * 100 * 2 * 128 * 2


def test_stage_calls_validate_before_any_hip_call():
    assert B.layer_prefill(None, 1, 1, 4, 1, 1, 2, 1, 1 << 20, 0) == B.W4_EINVAL
    assert B.layer_prefill_kv(None, 1, 1, 4, 0, 1, 1, 2, 1, 1 << 20, 0) == B.W4_EINVAL
    assert B.layer_decode(None, 1, 1, 1, 8, None, 1, 1, 1, 2, 1, 1 << 20, 0) == B.W4_EINVAL
    assert B.layer_prefill_chunked(None, 1, 1, 4, 2, 1, 1, 2, 1, 1 << 20, 0) == B.W4_EINVAL
    assert B.layer_prefill_chunked_workspace_size(None, 4, 2) == 0
    assert "null layer" in B.layer_last_error()
    assert B.layer_workspace_size(None, 0, 1, 16, 0) == 0
    assert B.layer_debug_dequant(None, 0, 1, stream=0) == B.W4_EINVAL
    assert B.layer_profile_kernel(None, 0, 1) == B.W4_EINVAL


def test_stack_calls_validate_before_any_hip_call():
    assert B.stack_workspace_size([], 2, 1, 1, 8) == 0
    assert B.stack_workspace_size([None], 0, 1, 16, 0) == 0
    assert B.stack_prefill([], 1, 1, 4, 0, [], [], 2, 1, 1 << 20, 0) == B.W4_EINVAL
    assert B.stack_prefill([None, None], 1, 1, 4, 0, [1, 1], [1, 1], 2, 1, 1 << 20, 0) == B.W4_EINVAL
    assert "null layer" in B.layer_last_error()
    assert B.stack_decode([], 1, 1, 1, 8, None, 1, [], [], 2, 1, 1 << 20, 0) == B.W4_EINVAL


def test_kv_append_validation():
    cfg = synth.CONFIGS["tiny"]
    rc, d = B.kv_layout(cfg, 2)
    assert B.kv_append(d, 1, 1, 1, 1, 2, 4, [0, cfg.max_seq - 3], stream=0) == B.W4_ECAPACITY
    assert B.kv_append(d, 1, 1, 1, 1, 3, 4, [0, 0, 0], stream=0) == B.W4_ECAPACITY
    assert B.kv_append(d, 1, 1, 1, 1, 2, 0, [0, 0], stream=0) == B.W4_EINVAL
    assert B.kv_append(d, 1, 1, 1, 1, 2, 4, [-1, 0], stream=0) == B.W4_ECAPACITY


@pytest.mark.parametrize("field,value,code", [
    ("head_dim", 96, B.W4_EUNSUPPORTED), ("n_kv_heads", 3, B.W4_EUNSUPPORTED),
    ("group_size", 48, B.W4_EUNSUPPORTED), ("hidden", 200, B.W4_EUNSUPPORTED),
    ("ffn", 690, B.W4_EUNSUPPORTED), ("hidden", 0, B.W4_EINVAL), ("max_seq", 0, B.W4_EINVAL),
    ("n_heads", 36, B.W4_EUNSUPPORTED)])
def test_layer_create_rejects_bad_configs(field, value, code):
    cfg = synth.replace(synth.CONFIGS["tiny"], **{field: value})
    w = synth.make_layer(synth.CONFIGS["tiny"])
    rc, h = B.layer_create(cfg, w)
    assert rc == code, (field, value, rc, B.layer_last_error())
    assert not h


def test_bandwidth_utilisation_definition():
    """Bandwidth utilisation as Sec. 5.1 defines it (tokens/s x model size /
    peak bandwidth) reproduces Table 2 within its printed rounding."""
    for row in read_golden("table2_bw_util.txt"):
        size, tps, printed = float(row[1]), float(row[2]), float(row[3])
        util = 100.0 * tps * size / 64.0
        assert abs(util - printed) < 0.5, row


def test_lm_validation_before_any_hip_call():
    cfg = synth.CONFIGS["tiny"]
    lm = synth.make_lm(cfg, 128)
    H, G = cfg.hidden, cfg.group_size
    assert B.lm_create(96, H, G, 1e-6, 8, lm)[0] == B.W4_EUNSUPPORTED          # vocab % 64
    assert B.lm_create(128, H, 48, 1e-6, 8, lm)[0] == B.W4_EUNSUPPORTED        # group size
    assert B.lm_create(128, 7808, G, 1e-6, 8, lm)[0] == B.W4_EUNSUPPORTED      # hidden too large
    assert B.lm_create(128, H, G, 1e-6, 65, lm)[0] == B.W4_EUNSUPPORTED        # max_batch
    assert B.lm_create(128, H, G, -1.0, 8, lm)[0] == B.W4_EINVAL               # eps
    bad = dict(lm, head=dict(lm["head"], scales=lm["head"]["scales"].copy()))
    bad["head"]["scales"][1, 5] = np.float16(np.inf)
    assert B.lm_create(128, H, G, 1e-6, 8, bad)[0] == B.W4_EINVAL
    assert "scale" in B.layer_last_error()
    assert B.lm_embed(None, 0, 1, 0, 0) == B.W4_EINVAL
    assert B.lm_head(None, 0, 1, 0, None, 0, 0, 0) == B.W4_EINVAL
    assert B.lm_head_workspace_size(None, 1) == 0
    assert B.lm_error(None)[0] == B.W4_EINVAL
    assert B.lm_destroy(None) == B.W4_EINVAL


def test_layer_create_weight_format_checks_before_any_hip_call():
    """An unknown weight format, and a format whose weight pointers are
    missing, are rejected on the host (no device needed)."""
    import ctypes
    cfg = synth.CONFIGS["tiny"]
    for fmt, code in ((7, B.W4_EINVAL), (-1, B.W4_EINVAL)):
        c = B.make_config(cfg, fmt)
        wh = B.layer_weights_host()
        h = ctypes.c_void_p()
        assert B._lib.layer_create(ctypes.byref(c), ctypes.byref(wh), ctypes.byref(h)) == code
        assert not h.value
    w8 = synth.make_layer(cfg, fmt="int8")
    for fmt in (B.W4_WEIGHTS_INT8, B.W4_WEIGHTS_BF16):
        c = B.make_config(cfg, fmt)
        wh = B.layer_weights_host()
        keep = []
        for name in synth.LINEARS:          # only the INT4 fields set: the format's own are missing
            q = np.zeros((cfg.linear_shape(name)[0] // 8, cfg.linear_shape(name)[1]), np.int32)
            s = np.ascontiguousarray(w8[name]["scales"]).view(np.uint16)
            keep += [q, s]
            setattr(wh, name, B.qlinear_host(q.ctypes.data, s.ctypes.data, None, None, None))
        h = ctypes.c_void_p()
        assert B._lib.layer_create(ctypes.byref(c), ctypes.byref(wh), ctypes.byref(h)) == B.W4_EINVAL
        assert "null weight pointer" in B.layer_last_error()


def test_binding_rejects_mixed_formats():
    cfg = synth.CONFIGS["tiny"]
    w = synth.make_layer(cfg, fmt="int8")
    w["down"] = synth.make_linear(cfg, "down", fmt="bf16")
    with pytest.raises(ValueError):
        B.layer_create(cfg, w)
