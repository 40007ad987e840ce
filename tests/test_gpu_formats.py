"""The paper's other direct-through weight modes (Sec. 3.2) on the GPU:
INT8 symmetric, INT8 asymmetric (per-channel scales) and BF16 weights, through
the prefill GEMM and the decode GEMV with their own fragment unpack.  Device
weights bit-exact against the oracle's dequantisation (BF16: up to the fp16
grid below 2^-17); all three stages within the parity bar (max-abs 2e-2,
relative Frobenius 1e-2) against the oracle on the same seeded inputs, from the
tiny layer to the Llama-3-8B-shaped layer."""
import functools

import numpy as np
import pytest
import torch

from oracle import layer as O
from paper_2607_15865_amd import binding, synth
from gpu_helpers import assert_parity, bits_to_torch_f32, cache_values, log, to_cache_bits

pytestmark = pytest.mark.gpu

FORMATS = ("int8", "int8a", "bf16")


@functools.lru_cache(maxsize=2)
def _host(name, fmt):
    cfg = synth.CONFIGS[name]
    w = synth.make_layer(cfg, fmt=fmt)
    return cfg, w, O.dequant_layer(w, cfg)


_dev = {}


def _layer(name, fmt):
    key = (name, fmt)
    if key not in _dev:
        if len(_dev) >= 2:
            _dev.pop(next(iter(_dev))).close()
        cfg, w, _ = _host(name, fmt)
        _dev[key] = binding.Layer(cfg, w)
    return _dev[key]


def teardown_module(module):
    for lay in _dev.values():
        lay.close()
    _dev.clear()


def _x(cfg, tid, rows):
    bits = synth.activations(cfg, tid, rows)
    return bits, O.bf16_to_f64(bits)


@pytest.mark.parametrize("fmt", FORMATS)
@pytest.mark.parametrize("name", ["tiny", "qwen05b"])
def test_format_dequant_exact(name, fmt):
    cfg, w, W = _host(name, fmt)
    lay = _layer(name, fmt)
    for lin in synth.LINEARS:
        got = lay.debug_dequant(lin).cpu().numpy().astype(np.float64)
        ref = W[lin]
        if fmt == "bf16":
            # the device's fp16 holds every bf16 value of magnitude >= 2^-17
            # exactly; below it, values on the fp16 subnormal grid 2^-24
            # (rounded once there, and for the elements held times 16 once
            # more on the way back: error < 2^-24)
            big = np.abs(ref) >= 2.0 ** -17
            assert np.array_equal(got[big], ref[big]), f"{lin}: {np.sum(got[big] != ref[big])} mismatches"
            assert np.max(np.abs(got - ref)) < 2.0 ** -24
        else:
            assert np.array_equal(got, ref), f"{lin}: {np.sum(got != ref)} mismatches"
    log(f"dequant {name} {fmt}: exact")


@pytest.mark.parametrize("fmt", FORMATS)
@pytest.mark.parametrize("name,T,rows", [("tiny", 32, None), ("tiny", 77, None),
                                         ("llama8b", 512, [0, 1, 2, 63, 64, 255, 256, 510, 511])])
def test_format_prefill(name, T, rows, fmt):
    cfg, w, W = _host(name, fmt)
    lay = _layer(name, fmt)
    lay.set_decode_path(0)
    log(f"prefill {name} {fmt} T={T}")
    xb, xv = _x(cfg, synth.TID_X_PREFILL, T)
    pos = np.arange(T)
    k, v = lay.new_cache(1, 0)
    x = bits_to_torch_f32(xb)
    y = torch.empty_like(x)
    lay.prefill(x, torch.from_numpy(pos.astype(np.int32)).cuda(), k, v, y)
    torch.cuda.synchronize()
    assert lay.error() == 0
    yo, ko, vo = O.prefill(w, cfg, xv, pos, rows=rows, W=W)
    gy = y.cpu().numpy().astype(np.float64)
    assert_parity(gy if rows is None else gy[rows], yo, "y")
    gk = cache_values(k)[0][:, :T, :].transpose(1, 0, 2)
    gv = cache_values(v)[0][:, :T, :].transpose(1, 0, 2)
    assert_parity(gk, ko, "new K")
    assert_parity(gv, vo, "new V")


@pytest.mark.parametrize("fmt", FORMATS)
@pytest.mark.parametrize("name,T,L", [("tiny", 16, 32), ("tiny", 5, 100), ("llama8b", 128, 1024)])
def test_format_prefill_kv(name, T, L, fmt):
    """A chunk of T tokens after an L-token history (the oracle's own prefill
    of the history, given to both sides); T = 5 runs on the decode kernels."""
    cfg, w, W = _host(name, fmt)
    lay = _layer(name, fmt)
    lay.set_decode_path(0)
    log(f"prefill_kv {name} {fmt} T={T} L={L}")
    _, xh = _x(cfg, synth.TID_X_PREFILL, L)
    _, kh, vh = O.prefill(w, cfg, xh, np.arange(L), rows=[L - 1], W=W)
    kc = O.cache_write(np.zeros((cfg.n_kv_heads, cfg.max_seq, cfg.head_dim)), kh, 0)
    vc = O.cache_write(np.zeros_like(kc), vh, 0)
    k = torch.from_numpy(to_cache_bits(kc)[None]).cuda()
    v = torch.from_numpy(to_cache_bits(vc)[None]).cuda()
    xb, xv = _x(cfg, synth.TID_X_PREFILL_KV, T)
    pos = np.arange(L, L + T)
    x = bits_to_torch_f32(xb)
    y = torch.empty_like(x)
    lay.prefill_kv(x, torch.from_numpy(pos.astype(np.int32)).cuda(), L, k, v, y)
    torch.cuda.synchronize()
    assert lay.error() == 0
    yo, ko, vo = O.prefill_kv(w, cfg, xv, pos, kc, vc, L, W=W)
    assert_parity(y.cpu().numpy(), yo, "y")
    gk = cache_values(k)[0][:, L:L + T, :].transpose(1, 0, 2)
    gv = cache_values(v)[0][:, L:L + T, :].transpose(1, 0, 2)
    assert_parity(gk, ko, "new K")
    assert_parity(gv, vo, "new V")


@pytest.mark.parametrize("fmt", FORMATS)
@pytest.mark.parametrize("name,B,ctx,path", [("tiny", 1, [48], 0), ("tiny", 4, [0, 9, 64, 126], 0),
                                             ("llama8b", 1, [2048], 0), ("llama8b", 3, [2048, 17, 4000], 1)])
def test_format_decode(name, B, ctx, path, fmt):
    """Decode against the N(0, 1) bf16 cache of the decode workloads, with
    positions that are not the cache slots."""
    cfg, w, W = _host(name, fmt)
    lay = _layer(name, fmt)
    lay.set_decode_path(path)
    log(f"decode {name} {fmt} B={B} ctx={ctx} path={path}")
    kb, vb = synth.kv_fill(cfg, B)
    kc, vc = O.bf16_to_f64(kb), O.bf16_to_f64(vb)
    ctx = np.array(ctx, dtype=np.int32)
    pos = ((7 * ctx + 5) % cfg.max_seq).astype(np.int32)      # positions in the RoPE table, not the slots
    xb, xv = _x(cfg, synth.TID_X_DECODE, B)
    k = torch.from_numpy(kb.view(np.int16)).cuda()
    v = torch.from_numpy(vb.view(np.int16)).cuda()
    x = bits_to_torch_f32(xb)
    y = torch.empty_like(x)
    lay.decode(x, torch.from_numpy(pos).cuda(), torch.from_numpy(ctx).cuda(), int(ctx.max()), k, v, y)
    torch.cuda.synchronize()
    assert lay.error() == 0
    yo, ko, vo = O.decode(w, cfg, xv, pos, kc, vc, ctx, W=W)
    assert_parity(y.cpu().numpy(), yo, "y")
    gk, gv = cache_values(k), cache_values(v)
    assert_parity(np.stack([gk[b][:, ctx[b], :] for b in range(B)]), ko, "new K")
    assert_parity(np.stack([gv[b][:, ctx[b], :] for b in range(B)]), vo, "new V")
    lay.set_decode_path(0)


@pytest.mark.parametrize("fmt", FORMATS)
def test_format_persistent_path_refused(fmt):
    """The persistent decode launch takes INT4 weights only: forcing it on an
    8- or 16-bit layer fails before any launch; the automatic choice runs the
    kernel sequence."""
    cfg, w, _ = _host("tiny", fmt)
    lay = _layer("tiny", fmt)
    lay.set_decode_path(2)
    k, v = lay.new_cache(1, 0)
    x = torch.zeros(1, cfg.hidden, device="cuda")
    y = torch.empty_like(x)
    c = torch.tensor([3], dtype=torch.int32, device="cuda")
    with pytest.raises(binding.W4Error) as e:
        lay.decode(x, c, c, 3, k, v, y)
    assert e.value.code == binding.W4_EUNSUPPORTED
    lay.set_decode_path(0)


def test_bf16_weight_range_checked():
    cfg = synth.CONFIGS["tiny"]
    w = synth.make_layer(cfg, fmt="bf16")
    w16 = w["o"]["w16"].copy()
    w16[3, 5] = 0x4580                        # 4096.0
    w["o"] = dict(w["o"], w16=w16)
    rc, h = binding.layer_create(cfg, w)
    assert rc == binding.W4_EINVAL and not h
    w16[3, 5] = 0x457F                        # 4080.0, the largest bf16 below 4096
    rc, h = binding.layer_create(cfg, w)
    assert rc == binding.W4_OK and h
    binding.layer_destroy(h)
