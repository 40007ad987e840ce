"""Pins of the oracle's INT8 and BF16 weight formats (the paper's
direct-through weight modes besides W4, Sec. 3.2): brute-force scalar loops
with hand-decoded fp16 scales, the sign-byte identity between the symmetric
and asymmetric INT8 readings, bf16 bit patterns of known value, and the
block's independence of the format that carries a given weight."""
import struct

import numpy as np
import pytest

from oracle import layer as O
from paper_2607_15865_amd import synth


def _fp16(bits: int) -> float:
    return struct.unpack("<e", int(bits).to_bytes(2, "little"))[0]


def _bf16(bits: int) -> float:
    return struct.unpack("<f", (int(bits) << 16).to_bytes(4, "little"))[0]


def _scales(rng, N):
    sbits = rng.integers(0, 1 << 16, size=N).astype(np.uint16)
    sbits[0] = 0x0001                         # smallest subnormal
    sbits[1 % N] = 0xBC00                     # -1
    exp = (sbits >> 10) & 0x1F
    sbits[exp == 0x1F] = 0x3C00               # no inf / nan scales
    return sbits


@pytest.mark.parametrize("K,N", [(5, 3), (16, 7)])
def test_int8_symmetric_brute_force(K, N):
    rng = np.random.default_rng(K * 31 + N)
    q = rng.integers(-128, 128, size=(K, N), dtype=np.int16).astype(np.int8)
    q[0, 0], q[-1, -1], q[1, 0] = -128, 127, 0
    sbits = _scales(rng, N)
    lin = dict(format="int8", K=K, N=N, q8=q, scales=sbits.view(np.float16), zeros=None)
    got = O.dequant(lin, 128)
    raw = q.view(np.uint8)
    for k in range(K):
        for n in range(N):
            b = int(raw[k, n])
            code = b - 256 if b >= 128 else b          # two's complement byte
            assert got[k, n] == _fp16(sbits[n]) * code


@pytest.mark.parametrize("K,N", [(5, 3), (16, 7)])
def test_int8_asymmetric_brute_force(K, N):
    rng = np.random.default_rng(K * 17 + N)
    u = rng.integers(0, 256, size=(K, N), dtype=np.int16).astype(np.uint8)
    u[0, 0], u[-1, -1] = 0, 255
    z = rng.integers(0, 256, size=N, dtype=np.int16).astype(np.uint8)
    z[0], z[-1] = 0, 255
    sbits = _scales(rng, N)
    lin = dict(format="int8", K=K, N=N, q8=u, scales=sbits.view(np.float16), zeros=z)
    got = O.dequant(lin, 128)
    for k in range(K):
        for n in range(N):
            assert got[k, n] == _fp16(sbits[n]) * (int(u[k, n]) - int(z[n]))


def test_int8_sign_byte_identity():
    """A symmetric code q is the asymmetric code q + 128 with zero point 128."""
    rng = np.random.default_rng(3)
    K, N = 64, 9
    q = rng.integers(-128, 128, size=(K, N), dtype=np.int16).astype(np.int8)
    s = (np.abs(rng.normal(0, 0.02, N)) / 128).astype(np.float16)
    sym = dict(format="int8", K=K, N=N, q8=q, scales=s, zeros=None)
    asym = dict(format="int8", K=K, N=N, q8=(q.view(np.uint8) ^ np.uint8(0x80)), scales=s,
                zeros=np.full(N, 128, dtype=np.uint8))
    assert np.array_equal(O.dequant(sym, 128), O.dequant(asym, 128))


def test_bf16_weights_exact():
    bits = np.array([[0x3F80, 0xBF80, 0x4049], [0x0001, 0x7F7F, 0x0000]], dtype=np.uint16)
    lin = dict(format="bf16", K=2, N=3, w16=bits)
    got = O.dequant(lin, 128)
    assert got[0, 0] == 1.0 and got[0, 1] == -1.0 and got[0, 2] == 3.140625
    assert got[1, 0] == 2.0 ** -133 and got[1, 2] == 0.0
    for k in range(2):
        for n in range(3):
            assert got[k, n] == _bf16(bits[k, n])


def test_unknown_format_rejected():
    with pytest.raises(ValueError):
        O.dequant(dict(format="int3", K=1, N=1), 128)


def test_generator_formats():
    cfg = synth.CONFIGS["tiny"]
    s8 = synth.make_linear(cfg, "down", fmt="int8")
    assert s8["q8"].dtype == np.int8 and s8["q8"].shape == (688, 256) and s8["zeros"] is None
    assert s8["q8"].min() == -128 and s8["q8"].max() == 127 and s8["scales"].shape == (256,)
    a8 = synth.make_linear(cfg, "down", fmt="int8a")
    assert a8["q8"].dtype == np.uint8 and a8["q8"].min() == 0 and a8["q8"].max() == 255
    assert a8["zeros"].min() >= 96 and a8["zeros"].max() <= 160
    b = synth.make_linear(cfg, "down", fmt="bf16")
    assert b["w16"].dtype == np.uint16 and b["w16"].shape == (688, 256)
    w = O.dequant(b, cfg.group_size)
    assert 0.009 < w.std() < 0.011


def test_block_depends_on_the_weights_only():
    """One set of weights carried by all four formats gives the same block.

    The int4 weights use one power-of-two scale per column (every group
    alike) and zero point 8, so s (q - 8) is exactly an int8 code times the
    same scale and exactly a bf16 value."""
    cfg = synth.CONFIGS["tiny"]
    rng = np.random.default_rng(11)
    w4, w8, w8a, wb = {}, {}, {}, {}
    for name in synth.LINEARS:
        K, N = cfg.linear_shape(name)
        ng = -(-K // cfg.group_size)
        q = rng.integers(0, 16, size=(K, N), dtype=np.uint8)
        col = np.ldexp(1.0, rng.integers(-10, -6, size=N)).astype(np.float16)
        w4[name] = dict(K=K, N=N, qweight=synth.pack_int4(q), scales=np.tile(col, (ng, 1)), zeros=None)
        c = q.astype(np.int16) - 8
        w8[name] = dict(format="int8", K=K, N=N, q8=c.astype(np.int8), scales=col, zeros=None)
        w8a[name] = dict(format="int8", K=K, N=N, q8=(c + 100).astype(np.uint8), scales=col,
                         zeros=np.full(N, 100, dtype=np.uint8))
        wv = c.astype(np.float64) * col.astype(np.float64)[None, :]
        wb[name] = dict(format="bf16", K=K, N=N, w16=synth.bf16_bits(wv))
        assert np.array_equal(O.bf16_to_f64(wb[name]["w16"]), wv)
    for w in (w4, w8, w8a, wb):
        w["attn_norm"] = synth.bf16_bits(rng.uniform(0.5, 1.5, cfg.hidden))
        w["mlp_norm"] = synth.bf16_bits(rng.uniform(0.5, 1.5, cfg.hidden))
    for w in (w8, w8a, wb):
        w["attn_norm"], w["mlp_norm"] = w4["attn_norm"], w4["mlp_norm"]
    T = 6
    x = O.bf16_to_f64(synth.activations(cfg, synth.TID_X_PREFILL, T))
    pos = np.arange(T)
    y4, k4, v4 = O.prefill(w4, cfg, x, pos)
    for w in (w8, w8a, wb):
        y, k, v = O.prefill(w, cfg, x, pos)
        assert np.array_equal(y, y4) and np.array_equal(k, k4) and np.array_equal(v, v4)
