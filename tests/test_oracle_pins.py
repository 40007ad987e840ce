"""Pins of the CPU oracle against what the paper and the mathematics fix:
hand-derived fixtures, brute force on tiny inputs, closed forms and special
cases.  None of these re-types the oracle's own formula."""
import math
import struct

import numpy as np
import pytest
import torch

from oracle import layer as O
from paper_2607_15865_amd import synth
from conftest import read_golden


# ------------------------------------------------------------ number formats

def test_bf16_decode_all_patterns():
    bits = np.arange(1 << 16, dtype=np.uint16)
    ours = O.bf16_to_f64(bits)
    ref = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).to(torch.float64).numpy()
    finite = np.isfinite(ref)
    assert np.array_equal(ours[finite], ref[finite])
    assert np.array_equal(np.isnan(ours), np.isnan(ref))


def test_round_bf16_matches_torch_on_fp32_values():
    rng = np.random.default_rng(7)
    v = rng.standard_normal(200000).astype(np.float32).astype(np.float64)
    v *= np.exp2(rng.integers(-140, 120, size=v.shape)).astype(np.float64)
    v = v.astype(np.float32).astype(np.float64)          # keep fp32-exact
    ref = torch.from_numpy(v).to(torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(O.round_bf16(v), ref)


def test_round_bf16_ties_to_even():
    # midpoints of consecutive bf16 values are exact in fp32; RNE picks the
    # neighbour with an even last bit
    rng = np.random.default_rng(3)
    b = rng.integers(0x0080, 0x7F00, size=5000).astype(np.uint16)
    lo = O.bf16_to_f64(b)
    hi = O.bf16_to_f64(b + 1)
    mid = (lo + hi) / 2
    even = np.where(b % 2 == 0, lo, hi)
    assert np.array_equal(O.round_bf16(mid), even)
    assert np.array_equal(O.round_bf16(-mid), -even)


def test_round_bf16_no_double_rounding():
    # 1 + 2^-8 + 2^-30 lies above the midpoint between 1 and 1 + 2^-7; a
    # detour through fp32 would land exactly on the midpoint and tie to 1.
    v = 1.0 + 2.0 ** -8 + 2.0 ** -30
    assert O.round_bf16(np.array([v]))[0] == 1.0 + 2.0 ** -7
    assert O.round_bf16(np.array([1.0 + 2.0 ** -8]))[0] == 1.0


def test_round_bf16_overflow_and_subnormal():
    big = 3.3895313892515355e38
    assert O.round_bf16(np.array([big]))[0] == big
    assert np.isinf(O.round_bf16(np.array([big * 1.01]))[0])
    tiny = 2.0 ** -133
    assert O.round_bf16(np.array([tiny * 1.4]))[0] == tiny
    assert O.round_bf16(np.array([tiny * 0.4]))[0] == 0.0


def test_generator_bf16_bits_match_torch():
    rng = np.random.default_rng(11)
    v = rng.standard_normal(100000).astype(np.float32)
    ref = torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(synth.bf16_bits(v), ref)


def _fp16_value_by_hand(bits: int) -> float:
    """binary16 decoded bit by bit: sign, 5-bit exponent (bias 15), 10-bit
    fraction, exponent field 0 meaning subnormal."""
    sign = -1.0 if (bits >> 15) & 1 else 1.0
    e = (bits >> 10) & 0x1F
    f = bits & 0x3FF
    if e == 0:
        return sign * (f / 1024.0) * 2.0 ** -14
    return sign * (1.0 + f / 1024.0) * 2.0 ** (e - 15)


def test_fp16_scale_fixture():
    for row in read_golden("fp16_scales.txt"):
        bits = int(row[0], 16)
        val, w0 = float(row[1]), float(row[2])
        assert _fp16_value_by_hand(bits) == val
        assert O.f16_to_f64(np.array([bits], dtype=np.uint16))[0] == val
        lin = dict(K=8, N=1, qweight=np.zeros((1, 1), dtype=np.int32),
                   scales=np.array([[bits]], dtype=np.uint16).view(np.float16), zeros=None)
        assert O.dequant(lin, 8)[0, 0] == w0


# ------------------------------------------------------------ int4 format

def test_int4_word_fixture():
    for row in read_golden("int4_words.txt"):
        word = int(row[0], 16)
        codes = [int(c) for c in row[1:]]
        qw = np.array([[word]], dtype=np.uint32).view(np.int32)
        assert list(O.unpack_int4(qw, 8)[:, 0]) == codes
        assert synth.pack_int4(np.array(codes, dtype=np.uint8)[:, None]).view(np.uint32)[0, 0] == word


@pytest.mark.parametrize("K,N", [(8, 1), (16, 3), (72, 5)])
def test_unpack_brute_force_bits(K, N):
    rng = np.random.default_rng(K * 10 + N)
    q = rng.integers(0, 16, size=(K, N), dtype=np.uint8)
    qw = synth.pack_int4(q)
    got = O.unpack_int4(qw, K)
    for k in range(K):
        for n in range(N):
            word = int(qw.view(np.uint32)[k // 8, n])
            code = 0
            for b in range(4):
                code |= ((word >> (4 * (k % 8) + b)) & 1) << b
            assert got[k, n] == code == q[k, n]


@pytest.mark.parametrize("with_zeros", [False, True])
def test_dequant_brute_force(with_zeros):
    K, N, G = 72, 5, 32                       # ragged last group of 8 rows
    rng = np.random.default_rng(5)
    q = rng.integers(0, 16, size=(K, N), dtype=np.uint8)
    ng = -(-K // G)
    sbits = rng.integers(0, 1 << 16, size=(ng, N)).astype(np.uint16)
    sbits[0, 0] = 0x0001                      # smallest subnormal
    sbits[1, 1] = 0x03FF                      # largest subnormal
    sbits[2, 2] = 0x0000                      # zero scale
    sbits[0, 3] = 0x8400                      # negative normal
    exp = (sbits >> 10) & 0x1F
    sbits[exp == 0x1F] = 0x3C00               # no inf/nan scales
    zeros = rng.integers(0, 16, size=(ng, N), dtype=np.uint8) if with_zeros else None
    lin = dict(K=K, N=N, qweight=synth.pack_int4(q), scales=sbits.view(np.float16), zeros=zeros)
    got = O.dequant(lin, G)
    for k in range(K):
        for n in range(N):
            s = _fp16_value_by_hand(int(sbits[k // G, n]))
            z = 8 if zeros is None else int(zeros[k // G, n])
            assert got[k, n] == s * (int(q[k, n]) - z)


def test_generator_distributions():
    cfg = synth.CONFIGS["tiny"]
    lin = synth.make_linear(cfg, "down")
    assert lin["q"].shape == (688, 256) and lin["qweight"].shape == (86, 256)
    assert lin["scales"].shape == (11, 256) and lin["scales"].dtype == np.float16
    assert lin["q"].min() == 0 and lin["q"].max() == 15
    assert np.all(lin["scales"].astype(np.float64) >= 0)
    # same seed -> same tensor, different tensor id -> different draws
    assert np.array_equal(synth.make_linear(cfg, "down")["qweight"], lin["qweight"])
    assert not np.array_equal(synth.make_linear(cfg, "up")["q"][:8], lin["q"][:8])


# ------------------------------------------------------------ operators

def test_rmsnorm_fixture_and_invariants():
    for row in read_golden("rmsnorm.txt"):
        eps, x0, x1, g0, g1, y0, y1 = map(float, row)
        y = O.rmsnorm(np.array([[x0, x1]]), np.array([g0, g1]), eps)
        assert np.allclose(y, [[y0, y1]], rtol=1e-14, atol=0)
    rng = np.random.default_rng(0)
    x = rng.standard_normal((4, 64))
    g = rng.uniform(0.5, 1.5, 64)
    assert np.allclose(O.rmsnorm(3.7 * x, g, 0.0), O.rmsnorm(x, g, 0.0), rtol=1e-13)
    y = O.rmsnorm(x, np.ones(64), 0.0)
    assert np.allclose(np.mean(y * y, axis=-1), 1.0, rtol=1e-13)


def test_rope_fixture():
    for row in read_golden("rope_d4.txt"):
        vals = list(map(float, row))
        pos, x, y = vals[0], np.array(vals[1:5]), np.array(vals[5:9])
        c, s = O.rope_cos_sin(np.array([pos]), 4, 10000.0)
        out = O.rope(x[None, None, :], c, s)[0, 0]
        assert np.allclose(out, y, rtol=0, atol=1e-15)


def test_rope_is_complex_rotation():
    # second formulation: pair (i, i + d/2) as the complex number
    # x_i + 1j x_{i+d/2}, multiplied by exp(1j * p * base^(-2i/d))
    d, base = 16, 500000.0
    rng = np.random.default_rng(2)
    x = rng.standard_normal((3, 2, d))
    pos = np.array([0, 7, 1234])
    c, s = O.rope_cos_sin(pos, d, base)
    got = O.rope(x, c, s)
    for t in range(3):
        for h in range(2):
            for i in range(d // 2):
                z = complex(x[t, h, i], x[t, h, i + d // 2])
                z *= complex(math.cos(pos[t] * base ** (-2 * i / d)), math.sin(pos[t] * base ** (-2 * i / d)))
                assert abs(got[t, h, i] - z.real) < 1e-12
                assert abs(got[t, h, i + d // 2] - z.imag) < 1e-12


def test_rope_relative_position():
    # <rope(q, m), rope(k, n)> depends on m - n only; norms are preserved
    d = 64
    rng = np.random.default_rng(4)
    q = rng.standard_normal((1, 1, d))
    k = rng.standard_normal((1, 1, d))

    def dot(m, n):
        cm, sm = O.rope_cos_sin(np.array([m]), d, 1e4)
        cn, sn = O.rope_cos_sin(np.array([n]), d, 1e4)
        return float(np.sum(O.rope(q, cm, sm) * O.rope(k, cn, sn)))

    assert abs(dot(10, 3) - dot(1010, 1003)) < 1e-9
    assert abs(dot(5, 5) - float(np.sum(q * k))) < 1e-12
    c, s = O.rope_cos_sin(np.array([99]), d, 1e4)
    r = O.rope(q, c, s)
    assert abs(np.linalg.norm(r) - np.linalg.norm(q)) < 1e-12


def test_attention_fixture():
    for row in read_golden("attention_small.txt"):
        qv, k0, k1, v0, v1, out = map(float, row)
        q = np.array([[[qv]]])
        k = np.array([[[k0]], [[k1]]])
        v = np.array([[[v0]], [[v1]]])
        got = O.attention(q, k, v, np.array([1]))
        assert abs(got[0, 0, 0] - out) < 1e-14


def _attention_brute(q, k, v, slots, bias):
    T, nq, d = q.shape
    S, nkv, _ = k.shape
    out = np.zeros_like(q)
    for t in range(T):
        for h in range(nq):
            g = h // (nq // nkv)
            sc = []
            for j in range(S):
                if j > slots[t]:
                    continue
                val = sum(q[t, h, e] * k[j, g, e] for e in range(d)) / math.sqrt(d)
                sc.append((j, val + (bias[t][j] if bias is not None else 0.0)))
            m = max(s for _, s in sc)
            if m == -math.inf:
                continue
            wts = [(j, math.exp(s - m)) for j, s in sc]
            tot = sum(w for _, w in wts)
            for e in range(d):
                out[t, h, e] = sum(w * v[j, g, e] for j, w in wts) / tot
    return out


def test_attention_brute_force_gqa_causal_bias():
    rng = np.random.default_rng(9)
    T, S, nq, nkv, d = 3, 5, 4, 2, 4
    q = rng.standard_normal((T, nq, d))
    k = rng.standard_normal((S, nkv, d))
    v = rng.standard_normal((S, nkv, d))
    slots = np.array([2, 3, 4])
    bias = rng.standard_normal((T, S))
    bias[1, 0] = -np.inf
    got = O.attention(q, k, v, slots, bias)
    ref = _attention_brute(q, k, v, slots, bias)
    assert np.allclose(got, ref, rtol=0, atol=1e-13)


def test_attention_special_cases():
    rng = np.random.default_rng(1)
    d = 8
    q = rng.standard_normal((1, 4, d))
    k = rng.standard_normal((1, 2, d))
    v = rng.standard_normal((1, 2, d))
    # a single visible key: the output is that key's value
    out = O.attention(q, k, v, np.array([0]))
    assert np.allclose(out[0, :2], v[0, 0]) and np.allclose(out[0, 2:], v[0, 1])
    # identical keys: the output is the mean of the values
    k5 = np.repeat(k, 5, axis=0)
    v5 = rng.standard_normal((5, 2, d))
    out = O.attention(q, k5, v5, np.array([4]))
    assert np.allclose(out[0, 0], v5[:, 0].mean(0), atol=1e-14)
    # every key masked: zero output
    out = O.attention(q, k5, v5, np.array([4]), np.full((1, 5), -np.inf))
    assert np.all(out == 0)
    # GQA equals multi-head attention with each kv head repeated r times
    qq = rng.standard_normal((3, 4, d))
    kk = rng.standard_normal((3, 2, d))
    vv = rng.standard_normal((3, 2, d))
    gqa = O.attention(qq, kk, vv, np.arange(3))
    mha = O.attention(qq, np.repeat(kk, 2, axis=1), np.repeat(vv, 2, axis=1), np.arange(3))
    assert np.allclose(gqa, mha, atol=1e-14)


def test_silu_values():
    assert O.silu(np.array([0.0]))[0] == 0.0
    assert abs(O.silu(np.array([1.0]))[0] - 1.0 / (1.0 + math.exp(-1.0))) < 1e-15
    assert abs(O.silu(np.array([-30.0]))[0]) < 1e-11
