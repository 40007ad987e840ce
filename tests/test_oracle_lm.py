"""Pins of the model-ends oracle (embedding, LM head, greedy sampling)
against brute force on tiny inputs and closed forms.  None of these re-types
the oracle's own formula."""
import math
import struct
from fractions import Fraction

import numpy as np
import pytest

from oracle import lm as M
from paper_2607_15865_amd import synth


def bf16_val(bits: int) -> float:
    return struct.unpack(">f", struct.pack(">I", (int(bits) & 0xFFFF) << 16))[0]


def f16_val(bits: int) -> float:
    return struct.unpack("<e", struct.pack("<H", int(bits)))[0]


def nearest_bf16(v: float) -> float:
    """Nearest bf16 value by exact comparison of neighbouring candidates,
    ties to the even bit pattern."""
    if v == 0.0:
        return 0.0
    t = struct.unpack(">I", struct.pack(">f", v))[0] >> 16
    best = None
    for b in (t - 1, t, t + 1):
        c = bf16_val(b)
        if not math.isfinite(c):
            continue
        d = abs(Fraction(v) - Fraction(c))
        if best is None or d < best[0] or (d == best[0] and b % 2 == 0):
            best = (d, b, c)
    return best[2]


def tiny_lm(H=64, V=12, G=32, seed=0, with_zeros=False):
    cfg = synth.replace(synth.CONFIGS["tiny"], hidden=H, group_size=G, cfg_id=50 + seed)
    return cfg, synth.make_lm(cfg, V, with_zeros=with_zeros)


# ------------------------------------------------------------ embedding

def test_embed_brute_force():
    cfg, lm = tiny_lm(V=20)
    tok = np.array([3, 0, 19, 3, 7])
    e = M.embed(lm["embed"], tok)
    for i, t in enumerate(tok):
        for k in range(cfg.hidden):
            assert e[i, k] == bf16_val(lm["embed"][t, k])


def test_embed_known_patterns_and_range():
    table = np.array([[0x3F80, 0xC000], [0x0000, 0x4049]], dtype=np.uint16)
    assert M.embed(table, [0, 1]).tolist() == [[1.0, -2.0], [0.0, 3.140625]]
    with pytest.raises(ValueError):
        M.embed(table, [2])
    with pytest.raises(ValueError):
        M.embed(table, [-1])


# ------------------------------------------------------------ LM head

@pytest.mark.parametrize("with_zeros", [False, True])
def test_logits_brute_force(with_zeros):
    H, V, G, B = 64, 12, 32, 3
    cfg, lm = tiny_lm(H, V, G, with_zeros=with_zeros)
    head = lm["head"]
    rng = np.random.default_rng(11)
    x = (rng.standard_normal((B, H)) * 2.0).astype(np.float32)
    eps = 1e-5
    words = np.asarray(head["qweight"]).view(np.uint32)
    sc = np.asarray(head["scales"]).view(np.uint16)
    zs = head["zeros"]
    W = [[0.0] * V for _ in range(H)]
    for k in range(H):
        for v in range(V):
            code = (int(words[k // 8, v]) >> (4 * (k % 8))) & 0xF
            z = 8 if zs is None else int(zs[k // G, v])
            W[k][v] = f16_val(sc[k // G, v]) * (code - z)
    got = M.lm_logits(x, lm["final_norm"], head, G, eps)
    for b in range(B):
        xs = [float(t) for t in x[b]]
        ms = math.fsum(t * t for t in xs) / H
        r = 1.0 / math.sqrt(ms + eps)
        xn = [nearest_bf16(xs[k] * r * bf16_val(lm["final_norm"][k])) for k in range(H)]
        for v in range(V):
            ref = math.fsum(xn[k] * W[k][v] for k in range(H))
            assert got[b, v] == pytest.approx(ref, rel=1e-12, abs=1e-12)


def test_logits_closed_forms():
    H, V, G = 64, 5, 32
    cfg, lm = tiny_lm(H, V, G)
    gamma = np.full(H, 0x3F80, dtype=np.uint16)               # 1.0
    q = np.full((H, V), 9, dtype=np.uint8)                    # code - 8 = 1
    head = dict(K=H, N=V, q=q, qweight=synth.pack_int4(q),
                scales=np.full((H // G, V), 0.5, dtype=np.float16), zeros=None)
    # constant input, eps 0: the normalised row is all ones, logits = H * 0.5
    x = np.full((1, H), 3.0)
    assert np.array_equal(M.lm_logits(x, gamma, head, G, 0.0), np.full((1, V), H * 0.5))
    # a one-hot input selects one row of W, scaled by sqrt(H) (transposed
    # operands or a wrong row fail here)
    q2 = np.arange(H * V).reshape(H, V) % 16
    head2 = dict(K=H, N=V, q=q2, qweight=synth.pack_int4(q2.astype(np.uint8)),
                 scales=np.full((H // G, V), 0.25, dtype=np.float16), zeros=None)
    j = 37
    x = np.zeros((1, H))
    x[0, j] = -2.0
    got = M.lm_logits(x, gamma, head2, G, 0.0)
    assert np.array_equal(got[0], -math.sqrt(H) * 0.25 * (q2[j] - 8))


# ------------------------------------------------------------ greedy sampling

def test_greedy_brute_force_and_ties():
    rng = np.random.default_rng(5)
    L = rng.integers(-4, 5, size=(40, 17)).astype(np.float64)   # many ties
    got = M.greedy(L)
    for b in range(L.shape[0]):
        best = 0
        for v in range(1, L.shape[1]):
            if L[b, v] > L[b, best]:
                best = v
        assert got[b] == best
    assert M.greedy([[-np.inf, -np.inf]]).tolist() == [0]
    assert M.greedy([[-3.0, -1.0, -1.0, -2.0]]).tolist() == [1]


def test_make_lm_shapes_and_words_mode():
    cfg = synth.replace(synth.CONFIGS["tiny"], cfg_id=60)
    a = synth.make_lm(cfg, 128)
    b = synth.make_lm(cfg, 128, words=True)
    assert a["embed"].shape == (128, cfg.hidden) and a["embed"].dtype == np.uint16
    assert a["head"]["qweight"].shape == b["head"]["qweight"].shape == (cfg.hidden // 8, 128)
    assert np.array_equal(a["head"]["scales"], b["head"]["scales"])
    codes = (b["head"]["qweight"].view(np.uint32)[..., None] >> (4 * np.arange(8, dtype=np.uint32))) & 15
    assert codes.min() == 0 and codes.max() == 15
