"""Block- and stage-level pins of the CPU oracle: a scalar brute-force block on
a tiny layer, the special cases where the layer reduces to the identity, and
the equivalences the paper states between the three stages (Sec. 4.1-4.5)."""
import math

import numpy as np
import pytest

from oracle import layer as O
from paper_2607_15865_amd import synth
from test_oracle_pins import _fp16_value_by_hand

MICRO = synth.LayerConfig("micro", hidden=16, n_heads=4, n_kv_heads=2, head_dim=4, ffn=24,
                          group_size=8, rms_eps=1e-6, rope_base=10000.0, max_seq=16, max_batch=4,
                          cfg_id=99)


def _rb(v: float) -> float:
    """Nearest bf16 value with ties to even (Python's round() is half-even)."""
    if v == 0.0:
        return 0.0
    m, e = math.frexp(v)
    return math.ldexp(round(math.ldexp(m, 8)), e - 8)


def _bf16(bits: int) -> float:
    import struct
    return struct.unpack("<f", struct.pack("<I", int(bits) << 16))[0]


def _weight_by_hand(lin, G, k, n):
    word = int(lin["qweight"].view(np.uint32)[k // 8, n])
    code = (word >> (4 * (k % 8))) & 0xF
    s = _fp16_value_by_hand(int(lin["scales"].view(np.uint16)[k // G, n]))
    return s * (code - 8)


def _block_by_hand(w, cfg, x, pos, kh, vh):
    """The block of Listings 1-2 written as scalar loops over every index."""
    H, nq, nkv, d, F, G = cfg.hidden, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.ffn, cfg.group_size
    T, L = len(x), len(kh)
    Wm = {}
    for name in synth.LINEARS:
        K, N = cfg.linear_shape(name)
        Wm[name] = [[_weight_by_hand(w[name], G, k, n) for n in range(N)] for k in range(K)]

    def norm(row, gbits):
        ms = sum(v * v for v in row) / len(row)
        r = 1.0 / math.sqrt(ms + cfg.rms_eps)
        return [_rb(row[i] * r * _bf16(gbits[i])) for i in range(len(row))]

    def matvec(row, Wk):
        return [sum(row[k] * Wk[k][n] for k in range(len(row))) for n in range(len(Wk[0]))]

    def rot(vec, p):
        out = list(vec)
        for i in range(d // 2):
            ang = p * cfg.rope_base ** (-2.0 * i / d)
            a, b = vec[i], vec[i + d // 2]
            out[i] = a * math.cos(ang) - b * math.sin(ang)
            out[i + d // 2] = b * math.cos(ang) + a * math.sin(ang)
        return out

    qs, ks, vs = [], [], []
    for t in range(T):
        xn = norm(x[t], w["attn_norm"])
        q, k, v = matvec(xn, Wm["q"]), matvec(xn, Wm["k"]), matvec(xn, Wm["v"])
        qs.append([[_rb(c) for c in rot(q[h * d:(h + 1) * d], pos[t])] for h in range(nq)])
        ks.append([[_rb(c) for c in rot(k[g * d:(g + 1) * d], pos[t])] for g in range(nkv)])
        vs.append([[_rb(c) for c in v[g * d:(g + 1) * d]] for g in range(nkv)])
    keys = [[list(kh[j][g]) for g in range(nkv)] for j in range(L)] + ks
    vals = [[list(vh[j][g]) for g in range(nkv)] for j in range(L)] + vs
    ys = []
    for t in range(T):
        attn = []
        for h in range(nq):
            g = h // (nq // nkv)
            sc = [sum(qs[t][h][e] * keys[j][g][e] for e in range(d)) / math.sqrt(d) for j in range(L + t + 1)]
            m = max(sc)
            p = [math.exp(s - m) for s in sc]
            tot = sum(p)
            attn += [_rb(sum(p[j] * vals[j][g][e] for j in range(L + t + 1)) / tot) for e in range(d)]
        o = matvec(attn, Wm["o"])
        h_ = [x[t][i] + o[i] for i in range(H)]
        hn = norm(h_, w["mlp_norm"])
        a, b = matvec(hn, Wm["gate"]), matvec(hn, Wm["up"])
        gg = [_rb(a[f] / (1.0 + math.exp(-a[f])) * b[f]) for f in range(F)]
        dn = matvec(gg, Wm["down"])
        ys.append([h_[i] + dn[i] for i in range(H)])
    return np.array(ys), np.array(ks), np.array(vs)


def _micro_layer():
    w = synth.make_layer(MICRO)
    # make the sums big enough that a transposed or mis-indexed operand shows
    for name in synth.LINEARS:
        w[name]["scales"] = (w[name]["scales"].astype(np.float64) * 40).astype(np.float16)
    return w


def test_block_matches_scalar_loops():
    w = _micro_layer()
    rng = np.random.default_rng(0)
    T, L = 3, 2
    x = O.bf16_to_f64(synth.bf16_bits(rng.standard_normal((T, MICRO.hidden))))
    pos = np.array([5, 6, 9])
    kh = O.round_bf16(rng.standard_normal((MICRO.n_kv_heads, L, MICRO.head_dim)))
    vh = O.round_bf16(rng.standard_normal((MICRO.n_kv_heads, L, MICRO.head_dim)))
    y, k, v = O.block(w, MICRO, x, pos, kh, vh)
    yb, kb, vb = _block_by_hand(w, MICRO, x.tolist(), pos.tolist(), kh.transpose(1, 0, 2), vh.transpose(1, 0, 2))
    # bf16 rounding points agree exactly unless fp64 summation order moves a
    # value across a rounding boundary, which these inputs do not do
    assert np.array_equal(k, kb) and np.array_equal(v, vb)
    assert np.allclose(y, yb, rtol=0, atol=1e-10)


def _tiny():
    cfg = synth.CONFIGS["tiny"]
    w = synth.make_layer(cfg)
    return cfg, w, O.dequant_layer(w, cfg)


def test_zero_weights_give_identity():
    cfg, w, _ = _tiny()
    wz = dict(w)
    for name in synth.LINEARS:
        wz[name] = synth.zero_linear(w[name])
    x = O.bf16_to_f64(synth.activations(cfg, synth.TID_X_PREFILL, 8))
    y, k, v = O.prefill(wz, cfg, x, np.arange(8))
    assert np.array_equal(y, x)
    assert np.all(k == 0) and np.all(v == 0)


def test_zero_v_projection_keeps_residual():
    cfg, w, _ = _tiny()
    wz = dict(w)
    wz["v"] = synth.zero_linear(w["v"])
    wz["down"] = synth.zero_linear(w["down"])
    x = O.bf16_to_f64(synth.activations(cfg, synth.TID_X_PREFILL, 8))
    y, _, _ = O.prefill(wz, cfg, x, np.arange(8))
    assert np.array_equal(y, x)


def test_causality():
    cfg, w, W = _tiny()
    x = O.bf16_to_f64(synth.activations(cfg, synth.TID_X_PREFILL, 12))
    y1, k1, _ = O.prefill(w, cfg, x, np.arange(12), W=W)
    x2 = x.copy()
    x2[7:] = -x2[7:] * 3.0
    y2, k2, _ = O.prefill(w, cfg, x2, np.arange(12), W=W)
    assert np.array_equal(y1[:7], y2[:7]) and np.array_equal(k1[:7], k2[:7])
    assert not np.allclose(y1[7:], y2[7:])


def _cache(cfg, new_k, S=None):
    S = cfg.max_seq if S is None else S
    c = np.zeros((cfg.n_kv_heads, S, cfg.head_dim))
    return O.cache_write(c, new_k, 0)


def test_prefill_kv_equals_tail_of_prefill():
    """Prefill_kv of chunk C after history H equals the last rows of one
    prefill over H + C (Sec. 4.3: the history is concatenated in front)."""
    cfg, w, W = _tiny()
    Hn, Cn = 20, 12
    x = O.bf16_to_f64(synth.activations(cfg, synth.TID_X_PREFILL, Hn + Cn))
    pos = np.arange(Hn + Cn)
    y_full, k_full, v_full = O.prefill(w, cfg, x, pos, W=W)
    y_h, k_h, v_h = O.prefill(w, cfg, x[:Hn], pos[:Hn], W=W)
    kc, vc = _cache(cfg, k_h), _cache(cfg, v_h)
    y_c, k_c, v_c = O.prefill_kv(w, cfg, x[Hn:], pos[Hn:], kc, vc, Hn, W=W)
    assert np.allclose(y_c, y_full[Hn:], rtol=0, atol=1e-10)
    assert np.array_equal(k_c, k_full[Hn:]) and np.array_equal(v_c, v_full[Hn:])
    # stale entries beyond the history are never read
    kc2 = kc.copy(); kc2[:, Hn:, :] = 1e3
    y_c2, _, _ = O.prefill_kv(w, cfg, x[Hn:], pos[Hn:], kc2, vc, Hn, W=W)
    assert np.array_equal(y_c2, y_c)


def test_segmented_prefill_equals_one_prefill():
    """1 prefill + k prefill_kv segments reproduce one long prefill (the
    long-prompt segmentation of Sec. 4.1)."""
    cfg, w, W = _tiny()
    n = 40
    x = O.bf16_to_f64(synth.activations(cfg, synth.TID_X_PREFILL, n))
    pos = np.arange(n)
    y_full, k_full, _ = O.prefill(w, cfg, x, pos, W=W)
    kc = np.zeros((cfg.n_kv_heads, cfg.max_seq, cfg.head_dim)); vc = kc.copy()
    ys, start = [], 0
    for seg in (16, 8, 8, 8):
        if start == 0:
            y, k, v = O.prefill(w, cfg, x[:seg], pos[:seg], W=W)
        else:
            y, k, v = O.prefill_kv(w, cfg, x[start:start + seg], pos[start:start + seg], kc, vc, start, W=W)
        kc, vc = O.cache_write(kc, k, start), O.cache_write(vc, v, start)
        ys.append(y); start += seg
    assert np.allclose(np.concatenate(ys), y_full, rtol=0, atol=1e-10)
    assert np.array_equal(kc[:, :n, :], k_full.transpose(1, 0, 2))


def test_decode_steps_equal_prefill_rows():
    """Decoding tokens one at a time against the growing cache gives the rows
    of a prefill over the same tokens, and builds the same cache (Sec. 4.4,
    4.5)."""
    cfg, w, W = _tiny()
    P, D = 24, 8
    x = O.bf16_to_f64(synth.activations(cfg, synth.TID_X_PREFILL, P + D))
    pos = np.arange(P + D)
    y_full, k_full, v_full = O.prefill(w, cfg, x, pos, W=W)
    _, k_p, v_p = O.prefill(w, cfg, x[:P], pos[:P], W=W)
    kc, vc = _cache(cfg, k_p)[None], _cache(cfg, v_p)[None]
    for s in range(D):
        t = P + s
        y, k, v = O.decode(w, cfg, x[t:t + 1], pos[t:t + 1], kc, vc, [t], W=W)
        assert np.allclose(y[0], y_full[t], rtol=0, atol=1e-10)
        kc = O.cache_write(kc[0], k, t)[None]
        vc = O.cache_write(vc[0], v, t)[None]
    assert np.array_equal(kc[0][:, :P + D], k_full.transpose(1, 0, 2))
    assert np.array_equal(vc[0][:, :P + D], v_full.transpose(1, 0, 2))


def _decode_inputs(cfg, B, ctx):
    kb, vb = synth.kv_fill(cfg, B)
    kc, vc = O.bf16_to_f64(kb), O.bf16_to_f64(vb)
    x = O.bf16_to_f64(synth.activations(cfg, synth.TID_X_DECODE, B))
    return x, kc, vc


def test_decode_mask_semantics():
    cfg, w, W = _tiny()
    ctx = 40
    x, kc, vc = _decode_inputs(cfg, 1, ctx)
    pos = np.array([ctx])
    y0, k0, v0 = O.decode(w, cfg, x, pos, kc, vc, [ctx], W=W)
    zero = np.zeros((1, cfg.max_seq))
    assert np.array_equal(O.decode(w, cfg, x, pos, kc, vc, [ctx], zero, W=W)[0], y0)
    # -inf at slot j is the same as deleting key j from the cache
    j = 13
    m = zero.copy(); m[0, j] = -np.inf
    y_m = O.decode(w, cfg, x, pos, kc, vc, [ctx], m, W=W)[0]
    kd = np.delete(kc, j, axis=2); vd = np.delete(vc, j, axis=2)
    y_d = O.decode(w, cfg, x, pos, kd, vd, [ctx - 1], W=W)[0]
    assert np.allclose(y_m, y_d, rtol=0, atol=1e-10)
    # a constant added to every visible score changes nothing
    y_c = O.decode(w, cfg, x, pos, kc, vc, [ctx], zero + 2.5, W=W)[0]
    assert np.allclose(y_c, y0, rtol=0, atol=1e-10)


def test_decode_batch_rows_are_independent():
    cfg, w, W = _tiny()
    B = 4
    x, kc, vc = _decode_inputs(cfg, B, 0)
    ctx = np.array([5, 60, 0, 127])
    pos = ctx + 3
    y, k, v = O.decode(w, cfg, x, pos, kc, vc, ctx, W=W)
    for b in range(B):
        yb, kb, vb = O.decode(w, cfg, x[b:b + 1], pos[b:b + 1], kc[b:b + 1], vc[b:b + 1], ctx[b:b + 1], W=W)
        assert np.array_equal(y[b], yb[0]) and np.array_equal(k[b], kb[0])
