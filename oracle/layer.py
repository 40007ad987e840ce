"""CPU oracle for the three-stage W4A16 decoder layer.

TEST INFRASTRUCTURE ONLY.  Only the tests, the package's smoke check and the
benchmark's CPU-baseline leg may import this module; the product path never
does, and this module imports nothing from the product path.

Plain, slow, obviously correct fp64 numpy.  Every function states the passage
of the paper it follows.  The block dataflow is the one the paper gives for a
Transformer block without and with history (Sec. 3.1, Listings 1 and 2):

    x = RMSNorm(input)                       input_layernorm
    q, k, v = x Wq, x Wk, x Wv               q/k/v projections
    cos, sin = table[position_ids]           Gather of a precomputed table
    q, k = Rope(q), Rope(k)
    k_all, v_all = Concat(history, k / v)    only with history
    attn = FAttention(q, k_all, v_all)       scaled dot product + causal mask
    h = input + attn Wo                      o_proj + residual
    out = h + MLP(RMSNorm(h))                post-attention norm, MLP, residual
    return out, k, v

The three stages (Sec. 4.1, Table 1) are that block with an empty history
(prefill, Sec. 4.2), with a history cache (prefill_kv, Sec. 4.3) and with a
single token per sequence plus an externally supplied attention mask (decode,
Sec. 4.4).  Where the paper leaves a detail open, the reading taken is named
at the function that depends on it.

Precision.  The paper fixes the precision of the deployed models as W4BF16,
4-bit weights with BF16 activations (Sec. 5.1), and shows the block's
hidden-state interface as f32 tensors (Listing 3).  Reading taken: the
activation tensors the block materialises between its operators are bf16,
rounded to nearest-even once when they are formed -- the normalised input of
the q/k/v and gate/up matmuls, q and k after RoPE, v, the attention output
entering o_proj, and the MLP hidden activation entering down; the K/V cache
therefore holds bf16 values.  Everything else (weights after dequantisation,
scores, softmax, sums, the residual stream h and the output y) is computed in
fp64 and not rounded.

Weight formats.  Besides the W4 format (4-bit codes, group scales), the
paper's direct-through modes INT8 (symmetric or asymmetric) and BF16 are
accepted per linear (``dequant``); the block's arithmetic does not depend on
the format, only on the fp64 weights it yields.

Pins: every function here is checked by tests/test_oracle_*.py against
brute-force loops on tiny inputs, closed forms and the stage invariants the
paper implies; none is "parity unpinned".
"""
from __future__ import annotations

import contextlib

import numpy as np

F64 = np.float64      # the working precision (fp64; see working_precision)


@contextlib.contextmanager
def working_precision(dtype):
    """Timing only: run the oracle's arithmetic in ``dtype`` (np.float32 is
    the fp32 mode timed as a CPU baseline).  Every comparison with the GPU
    path and every pin uses the default fp64."""
    global F64
    old = F64
    F64 = dtype
    try:
        yield
    finally:
        F64 = old


# ------------------------------------------------------------ storage formats

def bf16_to_f64(bits) -> np.ndarray:
    """bfloat16 bit patterns -> exact fp64 values (bf16 is the top half of fp32)."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(F64)


def f16_to_f64(a) -> np.ndarray:
    """fp16 values (numpy float16 array or uint16 bits) -> exact fp64 values."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.float16)
    return a.astype(F64)


def unpack_int4(qweight, K: int) -> np.ndarray:
    """Codes q[k][n] from the canonical packing: word r of column n holds
    code k = 8r + j in bits 4j .. 4j+3 (reading of the weight format the
    paper passes through for GPTQ-style checkpoints, Sec. 3.2)."""
    w = np.asarray(qweight).view(np.uint32)
    k = np.arange(K)
    shift = (4 * (k % 8)).astype(np.uint32)
    return ((w[k // 8, :] >> shift[:, None]) & np.uint32(0xF)).astype(np.int64)


def dequant_int8(lin: dict) -> np.ndarray:
    """W[k][n] = s[n] * (q[k][n] - z[n]) in fp64 (exact) for an INT8 linear.

    The paper compiles INT8 weights symmetric or asymmetric (Sec. 3.2).
    Readings taken: one scale per output channel (fp16, ``scales[n]``);
    symmetric weights hold signed codes -128 .. 127 (``q8`` as int8) with
    zero point 0; asymmetric weights hold unsigned codes 0 .. 255 (``q8`` as
    uint8) and a zero point per output channel (``zeros[n]``, 0 .. 255).
    """
    s = f16_to_f64(lin["scales"]).reshape(-1)
    if lin.get("zeros") is None:
        q = np.asarray(lin["q8"]).view(np.int8).astype(F64)
        return s[None, :] * q
    q = np.asarray(lin["q8"]).view(np.uint8).astype(F64)
    z = np.asarray(lin["zeros"], dtype=F64).reshape(-1)
    return s[None, :] * (q - z[None, :])


def dequant(lin: dict, group_size: int) -> np.ndarray:
    """The fp64 weight W[K][N] of a linear in any of the layer's formats.

    ``format`` "int4" (the default): W[k][n] = s[k // G][n] * (q[k][n] -
    z[k // G][n]) (exact).  The W4A16 matmul carries the weight's
    quantisation scales (and zero points) alongside the packed codes
    (Sec. 3.2).  Reading taken: groups run along K, the last group may be
    shorter, the zero point is 8 unless per-group zero points are supplied.
    ``format`` "int8": dequant_int8.  ``format`` "bf16": the unquantised
    weights of the paper's BF16 mode (Sec. 3.2), bf16 bit patterns
    ``w16[K][N]`` taken exactly.
    """
    fmt = lin.get("format", "int4")
    if fmt == "int8":
        return dequant_int8(lin)
    if fmt == "bf16":
        return bf16_to_f64(lin["w16"])
    if fmt != "int4":
        raise ValueError(f"unknown weight format {fmt!r}")
    K, N = lin["K"], lin["N"]
    q = unpack_int4(lin["qweight"], K)
    g = np.arange(K) // group_size
    s = f16_to_f64(lin["scales"])[g, :]
    z = 8.0 if lin.get("zeros") is None else np.asarray(lin["zeros"], dtype=F64)[g, :]
    return s * (q.astype(F64) - z)


def round_bf16(a) -> np.ndarray:
    """Nearest bfloat16 value of each fp64 element (8 significant bits, ties
    to even), returned in fp64.  Values below the bf16 normal range round
    on the subnormal grid 2^-133; values beyond the largest finite bf16
    become infinities."""
    a = np.asarray(a, dtype=F64)
    m, e = np.frexp(a)                        # a = m * 2^e, 0.5 <= |m| < 1
    e = np.maximum(e, -125)                   # subnormal range: fixed quantum
    q = np.ldexp(np.rint(np.ldexp(a, 8 - e)), e - 8)
    big = np.abs(q) > 3.3895313892515355e38   # largest finite bf16
    return np.where(big, np.copysign(np.inf, a), q)


# ------------------------------------------------------------ operators

def rmsnorm(x: np.ndarray, gamma: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm (top.RMSNorm, Sec. 2.2): x / sqrt(mean(x^2) + eps) * gamma over
    the hidden axis.  Reading taken: eps inside the square root and a
    multiplicative weight gamma."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * gamma


def rope_cos_sin(pos: np.ndarray, head_dim: int, base: float):
    """cos/sin of the rotary angles for the given positions (the table the
    paper precomputes once and gathers by position_ids, Sec. 4.6.2).
    Angle of pair i at position p: p * base^(-2i/d), i < d/2."""
    i = np.arange(head_dim // 2, dtype=F64)
    theta = np.power(F64(base), -2.0 * i / head_dim)
    ang = np.asarray(pos, dtype=F64)[:, None] * theta[None, :]
    return np.cos(ang), np.sin(ang)


def rope(x: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """top.Rope (Sec. 2.2, Listing 1) on x[T][heads][d].  Reading taken: the
    rotate-half pairing, element i rotates with element i + d/2."""
    half = x.shape[-1] // 2
    x1, x2 = x[..., :half], x[..., half:]
    c, s = cos[:, None, :], sin[:, None, :]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def attention(q, k_all, v_all, q_slot, bias=None):
    """top.FAttention (Sec. 2.2): softmax(q k^T / sqrt(d) + bias) v with the
    causal mask, for q[T][nq][d] and k_all, v_all[S][nkv][d].

    Query t sits at cache slot q_slot[t] and sees keys j <= q_slot[t].
    Readings taken: scale 1/sqrt(d); query head h reads kv head h // (nq/nkv);
    ``bias`` (additive, [T][S]) is the decode stage's external mask; a query
    whose every visible key is masked to -inf gets a zero output.
    """
    T, nq, d = q.shape
    S, nkv, _ = k_all.shape
    r = nq // nkv
    out = np.zeros((T, nq, d), dtype=F64)
    visible = np.arange(S)[None, :] <= np.asarray(q_slot)[:, None]
    for h in range(nq):
        g = h // r
        s = q[:, h, :] @ k_all[:, g, :].T / np.sqrt(F64(d))
        if bias is not None:
            s = s + bias
        s = np.where(visible, s, -np.inf)
        for t in range(T):
            row = s[t]
            m = np.max(row)
            if not np.isfinite(m):
                continue                       # fully masked: output 0
            p = np.exp(row - m)
            p = p / np.sum(p)
            out[t, h, :] = p @ v_all[:, g, :]
    return out


def silu(z):
    return z / (1.0 + np.exp(-z))


# ------------------------------------------------------------ the block

def dequant_layer(w: dict, cfg) -> dict:
    """All seven linears of a layer dequantised to fp64 [K][N]."""
    return {n: dequant(w[n], cfg.group_size) for n in ("q", "k", "v", "o", "gate", "up", "down")}


def block(w: dict, cfg, x, pos, k_hist=None, v_hist=None, bias=None,
          rows=None, W=None):
    """One decoder block over T new tokens after L history tokens.

    x: hidden states [T][H] (values); pos: position_ids [T];
    k_hist, v_hist: fp64 [nkv][L][d] (post-RoPE keys, values) or None;
    bias: additive attention mask [T][L+T] or None;
    rows: optional subset of query rows whose outputs are wanted (keys and
    values are still formed for every row, as causality requires).
    Returns y [T or len(rows)][H], and the new k, v [T][nkv][d] (bf16
    values, as they enter the cache).
    Follows Listing 1 (no history) and Listing 2 (history) of Sec. 3.1; the
    bf16 rounding points are the ones named in the module docstring.
    """
    H, nq, nkv, d = cfg.hidden, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim
    W = dequant_layer(w, cfg) if W is None else W
    x = np.asarray(x, dtype=F64)
    T = x.shape[0]
    L = 0 if k_hist is None else k_hist.shape[1]
    sel = np.arange(T) if rows is None else np.asarray(rows)

    xn = round_bf16(rmsnorm(x, bf16_to_f64(w["attn_norm"]), cfg.rms_eps))
    q = (xn[sel] @ W["q"]).reshape(len(sel), nq, d)
    k = (xn @ W["k"]).reshape(T, nkv, d)
    v = round_bf16((xn @ W["v"]).reshape(T, nkv, d))
    cos, sin = rope_cos_sin(pos, d, cfg.rope_base)
    q = round_bf16(rope(q, cos[sel], sin[sel]))
    k = round_bf16(rope(k, cos, sin))

    if L:
        k_all = np.concatenate([k_hist.transpose(1, 0, 2), k], axis=0)
        v_all = np.concatenate([v_hist.transpose(1, 0, 2), v], axis=0)
    else:
        k_all, v_all = k, v
    b = None if bias is None else np.asarray(bias, dtype=F64)[sel]
    a = round_bf16(attention(q, k_all, v_all, L + sel, b).reshape(len(sel), nq * d))

    h = x[sel] + a @ W["o"]
    hn = round_bf16(rmsnorm(h, bf16_to_f64(w["mlp_norm"]), cfg.rms_eps))
    g = round_bf16(silu(hn @ W["gate"]) * (hn @ W["up"]))
    y = h + g @ W["down"]
    return y, k, v


# ------------------------------------------------------------ the three stages

def prefill(w, cfg, x, pos, rows=None, W=None):
    """Prefill (Sec. 4.2): the whole prompt, no history.  Returns y and the
    new keys/values [T][nkv][d], which fill cache slots 0 .. T-1."""
    return block(w, cfg, x, pos, rows=rows, W=W)


def prefill_kv(w, cfg, x, pos, k_cache, v_cache, hist_len, rows=None, W=None):
    """Prefill_kv (Sec. 4.3): a new chunk after hist_len cached tokens.

    k_cache, v_cache: fp64 [nkv][S][d]; only slots < hist_len are read.  The
    new keys/values belong in slots hist_len .. hist_len+T-1 (the in-place
    Concat of Sec. 4.6.3)."""
    kh = k_cache[:, :hist_len, :]
    vh = v_cache[:, :hist_len, :]
    return block(w, cfg, x, pos, kh, vh, rows=rows, W=W)


def decode(w, cfg, x, pos, k_cache, v_cache, ctx_lens, mask=None, W=None):
    """Decode (Sec. 4.4): one token per sequence against its cache.

    x [B][H]; pos [B]; k_cache, v_cache fp64 [B][nkv][S][d];
    ctx_lens [B] valid history per sequence; mask: additive [B][S] or None.
    Sequence b's new token goes to slot ctx_lens[b] and sees slots
    0 .. ctx_lens[b], with mask[b][j] added to the score of slot j.
    Returns y [B][H], k_new, v_new [B][nkv][d]."""
    W = dequant_layer(w, cfg) if W is None else W
    B = len(ctx_lens)
    ys, ks, vs = [], [], []
    for b in range(B):
        c = int(ctx_lens[b])
        bias = None if mask is None else np.asarray(mask, dtype=F64)[b:b + 1, :c + 1]
        y, k, v = block(w, cfg, np.asarray(x, dtype=F64)[b:b + 1], np.asarray(pos)[b:b + 1],
                        k_cache[b][:, :c, :], v_cache[b][:, :c, :], bias, W=W)
        ys.append(y[0]); ks.append(k[0]); vs.append(v[0])
    return np.stack(ys), np.stack(ks), np.stack(vs)


def cache_write(cache, new, start):
    """Copy of cache [nkv][S][d] with new [T][nkv][d] written at slots
    start .. start+T-1 (the in-place Concat, Sec. 4.6.3)."""
    out = np.array(cache, dtype=F64, copy=True)
    out[:, start:start + new.shape[0], :] = np.asarray(new).transpose(1, 0, 2)
    return out
