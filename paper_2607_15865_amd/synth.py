"""Seeded synthetic inputs for the three-stage W4A16 decoder layer.

This module only draws random numbers and encodes them into the storage
formats the layer consumes (bf16 bit patterns, fp16 scales, int4 nibbles
packed into 32-bit words).  It performs none of the layer's arithmetic, so
both the CPU oracle and the GPU path can take their inputs from here.

Workload shapes follow the model families the paper deploys (Qwen and Llama
decoders, Sec. 1 and Sec. 5); the paper's own Qwen3.5 checkpoints are not
available, so seeded random layers of the same shapes stand in for them.

Weight format (canonical, GPTQ-style "already quantized" weights that the
paper passes straight through the lowering, Sec. 3.2):
  * ``q[k][n]`` are unsigned 4-bit codes in [0, 15];
  * ``qweight[r][n]`` (int32) holds codes k = 8r .. 8r+7 of column n, code
    8r+j in bits 4j .. 4j+3;
  * ``scales[g][n]`` (fp16) is the scale of group g = k // group_size;
  * the zero point is 8 unless a ``zeros[g][n]`` array is given.
The paper's other direct-through weight modes (Sec. 3.2) are drawn too:
INT8 symmetric / asymmetric with per-channel scales, and BF16 (make_linear).
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional

import numpy as np

LINEARS = ("q", "k", "v", "o", "gate", "up", "down")

# Tensor ids of the per-tensor random streams.
TID_X_PREFILL = 0
TID_X_PREFILL_KV = 1
TID_X_DECODE = 2          # per decode step s: 2 + 1000 * s
TID_K_FILL = 3
TID_V_FILL = 4
TID_MASK = 5
TID_GAMMA1 = 10
TID_GAMMA2 = 11
TID_QVALS = 20            # + linear index
TID_SCALES = 30           # + linear index
TID_ZEROS = 40            # + linear index
TID_EMBED = 60            # model ends: embedding table, final norm, LM head
TID_FINAL_NORM = 61
TID_HEAD_QVALS = 62
TID_HEAD_SCALES = 63
TID_HEAD_ZEROS = 64
TID_TOKENS = 65


@dataclasses.dataclass(frozen=True)
class LayerConfig:
    name: str
    hidden: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    group_size: int
    rms_eps: float
    rope_base: float
    max_seq: int
    max_batch: int = 8
    cfg_id: int = 0

    def linear_shape(self, which: str):
        """(K, N) of a linear: y[M][N] = x[M][K] @ W[K][N]."""
        h, qd, kvd, f = (self.hidden, self.n_heads * self.head_dim,
                         self.n_kv_heads * self.head_dim, self.ffn)
        return {"q": (h, qd), "k": (h, kvd), "v": (h, kvd), "o": (qd, h),
                "gate": (h, f), "up": (h, f), "down": (f, h)}[which]


CONFIGS: Dict[str, LayerConfig] = {
    # Tiny decoder layer used for parity at sizes the oracle finishes quickly.
    "tiny": LayerConfig("tiny", 256, 4, 2, 64, 688, 64, 1e-6, 1e4, 128, 8, 0),
    # Qwen2.5-0.5B-shaped layer.
    "qwen05b": LayerConfig("qwen05b", 896, 14, 2, 64, 4864, 128, 1e-6, 1e4, 1024, 8, 1),
    # Llama-3-8B-shaped layer.
    "llama8b": LayerConfig("llama8b", 4096, 32, 8, 128, 14336, 128, 1e-6, 5e5, 4096, 8, 2),
    # Qwen2.5-7B-shaped layer.
    "qwen7b": LayerConfig("qwen7b", 3584, 28, 4, 128, 18944, 128, 1e-6, 1e4, 8448, 8, 3),
}

# The runs each configuration is exercised with: prefill length, the
# prefill_kv chunk and its history, decode context lengths and batches.
RUNS = {
    "tiny": dict(prefill_T=32, pkv_T=16, pkv_hist=32, decode_ctx=48, decode_steps=16, decode_B=(1,)),
    "qwen05b": dict(prefill_T=256, pkv_T=64, pkv_hist=256, decode_ctx=512, decode_steps=1, decode_B=(1,)),
    "llama8b": dict(prefill_T=512, pkv_T=128, pkv_hist=1024, decode_ctx=2048, decode_steps=1, decode_B=(1,)),
    "qwen7b": dict(prefill_T=2048, pkv_T=None, pkv_hist=None, decode_ctx=8192, decode_steps=1, decode_B=(1, 8)),
}


def rng_for(cfg_id: int, layer: int, tensor_id: int) -> np.random.Generator:
    return np.random.default_rng([0x5EED, int(cfg_id), int(layer), int(tensor_id)])


# ---------------------------------------------------------------- encodings

def bf16_bits(x) -> np.ndarray:
    """Round to bfloat16 (round to nearest, ties to even) and return the bits.

    The value is first rounded to fp32 (exact for every draw used here except
    in the last fp32 bit), then the upper 16 bits are kept with RNE.
    """
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    nan = np.isnan(f)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)
    if nan.any():
        r = np.where(nan, np.uint16(0x7FC0), r)
    return r


def pack_int4(q: np.ndarray) -> np.ndarray:
    """Pack codes q[K][N] (0..15, K % 8 == 0) into qweight[K/8][N] int32."""
    q = np.asarray(q)
    K, N = q.shape
    if K % 8:
        raise ValueError("K must be a multiple of 8")
    qu = q.astype(np.uint32).reshape(K // 8, 8, N)
    words = np.zeros((K // 8, N), dtype=np.uint32)
    for j in range(8):
        words |= qu[:, j, :] << np.uint32(4 * j)
    return words.view(np.int32)


# ---------------------------------------------------------------- draws

WEIGHT_FORMATS = ("int4", "int8", "int8a", "bf16")


def make_linear(cfg: LayerConfig, which: str, layer: int = 0,
                with_zeros: bool = False, fmt: str = "int4") -> dict:
    """One linear in weight format ``fmt``:

    * "int4": codes uniform in [0, 15], fp16 scales |N(0, 0.02)| / 8 per
      group, zero point 8 (or per-group zero points uniform in [0, 15]);
    * "int8" (symmetric): signed codes uniform in [-128, 127], one fp16 scale
      |N(0, 0.02)| / 128 per output channel;
    * "int8a" (asymmetric): unsigned codes uniform in [0, 255], per-channel
      zero points uniform in [96, 160] and scales as "int8";
    * "bf16": N(0, 0.01) weights as bf16 bit patterns.
    The 8-bit and bf16 draws give weights of about the magnitude of the
    4-bit ones."""
    j = LINEARS.index(which)
    K, N = cfg.linear_shape(which)
    if fmt in ("int8", "int8a"):
        s = np.abs(rng_for(cfg.cfg_id, layer, TID_SCALES + j).normal(0.0, 0.02, size=N)) / 128.0
        g = rng_for(cfg.cfg_id, layer, TID_QVALS + j)
        if fmt == "int8":
            q8 = g.integers(-128, 128, size=(K, N), dtype=np.int16).astype(np.int8)
            zeros = None
        else:
            q8 = g.integers(0, 256, size=(K, N), dtype=np.int16).astype(np.uint8)
            zeros = rng_for(cfg.cfg_id, layer, TID_ZEROS + j).integers(96, 161, size=N, dtype=np.int16).astype(np.uint8)
        return dict(format="int8", K=K, N=N, q8=q8, scales=s.astype(np.float16), zeros=zeros)
    if fmt == "bf16":
        w16 = bf16_bits(rng_for(cfg.cfg_id, layer, TID_QVALS + j).normal(0.0, 0.01, size=(K, N)))
        return dict(format="bf16", K=K, N=N, w16=w16)
    if fmt != "int4":
        raise ValueError(f"unknown weight format {fmt!r}")
    ng = -(-K // cfg.group_size)
    q = rng_for(cfg.cfg_id, layer, TID_QVALS + j).integers(0, 16, size=(K, N), dtype=np.uint8)
    s = (np.abs(rng_for(cfg.cfg_id, layer, TID_SCALES + j).normal(0.0, 0.02, size=(ng, N))) / 8.0)
    scales = s.astype(np.float16)
    zeros = None
    if with_zeros:
        zeros = rng_for(cfg.cfg_id, layer, TID_ZEROS + j).integers(0, 16, size=(ng, N), dtype=np.uint8)
    return dict(K=K, N=N, q=q, qweight=pack_int4(q), scales=scales, zeros=zeros)


def make_layer(cfg: LayerConfig, layer: int = 0, with_zeros: bool = False, fmt: str = "int4") -> dict:
    """All weights of one decoder layer in the canonical host format (every
    linear in weight format ``fmt``, see make_linear)."""
    w = {name: make_linear(cfg, name, layer, with_zeros, fmt) for name in LINEARS}
    w["attn_norm"] = bf16_bits(rng_for(cfg.cfg_id, layer, TID_GAMMA1).uniform(0.5, 1.5, cfg.hidden))
    w["mlp_norm"] = bf16_bits(rng_for(cfg.cfg_id, layer, TID_GAMMA2).uniform(0.5, 1.5, cfg.hidden))
    return w


def make_layer_words(cfg: LayerConfig, layer: int = 0) -> dict:
    """All weights of one layer drawn as packed words: each int32 word of a
    qweight is uniform, so its eight codes are independent and uniform in
    [0, 15] (the distribution of make_layer, drawn about 8x faster).  Scales
    and norm weights as make_layer.  For throughput runs over many layers."""
    w = {}
    for j, name in enumerate(LINEARS):
        K, N = cfg.linear_shape(name)
        ng = -(-K // cfg.group_size)
        words = rng_for(cfg.cfg_id, layer, TID_QVALS + j).integers(0, 1 << 32, size=(K // 8, N), dtype=np.uint32)
        s = np.abs(rng_for(cfg.cfg_id, layer, TID_SCALES + j).normal(0.0, 0.02, size=(ng, N))) / 8.0
        w[name] = dict(K=K, N=N, qweight=words.view(np.int32), scales=s.astype(np.float16), zeros=None)
    w["attn_norm"] = bf16_bits(rng_for(cfg.cfg_id, layer, TID_GAMMA1).uniform(0.5, 1.5, cfg.hidden))
    w["mlp_norm"] = bf16_bits(rng_for(cfg.cfg_id, layer, TID_GAMMA2).uniform(0.5, 1.5, cfg.hidden))
    return w


def normal_bf16(cfg_id: int, layer: int, tensor_id: int, shape) -> np.ndarray:
    """bf16 bits of N(0, 1) draws."""
    return bf16_bits(rng_for(cfg_id, layer, tensor_id).standard_normal(size=shape))


def activations(cfg: LayerConfig, tensor_id: int, rows: int, layer: int = 0) -> np.ndarray:
    """Hidden states x[rows][hidden] as bf16 bits, N(0, 1)."""
    return normal_bf16(cfg.cfg_id, layer, tensor_id, (rows, cfg.hidden))


def kv_fill(cfg: LayerConfig, batch: int, layer: int = 0):
    """A full K and V cache [B][n_kv][max_seq][d] of N(0, 1) bf16 bits."""
    shape = (batch, cfg.n_kv_heads, cfg.max_seq, cfg.head_dim)
    return (normal_bf16(cfg.cfg_id, layer, TID_K_FILL, shape),
            normal_bf16(cfg.cfg_id, layer, TID_V_FILL, shape))


def replace(cfg: LayerConfig, **kw) -> LayerConfig:
    return dataclasses.replace(cfg, **kw)


def zero_linear(lin: dict) -> dict:
    """The same linear with every code at the zero point (W == 0)."""
    q = np.full_like(lin["q"], 8)
    out = dict(lin)
    out.update(q=q, qweight=pack_int4(q), zeros=None)
    return out


def as_optional(a: Optional[np.ndarray]):
    return None if a is None else np.ascontiguousarray(a)


def make_lm(cfg: LayerConfig, vocab: int, with_zeros: bool = False, words: bool = False) -> dict:
    """The two ends of a model with cfg's hidden size: a bf16 embedding
    table [vocab][hidden] of N(0, 1) draws, a final RMSNorm weight (bf16,
    uniform in [0.5, 1.5]) and a 4-bit LM head [hidden][vocab] drawn like
    the layer's linears (codes uniform in [0, 15], fp16 scales
    |N(0, 0.02)| / 8, zero point 8 unless zero points are drawn).  With
    words=True the head's packed words are drawn directly, as in
    make_layer_words (no "q" array), and the embedding table repeats 8192
    drawn rows."""
    H, G = cfg.hidden, cfg.group_size
    ng = -(-H // G)
    s = np.abs(rng_for(cfg.cfg_id, 0, TID_HEAD_SCALES).normal(0.0, 0.02, size=(ng, vocab))) / 8.0
    zeros = None
    if with_zeros:
        zeros = rng_for(cfg.cfg_id, 0, TID_HEAD_ZEROS).integers(0, 16, size=(ng, vocab), dtype=np.uint8)
    if words:
        w = rng_for(cfg.cfg_id, 0, TID_HEAD_QVALS).integers(0, 1 << 32, size=(H // 8, vocab), dtype=np.uint32)
        head = dict(K=H, N=vocab, qweight=w.view(np.int32), scales=s.astype(np.float16), zeros=zeros)
    else:
        q = rng_for(cfg.cfg_id, 0, TID_HEAD_QVALS).integers(0, 16, size=(H, vocab), dtype=np.uint8)
        head = dict(K=H, N=vocab, q=q, qweight=pack_int4(q), scales=s.astype(np.float16), zeros=zeros)
    if words:   # throughput runs: 8192 distinct embedding rows, repeated
        base = normal_bf16(cfg.cfg_id, 0, TID_EMBED, (min(vocab, 8192), H))
        embed = np.tile(base, (-(-vocab // base.shape[0]), 1))[:vocab]
    else:
        embed = normal_bf16(cfg.cfg_id, 0, TID_EMBED, (vocab, H))
    return dict(vocab=vocab, embed=embed,
                final_norm=bf16_bits(rng_for(cfg.cfg_id, 0, TID_FINAL_NORM).uniform(0.5, 1.5, H)),
                head=head)


def tokens(cfg: LayerConfig, vocab: int, n: int, seed: int = 0) -> np.ndarray:
    """n token ids uniform in [0, vocab) (int32)."""
    return rng_for(cfg.cfg_id, seed, TID_TOKENS).integers(0, vocab, size=n).astype(np.int32)
