"""CPU oracle for the two ends of the model around the decoder layers.

TEST INFRASTRUCTURE ONLY.  Only the tests, the package's smoke check and the
benchmark's CPU-baseline leg may import this module; the product path never
does, and this module imports nothing from the product path.

The paper's runtime loop (Sec. 2, the inference procedure; Sec. 4.5, runtime
orchestration) brackets the decoder layers with three steps: the token ids
are turned into hidden states by the word-embedding module, the last hidden
state goes through the language-model head to give logits, and the next
token is sampled from the logits and fed back.  Readings taken where the
paper leaves the details open:

  * the embedding is a table lookup, row t of a bf16 table [vocab][hidden];
  * the LM head is the model's final RMSNorm followed by a 4-bit
    group-quantised linear [hidden][vocab] in the same canonical format as
    the layer's linears; the normalised input is rounded to bf16 once, as
    every normalised matmul input of the block is (module docstring of
    oracle.layer), and the logits are fp64;
  * sampling is greedy: the index of the largest logit, the lowest index
    among equal maxima.

Pins: tests/test_oracle_lm.py checks each function against brute-force
loops on tiny inputs and closed forms; none is "parity unpinned".
"""
from __future__ import annotations

import numpy as np

from oracle.layer import bf16_to_f64, dequant, rmsnorm, round_bf16

F64 = np.float64


def embed(table_bits, tokens) -> np.ndarray:
    """Word embedding (first step of the runtime loop, Sec. 2): hidden state
    of token t = row t of the bf16 table, as exact fp64 values."""
    table_bits = np.asarray(table_bits, dtype=np.uint16)
    tokens = np.asarray(tokens, dtype=np.int64)
    V = table_bits.shape[0]
    if tokens.size and (tokens.min() < 0 or tokens.max() >= V):
        raise ValueError("token id outside the vocabulary")
    return bf16_to_f64(table_bits[tokens])


def lm_logits(x, final_norm_bits, head: dict, group_size: int, eps: float) -> np.ndarray:
    """LM head (the runtime loop's logits step, Sec. 2): logits[b][v] =
    sum_k bf16(RMSNorm(x[b]))[k] * W[k][v] with the head weight dequantised
    exactly (Sec. 3.2).  x: fp32/fp64 hidden states [B][hidden]."""
    x = np.asarray(x, dtype=F64)
    xn = round_bf16(rmsnorm(x, bf16_to_f64(final_norm_bits), eps))
    return xn @ dequant(head, group_size)


def greedy(logits) -> np.ndarray:
    """Greedy sampling (the runtime loop's sampling step, Sec. 2): per row
    the index of the largest logit, the lowest index among equal maxima."""
    return np.argmax(np.asarray(logits, dtype=F64), axis=-1).astype(np.int64)
