"""Failures the host cannot see, made visible through the device error
flags (layer_error, lm_error, and the -1 picks of the native loop step):

* an activation whose bf16 value is beyond the fp16 range where the fp16
  matrix operands are formed (the normalised inputs, the attention output,
  the SwiGLU output) -- forced with scaled weights or cache values;
* a wait of the persistent decode that gives up -- forced from the host with
  a tiny poll budget, so every wait still ends and the launch runs to its
  end (Sec. 4.4 is the stage the loop runs most often).

Each test reads, and so clears, the flags it raises."""
import copy

import numpy as np
import pytest
import torch

from paper_2607_15865_amd import binding, synth
from gpu_helpers import bits_to_torch_f32, host_layer, log

pytestmark = pytest.mark.gpu

BIG_BF16 = 0x47C3        # bf16 99840
BIG_F16 = np.float16(60000.0)


def scaled_layer(which):
    cfg, w = host_layer("tiny")
    w = copy.deepcopy(w)
    if which == "attn_norm":
        w["attn_norm"] = np.full(cfg.hidden, BIG_BF16, dtype=np.uint16)
    elif which == "mlp_norm":
        w["mlp_norm"] = np.full(cfg.hidden, BIG_BF16, dtype=np.uint16)
    elif which == "v":
        w["v"]["scales"] = np.full_like(w["v"]["scales"], BIG_F16)
    elif which == "gate_up":
        for n in ("gate", "up"):
            w[n]["scales"] = np.full_like(w[n]["scales"], BIG_F16)
    return cfg, binding.Layer(cfg, w)


def run_prefill(cfg, lay, T=16):
    xb = synth.activations(cfg, synth.TID_X_PREFILL, T)
    x = bits_to_torch_f32(xb)
    y = torch.empty_like(x)
    k, v = lay.new_cache(1, 0)
    lay.prefill(x, torch.arange(T, dtype=torch.int32, device="cuda"), k, v, y)


def run_decode(cfg, lay, B, path, big_cache=False):
    lay.set_decode_path(path)
    kb, vb = synth.kv_fill(cfg, B)
    if big_cache:
        vb = np.full_like(vb, BIG_BF16)
    k = torch.from_numpy(kb.view(np.int16).copy()).cuda()
    v = torch.from_numpy(vb.view(np.int16).copy()).cuda()
    xb = synth.activations(cfg, synth.TID_X_DECODE, B)
    x = bits_to_torch_f32(xb)
    y = torch.empty_like(x)
    c = torch.full((B,), 50, dtype=torch.int32, device="cuda")
    lay.decode(x, c, c, 50, k, v, y)
    lay.set_decode_path(0)


@pytest.mark.parametrize("which", ["attn_norm", "mlp_norm", "v", "gate_up"])
def test_f16_range_flag_prefill(which):
    cfg, lay = scaled_layer(which)
    assert lay.error() == 0
    run_prefill(cfg, lay)
    f = lay.error()
    log(f"prefill with scaled {which}: flag {f}")
    assert f & binding.W4_FLAG_F16_RANGE
    assert lay.error() == 0          # read and cleared
    lay.close()


@pytest.mark.parametrize("which,B,path", [("attn_norm", 1, 2), ("attn_norm", 1, 1), ("attn_norm", 5, 0),
                                         ("mlp_norm", 1, 2), ("mlp_norm", 2, 1), ("mlp_norm", 4, 1),
                                         ("gate_up", 1, 2), ("gate_up", 3, 1)])
def test_f16_range_flag_decode(which, B, path):
    cfg, lay = scaled_layer(which)
    run_decode(cfg, lay, B, path)
    f = lay.error()
    log(f"decode B={B} path {path} with scaled {which}: flag {f}")
    assert f & binding.W4_FLAG_F16_RANGE
    lay.close()


@pytest.mark.parametrize("B,path", [(1, 2), (2, 1), (4, 0)])
def test_f16_range_flag_attention_output(B, path):
    """A cache of values near 1e5: the attention output (a convex combination
    of the values) is beyond the fp16 range."""
    cfg, w = host_layer("tiny")
    lay = binding.Layer(cfg, w)
    run_decode(cfg, lay, B, path, big_cache=True)
    f = lay.error()
    log(f"decode B={B} path {path} with a large V cache: flag {f}")
    assert f & binding.W4_FLAG_F16_RANGE
    # the same layer on the synthetic cache raises nothing
    run_decode(cfg, lay, B, path)
    assert lay.error() == 0
    lay.close()


def test_f16_range_flag_lm_head():
    cfg = synth.CONFIGS["tiny"]
    V = 1024
    lw = synth.make_lm(cfg, V)
    lw = dict(lw, final_norm=np.full(cfg.hidden, BIG_BF16, dtype=np.uint16))
    lmh = binding.LM(cfg, lw, max_batch=2)
    x = torch.ones(2, cfg.hidden, device="cuda")
    logits = torch.empty(2, V, device="cuda")
    lmh.head(x, logits, None)
    f = lmh.error()
    assert f & binding.W4_FLAG_F16_RANGE and lmh.error() == 0
    lmh.close()


def test_wait_timeout_flag_and_sentinel_picks():
    """A persistent decode whose waits give up at once: the launch ends, the
    layer flags W4_FLAG_WAIT_TIMEOUT, and a native loop step over that layer
    turns its picks into -1.  With the default budget the same calls raise
    nothing."""
    cfg, w = host_layer("tiny")
    lay = binding.Layer(cfg, w)
    binding.check(binding.layer_set_decode_spin_limit(lay.handle, 1))
    run_decode(cfg, lay, 1, 2)
    f = lay.error()
    log(f"persistent decode with a poll budget of 1: flag {f}")
    assert f & binding.W4_FLAG_WAIT_TIMEOUT

    V, B, ctx = 1024, 2, 30
    lmh = binding.LM(cfg, synth.make_lm(cfg, V), max_batch=B)
    k, v = lay.new_cache(B, 0)
    tok = torch.from_numpy(synth.tokens(cfg, V, B)).cuda()
    logits = torch.empty(B, V, device="cuda")
    c = torch.full((B,), ctx, dtype=torch.int32, device="cuda")
    n = binding.model_decode_workspace_size([lay.handle], lmh.handle, B, ctx)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    binding.check(binding.model_decode_greedy([lay.handle], lmh.handle, tok, c, c, ctx, B, [k], [v], logits, tok,
                                              ws, n))
    torch.cuda.synchronize()
    picks = tok.cpu().numpy()
    log(f"  picks after a timed-out step: {picks}")
    assert (picks == -1).all()
    assert lay.error() & binding.W4_FLAG_WAIT_TIMEOUT
    lmh.error()      # (the outputs of the timed-out step are not valid: clear whatever they raised)
    # a clean step with the default budget
    binding.check(binding.layer_set_decode_spin_limit(lay.handle, 0))
    tok = torch.from_numpy(synth.tokens(cfg, V, B)).cuda()
    binding.check(binding.model_decode_greedy([lay.handle], lmh.handle, tok, c, c, ctx, B, [k], [v], logits, tok,
                                              ws, n))
    torch.cuda.synchronize()
    assert (tok.cpu().numpy() >= 0).all() and lay.error() == 0 and lmh.error() == 0
    lmh.close()
    lay.close()


def test_sentinel_picks_past_the_first_64_flags():
    """The pick guard reads up to 64 error words per launch; a model of 70
    layers needs a second launch.  Only the last layer (the 71st word after
    the LM's) times out: the picks still turn into -1, and a clean step over
    the same layers picks valid tokens."""
    cfg, w = host_layer("tiny")
    n_layers, V, B, ctx = 70, 1024, 1, 12
    lays = [binding.Layer(cfg, w) for _ in range(n_layers)]
    lmh = binding.LM(cfg, synth.make_lm(cfg, V), max_batch=B)
    caches = [l.new_cache(B, 0) for l in lays]
    logits = torch.empty(B, V, device="cuda")
    c = torch.full((B,), ctx, dtype=torch.int32, device="cuda")
    hs = [l.handle for l in lays]
    n = binding.model_decode_workspace_size(hs, lmh.handle, B, ctx)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")

    def step():
        tok = torch.from_numpy(synth.tokens(cfg, V, B)).cuda()
        binding.check(binding.model_decode_greedy(hs, lmh.handle, tok, c, c, ctx, B, [k for k, _ in caches],
                                                  [v for _, v in caches], logits, tok, ws, n))
        torch.cuda.synchronize()
        return tok.cpu().numpy()

    picks = step()
    assert (picks >= 0).all() and all(l.error() == 0 for l in lays) and lmh.error() == 0
    binding.check(binding.layer_set_decode_spin_limit(lays[-1].handle, 1))
    picks = step()
    log(f"  70 layers, the last one timed out: picks {picks}")
    assert (picks == -1).all()
    assert lays[-1].error() & binding.W4_FLAG_WAIT_TIMEOUT
    assert all(l.error() == 0 for l in lays[:-1])
    lmh.error()      # (the outputs of the timed-out step are not valid)
    binding.check(binding.layer_set_decode_spin_limit(lays[-1].handle, 0))
    picks = step()
    assert (picks >= 0).all() and lays[-1].error() == 0 and lmh.error() == 0
    lmh.close()
    for l in lays:
        l.close()


def test_range_flag_turns_picks_into_minus_one():
    cfg, lay = scaled_layer("attn_norm")
    V, B, ctx = 1024, 1, 10
    lmh = binding.LM(cfg, synth.make_lm(cfg, V), max_batch=B)
    k, v = lay.new_cache(B, 0)
    tok = torch.from_numpy(synth.tokens(cfg, V, B)).cuda()
    logits = torch.empty(B, V, device="cuda")
    c = torch.full((B,), ctx, dtype=torch.int32, device="cuda")
    n = binding.model_decode_workspace_size([lay.handle], lmh.handle, B, ctx)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    binding.check(binding.model_decode_greedy([lay.handle], lmh.handle, tok, c, c, ctx, B, [k], [v], logits, tok,
                                              ws, n))
    torch.cuda.synchronize()
    assert int(tok.item()) == -1
    assert lay.error() & binding.W4_FLAG_F16_RANGE
    lmh.error()
    lmh.close()
    lay.close()
