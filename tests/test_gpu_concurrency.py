"""Stage calls that share one layer handle.

The handle holds no device state that a prefill call changes: the split-K
arrival counters of the GEMMs live in the caller's workspace as tagged words
that need no clearing.  So prefill calls in flight together on two streams,
each with its own workspace, caches and output, give the same bits as the
same calls made one after another; and a workspace that a decode call left
full of its own tagged words serves a prefill_kv call without clearing."""
import numpy as np
import pytest
import torch

from paper_2607_15865_amd import binding, synth
from gpu_helpers import bits_to_torch_f32, device_layer, host_layer, log

pytestmark = pytest.mark.gpu


def _inputs(cfg, T, L, seed):
    kb, vb = synth.kv_fill(cfg, 1)
    k = torch.from_numpy(kb.view(np.int16).copy()).cuda()
    v = torch.from_numpy(vb.view(np.int16).copy()).cuda()
    x = bits_to_torch_f32(synth.activations(cfg, synth.TID_X_PREFILL_KV + seed, T))
    pos = torch.arange(L, L + T, dtype=torch.int32, device="cuda")
    return x, pos, k, v, torch.empty_like(x)


@pytest.mark.parametrize("name,T,L", [("llama8b", 128, 1024), ("tiny", 16, 32)])
def test_two_streams_match_serial_calls(name, T, L):
    cfg, _ = host_layer(name)
    lay = device_layer(name)
    h = lay.handle
    n = binding.layer_workspace_size(h, 1, 1, T, L)
    ins = [_inputs(cfg, T, L, s) for s in range(2)]
    wss = [torch.empty(n, dtype=torch.uint8, device="cuda") for _ in range(2)]
    ref = []
    for (x, pos, k, v, y), ws in zip(ins, wss):
        binding.check(binding.layer_prefill_kv(h, x, pos, T, L, k, v, y, ws, n))
        torch.cuda.synchronize()
        ref.append((y.cpu().numpy().copy(), k.cpu().numpy().copy(), v.cpu().numpy().copy()))
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    log(f"{name}: prefill_kv T={T} over {L} on two streams, 4 rounds")
    for _ in range(4):
        for (x, pos, k, v, y), ws, st in zip(ins, wss, streams):
            y.fill_(float("nan"))
        torch.cuda.synchronize()
        for (x, pos, k, v, y), ws, st in zip(ins, wss, streams):
            binding.check(binding.layer_prefill_kv(h, x, pos, T, L, k, v, y, ws, n, st))
        torch.cuda.synchronize()
        for (x, pos, k, v, y), (yr, kr, vr) in zip(ins, ref):
            assert np.array_equal(y.cpu().numpy(), yr)
            assert np.array_equal(k.cpu().numpy(), kr) and np.array_equal(v.cpu().numpy(), vr)


def test_workspace_after_decode_serves_prefill_kv():
    """Decode writes tagged words over its workspace; the next prefill_kv on
    the same memory must not mistake them for its own split-K counts."""
    name, T, L, ctx = "llama8b", 128, 1024, 2048
    cfg, _ = host_layer(name)
    lay = device_layer(name)
    h = lay.handle
    n = max(binding.layer_workspace_size(h, 1, 1, T, L), binding.layer_workspace_size(h, 2, 1, 1, ctx))
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    x, pos, k, v, y = _inputs(cfg, T, L, 0)
    binding.check(binding.layer_prefill_kv(h, x, pos, T, L, k, v, y, ws, n))
    torch.cuda.synchronize()
    yr = y.cpu().numpy().copy()
    kd, vd = lay.new_cache(1, 0)
    xd = bits_to_torch_f32(synth.activations(cfg, synth.TID_X_DECODE, 1))
    c = torch.full((1,), ctx, dtype=torch.int32, device="cuda")
    yd = torch.empty_like(xd)
    for _ in range(3):
        binding.check(binding.layer_decode(h, xd, c, c, ctx, None, 1, kd, vd, yd, ws, n))
        y.fill_(float("nan"))
        binding.check(binding.layer_prefill_kv(h, x, pos, T, L, k, v, y, ws, n))
        torch.cuda.synchronize()
        assert np.array_equal(y.cpu().numpy(), yr)
