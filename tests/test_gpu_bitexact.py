"""Bit-exact checks on the GPU: int4 unpacking and dequantisation of every
linear, the standalone KV append, and that each stage writes exactly the
cache slots it owns (the in-place Concat of Sec. 4.6.3)."""
import numpy as np
import pytest
import torch

from oracle import layer as O
from paper_2607_15865_amd import synth
from gpu_helpers import device_layer, host_layer, bits_to_torch_f32, log

pytestmark = pytest.mark.gpu

SENTINEL = 0x7F7F  # bf16 bit pattern never produced by the layer (3.39e38)


@pytest.mark.parametrize("name,zeros", [("tiny", False), ("tiny", True), ("qwen05b", False)])
def test_debug_dequant_exact(name, zeros):
    cfg, w = host_layer(name, 0, zeros)
    lay = device_layer(name, 0, zeros)
    for lin in synth.LINEARS:
        log(f"dequant {name} zeros={zeros} {lin}")
        got = lay.debug_dequant(lin).cpu().numpy().astype(np.float64)
        ref = O.dequant(w[lin], cfg.group_size)
        assert np.array_equal(got, ref), f"{lin}: {np.sum(got != ref)} mismatches"


def test_kv_append_exact():
    from paper_2607_15865_amd import binding
    cfg = synth.CONFIGS["tiny"]
    B, T = 3, 5
    rc, desc = binding.kv_layout(cfg, B)
    assert rc == 0
    k, v = (torch.full((B, cfg.n_kv_heads, cfg.max_seq, cfg.head_dim), SENTINEL, dtype=torch.int16,
                       device="cuda") for _ in range(2))
    rng = np.random.default_rng(0)
    kn = rng.integers(0, 1 << 16, size=(B, T, cfg.n_kv_heads, cfg.head_dim)).astype(np.uint16)
    vn = rng.integers(0, 1 << 16, size=(B, T, cfg.n_kv_heads, cfg.head_dim)).astype(np.uint16)
    kd = torch.from_numpy(kn.view(np.int16)).cuda()
    vd = torch.from_numpy(vn.view(np.int16)).cuda()
    starts = [0, 17, cfg.max_seq - T]
    binding.check(binding.kv_append(desc, k, v, kd, vd, B, T, starts))
    torch.cuda.synchronize()
    kh = k.cpu().numpy().view(np.uint16)
    vh = v.cpu().numpy().view(np.uint16)
    for b in range(B):
        s = starts[b]
        assert np.array_equal(kh[b, :, s:s + T, :], kn[b].transpose(1, 0, 2))
        assert np.array_equal(vh[b, :, s:s + T, :], vn[b].transpose(1, 0, 2))
        rest = np.ones(cfg.max_seq, bool)
        rest[s:s + T] = False
        assert np.all(kh[b, :, rest, :] == SENTINEL) and np.all(vh[b, :, rest, :] == SENTINEL)
    # out-of-range slots are refused before anything runs
    assert binding.kv_append(desc, k, v, kd, vd, B, T, [0, 0, cfg.max_seq - T + 1]) == binding.W4_ECAPACITY


def test_prefill_kv_writes_only_its_slots():
    cfg, w = host_layer("tiny")
    lay = device_layer("tiny")
    L, T = 20, 12
    k, v = lay.new_cache(1, SENTINEL)
    rng = np.random.default_rng(1)
    hist_bits = rng.integers(0, 0x3F00, size=(cfg.n_kv_heads, L, cfg.head_dim)).astype(np.uint16)
    k[0, :, :L, :] = torch.from_numpy(hist_bits.view(np.int16)).cuda()
    v[0, :, :L, :] = torch.from_numpy(hist_bits[::-1].copy().view(np.int16)).cuda()
    x = bits_to_torch_f32(synth.activations(cfg, synth.TID_X_PREFILL_KV, T))
    pos = torch.arange(L, L + T, dtype=torch.int32, device="cuda")
    y = torch.empty_like(x)
    lay.prefill_kv(x, pos, L, k, v, y)
    torch.cuda.synchronize()
    kh = k.cpu().numpy().view(np.uint16)
    vh = v.cpu().numpy().view(np.uint16)
    assert np.array_equal(kh[0, :, :L], hist_bits) and np.array_equal(vh[0, :, :L], hist_bits[::-1])
    assert np.all(kh[0, :, L + T:] == SENTINEL) and np.all(vh[0, :, L + T:] == SENTINEL)
    assert not np.any(kh[0, :, L:L + T] == SENTINEL) and not np.any(vh[0, :, L:L + T] == SENTINEL)


def test_decode_writes_only_slot_ctx():
    cfg, w = host_layer("tiny")
    lay = device_layer("tiny")
    B = 4
    ctx = np.array([0, 5, 77, cfg.max_seq - 1 - 3], dtype=np.int32)
    kb, vb = synth.kv_fill(cfg, B)
    for b in range(B):
        kb[b, :, ctx[b]:, :] = SENTINEL
        vb[b, :, ctx[b]:, :] = SENTINEL
    k = torch.from_numpy(kb.view(np.int16)).cuda()
    v = torch.from_numpy(vb.view(np.int16)).cuda()
    x = bits_to_torch_f32(synth.activations(cfg, synth.TID_X_DECODE, B))
    y = torch.empty_like(x)
    lay.decode(x, torch.from_numpy(ctx).cuda(), torch.from_numpy(ctx).cuda(), int(ctx.max()), k, v, y)
    torch.cuda.synchronize()
    kh = k.cpu().numpy().view(np.uint16)
    vh = v.cpu().numpy().view(np.uint16)
    for b in range(B):
        c = ctx[b]
        assert np.array_equal(kh[b, :, :c], kb[b, :, :c]) and np.array_equal(vh[b, :, :c], vb[b, :, :c])
        assert np.all(kh[b, :, c + 1:] == SENTINEL) and np.all(vh[b, :, c + 1:] == SENTINEL)
        assert not np.any(kh[b, :, c] == SENTINEL) and not np.any(vh[b, :, c] == SENTINEL)
