"""Parity of the kernel variants for the other weight formats: uint8 zero
points (the AWQ-style asymmetric form) and groups of 32 along K.  They run
the GEMM and GEMV variants that the default layers (groups of 64 and 128,
zero point 8) never reach; decode then takes the kernel-sequence path.  Each
case chains prefill (ragged T), prefill_kv and a two-sequence decode against
the oracle."""
import numpy as np
import pytest
import torch

from oracle import layer as O
from paper_2607_15865_amd import binding, synth
from gpu_helpers import assert_parity, bits_to_torch_f32, cache_values, log, to_cache_bits

pytestmark = pytest.mark.gpu

VARIANTS = [("tiny", 64, True, 77), ("tiny", 32, False, 77), ("tiny", 32, True, 33), ("qwen05b", 32, True, 200)]


@pytest.mark.parametrize("name,G,zeros,T", VARIANTS)
def test_variant_chain(name, G, zeros, T):
    cfg = synth.replace(synth.CONFIGS[name], group_size=G)
    w = synth.make_layer(cfg, 0, zeros)
    W = O.dequant_layer(w, cfg)
    lay = binding.Layer(cfg, w)
    try:
        log(f"{name} G={G} zeros={zeros}: prefill T={T}")
        xb = synth.activations(cfg, synth.TID_X_PREFILL, T)
        k, v = lay.new_cache(1, 0)
        x = bits_to_torch_f32(xb)
        y = torch.empty_like(x)
        lay.prefill(x, torch.arange(T, dtype=torch.int32, device="cuda"), k, v, y)
        torch.cuda.synchronize()
        yo, ko, vo = O.prefill(w, cfg, O.bf16_to_f64(xb), np.arange(T), W=W)
        assert_parity(y.cpu().numpy(), yo, "prefill y")
        kc = O.cache_write(np.zeros((cfg.n_kv_heads, cfg.max_seq, cfg.head_dim)), ko, 0)
        vc = O.cache_write(np.zeros_like(kc), vo, 0)
        assert_parity(cache_values(k)[0][:, :T, :].transpose(1, 0, 2), ko, "prefill new K")

        T2 = 16
        log(f"  prefill_kv T={T2} over {T}")
        k = torch.from_numpy(to_cache_bits(kc)[None]).cuda()
        v = torch.from_numpy(to_cache_bits(vc)[None]).cuda()
        xb2 = synth.activations(cfg, synth.TID_X_PREFILL_KV, T2)
        x2 = bits_to_torch_f32(xb2)
        y2 = torch.empty_like(x2)
        pos2 = np.arange(T, T + T2)
        lay.prefill_kv(x2, torch.from_numpy(pos2.astype(np.int32)).cuda(), T, k, v, y2)
        torch.cuda.synchronize()
        yo2, ko2, vo2 = O.prefill_kv(w, cfg, O.bf16_to_f64(xb2), pos2, kc, vc, T, W=W)
        assert_parity(y2.cpu().numpy(), yo2, "prefill_kv y")
        assert_parity(cache_values(v)[0][:, T:T + T2, :].transpose(1, 0, 2), vo2, "prefill_kv new V")

        B, ctx = 2, np.array([T + T2, 50], dtype=np.int32)
        kb, vb = synth.kv_fill(cfg, B)
        xb3 = synth.activations(cfg, synth.TID_X_DECODE, B)
        for path in (0, 1):
            log(f"  decode B={B} ctx={ctx.tolist()} path={path}")
            lay.set_decode_path(path)
            kd = torch.from_numpy(kb.view(np.int16).copy()).cuda()
            vd = torch.from_numpy(vb.view(np.int16).copy()).cuda()
            x3 = bits_to_torch_f32(xb3)
            y3 = torch.empty_like(x3)
            c = torch.from_numpy(ctx).cuda()
            lay.decode(x3, c, c, int(ctx.max()), kd, vd, y3)
            torch.cuda.synchronize()
            yo3, ko3, _ = O.decode(w, cfg, O.bf16_to_f64(xb3), ctx, O.bf16_to_f64(kb), O.bf16_to_f64(vb), ctx, W=W)
            assert_parity(y3.cpu().numpy(), yo3, f"decode y (path {path})")
            gk = cache_values(kd)
            assert_parity(np.stack([gk[b][:, ctx[b], :] for b in range(B)]), ko3, f"decode new K (path {path})")
        lay.set_decode_path(0)
    finally:
        lay.close()
