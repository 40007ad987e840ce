"""A stack of layers (Sec. 4.5 runtime orchestration) run through
stack_prefill / stack_decode on the GPU, against the oracle layers chained
on their own caches: prefill, prefill_kv, then decode steps, each layer with
its own seeded weights and caches.  Outputs after every call are held to the
parity bound."""
import numpy as np
import pytest
import torch

from oracle import layer as O
from paper_2607_15865_amd import binding, synth
from gpu_helpers import assert_parity, bits_to_torch_f32, cache_values, host_layer, log, oracle_weights

pytestmark = pytest.mark.gpu


def test_stack_chain_matches_chained_oracle_layers():
    name, nl = "tiny", 3
    cfg = synth.CONFIGS[name]
    hw = [host_layer(name, layer=l)[1] for l in range(nl)]
    W = [oracle_weights(name, layer=l) for l in range(nl)]
    layers = [binding.Layer(cfg, hw[l]) for l in range(nl)]
    st = binding.Stack(layers)
    caches = [l.new_cache(1, 0) for l in layers]
    kcs, vcs = [c[0] for c in caches], [c[1] for c in caches]
    okc = [np.zeros((cfg.n_kv_heads, cfg.max_seq, cfg.head_dim)) for _ in range(nl)]
    ovc = [np.zeros_like(okc[0]) for _ in range(nl)]

    def oracle_chain(fn, xv):
        for l in range(nl):
            xv = fn(l, xv)
        return xv

    P, C, D = 32, 16, 4
    # prefill
    xb = synth.activations(cfg, synth.TID_X_PREFILL, P)
    x = bits_to_torch_f32(xb)
    y = torch.empty_like(x)
    st.prefill(x, torch.arange(P, dtype=torch.int32, device="cuda"), 0, kcs, vcs, y)

    def pf(l, xv):
        yo, ko, vo = O.prefill(hw[l], cfg, xv, np.arange(P), W=W[l])
        okc[l], ovc[l] = O.cache_write(okc[l], ko, 0), O.cache_write(ovc[l], vo, 0)
        return yo
    yo = oracle_chain(pf, O.bf16_to_f64(xb))
    assert_parity(y.cpu().numpy(), yo, "stack prefill y")
    # prefill_kv
    xb = synth.activations(cfg, synth.TID_X_PREFILL_KV, C)
    x = bits_to_torch_f32(xb)
    y = torch.empty_like(x)
    st.prefill(x, torch.arange(P, P + C, dtype=torch.int32, device="cuda"), P, kcs, vcs, y)

    def pkv(l, xv):
        yo, ko, vo = O.prefill_kv(hw[l], cfg, xv, np.arange(P, P + C), okc[l], ovc[l], P, W=W[l])
        okc[l], ovc[l] = O.cache_write(okc[l], ko, P), O.cache_write(ovc[l], vo, P)
        return yo
    yo = oracle_chain(pkv, O.bf16_to_f64(xb))
    assert_parity(y.cpu().numpy(), yo, "stack prefill_kv y")
    # decode steps
    for s in range(D):
        t = P + C + s
        xb = synth.activations(cfg, synth.TID_X_DECODE + 1000 * s, 1)
        x = bits_to_torch_f32(xb)
        y = torch.empty_like(x)
        td = torch.tensor([t], dtype=torch.int32, device="cuda")
        st.decode(x, td, td, t, kcs, vcs, y)

        def dec(l, xv):
            yo, ko, vo = O.decode(hw[l], cfg, xv, [t], okc[l][None], ovc[l][None], [t], W=W[l])
            okc[l], ovc[l] = O.cache_write(okc[l], ko, t), O.cache_write(ovc[l], vo, t)
            return yo
        yo = oracle_chain(dec, O.bf16_to_f64(xb))
        assert_parity(y.cpu().numpy(), yo, f"stack decode step {s} y")
    torch.cuda.synchronize()
    n = P + C + D
    for l in range(nl):
        assert_parity(cache_values(kcs[l])[0][:, :n], okc[l][:, :n], f"layer {l} cache K")
        assert_parity(cache_values(vcs[l])[0][:, :n], ovc[l][:, :n], f"layer {l} cache V")


def test_stack_of_one_equals_the_layer_call():
    """stack_* with one layer is the single-layer call: bit-identical."""
    name = "tiny"
    cfg, w = host_layer(name)
    lay = binding.Layer(cfg, w)
    st = binding.Stack([lay])
    P = 24
    xb = synth.activations(cfg, synth.TID_X_PREFILL, P)
    x = bits_to_torch_f32(xb)
    pos = torch.arange(P, dtype=torch.int32, device="cuda")
    k1, v1 = lay.new_cache(1, 0)
    k2, v2 = lay.new_cache(1, 0)
    y1, y2 = torch.empty_like(x), torch.empty_like(x)
    lay.prefill(x, pos, k1, v1, y1)
    st.prefill(x, pos, 0, [k2], [v2], y2)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2) and torch.equal(k1, k2) and torch.equal(v1, v2)


def test_stack_decode_positions_not_slots():
    """stack_decode at B = 3 (the kernel sequence) and B = 2 (the persistent
    launch) with positions unrelated to the context lengths, each row
    against the chained oracle layers on its own cache."""
    name, nl = "tiny", 2
    cfg = synth.CONFIGS[name]
    hw = [host_layer(name, layer=l)[1] for l in range(nl)]
    W = [oracle_weights(name, layer=l) for l in range(nl)]
    layers = [binding.Layer(cfg, hw[l]) for l in range(nl)]
    st = binding.Stack(layers)
    for B, ctx, pos in ((3, [40, 0, 100], [3, 77, 120]), (2, [64, 5], [0, 127])):
        ctx = np.array(ctx, dtype=np.int32)
        pos = np.array(pos, dtype=np.int32)
        log(f"stack decode B={B} ctx={ctx} pos={pos}")
        fills = [synth.kv_fill(cfg, B, layer=l) for l in range(nl)]
        kcs = [torch.from_numpy(f[0].view(np.int16).copy()).cuda() for f in fills]
        vcs = [torch.from_numpy(f[1].view(np.int16).copy()).cuda() for f in fills]
        xb = synth.activations(cfg, synth.TID_X_DECODE, B)
        x = bits_to_torch_f32(xb)
        y = torch.empty_like(x)
        st.decode(x, torch.from_numpy(pos).cuda(), torch.from_numpy(ctx).cuda(), int(ctx.max()), kcs, vcs, y)
        torch.cuda.synchronize()
        xv = O.bf16_to_f64(xb)
        for l in range(nl):
            kc, vc = O.bf16_to_f64(fills[l][0]), O.bf16_to_f64(fills[l][1])
            xv, ko, vo = O.decode(hw[l], cfg, xv, pos, kc, vc, ctx, W=W[l])
            gk = cache_values(kcs[l])
            assert_parity(np.stack([gk[b][:, ctx[b], :] for b in range(B)]), ko, f"layer {l} new K")
        assert_parity(y.cpu().numpy(), xv, f"stack decode B={B} y")


def test_stack_llama8b_four_layers_rel_frobenius():
    """Four Llama-3-8B-shaped layers with their own seeded weights: prefill
    of 64 tokens, then 3 decode steps through stack_decode, positions
    shifted from the slots.  By causality the oracle runs each layer once
    as a prefill of all 67 tokens (a decode step of a token equals that
    token's row of a prefill over the whole sequence) and hands its output
    to the next layer.  The relative Frobenius error of the last layer's
    output is reported and held to the parity bound (the residual stream
    grows through the layers; the max-abs error is reported)."""
    name, nl, P, D, shift = "llama8b", 4, 64, 3, 100
    cfg = synth.CONFIGS[name]
    hws = [host_layer(name, layer=l)[1] for l in range(nl)]
    layers = [binding.Layer(cfg, hws[l]) for l in range(nl)]
    st = binding.Stack(layers)
    caches = [l.new_cache(1, 0) for l in layers]
    kcs, vcs = [c[0] for c in caches], [c[1] for c in caches]
    xp = synth.activations(cfg, synth.TID_X_PREFILL, P)
    xd = [synth.activations(cfg, synth.TID_X_DECODE + 1000 * s, 1) for s in range(D)]
    x = bits_to_torch_f32(xp)
    y = torch.empty_like(x)
    st.prefill(x, torch.arange(shift, shift + P, dtype=torch.int32, device="cuda"), 0, kcs, vcs, y)
    ys = [y.cpu().numpy()]
    for s in range(D):
        t = P + s
        x1 = bits_to_torch_f32(xd[s])
        y1 = torch.empty_like(x1)
        st.decode(x1, torch.tensor([t + shift], dtype=torch.int32, device="cuda"),
                  torch.tensor([t], dtype=torch.int32, device="cuda"), t, kcs, vcs, y1)
        ys.append(y1.cpu().numpy())
    torch.cuda.synchronize()
    got = np.concatenate(ys, axis=0).astype(np.float64)
    xv = O.bf16_to_f64(np.concatenate([xp] + xd, axis=0))
    pos = np.arange(P + D) + shift
    for l in range(nl):
        W = O.dequant_layer(hws[l], cfg)
        xv = O.prefill(hws[l], cfg, xv, pos, W=W)[0]
        del W
    err = np.abs(got - xv)
    rel = float(np.linalg.norm(got - xv) / np.linalg.norm(xv))
    log(f"  4-layer llama8b stack: rel-fro {rel:.3e}  max-abs {err.max():.3e}  "
        f"(prefill rows {np.linalg.norm(got[:P] - xv[:P]) / np.linalg.norm(xv[:P]):.3e}, "
        f"decode rows {np.linalg.norm(got[P:] - xv[P:]) / np.linalg.norm(xv[P:]):.3e})  |y| max {np.abs(xv).max():.1f}")
    assert np.all(np.isfinite(got))
    assert rel <= 1e-2
    for l in layers:
        l.close()
