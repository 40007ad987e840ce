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
