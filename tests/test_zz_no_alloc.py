"""layer_decode_noalloc (decode on the library's static scratch array, for
callers that cannot allocate) against layer_decode on a caller workspace:
two calls in a row on one device, the second with a smaller input, each on
its own inputs and caches.  y to the parity bar of the oracle comparisons
(the kernel sequence adds k-split partials in a timing-dependent order), the
new cache entries bit for bit, and a call whose scratch need exceeds the
array is refused before any launch."""
import numpy as np
import pytest
import torch

from paper_2607_15865_amd import binding, synth
from gpu_helpers import assert_parity, bits_to_torch_f32, device_layer, host_layer, log

pytestmark = pytest.mark.gpu


def _inputs(cfg, B, ctx, seed):
    kb, vb = synth.kv_fill(cfg, B)
    xb = synth.activations(cfg, synth.TID_X_DECODE + 1000 * seed, B)
    rng = np.random.default_rng(seed)
    pos = rng.integers(0, cfg.max_seq, B).astype(np.int32)
    return kb, vb, xb, np.array(ctx, dtype=np.int32), pos


def _run(lay, cfg, kb, vb, xb, ctx, pos, noalloc):
    B = len(ctx)
    k = torch.from_numpy(kb.view(np.int16).copy()).cuda()
    v = torch.from_numpy(vb.view(np.int16).copy()).cuda()
    x = bits_to_torch_f32(xb)
    y = torch.full_like(x, float("nan"))
    c, p = torch.from_numpy(ctx).cuda(), torch.from_numpy(pos).cuda()
    if noalloc:
        binding.check(binding.layer_decode_noalloc(lay.handle, x, p, c, int(ctx.max()), None, B, k, v, y))
    else:
        lay.decode(x, p, c, int(ctx.max()), k, v, y)
    torch.cuda.synchronize()
    return y.cpu().numpy(), k.cpu().numpy(), v.cpu().numpy()


@pytest.mark.parametrize("name,first,second", [
    ("tiny", [100, 3, 127, 64, 0], [50]),                      # kernel sequence, then the persistent launch
    ("llama8b", [2048, 17, 4000], [2048]),
    ("qwen7b", [8192, 300, 5000, 8191, 1, 2, 3, 4], [7000, 10]),
])
def test_noalloc_matches_workspace_decode(name, first, second):
    cfg, _ = host_layer(name)
    lay = device_layer(name)
    assert binding.layer_decode_noalloc_max_bytes() == 32 << 20
    for i, ctx in enumerate((first, second)):
        kb, vb, xb, c, p = _inputs(cfg, len(ctx), ctx, 7 + i)
        log(f"noalloc {name} call {i}: B={len(ctx)} ctx={c} pos={p}")
        ya, ka, va = _run(lay, cfg, kb, vb, xb, c, p, noalloc=True)
        yb, kb2, vb2 = _run(lay, cfg, kb, vb, xb, c, p, noalloc=False)
        assert_parity(ya, yb, f"call {i} y (noalloc vs workspace)")
        assert np.array_equal(ka, kb2) and np.array_equal(va, vb2)


def test_noalloc_refuses_beyond_the_array():
    """A decode whose scratch need exceeds the static array: W4_EWORKSPACE
    before any launch (the output keeps its contents)."""
    cfg = synth.replace(synth.CONFIGS["tiny"], max_seq=320000)
    _, w = host_layer("tiny")
    lay = binding.Layer(cfg, w)
    B, ctx = 8, 319999
    assert binding.layer_workspace_size(lay.handle, 2, B, 1, ctx) > binding.layer_decode_noalloc_max_bytes()
    x = torch.zeros(B, cfg.hidden, device="cuda")
    y = torch.full_like(x, 4.0)
    c = torch.full((B,), ctx, dtype=torch.int32, device="cuda")
    kc = torch.zeros(16, dtype=torch.int16, device="cuda")
    rc = binding.layer_decode_noalloc(lay.handle, x, c, c, ctx, None, B, kc, kc, y)
    assert rc == binding.W4_EWORKSPACE, rc
    assert "scratch" in binding.layer_last_error()
    torch.cuda.synchronize()
    assert bool((y == 4.0).all())
    lay.close()
