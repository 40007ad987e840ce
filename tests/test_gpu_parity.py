"""Parity of the three stages on the GPU against the CPU oracle, element by
element on the same seeded inputs: y (fp32) and the new cache entries, within
max-abs 2e-2 and relative Frobenius 1e-2.  Sizes run from the tiny layer
(several tiles and ragged tails) to the full Qwen/Llama-shaped layers, where
the oracle evaluates a sample of rows."""
import numpy as np
import pytest
import torch

from oracle import layer as O
from paper_2607_15865_amd import binding, synth
from gpu_helpers import (assert_parity, bits_to_torch_f32, cache_values, device_layer, host_layer, log,
                         oracle_weights, to_cache_bits)

pytestmark = pytest.mark.gpu


def _x(cfg, tid, rows):
    bits = synth.activations(cfg, tid, rows)
    return bits, O.bf16_to_f64(bits)


def _check_new_kv(k, v, ok, ov, start, T, seq=0, rows=None):
    gk = cache_values(k)[seq][:, start:start + T, :].transpose(1, 0, 2)
    gv = cache_values(v)[seq][:, start:start + T, :].transpose(1, 0, 2)
    if rows is not None:
        gk, gv, ok, ov = gk[rows], gv[rows], ok[rows], ov[rows]
    assert_parity(gk, ok, "new K")
    assert_parity(gv, ov, "new V")
    # bf16 rounding of K: a wrong rounding mode (truncation) moves about half
    # of the entries off the oracle's bf16 value; with exact weights and fp32
    # accumulation only entries within about 1e-6 of a rounding boundary may
    # differ.
    flips = np.mean(gk != ok)
    log(f"  new K entries differing from the oracle's bf16 value: {flips:.2e}")
    assert flips < 0.05


PREFILL_CASES = [("tiny", 32, None), ("tiny", 1, None), ("tiny", 77, None), ("qwen05b", 256, None),
                 ("llama8b", 512, None), ("qwen7b", 2048, [0, 1, 2, 3, 7, 31, 32, 127, 128, 129, 511, 1000, 1023,
                                                          1024, 1535, 2000, 2046, 2047])]


@pytest.mark.parametrize("name,T,rows", PREFILL_CASES)
def test_prefill(name, T, rows):
    cfg, w = host_layer(name)
    W = oracle_weights(name)
    lay = device_layer(name)
    log(f"prefill {name} T={T}")
    xb, xv = _x(cfg, synth.TID_X_PREFILL, T)
    pos = np.arange(T)
    k, v = lay.new_cache(1, 0)
    x = bits_to_torch_f32(xb)
    y = torch.empty_like(x)
    lay.prefill(x, torch.from_numpy(pos.astype(np.int32)).cuda(), k, v, y)
    torch.cuda.synchronize()
    yo, ko, vo = O.prefill(w, cfg, xv, pos, rows=rows, W=W)
    gy = y.cpu().numpy().astype(np.float64)
    assert_parity(gy if rows is None else gy[rows], yo, "y")
    _check_new_kv(k, v, ko, vo, 0, T)


PKV_CASES = [("tiny", 16, 32), ("tiny", 5, 100), ("qwen05b", 64, 256), ("llama8b", 128, 1024)]


@pytest.mark.parametrize("name,T,L", PKV_CASES)
def test_prefill_kv(name, T, L):
    """History = the oracle's own prefill of L tokens (bf16 values), given to
    both sides; then a chunk of T new tokens."""
    cfg, w = host_layer(name)
    W = oracle_weights(name)
    lay = device_layer(name)
    log(f"prefill_kv {name} T={T} L={L}")
    xh_bits, xh = _x(cfg, synth.TID_X_PREFILL, L)
    _, kh, vh = O.prefill(w, cfg, xh, np.arange(L), rows=[L - 1], W=W)
    kc = np.zeros((cfg.n_kv_heads, cfg.max_seq, cfg.head_dim))
    kc = O.cache_write(kc, kh, 0)
    vc = O.cache_write(np.zeros_like(kc), vh, 0)
    k = torch.from_numpy(to_cache_bits(kc)[None]).cuda()
    v = torch.from_numpy(to_cache_bits(vc)[None]).cuda()
    xb, xv = _x(cfg, synth.TID_X_PREFILL_KV, T)
    pos = np.arange(L, L + T)
    x = bits_to_torch_f32(xb)
    y = torch.empty_like(x)
    lay.prefill_kv(x, torch.from_numpy(pos.astype(np.int32)).cuda(), L, k, v, y)
    torch.cuda.synchronize()
    yo, ko, vo = O.prefill_kv(w, cfg, xv, pos, kc, vc, L, W=W)
    assert_parity(y.cpu().numpy(), yo, "y")
    _check_new_kv(k, v, ko, vo, L, T)


# Decode path 0 runs T <= 2 as one persistent launch and T <= 8 on the decode
# kernel sequence, the tokens as rows sharing one cache (rows that straddle a
# key-chunk boundary: tiny 4 over 94); path 2 runs T <= 4 as the persistent
# launch; path 1 keeps the prefill kernels.
VERIFY_CASES = [("tiny", 2, 120), ("tiny", 4, 94), ("tiny", 3, 0), ("tiny", 8, 100), ("qwen05b", 3, 1000),
                ("qwen05b", 4, 1019), ("llama8b", 2, 3000), ("llama8b", 4, 4000), ("llama8b", 8, 2048),
                ("qwen7b", 2, 8190), ("qwen7b", 5, 8000)]


@pytest.mark.parametrize("name,T,L", VERIFY_CASES)
def test_prefill_kv_verify(name, T, L):
    """Speculative-decode verification (the extension named as future work in
    Sec. 6): prefill_kv of T = 2..8 draft tokens over a long history, with
    the N(0,1) bf16 cache of the decode workloads as the history."""
    cfg, w = host_layer(name)
    W = oracle_weights(name)
    lay = device_layer(name)
    log(f"prefill_kv verify {name} T={T} L={L}")
    kb, vb = synth.kv_fill(cfg, 1)
    kc, vc = O.bf16_to_f64(kb)[0], O.bf16_to_f64(vb)[0]
    k = torch.from_numpy(kb.view(np.int16).copy()).cuda()
    v = torch.from_numpy(vb.view(np.int16).copy()).cuda()
    xb, xv = _x(cfg, synth.TID_X_PREFILL_KV, T)
    pos = np.arange(L, L + T)
    x = bits_to_torch_f32(xb)
    y = torch.empty_like(x)
    yo, ko, vo = O.prefill_kv(w, cfg, xv, pos, kc, vc, L, W=W)
    for path in ((0, 1, 2) if T <= 4 else (0, 1)):
        lay.set_decode_path(path)
        lay.prefill_kv(x, torch.from_numpy(pos.astype(np.int32)).cuda(), L, k, v, y)
        torch.cuda.synchronize()
        assert_parity(y.cpu().numpy(), yo, f"y (path {path})")
        _check_new_kv(k, v, ko, vo, L, T)
    lay.set_decode_path(0)
    # the history is untouched
    assert np.array_equal(k.cpu().numpy()[0][:, :L, :], kb.view(np.int16)[0][:, :L, :])


CHUNKED_CASES = [("tiny", 100, 32), ("qwen05b", 1000, 256), ("llama8b", 2048, 512)]


@pytest.mark.parametrize("name,T,chunk", CHUNKED_CASES)
def test_prefill_chunked(name, T, chunk):
    """A long prompt in segments (the third scenario of Sec. 4.1): one prefill
    of `chunk` tokens, then prefill_kv chunks over the tokens before them (the
    last one ragged), against the oracle's one-shot prefill of all T tokens."""
    cfg, w = host_layer(name)
    W = oracle_weights(name)
    lay = device_layer(name)
    log(f"prefill_chunked {name} T={T} chunk={chunk}")
    rows = None
    if T > 256:
        rows = sorted({0, 1, chunk - 1, chunk, chunk + 1, 2 * chunk - 1, 2 * chunk, T // 2, T - chunk, T - 2, T - 1})
    xb, xv = _x(cfg, synth.TID_X_PREFILL, T)
    k, v = lay.new_cache(1, 0)
    x = bits_to_torch_f32(xb)
    y = torch.empty_like(x)
    lay.prefill_chunked(x, torch.arange(T, dtype=torch.int32, device="cuda"), chunk, k, v, y)
    torch.cuda.synchronize()
    yo, ko, vo = O.prefill(w, cfg, xv, np.arange(T), rows=rows, W=W)
    gy = y.cpu().numpy().astype(np.float64)
    assert_parity(gy if rows is None else gy[rows], yo, "y")
    _check_new_kv(k, v, ko, vo, 0, T)


def test_prefill_chunked_validation():
    """Argument errors of the segmentation driver are reported before any
    segment is enqueued: the output keeps its contents."""
    cfg, _ = host_layer("tiny")
    lay = device_layer("tiny")
    h = lay.handle
    T, chunk = 40, 16
    n = binding.layer_prefill_chunked_workspace_size(h, T, chunk)
    assert n > 0 and binding.layer_prefill_chunked_workspace_size(h, T, 0) == 0
    x = torch.zeros(T, cfg.hidden, device="cuda")
    y = torch.full_like(x, 7.0)
    pos = torch.arange(T, dtype=torch.int32, device="cuda")
    k, v = lay.new_cache(1, 0)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    assert binding.layer_prefill_chunked(h, x, pos, T, 0, k, v, y, ws, n) == binding.W4_EINVAL
    assert binding.layer_prefill_chunked(h, x, pos, T, chunk, k, v, y, ws, n - 1) == binding.W4_EWORKSPACE
    assert binding.layer_prefill_chunked(h, x, pos, cfg.max_seq + 1, chunk, k, v, y, ws, n) == binding.W4_ECAPACITY
    assert binding.layer_prefill_chunked(h, x, pos, T, chunk, k, v, x, ws, n) == binding.W4_EINVAL
    torch.cuda.synchronize()
    assert bool((y == 7.0).all())


DECODE_CASES = [("tiny", 1, [48], 0), ("tiny", 1, [48], 1), ("tiny", 4, [0, 9, 64, 126], 0),
                ("tiny", 4, [0, 9, 64, 126], 1), ("tiny", 3, [127, 2, 40], 2), ("qwen05b", 1, [512], 0),
                ("qwen05b", 2, [512, 100], 2), ("qwen05b", 2, [512, 100], 1), ("llama8b", 1, [2048], 0), ("llama8b", 1, [2048], 1),
                ("llama8b", 2, [2048, 1500], 2), ("llama8b", 3, [3000, 17, 2048], 2),
                ("llama8b", 4, [2048, 1, 4095, 700], 2), ("qwen7b", 1, [8192], 0), ("qwen7b", 1, [8192], 2),
                ("qwen7b", 2, [8192, 3000], 2),
                ("qwen7b", 8, [8192, 17, 4000, 8191, 1, 2048, 6000, 8100], 0)]


@pytest.mark.parametrize("name,B,ctx,path", DECODE_CASES)
def test_decode(name, B, ctx, path):
    """Decode against an N(0,1) bf16 cache (the synthetic cache of the decode
    workloads); path 0 automatic, 1 separate kernels, 2 persistent launch."""
    cfg, w = host_layer(name)
    W = oracle_weights(name)
    lay = device_layer(name)
    lay.set_decode_path(path)
    log(f"decode {name} B={B} ctx={ctx} path={path}")
    kb, vb = synth.kv_fill(cfg, B)
    kc, vc = O.bf16_to_f64(kb), O.bf16_to_f64(vb)
    ctx = np.array(ctx, dtype=np.int32)
    pos = ctx.copy()
    xb, xv = _x(cfg, synth.TID_X_DECODE, B)
    k = torch.from_numpy(kb.view(np.int16)).cuda()
    v = torch.from_numpy(vb.view(np.int16)).cuda()
    x = bits_to_torch_f32(xb)
    y = torch.empty_like(x)
    ctx_d = torch.from_numpy(ctx).cuda()
    lay.decode(x, torch.from_numpy(pos).cuda(), ctx_d, int(ctx.max()), k, v, y)
    torch.cuda.synchronize()
    yo, ko, vo = O.decode(w, cfg, xv, pos, kc, vc, ctx, W=W)
    assert_parity(y.cpu().numpy(), yo, "y")
    gk, gv = cache_values(k), cache_values(v)
    gkn = np.stack([gk[b][:, ctx[b], :] for b in range(B)])
    gvn = np.stack([gv[b][:, ctx[b], :] for b in range(B)])
    assert_parity(gkn, ko, "new K")
    assert_parity(gvn, vo, "new V")
    lay.set_decode_path(0)


def test_decode_mask():
    """The external decode mask: all-zero equals no mask; -inf at slot j
    removes key j; a row with every visible slot masked gives a zero
    attention output (y = h)."""
    name = "qwen05b"
    cfg, w = host_layer(name)
    W = oracle_weights(name)
    lay = device_layer(name)
    B = 3
    kb, vb = synth.kv_fill(cfg, B)
    kc, vc = O.bf16_to_f64(kb), O.bf16_to_f64(vb)
    ctx = np.array([300, 511, 64], dtype=np.int32)
    xb, xv = _x(cfg, synth.TID_X_DECODE, B)
    mask = np.zeros((B, cfg.max_seq), dtype=np.float32)
    rng = np.random.default_rng(5)
    mask[0, rng.choice(300, 40, replace=False)] = -np.inf
    mask[1, :] = rng.normal(0, 2, cfg.max_seq).astype(np.float32)
    mask[2, :65] = -np.inf
    yo, _, _ = O.decode(w, cfg, xv, ctx, kc, vc, ctx, mask.astype(np.float64), W=W)
    yz, _, _ = O.decode(w, cfg, xv, ctx, kc, vc, ctx, W=W)
    for path in (2, 0):            # the persistent launch, then the automatic choice (kernels for 3 rows)
        lay.set_decode_path(path)
        outs = []
        for m in (None, np.zeros_like(mask), mask):
            k = torch.from_numpy(kb.view(np.int16)).cuda()
            v = torch.from_numpy(vb.view(np.int16)).cuda()
            x = bits_to_torch_f32(xb)
            y = torch.empty_like(x)
            md = None if m is None else torch.from_numpy(m).cuda()
            lay.decode(x, torch.from_numpy(ctx).cuda(), torch.from_numpy(ctx).cuda(), int(ctx.max()), k, v, y, md)
            torch.cuda.synchronize()
            outs.append(y.cpu().numpy())
        if path == 2:
            # the persistent launch is deterministic: a zero mask is bit-identical to none
            assert np.array_equal(outs[0], outs[1])
        assert_parity(outs[1], yz, f"y zero mask (path {path})")
        assert_parity(outs[2], yo, f"y masked (path {path})")
    lay.set_decode_path(0)


@pytest.mark.parametrize("path,B", [(1, 8), (2, 4)])
def test_decode_batch_rows_match_single(path, B):
    """Rows of a batch are independent: each row of a B-row call equals the
    same row run alone on the same path (separate kernels up to B = 8, the
    persistent launch up to B = 4)."""
    name = "tiny"
    cfg, w = host_layer(name)
    lay = device_layer(name)
    lay.set_decode_path(path)
    kb, vb = synth.kv_fill(cfg, B)
    ctx = np.array([3, 100, 50, 127 - 1, 0, 64, 65, 31], dtype=np.int32)[:B]
    xb, _ = _x(cfg, synth.TID_X_DECODE, B)
    x = bits_to_torch_f32(xb)

    def run(sel):
        k = torch.from_numpy(kb[sel].view(np.int16).copy()).cuda()
        v = torch.from_numpy(vb[sel].view(np.int16).copy()).cuda()
        c = torch.from_numpy(ctx[sel].copy()).cuda()
        y = torch.empty((len(sel), cfg.hidden), dtype=torch.float32, device="cuda")
        lay.decode(x[sel].contiguous(), c, c, int(ctx[sel].max()), k, v, y)
        torch.cuda.synchronize()
        return y.cpu().numpy()

    yall = run(list(range(B)))
    for b in range(B):
        yb = run([b])
        assert np.max(np.abs(yb[0] - yall[b])) < 1e-4, b
    lay.set_decode_path(0)


@pytest.mark.parametrize("name,ctx", [("tiny", 100), ("llama8b", 2048)])
def test_decode_persistent_deterministic(name, ctx):
    """The persistent launch forms every sum in a fixed order: repeated calls
    on the same input are bit-identical (a raced or stale partial sum shows
    up here), and both decode paths stay within the oracle tolerance of each
    other.  The two paths may differ by a few bf16 rounding decisions, since
    they add the same fp32 terms in different orders."""
    cfg, w = host_layer(name)
    lay = device_layer(name)
    B = 1
    kb, vb = synth.kv_fill(cfg, B)
    xb, _ = _x(cfg, synth.TID_X_DECODE, B)
    x = bits_to_torch_f32(xb)
    c = torch.full((B,), ctx, dtype=torch.int32, device="cuda")
    outs = []
    for path in (1, 2, 2, 2):
        lay.set_decode_path(path)
        k = torch.from_numpy(kb.view(np.int16).copy()).cuda()
        v = torch.from_numpy(vb.view(np.int16).copy()).cuda()
        y = torch.empty_like(x)
        lay.decode(x, c, c, ctx, k, v, y)
        torch.cuda.synchronize()
        outs.append(y.cpu().numpy())
    lay.set_decode_path(0)
    log(f"  separate vs persistent: max |diff| = {np.max(np.abs(outs[0] - outs[1])):.2e}")
    assert_parity(outs[1].astype(np.float64), outs[0].astype(np.float64), "persistent vs separate")
    assert np.array_equal(outs[1], outs[2]) and np.array_equal(outs[1], outs[3])


def test_chain_prefill_prefill_kv_decode():
    """The paper's runtime order (Sec. 4.5) on the GPU's own caches: prefill 32
    tokens, prefill_kv 16 more, then 16 decode steps, against the oracle
    running the same chain on its own caches."""
    name = "tiny"
    cfg, w = host_layer(name)
    W = oracle_weights(name)
    lay = device_layer(name)
    P, C, D = 32, 16, 16
    k, v = lay.new_cache(1, 0)
    kc = np.zeros((cfg.n_kv_heads, cfg.max_seq, cfg.head_dim))
    vc = np.zeros_like(kc)
    xb, xv = _x(cfg, synth.TID_X_PREFILL, P)
    x = bits_to_torch_f32(xb)
    y = torch.empty_like(x)
    lay.prefill(x, torch.arange(P, dtype=torch.int32, device="cuda"), k, v, y)
    yo, ko, vo = O.prefill(w, cfg, xv, np.arange(P), W=W)
    kc, vc = O.cache_write(kc, ko, 0), O.cache_write(vc, vo, 0)
    assert_parity(y.cpu().numpy(), yo, "prefill y")
    xb, xv = _x(cfg, synth.TID_X_PREFILL_KV, C)
    x = bits_to_torch_f32(xb)
    y = torch.empty_like(x)
    lay.prefill_kv(x, torch.arange(P, P + C, dtype=torch.int32, device="cuda"), P, k, v, y)
    yo, ko, vo = O.prefill_kv(w, cfg, xv, np.arange(P, P + C), kc, vc, P, W=W)
    kc, vc = O.cache_write(kc, ko, P), O.cache_write(vc, vo, P)
    assert_parity(y.cpu().numpy(), yo, "prefill_kv y")
    for s in range(D):
        t = P + C + s
        xb = synth.activations(cfg, synth.TID_X_DECODE + 1000 * s, 1)
        x = bits_to_torch_f32(xb)
        y = torch.empty_like(x)
        td = torch.tensor([t], dtype=torch.int32, device="cuda")
        lay.decode(x, td, td, t, k, v, y)
        yo, ko, vo = O.decode(w, cfg, O.bf16_to_f64(xb), [t], kc[None], vc[None], [t], W=W)
        kc, vc = O.cache_write(kc, ko, t), O.cache_write(vc, vo, t)
        assert_parity(y.cpu().numpy(), yo, f"decode step {s} y")
    torch.cuda.synchronize()
    n = P + C + D
    assert_parity(cache_values(k)[0][:, :n], kc[:, :n], "cache K")
    assert_parity(cache_values(v)[0][:, :n], vc[:, :n], "cache V")


# Position ids feed only RoPE; the cache slot of a token is fixed by the
# history length (Table 1 lists the positions as an input of their own, and
# the cos/sin table is gathered by them, Sec. 4.6.2).  These cases give
# positions that differ from the slots (shifted, permuted, per row unrelated
# to the context), so a kernel that rotated by slot, or wrote the cache at the
# position, fails them.
def _positions(kind, n, lo, hi, seed):
    if kind == "shift":
        return np.arange(lo, lo + n)
    rng = np.random.default_rng(seed)
    return rng.choice(np.arange(lo, hi), n, replace=False)


POS_PREFILL_CASES = [("tiny", 32, "shift", 90), ("tiny", 20, "perm", 0), ("qwen05b", 256, "shift", 700),
                     ("llama8b", 128, "perm", 0)]


@pytest.mark.parametrize("name,T,kind,lo", POS_PREFILL_CASES)
def test_prefill_positions_not_slots(name, T, kind, lo):
    cfg, w = host_layer(name)
    W = oracle_weights(name)
    lay = device_layer(name)
    pos = _positions(kind, T, lo, cfg.max_seq, 11 + T)
    assert not np.array_equal(pos, np.arange(T))
    log(f"prefill {name} T={T} positions {kind} {pos[:4]}...")
    xb, xv = _x(cfg, synth.TID_X_PREFILL, T)
    k, v = lay.new_cache(1, 0)
    x = bits_to_torch_f32(xb)
    y = torch.empty_like(x)
    lay.prefill(x, torch.from_numpy(pos.astype(np.int32)).cuda(), k, v, y)
    torch.cuda.synchronize()
    yo, ko, vo = O.prefill(w, cfg, xv, pos, W=W)
    assert_parity(y.cpu().numpy(), yo, "y")
    _check_new_kv(k, v, ko, vo, 0, T)
    # slots past T are untouched (the cache was zeros)
    assert not k.cpu().numpy()[0][:, T:, :].any() and not v.cpu().numpy()[0][:, T:, :].any()


# prefill_kv on the prefill kernels (T = 16, 128) and on the decode kernels
# (T = 2: persistent launch; 4 with path 2: persistent; 6: kernel sequence)
POS_PKV_CASES = [("tiny", 16, 32, 0), ("tiny", 2, 40, 0), ("tiny", 4, 40, 2), ("tiny", 6, 40, 0),
                 ("llama8b", 128, 1024, 0), ("llama8b", 2, 1500, 0)]


@pytest.mark.parametrize("name,T,L,path", POS_PKV_CASES)
def test_prefill_kv_positions_not_slots(name, T, L, path):
    cfg, w = host_layer(name)
    W = oracle_weights(name)
    lay = device_layer(name)
    lay.set_decode_path(path)
    pos = _positions("perm", T, 0, cfg.max_seq, 5 + T + L)
    log(f"prefill_kv {name} T={T} L={L} path={path} positions {pos}")
    kb, vb = synth.kv_fill(cfg, 1)
    kc, vc = O.bf16_to_f64(kb)[0], O.bf16_to_f64(vb)[0]
    k = torch.from_numpy(kb.view(np.int16).copy()).cuda()
    v = torch.from_numpy(vb.view(np.int16).copy()).cuda()
    xb, xv = _x(cfg, synth.TID_X_PREFILL_KV, T)
    x = bits_to_torch_f32(xb)
    y = torch.empty_like(x)
    lay.prefill_kv(x, torch.from_numpy(pos.astype(np.int32)).cuda(), L, k, v, y)
    torch.cuda.synchronize()
    lay.set_decode_path(0)
    yo, ko, vo = O.prefill_kv(w, cfg, xv, pos, kc, vc, L, W=W)
    assert_parity(y.cpu().numpy(), yo, "y")
    _check_new_kv(k, v, ko, vo, L, T)
    kk = k.cpu().numpy()[0]
    ref = kb.view(np.int16)[0]
    assert np.array_equal(kk[:, :L, :], ref[:, :L, :]) and np.array_equal(kk[:, L + T:, :], ref[:, L + T:, :])


POS_DECODE_CASES = [("tiny", 4, [0, 9, 64, 126], 0), ("tiny", 4, [0, 9, 64, 126], 1), ("tiny", 4, [0, 9, 64, 126], 2),
                    ("tiny", 1, [48], 0), ("llama8b", 1, [2048], 0), ("llama8b", 2, [2048, 300], 0),
                    ("llama8b", 4, [2048, 1, 4000, 700], 1), ("qwen7b", 2, [8192, 3000], 2)]


@pytest.mark.parametrize("name,B,ctx,path", POS_DECODE_CASES)
def test_decode_positions_not_slots(name, B, ctx, path):
    """Decode rows whose positions are unrelated to their context lengths:
    each row writes slot ctx[b] and attends slots 0..ctx[b], rotated by
    pos[b]."""
    cfg, w = host_layer(name)
    W = oracle_weights(name)
    lay = device_layer(name)
    lay.set_decode_path(path)
    ctx = np.array(ctx, dtype=np.int32)
    rng = np.random.default_rng(B * 7 + int(ctx.sum()))
    pos = rng.integers(0, cfg.max_seq, B).astype(np.int32)
    pos = np.where(pos == ctx, (pos + 1) % cfg.max_seq, pos).astype(np.int32)
    log(f"decode {name} B={B} ctx={ctx} pos={pos} path={path}")
    kb, vb = synth.kv_fill(cfg, B)
    kc, vc = O.bf16_to_f64(kb), O.bf16_to_f64(vb)
    xb, xv = _x(cfg, synth.TID_X_DECODE, B)
    k = torch.from_numpy(kb.view(np.int16).copy()).cuda()
    v = torch.from_numpy(vb.view(np.int16).copy()).cuda()
    x = bits_to_torch_f32(xb)
    y = torch.empty_like(x)
    lay.decode(x, torch.from_numpy(pos).cuda(), torch.from_numpy(ctx).cuda(), int(ctx.max()), k, v, y)
    torch.cuda.synchronize()
    lay.set_decode_path(0)
    yo, ko, vo = O.decode(w, cfg, xv, pos, kc, vc, ctx, W=W)
    assert_parity(y.cpu().numpy(), yo, "y")
    gk, gv = cache_values(k), cache_values(v)
    assert_parity(np.stack([gk[b][:, ctx[b], :] for b in range(B)]), ko, "new K")
    assert_parity(np.stack([gv[b][:, ctx[b], :] for b in range(B)]), vo, "new V")
    # only slot ctx[b] of each row changed
    kk = k.cpu().numpy()
    for b in range(B):
        diff = np.argwhere((kk[b] != kb.view(np.int16)[b]).any(axis=(0, 2))).ravel()
        assert set(diff.tolist()) <= {int(ctx[b])}, (b, diff[:8])
