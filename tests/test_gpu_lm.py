"""The model ends on the GPU (embedding, LM head, greedy sampling; the
runtime loop of Sec. 2 / Sec. 4.5) against the oracle: the embedding
bit-exact, the logits to the parity bound, the greedy pick exactly the
argmax of the GPU's own logits and, against the oracle's logits, within the
parity bound of the largest one (near-ties may pick either).  A greedy loop
over a small two-layer model closes the cycle embed -> layers -> head ->
pick -> embed on the device, checked step by step against the oracle fed
the same tokens."""
import functools

import numpy as np
import pytest
import torch

from oracle import layer as O
from oracle import lm as M
from paper_2607_15865_amd import binding, synth
from gpu_helpers import MAX_ABS, assert_parity, host_layer, log, oracle_weights

pytestmark = pytest.mark.gpu


@functools.lru_cache(maxsize=2)
def host_lm(name, vocab, group=None, with_zeros=False, words=False):
    cfg = synth.CONFIGS[name]
    if group:
        cfg = synth.replace(cfg, group_size=group)
    return cfg, synth.make_lm(cfg, vocab, with_zeros=with_zeros, words=words)


def sub_head(head, cols):
    z = head.get("zeros")
    return dict(K=head["K"], N=len(cols), qweight=np.ascontiguousarray(head["qweight"][:, cols]),
                scales=np.ascontiguousarray(head["scales"][:, cols]),
                zeros=None if z is None else np.ascontiguousarray(z[:, cols]))


def check_pick(gl, ol, tok, what):
    """gl: GPU logits [V] (fp32), ol: oracle logits at the same columns."""
    assert tok == int(np.argmax(gl)), f"{what}: pick {tok} is not the argmax of the GPU logits"
    assert ol[tok] >= ol.max() - 2 * MAX_ABS, f"{what}: oracle logit {ol[tok]} vs max {ol.max()}"


def test_embed_bitexact_and_out_of_range():
    cfg, lw = host_lm("tiny", 1024)
    lmh = binding.LM(cfg, lw, max_batch=16)
    tok = np.array([0, 1023, 5, 5, 777, 300, 2, 1000, 64, 17, 512], dtype=np.int32)
    t = torch.from_numpy(tok).cuda()
    x = torch.full((len(tok), cfg.hidden), 7.0, device="cuda")
    lmh.embed(t, x)
    assert np.array_equal(x.cpu().numpy().astype(np.float64), M.embed(lw["embed"], tok))
    assert lmh.error() == 0
    bad = torch.tensor([3, -1, 1024], dtype=torch.int32, device="cuda")
    xb = torch.full((3, cfg.hidden), 7.0, device="cuda")
    lmh.embed(bad, xb)
    xbh = xb.cpu().numpy()
    assert np.array_equal(xbh[0], M.embed(lw["embed"], [3])[0]) and not xbh[1:].any()
    assert lmh.error() == binding.W4_FLAG_TOKEN_ID and lmh.error() == 0
    lmh.close()


HEAD_CASES = [
    # name, vocab, group, zeros, B: one argmax block, two with a ragged tail,
    # groups of 32, zero points, more rows than one GEMV launch takes
    ("tiny", 1024, None, False, 1),
    ("tiny", 8384, None, False, 3),
    ("tiny", 2048, 32, False, 2),
    ("tiny", 2048, None, True, 2),
    ("tiny", 1024, None, False, 11),
]


@pytest.mark.parametrize("name,vocab,group,zeros,B", HEAD_CASES)
def test_head_parity(name, vocab, group, zeros, B):
    log(f"lm head {name} vocab {vocab} group {group} zeros {zeros} B {B}")
    cfg, lw = host_lm(name, vocab, group, zeros)
    lmh = binding.LM(cfg, lw, max_batch=16)
    rng = np.random.default_rng(vocab + B)
    x = (rng.standard_normal((B, cfg.hidden)) * 1.5).astype(np.float32)
    logits = torch.empty(B, vocab, device="cuda")
    nxt = torch.full((B,), -1, dtype=torch.int32, device="cuda")
    lmh.head(torch.from_numpy(x).cuda(), logits, nxt)
    gl = logits.cpu().numpy()
    ol = M.lm_logits(x, lw["final_norm"], lw["head"], cfg.group_size, cfg.rms_eps)
    assert_parity(gl, ol, "logits")
    picks = nxt.cpu().numpy()
    for b in range(B):
        check_pick(gl[b], ol[b], int(picks[b]), f"row {b}")
    # logits only
    logits2 = torch.empty_like(logits)
    lmh.head(torch.from_numpy(x).cuda(), logits2, None)
    assert torch.equal(logits, logits2)
    lmh.close()


def test_head_ties_pick_lowest_index():
    """Exact ties (every weight 0.5 or 1.0 times a normalised row of ones,
    so every logit is an exact sum): all columns equal pick token 0; equal
    maxima inside one argmax block, then in two blocks, pick the lowest."""
    cfg = synth.CONFIGS["tiny"]
    V, H, G = 16384, cfg.hidden, cfg.group_size
    x = torch.ones(1, H, device="cuda")
    logits = torch.empty(1, V, device="cuda")
    nxt = torch.empty(1, dtype=torch.int32, device="cuda")

    def pick(big):
        q = np.full((H, V), 9, dtype=np.uint8)            # weight 0.5
        q[:, big] = 10                                    # weight 1.0
        head = dict(K=H, N=V, qweight=synth.pack_int4(q),
                    scales=np.full((H // G, V), 0.5, dtype=np.float16), zeros=None)
        lw = dict(vocab=V, embed=np.zeros((V, H), dtype=np.uint16),
                  final_norm=np.full(H, 0x3F80, dtype=np.uint16), head=head)
        lmh = binding.LM(cfg, lw)
        lmh.head(x, logits, nxt)
        lmh.close()
        return int(nxt.item())

    assert pick([]) == 0
    assert pick([12000, 9000]) == 9000
    assert pick([12000, 9000, 5000]) == 5000
    assert pick([V - 1]) == V - 1


@pytest.mark.parametrize("name,V,B", [("llama8b", 128256, 2), ("qwen7b", 152064, 3)])
def test_head_full_size_sampled(name, V, B):
    """Full-size ends (Llama-3-8B: hidden 4096, vocab 128256; Qwen2.5-7B:
    hidden 3584, vocab 152064): logits of 512 sampled columns plus the
    GPU's 16 best and both ends of the vocabulary against the oracle on
    those columns; the pick exactly the argmax of the GPU logits."""
    cfg, lw = host_lm(name, V, words=True)
    log(f"lm head {name} vocab {V} B {B}")
    lmh = binding.LM(cfg, lw)
    rng = np.random.default_rng(3)
    x = (rng.standard_normal((B, cfg.hidden)) * 2.0).astype(np.float32)
    logits = torch.empty(B, V, device="cuda")
    nxt = torch.empty(B, dtype=torch.int32, device="cuda")
    lmh.head(torch.from_numpy(x).cuda(), logits, nxt)
    gl = logits.cpu().numpy()
    picks = nxt.cpu().numpy()
    for b in range(B):
        cols = np.unique(np.concatenate([rng.choice(V, 512, replace=False), np.argsort(-gl[b])[:16],
                                         [0, V - 1]]))
        ol = M.lm_logits(x[b:b + 1], lw["final_norm"], sub_head(lw["head"], cols), cfg.group_size,
                         cfg.rms_eps)[0]
        assert_parity(gl[b, cols], ol, f"row {b} sampled logits")
        assert int(picks[b]) == int(np.argmax(gl[b]))
        j = int(np.searchsorted(cols, picks[b]))
        assert ol[j] >= ol.max() - 2 * MAX_ABS
    lmh.close()


def test_greedy_loop_two_layers():
    """embed -> 2-layer stack -> head -> pick -> embed, 8 prompt tokens and 6
    generated ones, all on the device; the oracle runs the same token
    sequence through its layers (decode == prefill over the whole sequence
    by causality) and its head."""
    name, nl, V, T, D = "tiny", 2, 1024, 8, 6
    cfg = synth.CONFIGS[name]
    _, lw = host_lm(name, V)
    hw = [host_layer(name, layer=l)[1] for l in range(nl)]
    W = [oracle_weights(name, layer=l) for l in range(nl)]
    layers = [binding.Layer(cfg, hw[l]) for l in range(nl)]
    st = binding.Stack(layers)
    caches = [l.new_cache(1, 0) for l in layers]
    kcs, vcs = [c[0] for c in caches], [c[1] for c in caches]
    lmh = binding.LM(cfg, lw)
    H = cfg.hidden
    prompt = synth.tokens(cfg, V, T)
    x = torch.empty(T, H, device="cuda")
    lmh.embed(torch.from_numpy(prompt).cuda(), x)
    y = torch.empty_like(x)
    st.prefill(x, torch.arange(T, dtype=torch.int32, device="cuda"), 0, kcs, vcs, y)
    logits = torch.empty(1, V, device="cuda")
    nxt = torch.empty(1, dtype=torch.int32, device="cuda")
    lmh.head(y[T - 1:T], logits, nxt)
    g_logits, g_tok = [logits.cpu().numpy()[0]], [int(nxt.item())]
    x1 = torch.empty(1, H, device="cuda")
    y1 = torch.empty_like(x1)
    for s in range(D):
        t = T + s
        lmh.embed(nxt, x1)
        td = torch.tensor([t], dtype=torch.int32, device="cuda")
        st.decode(x1, td, td, t, kcs, vcs, y1)
        lmh.head(y1, logits, nxt)
        g_logits.append(logits.cpu().numpy()[0])
        g_tok.append(int(nxt.item()))
    log(f"  generated {g_tok}")
    seq = np.concatenate([prompt, np.array(g_tok[:D], dtype=np.int32)])
    xv = M.embed(lw["embed"], seq)
    for l in range(nl):
        xv = O.prefill(hw[l], cfg, xv, np.arange(len(seq)), W=W[l])[0]
    ol = M.lm_logits(xv[T - 1:], lw["final_norm"], lw["head"], cfg.group_size, cfg.rms_eps)
    for i in range(D + 1):
        assert_parity(g_logits[i], ol[i], f"step {i} logits")
        check_pick(g_logits[i], ol[i], g_tok[i], f"step {i}")
    lmh.close()
    for l in layers:
        l.close()


def test_greedy_loop_batch_of_two():
    """Two sequences decoded together: one prefill per prompt into its own
    cache row, then 4 steps of embed -> 2-layer stack decode at B = 2 ->
    head + pick for both rows at once; each sequence against the oracle fed
    its own tokens."""
    name, nl, V, T, D, B = "tiny", 2, 1024, 6, 4, 2
    cfg = synth.CONFIGS[name]
    _, lw = host_lm(name, V)
    hw = [host_layer(name, layer=l)[1] for l in range(nl)]
    W = [oracle_weights(name, layer=l) for l in range(nl)]
    layers = [binding.Layer(cfg, hw[l]) for l in range(nl)]
    st = binding.Stack(layers)
    caches = [l.new_cache(B, 0) for l in layers]
    lmh = binding.LM(cfg, lw)
    H = cfg.hidden
    prompts = [synth.tokens(cfg, V, T, seed=10 + b) for b in range(B)]
    nxt = torch.empty(B, dtype=torch.int32, device="cuda")
    logits = torch.empty(B, V, device="cuda")
    y_last = torch.empty(B, H, device="cuda")
    for b in range(B):   # each prompt into cache row b (a one-sequence view of that row)
        kcs = [c[0][b:b + 1] for c in caches]
        vcs = [c[1][b:b + 1] for c in caches]
        x = torch.empty(T, H, device="cuda")
        lmh.embed(torch.from_numpy(prompts[b]).cuda(), x)
        y = torch.empty_like(x)
        st.prefill(x, torch.arange(T, dtype=torch.int32, device="cuda"), 0, kcs, vcs, y)
        y_last[b] = y[T - 1]
    lmh.head(y_last, logits, nxt)
    g_logits, g_tok = [logits.cpu().numpy()], [nxt.cpu().numpy().copy()]
    kcs, vcs = [c[0] for c in caches], [c[1] for c in caches]
    x1 = torch.empty(B, H, device="cuda")
    y1 = torch.empty_like(x1)
    for s in range(D):
        t = T + s
        lmh.embed(nxt, x1)
        td = torch.full((B,), t, dtype=torch.int32, device="cuda")
        st.decode(x1, td, td, t, kcs, vcs, y1)
        lmh.head(y1, logits, nxt)
        g_logits.append(logits.cpu().numpy())
        g_tok.append(nxt.cpu().numpy().copy())
    for b in range(B):
        toks = [int(g[b]) for g in g_tok]
        log(f"  sequence {b}: generated {toks}")
        seq = np.concatenate([prompts[b], np.array(toks[:D], dtype=np.int32)])
        xv = M.embed(lw["embed"], seq)
        for l in range(nl):
            xv = O.prefill(hw[l], cfg, xv, np.arange(len(seq)), W=W[l])[0]
        ol = M.lm_logits(xv[T - 1:], lw["final_norm"], lw["head"], cfg.group_size, cfg.rms_eps)
        for i in range(D + 1):
            assert_parity(g_logits[i][b], ol[i], f"seq {b} step {i} logits")
            check_pick(g_logits[i][b], ol[i], toks[i], f"seq {b} step {i}")
    lmh.close()
    for l in layers:
        l.close()


def test_lm_argument_errors_launch_nothing():
    """Capacity, workspace and null-pointer errors are reported before any
    launch: the output buffers keep their contents."""
    cfg, lw = host_lm("tiny", 1024)
    lmh = binding.LM(cfg, lw, max_batch=2)
    h = lmh.handle
    x = torch.ones(3, cfg.hidden, device="cuda")
    logits = torch.full((3, 1024), 5.0, device="cuda")
    nxt = torch.full((3,), -7, dtype=torch.int32, device="cuda")
    need = binding.lm_head_workspace_size(h, 2)
    assert need > 0 and binding.lm_head_workspace_size(h, 3) == 0 and binding.lm_head_workspace_size(h, 0) == 0
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    assert binding.lm_head(h, x, 3, logits, nxt, ws, need) == binding.W4_ECAPACITY
    assert binding.lm_head(h, x, 2, logits, nxt, ws, need - 1) == binding.W4_EWORKSPACE
    assert binding.lm_head(h, x, 2, logits, nxt, None, 0) == binding.W4_EWORKSPACE
    assert binding.lm_head(h, x, 0, logits, nxt, ws, need) == binding.W4_EINVAL
    assert binding.lm_head(h, None, 2, logits, nxt, ws, need) == binding.W4_EINVAL
    assert binding.lm_embed(h, nxt, 0, x) == binding.W4_EINVAL
    assert binding.lm_embed(h, None, 1, x) == binding.W4_EINVAL
    torch.cuda.synchronize()
    assert bool((logits == 5.0).all()) and bool((nxt == -7).all())
    assert binding.lm_head(h, x, 2, logits, nxt, ws, need) == binding.W4_OK
    torch.cuda.synchronize()
    assert bool((nxt[:2] >= 0).all()) and int(nxt[2]) == -7
    lmh.close()


def test_model_decode_greedy_matches_composed_calls():
    """The native loop step (embed -> stack decode -> head + pick in one
    call, the picks fed back in place) gives bit for bit the logits and
    tokens of the same calls made one by one, which the two-layer loop test
    holds against the oracle."""
    name, nl, V, T, D = "tiny", 2, 1024, 8, 5
    cfg = synth.CONFIGS[name]
    _, lw = host_lm(name, V)
    hw = [host_layer(name, layer=l)[1] for l in range(nl)]
    layers = [binding.Layer(cfg, hw[l]) for l in range(nl)]
    st = binding.Stack(layers)
    lmh = binding.LM(cfg, lw)
    handles = [l.handle for l in layers]
    prompt = torch.from_numpy(synth.tokens(cfg, V, T)).cuda()
    runs = []
    for native in (False, True):
        caches = [l.new_cache(1, 0) for l in layers]
        kcs, vcs = [c[0] for c in caches], [c[1] for c in caches]
        x = torch.empty(T, cfg.hidden, device="cuda")
        y = torch.empty_like(x)
        lmh.embed(prompt, x)
        st.prefill(x, torch.arange(T, dtype=torch.int32, device="cuda"), 0, kcs, vcs, y)
        logits = torch.empty(1, V, device="cuda")
        tok = torch.empty(1, dtype=torch.int32, device="cuda")
        lmh.head(y[T - 1:T], logits, tok)
        outs = []
        max_ctx = T + D
        n = binding.model_decode_workspace_size(handles, lmh.handle, 1, max_ctx)
        assert n > 0
        ws = torch.empty(n, dtype=torch.uint8, device="cuda")
        x1, y1 = torch.empty(1, cfg.hidden, device="cuda"), torch.empty(1, cfg.hidden, device="cuda")
        for s in range(D):
            td = torch.tensor([T + s], dtype=torch.int32, device="cuda")
            if native:
                binding.check(binding.model_decode_greedy(handles, lmh.handle, tok, td, td, max_ctx, 1, kcs, vcs,
                                                          logits, tok, ws, n))
            else:
                lmh.embed(tok, x1)
                st.decode(x1, td, td, max_ctx, kcs, vcs, y1)
                lmh.head(y1, logits, tok)
            outs.append((logits.cpu().numpy().copy(), int(tok.item())))
        runs.append(outs)
    for s in range(D):
        assert runs[0][s][1] == runs[1][s][1], f"step {s} tokens differ"
        assert np.array_equal(runs[0][s][0], runs[1][s][0]), f"step {s} logits differ"
    # argument checks happen before any launch
    assert binding.model_decode_workspace_size(handles, lmh.handle, 1, cfg.max_seq) == 0
    assert binding.model_decode_greedy(handles, lmh.handle, tok, td, td, cfg.max_seq, 1, kcs, vcs, logits, tok, ws,
                                       n) == binding.W4_ECAPACITY
    assert binding.model_decode_greedy(handles, lmh.handle, tok, td, td, T + D, 1, kcs, vcs, logits, tok, ws,
                                       n - 1) == binding.W4_EWORKSPACE
    assert binding.model_decode_greedy(handles, None, tok, td, td, T + D, 1, kcs, vcs, logits, tok, ws,
                                       n) == binding.W4_EINVAL
    lmh.close()
    for l in layers:
        l.close()


def test_model_decode_greedy_batch_positions_not_slots():
    """The native loop step at B = 4 (the layers' kernel-sequence decode,
    a head launch over four rows), each sequence at its own context with
    a position unrelated to it: every row's logits against the oracle
    layers decoding that row on its own cache, and its pick."""
    name, nl, V, B = "tiny", 2, 1024, 4
    cfg = synth.CONFIGS[name]
    _, lw = host_lm(name, V)
    hw = [host_layer(name, layer=l)[1] for l in range(nl)]
    W = [oracle_weights(name, layer=l) for l in range(nl)]
    layers = [binding.Layer(cfg, hw[l]) for l in range(nl)]
    lmh = binding.LM(cfg, lw)
    handles = [l.handle for l in layers]
    ctx = np.array([17, 0, 90, 55], dtype=np.int32)
    pos = np.array([100, 31, 2, 127], dtype=np.int32)
    fills = [synth.kv_fill(cfg, B, layer=l) for l in range(nl)]
    kcs = [torch.from_numpy(f[0].view(np.int16).copy()).cuda() for f in fills]
    vcs = [torch.from_numpy(f[1].view(np.int16).copy()).cuda() for f in fills]
    toks = synth.tokens(cfg, V, B, seed=99)
    tok = torch.from_numpy(toks.copy()).cuda()
    logits = torch.empty(B, V, device="cuda")
    max_ctx = int(ctx.max())
    n = binding.model_decode_workspace_size(handles, lmh.handle, B, max_ctx)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    binding.check(binding.model_decode_greedy(handles, lmh.handle, tok, torch.from_numpy(pos).cuda(),
                                              torch.from_numpy(ctx).cuda(), max_ctx, B, kcs, vcs, logits, tok,
                                              ws, n))
    gl, picks = logits.cpu().numpy(), tok.cpu().numpy()
    xv = M.embed(lw["embed"], toks)
    for l in range(nl):
        xv = O.decode(hw[l], cfg, xv, pos, O.bf16_to_f64(fills[l][0]), O.bf16_to_f64(fills[l][1]), ctx, W=W[l])[0]
    ol = M.lm_logits(xv, lw["final_norm"], lw["head"], cfg.group_size, cfg.rms_eps)
    for b in range(B):
        assert_parity(gl[b], ol[b], f"row {b} logits")
        check_pick(gl[b], ol[b], int(picks[b]), f"row {b}")
    lmh.close()
    for l in layers:
        l.close()


def test_model_decode_greedy_rejects_before_launch():
    """Rejected steps leave logits and tokens as they were: a batch above 8
    (W4_EUNSUPPORTED), a forced persistent path that cannot serve the batch,
    a context beyond max_seq, a short workspace."""
    name, nl, V = "tiny", 2, 1024
    cfg = synth.replace(synth.CONFIGS[name], max_batch=16)
    _, lw = host_lm(name, V)
    hw = [host_layer(name, layer=l)[1] for l in range(nl)]
    layers = [binding.Layer(cfg, hw[l]) for l in range(nl)]
    lmh = binding.LM(cfg, lw, max_batch=16)
    handles = [l.handle for l in layers]
    B = 9
    kcs = [l.new_cache(B, 0)[0] for l in layers]
    vcs = [l.new_cache(B, 0)[1] for l in layers]
    tok = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    logits = torch.full((B, V), 5.0, device="cuda")
    td = torch.full((B,), 3, dtype=torch.int32, device="cuda")
    ws = torch.empty(1 << 24, dtype=torch.uint8, device="cuda")
    assert binding.model_decode_workspace_size(handles, lmh.handle, B, 3) == 0
    assert binding.model_decode_greedy(handles, lmh.handle, tok, td, td, 3, B, kcs, vcs, logits, tok, ws,
                                       ws.numel()) == binding.W4_EUNSUPPORTED
    layers[1].set_decode_path(2)       # the persistent launch takes at most 4 rows
    assert binding.model_decode_workspace_size(handles, lmh.handle, 5, 3) == 0
    assert binding.model_decode_greedy(handles, lmh.handle, tok, td, td, 3, 5, kcs, vcs, logits, tok, ws,
                                       ws.numel()) == binding.W4_EUNSUPPORTED
    layers[1].set_decode_path(0)
    assert binding.model_decode_greedy(handles, lmh.handle, tok, td, td, cfg.max_seq, 2, kcs, vcs, logits, tok, ws,
                                       ws.numel()) == binding.W4_ECAPACITY
    need = binding.model_decode_workspace_size(handles, lmh.handle, 2, 3)
    assert need > 0
    assert binding.model_decode_greedy(handles, lmh.handle, tok, td, td, 3, 2, kcs, vcs, logits, tok, ws,
                                       need - 1) == binding.W4_EWORKSPACE
    # stack_decode checks every layer before the first one runs
    x = torch.zeros(5, cfg.hidden, device="cuda")
    y = torch.full_like(x, 3.0)
    layers[1].set_decode_path(2)
    assert binding.stack_decode(handles, x, td, td, 3, None, 5, kcs, vcs, y, ws, ws.numel()) == binding.W4_EUNSUPPORTED
    layers[1].set_decode_path(0)
    torch.cuda.synchronize()
    assert bool((logits == 5.0).all()) and bool((tok == -7).all()) and bool((y == 3.0).all())
    assert not kcs[0].any() and not vcs[0].any()
    lmh.close()
    for l in layers:
        l.close()
