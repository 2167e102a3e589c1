"""Streams and graph capture through the C ABI: device calls only enqueue on the caller's stream,
handles may be shared by calls on several streams at once, and the quantizer and the layer (also
split over K with a workspace) can be captured in a HIP graph and replayed, from the very first
call that uses a new plan and codebook (their device tables are set up when the handles are
created).  Every kernel is deterministic, so each result is compared bit for bit with the same
call made eagerly on the default stream."""

import numpy as np
import pytest
import torch

import paper_2607_02461_amd as oq

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _bf16(M, K, seed, scale=1.0):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    return (torch.randn((M, K), generator=g, device=DEV) * scale).to(torch.bfloat16)


def _layer(X, W, plan, cb, bias=None, gelu=False, out_dtype=torch.float32):
    xc, xn = oq.rpbh_quantize_act(plan, cb, X)
    wc, wn = oq.quantize_weights_offline(plan, cb, W)
    Y = oq.orbit_qlinear_ex(cb, xc, xn, cb, wc, wn, bias=bias, gelu=gelu, out_dtype=out_dtype)
    return xc, xn, wc, wn, Y


def test_two_streams_share_handles():
    # two layers on two non-default streams at once, the same plan and codebook handles, against
    # the same calls made one after the other on the default stream
    K = 3072
    plan, cb = oq.rpbh_plan(K, 128, 0), oq.lloydmax_codebook(4, K)
    Xs = [_bf16(4099, K, 1), _bf16(2311, K, 2, scale=3.0)]
    Ws = [_bf16(3072, K, 3, scale=0.02), _bf16(5000, K, 4, scale=0.02)]
    ref = [_layer(X, W, plan, cb) for X, W in zip(Xs, Ws)]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    out = [None, None]
    for i in range(2):
        streams[i].wait_stream(torch.cuda.current_stream())
    for _ in range(3):   # several rounds, so the two streams' kernels overlap
        for i in range(2):
            with torch.cuda.stream(streams[i]):
                out[i] = _layer(Xs[i], Ws[i], plan, cb)
    torch.cuda.synchronize()
    for i in range(2):
        for a, b in zip(out[i], ref[i]):
            assert torch.equal(a, b), f"stream {i}: results differ from the default-stream call"


def test_graph_capture_and_replay():
    # quantize + fused layer (bias, GELU, bf16 output) captured once, replayed on new input
    # contents with eager work between replays; every replay equals the eager result
    K, M, N = 5120, 3000, 4096
    plan, cb = oq.rpbh_plan(K, 128, 0), oq.lloydmax_codebook(4, K)
    W = _bf16(N, K, 9, scale=0.015)
    wc, wn = oq.quantize_weights_offline(plan, cb, W)
    bias = (torch.randn(N, device=DEV) * 0.1).to(torch.bfloat16)
    X = _bf16(M, K, 10)
    xc = torch.empty((M, K // 2), dtype=torch.uint8, device=DEV)
    xn = torch.empty((M,), dtype=torch.float32, device=DEV)
    Y = torch.empty((M, N), dtype=torch.bfloat16, device=DEV)

    def step():
        oq.rpbh_quantize_act(plan, cb, X, 1e-10, xc, xn)
        oq.orbit_qlinear_ex(cb, xc, xn, cb, wc, wn, bias=bias, gelu=True, out_dtype=torch.bfloat16, out=Y)

    step()                       # eager first call
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):   # warm-up on the capture stream, as torch recommends
        step()
    torch.cuda.current_stream().wait_stream(s)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    for r in range(4):
        X.copy_(_bf16(M, K, 100 + r, scale=1.0 + r))
        g.replay()
        torch.cuda.synchronize()
        got = (xc.clone(), xn.clone(), Y.clone())
        _ = _bf16(1024, 1024, 7).float().sum()       # unrelated eager work between replays
        step()                                        # the same step, eagerly
        torch.cuda.synchronize()
        for a, b, name in zip(got, (xc, xn, Y), ("codes", "norms", "Y")):
            assert torch.equal(a, b), f"replay {r}: {name} differ from the eager step"


def test_graph_capture_of_split_layer():
    # c1's layer split over K with a workspace (two kernels, no memset) captured with its
    # quantizer, replayed on new inputs; every replay equals the eager step
    K, M, N = 3072, 256, 3072
    plan, cb = oq.rpbh_plan(K, 128, 0), oq.lloydmax_codebook(4, K)
    W = _bf16(N, K, 19, scale=0.02)
    wc, wn = oq.quantize_weights_offline(plan, cb, W)
    bias = (torch.randn(N, device=DEV) * 0.1).to(torch.bfloat16)
    X = _bf16(M, K, 20)
    xc = torch.empty((M, K // 2), dtype=torch.uint8, device=DEV)
    xn = torch.empty((M,), dtype=torch.float32, device=DEV)
    Y = torch.empty((M, N), dtype=torch.bfloat16, device=DEV)
    n = oq.orbit_qlinear_workspace_size(M, N, K)
    assert n > 0
    ws = torch.empty(n, dtype=torch.uint8, device=DEV)

    def step():
        oq.rpbh_quantize_act(plan, cb, X, 1e-10, xc, xn)
        oq.orbit_qlinear_ws(cb, xc, xn, cb, wc, wn, ws, bias=bias, gelu=True, out_dtype=torch.bfloat16, out=Y)

    step()
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()
    torch.cuda.current_stream().wait_stream(s)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    for r in range(4):
        X.copy_(_bf16(M, K, 200 + r, scale=1.0 + r))
        g.replay()
        torch.cuda.synchronize()
        got = (xc.clone(), xn.clone(), Y.clone())
        ws.fill_(255)                                 # stale workspace between replays
        step()
        torch.cuda.synchronize()
        for a, b, name in zip(got, (xc, xn, Y), ("codes", "norms", "Y")):
            assert torch.equal(a, b), f"replay {r}: {name} differ from the eager step"


def test_split_layers_on_two_streams_with_their_own_workspaces():
    # two small layers split over K run at once on two streams, each with its own workspace,
    # against the same calls one after the other on the default stream
    K = 3072
    plan, cb = oq.rpbh_plan(K, 128, 0), oq.lloydmax_codebook(4, K)
    shapes = [(256, 3072), (64, 2000)]
    ops = []
    for i, (M, N) in enumerate(shapes):
        xc, xn = oq.rpbh_quantize_act(plan, cb, _bf16(M, K, 30 + i))
        wc, wn = oq.quantize_weights_offline(plan, cb, _bf16(N, K, 40 + i, scale=0.02))
        n = oq.orbit_qlinear_workspace_size(M, N, K)
        assert n > 0
        ops.append((xc, xn, wc, wn, torch.empty(n, dtype=torch.uint8, device=DEV)))
    ref = [oq.orbit_qlinear_ws(cb, xc, xn, cb, wc, wn, ws) for xc, xn, wc, wn, ws in ops]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    out = [None, None]
    for _ in range(3):
        for i, (xc, xn, wc, wn, ws) in enumerate(ops):
            with torch.cuda.stream(streams[i]):
                out[i] = oq.orbit_qlinear_ws(cb, xc, xn, cb, wc, wn, ws)
    torch.cuda.synchronize()
    for i in range(2):
        assert torch.equal(out[i], ref[i]), f"stream {i}: results differ from the default-stream call"


def test_first_call_of_new_handles_is_captured():
    # handles created just before the capture, with no eager call of theirs: the weight pass, the
    # quantizer and the layer record only kernel launches, and every replay (with eager work and
    # overwritten outputs between replays) equals the same calls made eagerly afterwards
    K, M, N = 3072, 1000, 2048
    plan = oq.rpbh_plan(K, 128, 11)
    cb_a, cb_w = oq.lloydmax_codebook(4, K), oq.lloydmax_codebook(3, K)
    X, W = _bf16(M, K, 50), _bf16(N, K, 51, scale=0.02)
    wc = torch.empty((N, K * 3 // 8), dtype=torch.uint8, device=DEV)
    wn = torch.empty((N,), dtype=torch.bfloat16, device=DEV)
    xc = torch.empty((M, K // 2), dtype=torch.uint8, device=DEV)
    xn = torch.empty((M,), dtype=torch.float32, device=DEV)
    Y = torch.empty((M, N), dtype=torch.float32, device=DEV)

    def step(outs):
        wc_, wn_, xc_, xn_, Y_ = outs
        oq.quantize_weights_offline(plan, cb_w, W, 1e-10, wc_, wn_)
        oq.rpbh_quantize_act(plan, cb_a, X, 1e-10, xc_, xn_)
        oq.orbit_qlinear(cb_a, xc_, xn_, cb_w, wc_, wn_, out=Y_)

    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step((wc, wn, xc, xn, Y))
    torch.cuda.synchronize()
    replays = []
    for r in range(3):
        for t in (wc, xc):
            t.fill_(0xA5)
        for t in (wn, xn, Y):
            t.fill_(float("nan"))
        _ = _bf16(512, 512, 60 + r).float().sum()     # unrelated eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        replays.append([t.clone() for t in (wc, wn, xc, xn, Y)])
    eager = [torch.empty_like(t) for t in (wc, wn, xc, xn, Y)]
    step(eager)
    torch.cuda.synchronize()
    for r, got in enumerate(replays):
        for a, b, name in zip(got, eager, ("weight codes", "weight norms", "codes", "norms", "Y")):
            assert torch.equal(a, b), f"replay {r}: {name} differ from the eager calls"
