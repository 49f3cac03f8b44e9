"""The layer captured in a HIP graph: the library enqueues only kernels on the caller's stream
(no allocation, memset or synchronisation), so a captured call replays.  Each replay, with
new inputs copied into the captured buffers and eager work in between, must equal an eager
call on the same inputs bit for bit (the kernels are deterministic)."""
import pytest
import torch

import workloads as W
from helpers import DEV, say

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.view(torch.int16).clone()


def test_moe_forward_graph_replays_match_eager():
    from paper_2602_07265_amd import xshare as X
    T, N, k, d, f, M = 24, 32, 4, 128, 256, 10
    cfg = dict(N=N, k=k, d=d, f=f, T=T, logits="domains", Q=3)
    w1, w3, w2 = W.expert_weights(N, d, f, 0, DEV)
    inputs = [(W.activations(T, d, s, DEV), torch.from_numpy(W.make_logits(cfg, s)[0]).to(DEV))
              for s in range(4)]
    p = X.params(N, k, 1, M)
    ws = torch.empty(X.moe_workspace_bytes(T, d, f, p), dtype=torch.uint8, device=DEV)
    x_s = inputs[0][0].clone()
    h_s = inputs[0][1].clone()
    y_s = torch.empty((T, d), dtype=torch.bfloat16, device=DEV)
    say("graph case moe_forward: capture")
    X.moe_forward(x_s, h_s, w1, w3, w2, k, 1, M, y=y_s, workspace=ws, routing_out=False)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        X.moe_forward(x_s, h_s, w1, w3, w2, k, 1, M, y=y_s, workspace=ws, routing_out=False)
    torch.cuda.synchronize()
    ws_eager = torch.empty_like(ws)
    for rep in range(3):
        for s, (x, h) in enumerate(inputs):
            say(f"graph case moe_forward: replay {rep} input {s}")
            x_s.copy_(x)
            h_s.copy_(h)
            g.replay()
            torch.cuda.synchronize()
            got = _bits(y_s)
            ref = X.moe_forward(x, h, w1, w3, w2, k, 1, M, workspace=ws_eager,
                                routing_out=False)["y"]
            torch.cuda.synchronize()
            assert torch.equal(got, _bits(ref)), f"replay {rep}, input {s}"


def test_moe_layer_graph_replays_match_eager():
    from paper_2602_07265_amd import xshare as X
    T, N, k, d, f, M = 16, 32, 4, 128, 256, 8
    w1, w3, w2 = W.expert_weights(N, d, f, 1, DEV)
    wg = W.router_weights(N, d, 1, DEV)
    sh = W.shared_weights(1, d, f, 1, DEV)
    xs = [W.activations_domains(T, d, 3, s, DEV) for s in range(3)]
    p = X.params(N, k, 1, M)
    ws = torch.empty(X.layer_workspace_bytes(T, d, f, p, None, X._shared(sh, d, f, DEV)),
                     dtype=torch.uint8, device=DEV)
    x_s = xs[0].clone()
    y_s = torch.empty((T, d), dtype=torch.bfloat16, device=DEV)
    say("graph case moe_layer: capture")
    X.moe_layer(x_s, wg, w1, w3, w2, k, 1, M, shared=sh, y=y_s, workspace=ws,
                routing_out=False, logits_out=False)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        X.moe_layer(x_s, wg, w1, w3, w2, k, 1, M, shared=sh, y=y_s, workspace=ws,
                    routing_out=False, logits_out=False)
    torch.cuda.synchronize()
    for rep in range(3):
        for s, x in enumerate(xs):
            say(f"graph case moe_layer: replay {rep} input {s}")
            x_s.copy_(x)
            g.replay()
            torch.cuda.synchronize()
            got = _bits(y_s)
            ref = X.moe_layer(x, wg, w1, w3, w2, k, 1, M, shared=sh, routing_out=False,
                              logits_out=False)["y"]
            torch.cuda.synchronize()
            assert torch.equal(got, _bits(ref)), f"replay {rep}, input {s}"


def test_concurrent_calls_on_two_streams_match_serial():
    """Calls are stateless: two layers in flight at once, on two streams (default priority)
    with their own workspaces, enqueued from one host thread and then from two, give the
    same bits as the same calls one after the other."""
    import threading

    from paper_2602_07265_amd import xshare as X
    T, N, k, d, f, M = 32, 64, 8, 256, 512, 16
    cfg = dict(N=N, k=k, d=d, f=f, T=T, logits="domains", Q=4)
    w1, w3, w2 = W.expert_weights(N, d, f, 2, DEV)
    inputs = [(W.activations(T, d, s, DEV), torch.from_numpy(W.make_logits(cfg, s)[0]).to(DEV))
              for s in range(2)]
    p = X.params(N, k, 1, M)
    nws = X.moe_workspace_bytes(T, d, f, p)
    say("concurrency case: serial reference")
    ref = [_bits(X.moe_forward(x, h, w1, w3, w2, k, 1, M, routing_out=False)["y"])
           for x, h in inputs]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    wss = [torch.empty(nws, dtype=torch.uint8, device=DEV) for _ in range(2)]
    ys = [torch.empty((T, d), dtype=torch.bfloat16, device=DEV) for _ in range(2)]

    def run(i, reps):
        for _ in range(reps):
            X.moe_forward(inputs[i][0], inputs[i][1], w1, w3, w2, k, 1, M, y=ys[i],
                          workspace=wss[i], routing_out=False, stream=streams[i])

    say("concurrency case: two streams, one thread")
    for _ in range(3):
        run(0, 2)
        run(1, 2)
    torch.cuda.synchronize()
    assert all(torch.equal(_bits(ys[i]), ref[i]) for i in range(2))
    say("concurrency case: two streams, two threads")
    for y in ys:
        y.zero_()
    threads = [threading.Thread(target=run, args=(i, 4)) for i in range(2)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    torch.cuda.synchronize()
    assert all(torch.equal(_bits(ys[i]), ref[i]) for i in range(2))
