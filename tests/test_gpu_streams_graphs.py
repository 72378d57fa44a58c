"""The PAM products on several HIP streams and host threads at once, and
inside HIP graphs.

The binding launches on the caller's current stream and takes split-K
workspaces from torch's stream-ordered allocator, so products may run
concurrently on different streams and may be captured into a HIP graph
(torch.cuda.CUDAGraph).  Every result is compared bitwise with the same
product run eagerly on one stream: the plans do not depend on the stream.
"""
import numpy as np
import pytest

import paper_2305_17190_amd as pam
from gpu_util import device, note, to_dev

pytestmark = pytest.mark.gpu


def _layer(seed, tokens=8192, d_in=256, d_out=192):
    g = np.random.default_rng(seed)
    x = to_dev(g.standard_normal((tokens, d_in)).astype(np.float32))
    w = to_dev((g.standard_normal((d_out, d_in)) * 0.05).astype(np.float32))
    dy = to_dev((g.standard_normal((tokens, d_out)) * 1e-3).astype(np.float32))
    return x, w, dy


def _products(x, w, dy, outs=None):
    """Y = X .^ W^T, dX = dY .^ W, dW = dY^T .^ X (dW: long K, few tiles: split K)."""
    y, dx, dw = outs if outs is not None else (None, None, None)
    y = pam.gemm(x, w, trans_b=True, out=y)
    dx = pam.gemm(dy, w, out=dx)
    dw = pam.gemm(dy, x, trans_a=True, out=dw)
    return y, dx, dw


def _same_bits(a, b):
    import torch
    return torch.equal(a.view(torch.int32), b.view(torch.int32))


def test_products_on_two_streams_at_once():
    import torch
    note("gemm on two streams concurrently (split-K dW on both)")
    assert pam.plan(192, 256, 8192)[2] > 1
    layers = [_layer(101), _layer(102)]
    want = [_products(*l) for l in layers]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]    # default priority
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    got = [None, None]
    for rep in range(3):
        for i, s in enumerate(streams):                      # interleaved enqueues
            with torch.cuda.stream(s):
                got[i] = _products(*layers[i])
        torch.cuda.synchronize()
        for i in range(2):
            for g, w_ in zip(got[i], want[i]):
                assert _same_bits(g, w_), f"stream {i} replay {rep}"


def test_linear_layer_products_in_a_hip_graph():
    import torch
    note("linear layer fwd + bwd products captured in a HIP graph, 4 replays")
    x, w, dy = _layer(103)
    outs = tuple(torch.empty(shape, device=device()) for shape in
                 ((x.shape[0], w.shape[0]), x.shape, w.shape))
    # warm-up on a side stream, as graph capture requires
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for _ in range(2):
            _products(x, w, dy, outs)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        _products(x, w, dy, outs)
    torch.cuda.synchronize()
    for rep in range(4):
        # new inputs in the captured buffers, eager work between replays
        nx, nw, ndy = _layer(200 + rep)
        x.copy_(nx)
        w.copy_(nw)
        dy.copy_(ndy)
        for o in outs:
            o.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        want = _products(nx, nw, ndy)
        torch.cuda.synchronize()
        for name, g, w_ in zip(("Y", "dX", "dW"), outs, want):
            assert _same_bits(g, w_), f"{name} differs from the eager product on replay {rep}"
    del graph


def test_attention_products_in_a_hip_graph():
    import torch
    note("batched attention products captured in a HIP graph, 3 replays")
    g = np.random.default_rng(104)
    q = to_dev(g.standard_normal((32, 256, 64)).astype(np.float32))
    k = to_dev(g.standard_normal((32, 256, 64)).astype(np.float32))
    p = to_dev(np.abs(g.standard_normal((32, 256, 256))).astype(np.float32) / 256)
    v = to_dev(g.standard_normal((32, 256, 64)).astype(np.float32))
    s_out = torch.empty((32, 256, 256), device=device())
    o_out = torch.empty((32, 256, 64), device=device())

    def run():
        pam.bmm(q, k, trans_b=True, out=s_out)     # S = Q .^ K^T
        pam.bmm(p, v, out=o_out)                    # O = P .^ V

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        run()
    torch.cuda.synchronize()
    for rep in range(3):
        q.mul_(1.5)
        v.add_(0.25)
        s_out.fill_(float("nan"))
        o_out.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        want_s = pam.bmm(q, k, trans_b=True)
        want_o = pam.bmm(p, v)
        torch.cuda.synchronize()
        assert _same_bits(s_out, want_s), f"S differs on replay {rep}"
        assert _same_bits(o_out, want_o), f"O differs on replay {rep}"
    del graph


def test_products_from_several_host_threads():
    # The library keeps no shared host state (its error text and device
    # check are per thread), and ctypes releases the interpreter lock during
    # each call, so host threads drive it concurrently, each on a stream of
    # its own; every result must equal the single-threaded product bitwise.
    import threading
    import torch
    note("gemm from 4 host threads, one stream each")
    layers = [_layer(300 + i, tokens=2048) for i in range(4)]
    want = [_products(*l) for l in layers]
    torch.cuda.synchronize()
    got = [None] * 4
    errors = []

    def work(i):
        try:
            s = torch.cuda.Stream()
            s.wait_stream(torch.cuda.default_stream())
            with torch.cuda.stream(s):
                for _ in range(3):
                    got[i] = _products(*layers[i])
            s.synchronize()
        except Exception as e:   # reported below, on the main thread
            errors.append((i, repr(e)))

    threads = [threading.Thread(target=work, args=(i,)) for i in range(4)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads), "a worker thread did not finish"
    assert not errors, errors
    torch.cuda.synchronize()
    for i in range(4):
        for name, g, w_ in zip(("Y", "dX", "dW"), got[i], want[i]):
            assert _same_bits(g, w_), f"thread {i} {name}"


def test_bfloat16_and_narrow_products_in_a_hip_graph():
    import torch
    note("bfloat16 and 7-bit-mantissa products (one split-K) captured in a HIP graph, 3 replays")
    g = np.random.default_rng(105)
    x = to_dev(g.standard_normal((4096, 256)).astype(np.float32))
    w = to_dev((g.standard_normal((192, 256)) * 0.05).astype(np.float32))
    dy = to_dev((g.standard_normal((4096, 192)) * 1e-3).astype(np.float32))
    x16, w16 = x.to(torch.bfloat16), w.to(torch.bfloat16)
    outs = (torch.empty((4096, 192), device=device()), torch.empty((192, 256), device=device()))
    assert pam.plan(192, 256, 4096)[2] > 1

    def run():
        pam.gemm(x16, w16, trans_b=True, out=outs[0])                       # bfloat16 operands
        pam.gemm(dy, x, trans_a=True, out=outs[1], mantissa_bits=7)         # narrow, split-K dW

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        run()
    torch.cuda.synchronize()
    for rep in range(3):
        x.mul_(1.25)
        x16.copy_(x.to(torch.bfloat16))
        dy.add_(1e-4)
        for o in outs:
            o.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        want = (pam.gemm(x16, w16, trans_b=True), pam.gemm(dy, x, trans_a=True, mantissa_bits=7))
        torch.cuda.synchronize()
        for name, o, w_ in zip(("bf16 Y", "narrow dW"), outs, want):
            assert _same_bits(o, w_), f"{name} differs on replay {rep}"
    del graph
