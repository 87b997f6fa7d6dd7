"""The torch.library registrations: shape propagation without a GPU, and on
the GPU, under torch.compile (graph capture of the custom ops, no code
generation) and under HIP-graph replay, the oracle's results: quantize and
pack bit for bit, the linear within its tolerance (and bitwise equal to the
direct calls)."""
import numpy as np
import pytest
import torch
from torch._subclasses.fake_tensor import FakeTensorMode

import oracle
from oracle.compare import linear_check
from paper_2605_08755_amd import inputs, laq
from paper_2605_08755_amd import torch_ops  # noqa: F401  (registers torch.ops.laq.*)


def test_fake_shapes():
    with FakeTensorMode():
        w = torch.empty(40, 384, dtype=torch.float16, device="cuda")
        x = torch.empty(3, 384, dtype=torch.float16, device="cuda")
        for bits in (3, 4):
            q, s, z = torch.ops.laq.quantize(w, bits)
            assert q.shape == (40, bits, 12) and q.dtype == torch.int32
            assert s.shape == (40, 3) and s.dtype == torch.float16
            assert z.shape == (40, 3) and z.dtype == torch.uint8
            q2 = torch.ops.laq.pack(w, s, z, bits)
            assert q2.shape == q.shape and q2.dtype == torch.int32
            y = torch.ops.laq.linear(x, q, s, z, bits)
            assert y.shape == (3, 40) and y.dtype == torch.float16


@pytest.mark.gpu
@pytest.mark.parametrize("bits", [3, 4])
def test_ops_match_direct_calls(bits):
    print("[gpu-case] torch ops", bits, flush=True)
    dev = torch.device("cuda:0")
    w_h = inputs.weights(96, 1024, cfg=30)
    x_h = inputs.activations(4, 1024, cfg=30)
    w = torch.from_numpy(w_h).to(dev)
    x = torch.from_numpy(x_h).to(dev)
    q, s, z = laq.quantize(w, bits)
    y = laq.linear(x, q, s, z, bits)

    def f(w, x):
        q, s, z = torch.ops.laq.quantize(w, bits)
        q2 = torch.ops.laq.pack(w, s, z, bits)
        return q, q2, torch.ops.laq.linear(x, q2, s, z, bits)

    cf = torch.compile(f, backend="aot_eager", fullgraph=True)
    qc, q2c, yc = cf(w, x)
    torch.cuda.synchronize()
    codes, os_, oz = oracle.quantize(w_h, bits)
    assert np.array_equal(qc.cpu().numpy().view(np.uint32), oracle.pack(codes, bits))
    assert np.array_equal(q2c.cpu().numpy().view(np.uint32), oracle.pack(codes, bits))
    r = linear_check(yc.cpu().numpy(), oracle.linear(x_h, codes, os_, oz))
    assert r["ok"], r
    assert torch.equal(qc, q) and torch.equal(q2c, q)
    assert torch.equal(yc, y)


@pytest.mark.gpu
def test_ops_in_graph_replay():
    print("[gpu-case] torch ops graph", flush=True)
    dev = torch.device("cuda:0")
    w_h = inputs.weights(257, 2560, cfg=31)
    x_h = inputs.activations(1, 2560, cfg=31)
    w = torch.from_numpy(w_h).to(dev)
    x = torch.from_numpy(x_h).to(dev)
    q, s, z = torch.ops.laq.quantize(w, 3)
    y_eager = torch.ops.laq.linear(x, q, s, z, 3)
    torch.cuda.synchronize()
    codes, os_, oz = oracle.quantize(w_h, 3)
    assert np.array_equal(s.cpu().numpy().view(np.uint16), os_) and np.array_equal(z.cpu().numpy(), oz)
    r = linear_check(y_eager.cpu().numpy(), oracle.linear(x_h, codes, os_, oz))
    assert r["ok"], r
    stream = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        y_graph = torch.ops.laq.linear(x, q, s, z, 3)
    for _ in range(3):
        y_graph.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y_graph, y_eager)
        # eager work between replays
        assert np.isfinite(laq.linear(x, q, s, z, 3).float().cpu().numpy()).all()
