"""The hot path captured into a HIP graph replays bit-identically.

The library enqueues kernels only (no memsets, no allocation, no host
synchronisation), so a caller can capture quantize -> qlinear -> dequant
into a graph.  Every replay, with eager work and synchronisations between
replays, must equal the eager result.
"""
import numpy as np
import pytest

from paper_2408_13933_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("M,K,w_bits,out_bits", [(300, 1024, 8, 8), (16, 1024, 8, 16),
                                                 (130, 1024, 4, 16), (130, 8192, 8, 8)])
def test_graph_replay_matches_eager(M, K, w_bits, out_bits):
    """The last case splits K through a workspace: its arrival counters
    return to zero inside the kernel, so replays need no memset."""
    import torch

    import paper_2408_13933_amd as mq

    layer = wl.Layer("g", M, K, 384, w_bits=w_bits, out_bits=out_bits)
    ld = wl.make_layer("graph", layer)
    dev = torch.device("cuda", 0)
    x = torch.from_numpy(ld.x).to(dev)
    w = torch.from_numpy(ld.w).to(dev)
    bias = torch.from_numpy(ld.bias).to(dev)
    wq, ws, cs = mq.mq_pack_weights(w, w_bits)
    a_scale, a_zp = mq.mq_act_params(*ld.act_range, 8)
    o_scale, o_zp = mq.mq_act_params(*ld.out_range, out_bits)
    a_q = torch.empty(x.shape, dtype=torch.int8, device=dev)
    y = torch.empty((M, 384), dtype=torch.int8 if out_bits == 8 else torch.int16, device=dev)
    deq = torch.empty((M, 384), dtype=torch.float32, device=dev)
    nws = mq.mq_qlinear_workspace_bytes(M, K, 384, w_bits, out_bits)
    work = torch.zeros(nws, dtype=torch.uint8, device=dev) if nws else None
    if K > 1024:
        assert nws > 0

    def step():
        mq.mq_quantize_act(x, a_scale, a_zp, 8, out=a_q)
        mq.mq_qlinear(a_q, wq, w_bits, ws, cs, a_scale, a_zp, o_scale, o_zp, out_bits,
                      bias=bias, out=y, workspace=work)
        mq.mq_dequant(y, o_scale, o_zp, out=deq)

    step()  # eager, also performs any one-time kernel set-up before capture
    torch.cuda.synchronize()
    y_ref, d_ref = y.cpu().numpy().copy(), deq.cpu().numpy().copy()

    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            step()
    torch.cuda.current_stream().wait_stream(s)
    for rep in range(4):
        y.fill_(0)
        deq.fill_(0)
        a_q.fill_(0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(y.cpu().numpy(), y_ref), f"replay {rep}"
        assert np.array_equal(deq.cpu().numpy().view(np.uint32), d_ref.view(np.uint32))
        step()  # eager work between replays
        torch.cuda.synchronize()


def test_graph_replay_asymmetric_split():
    """Asymmetric weights with the fused quantizer + row sums and a K split
    through a workspace, captured and replayed."""
    import torch

    import paper_2408_13933_amd as mq

    M, K, N = 130, 8192, 384
    layer = wl.Layer("g", M, K, N, w_bits=8, out_bits=16, asym=True)
    ld = wl.make_layer("graph_asym", layer)
    dev = torch.device("cuda", 0)
    x = torch.from_numpy(ld.x).to(dev)
    w = torch.from_numpy(ld.w).to(dev)
    bias = torch.from_numpy(ld.bias).to(dev)
    wq, ws, zw, cs = mq.mq_pack_weights_asym(w, 8)
    a_scale, a_zp = mq.mq_act_params(*ld.act_range, 8)
    o_scale, o_zp = mq.mq_act_params(*ld.out_range, 16)
    a_q = torch.empty(x.shape, dtype=torch.int8, device=dev)
    rs = torch.empty(M, dtype=torch.int32, device=dev)
    y = torch.empty((M, N), dtype=torch.int16, device=dev)
    nws = mq.mq_qlinear_workspace_bytes(M, K, N, 8, 16)
    assert nws > 0
    work = torch.zeros(nws, dtype=torch.uint8, device=dev)

    def step():
        mq.mq_quantize_act_rowsum(x, a_scale, a_zp, out=a_q, rowsum=rs)
        mq.mq_qlinear_asym(a_q, rs, wq, 8, ws, zw, cs, a_scale, a_zp, o_scale, o_zp, 16,
                           bias=bias, out=y, workspace=work)

    step()
    torch.cuda.synchronize()
    y_ref = y.cpu().numpy().copy()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            step()
    torch.cuda.current_stream().wait_stream(s)
    for rep in range(4):
        y.fill_(0)
        rs.fill_(0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(y.cpu().numpy(), y_ref), f"replay {rep}"
        step()
        torch.cuda.synchronize()


def test_block_graph_replay_matches_eager():
    """The whole decoder block (19 steps: projections with a split-K
    workspace, attention products with their sums, softmax, RoPE, tables)
    captured once and replayed four times, with eager work in between:
    every replay reproduces every intermediate of the eager run."""
    import torch

    from paper_2408_13933_amd import block as blk

    data = wl.make_block(256)
    g = blk.BlockGPU(data)
    g.run()
    torch.cuda.synchronize()
    ref = {k: v.cpu().numpy().copy() for k, v in g.out.items() if k not in blk.NOT_STORED}
    graph = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(graph, stream=s):
            g.run()
    torch.cuda.current_stream().wait_stream(s)
    low = np.tril(np.ones((256, 256), dtype=bool))
    for rep in range(4):
        for k, v in g.out.items():
            if k != "h0":
                v.fill_(7)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k, v in g.out.items():
            if k in blk.NOT_STORED:
                continue
            got = v.cpu().numpy()
            if k == "scores":  # only the causal lower triangle is computed
                assert np.array_equal(got[:, low], ref[k][:, low]), (rep, k)
            else:
                assert np.array_equal(got, ref[k]), (rep, k)
        g.stages()[0][1]()  # eager work between replays
