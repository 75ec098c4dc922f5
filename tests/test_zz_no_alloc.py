"""mq_qlinear_noalloc, the qlinear entry point that allocates nothing,
against mq_qlinear_ws (the same layer with a caller's split-K workspace)
and the CPU oracle: bit-exact, on consecutive calls of decreasing size that
share the library's static per-GPU array, across both weight widths and a
call that does not split at all."""
import numpy as np
import pytest

from paper_2408_13933_amd import workloads as wl
from tests.pipelines import oracle_layer

pytestmark = pytest.mark.gpu

# M, K, N, w_bits, out_bits, bias -- every prefill case splits K on the
# automatic choice; each call's input is smaller than the one before
SEQUENCE = [
    (300, 8192, 700, 8, 8, True),
    (130, 8192, 300, 8, 8, True),
    (200, 5632, 300, 4, 16, False),
    (64, 16384, 160, 8, 16, False),
    (16, 2048, 256, 8, 8, True),    # decode path: no split, no scratch
]


def _device_layer(ld, o):
    """Device copies of the oracle's packed weights and quantized inputs."""
    import torch

    dev = torch.device("cuda", 0)
    t = lambda v: torch.from_numpy(np.ascontiguousarray(v)).to(dev)
    return dict(a_q=t(o.a_q), w_q=t(o.w_q), w_scale=t(o.w_scale), w_colsum=t(o.w_colsum),
                bias=None if ld.bias is None else t(ld.bias))


def test_noalloc_matches_workspace_entry_point():
    import torch

    import paper_2408_13933_amd as mq

    for M, K, N, wb, ob, has_bias in SEQUENCE:
        layer = wl.Layer("x", M, K, N, w_bits=wb, out_bits=ob, bias=has_bias)
        ld = wl.make_layer("noalloc", layer)
        o = oracle_layer(ld)
        d = _device_layer(ld, o)
        need = mq.mq_qlinear_workspace_bytes(M, K, N, wb, ob)
        assert (need > 0) == (M > 16), (M, K, N, need)
        assert need <= mq.NOALLOC_SCRATCH_BYTES
        print(f"noalloc {M}x{K}x{N} w{wb} o{ob} split workspace {need} B", flush=True)
        args = (d["w_q"], wb, d["w_scale"], d["w_colsum"], o.a_scale, o.a_zp, o.out_scale,
                o.out_zp, ob)
        ws = torch.zeros(max(need, 256), dtype=torch.uint8, device="cuda")
        y_ws = mq.mq_qlinear(d["a_q"], *args, bias=d["bias"], workspace=ws)
        # poison the output so stale contents cannot pass
        y = torch.full((M, N), 77, dtype=torch.int8 if ob == 8 else torch.int16, device="cuda")
        mq.mq_qlinear_noalloc(d["a_q"], *args, bias=d["bias"], out=y)
        torch.cuda.synchronize()
        got, ref = y.cpu().numpy(), y_ws.cpu().numpy()
        assert np.array_equal(ref, o.y_q), "workspace entry point differs from the oracle"
        assert np.array_equal(got, ref), (M, K, N, int((got != ref).sum()))
    # the same first layer again after the smaller ones: the array keeps the
    # last call's contents, which must not leak into the result
    M, K, N, wb, ob, has_bias = SEQUENCE[0]
    ld = wl.make_layer("noalloc", wl.Layer("x", M, K, N, w_bits=wb, out_bits=ob, bias=has_bias))
    o = oracle_layer(ld)
    d = _device_layer(ld, o)
    y = mq.mq_qlinear_noalloc(d["a_q"], d["w_q"], wb, d["w_scale"], d["w_colsum"], o.a_scale,
                              o.a_zp, o.out_scale, o.out_zp, ob, bias=d["bias"])
    torch.cuda.synchronize()
    assert np.array_equal(y.cpu().numpy(), o.y_q)


def test_noalloc_rejects_split_beyond_scratch():
    """A shape whose K split needs more than the static array returns
    MQ_ERR_UNSUPPORTED and writes nothing."""
    import torch

    import paper_2408_13933_amd as mq

    M, K, N = 1024, 65536, 2048
    assert mq.mq_qlinear_workspace_bytes(M, K, N, 8, 16) > mq.NOALLOC_SCRATCH_BYTES
    a = torch.zeros((M, K), dtype=torch.int8, device="cuda")
    w = torch.zeros((N, K), dtype=torch.int8, device="cuda")
    s = torch.ones(N, device="cuda")
    c = torch.zeros(N, dtype=torch.int32, device="cuda")
    y = torch.full((M, N), 5, dtype=torch.int16, device="cuda")
    with pytest.raises(mq.MQError):
        mq.mq_qlinear_noalloc(a, w, 8, s, c, 0.1, 0, 0.1, 0, 16, out=y)
    torch.cuda.synchronize()
    assert bool((y == 5).all())
