"""GPU parity of the calibration-side kernels against the CPU oracle:
SmoothQuant's closed-form scales (Section 3.2) and the training form of
activation range learning (Section 4.2, Eq.(2)-(4)).

Tolerances: fp32 elementwise results are bit-exact (the same IEEE
operations in the same order); the fp64 sums of the range gradients are
compared within 1e-12 of the sum of the terms' magnitudes (summation
order differs); the scales go through fp64 pow, whose last bit is not
fixed by IEEE, so they may differ by one fp32 ulp.
"""
import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.gpu


def _mq():
    import paper_2408_13933_amd as mq
    return mq


def _torch():
    import torch
    return torch


def _dev(a, offset=0):
    torch = _torch()
    t = torch.from_numpy(np.ascontiguousarray(a))
    if offset == 0:
        return t.cuda()
    buf = torch.empty(a.size + offset, dtype=t.dtype, device="cuda")
    v = buf[offset:].view(a.shape)
    v.copy_(t)
    return v


def _arl_inputs(n, seed):
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal(n) * 3).astype(np.float32)
    x[: min(n, 5)] = [np.nan, np.inf, -np.inf, 0.0, 1e30][: min(n, 5)]
    if n > 40:  # exact rounding ties of x / alpha for alpha = 0.5
        x[10:40] = (np.arange(30) - 15 + 0.5).astype(np.float32) * np.float32(0.5)
    g = rng.standard_normal(n).astype(np.float32)
    return x, g


ARL_PARAMS = [(0.5, -130.0, 8), (0.02, -127.3, 8), (3e-4, -32768.0, 16), (0.3, -7.6, 4)]


@pytest.mark.parametrize("n,offset", [(1, 0), (1000, 1), (4097, 0), (2 ** 20 + 3, 0)])
@pytest.mark.parametrize("params", ARL_PARAMS, ids=lambda p: f"a{p[0]}-b{p[1]}-bw{p[2]}")
def test_arl_forward_backward_parity(n, offset, params):
    mq = _mq()
    alpha, beta, bits = params
    x, g = _arl_inputs(n, n + bits)
    gx_ = _dev(x, offset)
    y = mq.mq_arl_forward(gx_, alpha, beta, bits).cpu().numpy()
    ref = oracle.arl_forward(x, alpha, beta, bits)
    assert np.array_equal(y.view(np.uint32), ref.view(np.uint32))
    gx, grads = mq.mq_arl_backward(gx_, _dev(g, offset), alpha, beta, bits)
    o_gx, o_ga, o_gb = oracle.arl_backward(x, g, alpha, beta, bits)
    assert np.array_equal(gx.cpu().numpy().view(np.uint32), o_gx.view(np.uint32))
    ga, gb = grads[:2].cpu().numpy().tolist()
    q_max = 2 ** bits - 1
    with np.errstate(invalid="ignore", over="ignore"):
        t = x / np.float32(alpha)
        u = np.rint(t) - np.float32(beta)
        inside = (u >= 0) & (u <= q_max)
    absg = np.abs(g.astype(np.float64))
    mag_a = float(np.sum(absg * (q_max + abs(beta) + np.where(inside, np.abs(t), 0.0))))
    assert abs(ga - o_ga) <= 1e-12 * mag_a
    assert abs(gb - o_gb) <= 1e-12 * float(absg.sum()) * alpha
    # the same numel sums in the same order: repeated calls agree bit for bit
    _, grads2 = mq.mq_arl_backward(gx_, _dev(g, offset), alpha, beta, bits)
    assert grads2[:2].cpu().numpy().tolist() == [ga, gb]


def test_arl_in_place_and_empty():
    mq, torch = _mq(), _torch()
    x, _ = _arl_inputs(5000, 3)
    t = _dev(x)
    mq.mq_arl_forward(t, 0.1, -100.0, 8, out=t)
    assert np.array_equal(t.cpu().numpy(), oracle.arl_forward(x, 0.1, -100.0, 8))
    e = torch.zeros(0, device="cuda")
    gx, grads = mq.mq_arl_backward(e, e, 0.1, -100.0, 8)
    assert grads[:2].cpu().numpy().tolist() == [0.0, 0.0]


@pytest.mark.parametrize("M,K,N", [(2048, 2048, 5632), (37, 1000, 13), (0, 64, 20), (5, 3, 0),
                                   (300, 5632, 2048)])
def test_smooth_scales_parity(M, K, N):
    mq = _mq()
    rng = np.random.default_rng(M + K + N)
    x = (rng.standard_normal((M, K)) * rng.uniform(0.05, 40, K)).astype(np.float32)
    w = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    if M > 3 and K > 12:
        x[:, 2] = 0.0
        x[1, 7], x[2, 8] = np.nan, -np.inf
    if N > 3 and K > 12:
        w[:, 5] = 0.0
        w[0, 11] = np.inf
    for a in (0.0, 0.5, 0.85, 1.0):
        s, mx, mw = mq.mq_smooth_scales(_dev(x), _dev(w), a)
        o_s, o_mx, o_mw = oracle.smooth_scales(x, w, a)
        assert np.array_equal(mx.cpu().numpy(), o_mx)
        assert np.array_equal(mw.cpu().numpy(), o_mw)
        gs = s.cpu().numpy()
        if a in (0.0, 1.0):
            assert np.array_equal(gs, o_s)          # pow(v, 0) = 1, pow(v, 1) = v exactly
        else:
            assert np.all(np.abs(gs - o_s) <= np.spacing(o_s)), a
