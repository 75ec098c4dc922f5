"""GPU parity of the batched attention matmuls between 16-bit and 8-bit
activation codes (Section 5.6) against the CPU oracle: bit-exact on the
tiled MFMA kernel and on the generic kernel, for Q K^T and P V shapes with
grouped-query heads, strided head views and ragged sizes."""
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


def _params(rng, out_bits):
    a_scale = float(np.float32(rng.uniform(1e-5, 1e-4)))
    b_scale = float(np.float32(rng.uniform(0.01, 0.05)))
    out_scale = float(np.float32(rng.uniform(1e-3, 1e-2) * (1e-2 if out_bits == 16 else 1)))
    return (a_scale, int(rng.integers(-32768, 32768)), b_scale, int(rng.integers(-128, 128)),
            out_scale, int(rng.integers(-100, 100)), out_bits)


@pytest.mark.parametrize("T,D,H,G", [(200, 64, 8, 2), (128, 64, 4, 4), (17, 64, 2, 1),
                                     (300, 128, 6, 3), (40, 4, 2, 2), (33, 24, 3, 1)])
@pytest.mark.parametrize("out_bits", [16, 8])
def test_scores_qkt_parity(T, D, H, G, out_bits):
    """Q K^T on head views of the projections' [token][heads * D] outputs."""
    mq, torch = _mq(), _torch()
    rng = np.random.default_rng(T + D + H + out_bits)
    q = rng.integers(-32768, 32768, (T, H * D)).astype(np.int16)
    k = rng.integers(-128, 128, (G, T, D)).astype(np.int8).transpose(1, 0, 2).reshape(T, G * D)
    k = np.ascontiguousarray(k)
    prm = _params(rng, out_bits)
    qa = q.reshape(T, H, D).transpose(1, 0, 2)
    kb = k.reshape(T, G, D).transpose(1, 0, 2)
    ref = oracle.attn_matmul(np.ascontiguousarray(qa), np.ascontiguousarray(kb), *prm)
    gq = torch.from_numpy(q).cuda().view(T, H, D).permute(1, 0, 2)
    gk = torch.from_numpy(k).cuda().view(T, G, D).permute(1, 0, 2)
    for path in (mq.PATH_AUTO, mq.PATH_PREFILL, mq.PATH_GENERIC):
        y = mq.mq_attn_matmul(gq, gk, *prm, path=path).cpu().numpy()
        assert np.array_equal(y, ref), (path, int((y != ref).sum()))


@pytest.mark.parametrize("T,D,H,G", [(256, 64, 8, 2), (200, 64, 4, 2), (130, 128, 2, 1)])
def test_context_pv_parity(T, D, H, G):
    """P V: probability codes [H][T][T] times the transposed value codes,
    written into a [token][heads * D] context view."""
    mq, torch = _mq(), _torch()
    rng = np.random.default_rng(T * 3 + D + H)
    p = rng.integers(-32768, 32768, (H, T, T)).astype(np.int16)
    p[:, np.triu_indices(T, 1)[0], np.triu_indices(T, 1)[1]] = -32768  # causal zeros
    v = rng.integers(-128, 128, (T, G * D)).astype(np.int8)
    prm = _params(rng, 16)
    prm = (prm[0], -32768) + prm[2:]
    vt = np.ascontiguousarray(v.T).reshape(G, D, T)
    ref = oracle.attn_matmul(p, vt, *prm)
    gv = torch.from_numpy(v).cuda()
    gvt = mq.mq_transpose_i8(gv)
    assert np.array_equal(gvt.cpu().numpy(), v.T)
    gp = torch.from_numpy(p).cuda()
    for path in (mq.PATH_AUTO, mq.PATH_GENERIC):
        ctx = torch.zeros((T, H * D), dtype=torch.int16, device="cuda")
        view = ctx.view(T, H, D).permute(1, 0, 2)
        mq.mq_attn_matmul(gp, gvt.view(G, D, T), *prm, out=view, path=path)
        got = ctx.view(T, H, D).permute(1, 0, 2).cpu().numpy()
        assert np.array_equal(got, ref), (path, int((got != ref).sum()))


@pytest.mark.parametrize("M", [1, 5, 16, 33])
def test_attn_small_m_and_extremes(M):
    """Decode-sized query counts and codes at the ends of both ranges (sums
    beyond int32 saturate before the rescale)."""
    mq, torch = _mq(), _torch()
    rng = np.random.default_rng(M)
    H, G, N, K = 4, 2, 96, 1024
    a = np.where(rng.random((H, M, K)) < 0.5, -32768, 32767).astype(np.int16)
    b = np.where(rng.random((G, N, K)) < 0.5, -128, 127).astype(np.int8)
    a[:, 0] = 32767
    b[:, 0] = -128
    for prm in ((3e-5, -32768, 0.03, 127, 1e-2, 0, 16), (3e-5, 0, 0.03, 0, 40.0, 3, 8)):
        ref = oracle.attn_matmul(a, b, *prm)
        y = mq.mq_attn_matmul(torch.from_numpy(a).cuda(), torch.from_numpy(b).cuda(),
                              *prm).cpu().numpy()
        assert np.array_equal(y, ref)


@pytest.mark.parametrize("K", [128, 64, 16])
def test_attn_short_k_extremes(K):
    """K <= 128 without bias takes the int32 epilogue: its largest sums,
    |sum_k (a - a_zp)(b - b_zp)| up to 128 * 65535 * 255, must come out
    exact, with and without B's zero-point."""
    mq, torch = _mq(), _torch()
    rng = np.random.default_rng(K)
    H, G, M, N = 2, 1, 96, 160
    a = np.full((H, M, K), -32768, np.int16)
    b = np.full((G, N, K), 127, np.int8)
    a[:, 1::3] = np.where(rng.random((H, len(range(1, M, 3)), K)) < 0.5, -32768, 32767)
    b[:, 1::4] = np.where(rng.random((G, len(range(1, N, 4)), K)) < 0.5, -128, 127)
    for prm in ((3e-5, 32767, 0.03, -128, 200.0, 0, 16), (3e-5, 32767, 0.03, 0, 1e4, -3, 8),
                (3e-5, -5, 0.03, 77, 1e-2, 1, 16)):
        ref = oracle.attn_matmul(a, b, *prm)
        for path in (mq.PATH_AUTO, mq.PATH_PREFILL):
            y = mq.mq_attn_matmul(torch.from_numpy(a).cuda(), torch.from_numpy(b).cuda(), *prm,
                                  path=path).cpu().numpy()
            assert np.array_equal(y, ref), (prm, path, int((y != ref).sum()))


def test_attn_tinyllama_full_size_sampled_heads():
    """The 1024-token TinyLlama attention (32 query heads, 4 key/value
    heads, head dimension 64) through the tiled kernel; heads 0, 7, 8 and
    31 (groups 0, 0, 1, 3) against the oracle."""
    mq, torch = _mq(), _torch()
    rng = np.random.default_rng(1024)
    T, D, H, G = 1024, 64, 32, 4
    q = torch.from_numpy(rng.integers(-32768, 32768, (T, H * D)).astype(np.int16)).cuda()
    k = torch.from_numpy(rng.integers(-128, 128, (T, G * D)).astype(np.int8)).cuda()
    prm = _params(rng, 16)
    qa = q.view(T, H, D).permute(1, 0, 2)
    kb = k.view(T, G, D).permute(1, 0, 2)
    s = mq.mq_attn_matmul(qa, kb, *prm)
    heads = [0, 7, 8, 31]
    qa_np = qa.cpu().numpy()
    kb_np = kb.cpu().numpy()
    for h in heads:
        ref = oracle.attn_matmul(np.ascontiguousarray(qa_np[h:h + 1]),
                                 np.ascontiguousarray(kb_np[h // 8:h // 8 + 1]), *prm)
        assert np.array_equal(s[h:h + 1].cpu().numpy(), ref), h
    p = s  # int16 codes as the probabilities of the next product
    v = torch.from_numpy(rng.integers(-128, 128, (T, G * D)).astype(np.int8)).cuda()
    vt = mq.mq_transpose_i8(v).view(G, D, T)
    prm2 = _params(rng, 16)
    ctx = mq.mq_attn_matmul(p, vt, *prm2)
    p_np, vt_np = p.cpu().numpy(), vt.cpu().numpy()
    for h in heads:
        ref = oracle.attn_matmul(np.ascontiguousarray(p_np[h:h + 1]),
                                 np.ascontiguousarray(vt_np[h // 8:h // 8 + 1]), *prm2)
        assert np.array_equal(ctx[h:h + 1].cpu().numpy(), ref), h


@pytest.mark.parametrize("rows,cols", [(1, 1), (63, 65), (1024, 256), (7, 3000)])
def test_transpose_i8(rows, cols):
    mq, torch = _mq(), _torch()
    x = np.random.default_rng(rows).integers(-128, 128, (rows, cols + 5)).astype(np.int8)
    gx = torch.from_numpy(x).cuda()[:, :cols]
    assert np.array_equal(mq.mq_transpose_i8(gx).cpu().numpy(), x[:, :cols].T)


@pytest.mark.parametrize("T,D,H,G,b_zp", [(1024, 64, 8, 2, 0), (300, 64, 4, 2, 17),
                                          (200, 64, 2, 1, -5), (129, 128, 2, 2, 0)])
def test_causal_attention_parity(T, D, H, G, b_zp):
    """Q K^T with the causal output promise (entries past the diagonal may
    stay unwritten) and P V with causal probabilities (zero codes past the
    diagonal, which the kernel may skip): the lower triangle of the scores
    and the whole context equal the oracle's full products."""
    mq, torch = _mq(), _torch()
    rng = np.random.default_rng(T + D + H + b_zp)
    q = rng.integers(-32768, 32768, (H, T, D)).astype(np.int16)
    k = rng.integers(-128, 128, (G, T, D)).astype(np.int8)
    prm = _params(rng, 16)
    prm = prm[:3] + (b_zp,) + prm[4:]
    ref = oracle.attn_matmul(q, k, *prm)
    for path in (mq.PATH_AUTO, mq.PATH_GENERIC):
        s = torch.full((H, T, T), 12345, dtype=torch.int16, device="cuda")
        mq.mq_attn_matmul(torch.from_numpy(q).cuda(), torch.from_numpy(k).cuda(), *prm, out=s,
                          path=path, out_causal=0)
        got = s.cpu().numpy()
        low = np.tril(np.ones((T, T), dtype=bool))
        assert np.array_equal(got[:, low], ref[:, low]), path
    p = rng.integers(-32768, 32768, (H, T, T)).astype(np.int16)
    p[:, ~np.tril(np.ones((T, T), dtype=bool))] = -32768
    v = rng.integers(-128, 128, (G, D, T)).astype(np.int8)
    prm2 = (1.0 / 65535, -32768, 0.03, b_zp, 1e-3, 3, 8)
    ref2 = oracle.attn_matmul(p, v, *prm2)
    for path in (mq.PATH_AUTO, mq.PATH_GENERIC):
        ctx = mq.mq_attn_matmul(torch.from_numpy(p).cuda(), torch.from_numpy(v).cuda(), *prm2,
                                path=path, in_causal=0)
        assert np.array_equal(ctx.cpu().numpy(), ref2), path
