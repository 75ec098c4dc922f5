"""A whole decoder block on the GPU (paper_2408_13933_amd.block) against the
same block through the oracle: every stage compared, from the same float
inputs and static ranges.  Stages built from integer arithmetic and
correctly rounded fp64 operations must be bit-exact; the stages through
exp, cos and sin (RoPE, softmax, the SiLU table) may differ by one step at
rounding ties of their fp64 value, and a difference there can then move a
few codes downstream."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

TIE_STAGES = ("qr", "kr", "probs", "mul")  # "mul": through the SiLU table


@pytest.mark.parametrize("T", [128, 200])
def test_block_stages_match_the_oracle(T):
    from paper_2408_13933_amd import block as blk
    from paper_2408_13933_amd import workloads as wl
    from tests.pipelines import block_oracle

    data = wl.make_block(T)
    g = blk.BlockGPU(data)
    g.run()
    ref, fmt = block_oracle(data)
    assert fmt == g.fmt
    diverged = None
    for stage in blk.STAGE_BITS:
        if stage in blk.NOT_STORED:  # fused into the next step
            continue
        got = g.out[stage].cpu().numpy()
        exp = ref[stage]
        if stage == "scores":  # only the causal lower triangle is computed
            low = np.tril(np.ones((T, T), dtype=bool))
            got, exp = got[:, low], exp[:, low]
        assert got.shape == exp.shape and got.dtype == exp.dtype, stage
        diff = got.astype(np.int64) - exp.astype(np.int64)
        n_bad = int(np.count_nonzero(diff))
        if diverged is None:
            if n_bad == 0:
                continue
            assert stage in TIE_STAGES, (stage, n_bad)
            assert np.abs(diff).max() == 1 and n_bad <= max(1, got.size // 100000), (stage, n_bad)
            diverged = stage
        else:
            assert n_bad <= got.size // 1000 and np.abs(diff).max() <= 2, (stage, diverged, n_bad)
    print(f"T={T}: first stage that differs: {diverged}")
