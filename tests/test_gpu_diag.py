"""The matrix-core loop that the bench reports as the practical ceiling of the assignment's instruction: its
accumulator value and its FLOP count follow from the instruction's definition (a 32 x 32 x 16 product per
instruction, four chains per wave)."""
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("iters,a,b", [(0, 1.0, 1.0), (1, 1.0, 1.0), (100, 1.0, 1.0), (37, 0.5, -2.0)])
def test_mfma_loop_value_and_flops(fkv, iters, a, b):
    out, flops = fkv.fkv_diag_mfma_loop(3, iters, a=a, b=b)
    torch.cuda.synchronize()
    # each instruction adds sum_k a * b over k = 16 to every accumulator element; four chains
    assert float(out.item()) == 4 * 16 * iters * a * b
    assert flops == 3 * 4 * 4 * iters * 2 * 32 * 32 * 16


def test_mfma_loop_rejects_bad_arguments(fkv):
    out = torch.empty(1, dtype=torch.float32, device="cuda")
    with pytest.raises(fkv.FkvError):
        fkv.fkv_diag_mfma_loop(0, 10, out=out)
    with pytest.raises(fkv.FkvError):
        fkv.fkv_diag_mfma_loop(1, -1, out=out)


def test_mfma_loop_random_operands(fkv):
    """The random-operand form: a finite accumulator (the operands lie in [-1, 1)), the same value on a
    repeated call (it depends only on the launch), and the same FLOP count as the constant form."""
    out1, f1 = fkv.fkv_diag_mfma_loop(2, 50, random_operands=True)
    v1 = float(out1.item())
    out2, f2 = fkv.fkv_diag_mfma_loop(2, 50, random_operands=True)
    torch.cuda.synchronize()
    assert abs(v1) < 4 * 16 * 50 and v1 == float(out2.item()) and f1 == f2 == fkv.fkv_diag_mfma_loop(2, 50)[1]
