"""The Python binding validates shapes, dtypes and layouts before anything
reaches the library (CPU tensors: every check below fails before the device
check, so no launch can happen)."""
import pytest
import torch

from paper_2609_04910_amd import gauss_sum as gs

CPU = torch.device("cpu")


def pts(n, d, dtype=torch.float16):
    return torch.zeros((n, d), dtype=dtype)


def test_k_shape_must_match_v_rows_and_q_columns():
    q, v = pts(5, 8), torch.zeros((7, 2))
    for bad in (pts(6, 8), pts(7, 9), pts(3, 8)):
        with pytest.raises(ValueError, match="k must be 7 x 8"):
            gs.gauss_sum_fwd(q, bad, v, 1.0)
        with pytest.raises(ValueError, match="k must be 7 x 8"):
            gs.gauss_sum_bwd(q, bad, v, 1.0, torch.zeros((5, 2)))
        with pytest.raises(ValueError, match="k must be 7 x 8"):
            gs.gauss_sum_fwd_bwd(q, bad, v, 1.0, torch.zeros((5, 2)))


def test_inputs_must_be_contiguous_2d_and_share_dtype():
    q, k, v = pts(5, 8), pts(7, 8), torch.zeros((7, 2))
    with pytest.raises(ValueError, match="contiguous 2-d"):
        gs.gauss_sum_fwd(pts(8, 5).t(), k, v, 1.0)
    with pytest.raises(ValueError, match="contiguous 2-d"):
        gs.gauss_sum_fwd(q, k, torch.zeros(7), 1.0)
    with pytest.raises(TypeError, match="share a dtype"):
        gs.gauss_sum_fwd(q, pts(7, 8, torch.bfloat16), v, 1.0)
    # shapes fine: the device check comes last
    with pytest.raises(ValueError, match="GPU tensor"):
        gs.gauss_sum_fwd(q, k, v, 1.0)


def test_caller_outputs_checked_for_dtype_shape_layout():
    for bad, err in ((torch.zeros((5, 2), dtype=torch.float16), TypeError),
                     (torch.zeros((5, 3)), ValueError),
                     (torch.zeros((4, 2)), ValueError),
                     (torch.zeros((2, 5)).t(), ValueError)):
        with pytest.raises(err):
            gs._output(bad, "out", (5, 2), CPU)
    good = torch.zeros((5, 2))
    with pytest.raises(ValueError, match="dout"):
        gs._check_tensor(torch.zeros((5, 3)), "dout", (5, 2), CPU)
    # right shape and dtype but not on the GPU
    with pytest.raises(ValueError, match="GPU tensor"):
        gs._output(good, "out", (5, 2), torch.device("cuda", 0))


def test_workspace_must_be_a_contiguous_gpu_tensor():
    with pytest.raises(ValueError, match="workspace"):
        gs._workspace_arg(torch.zeros(64, dtype=torch.uint8), 64, torch.device("cuda", 0))


def test_batched_inputs_checked_before_device():
    q = torch.zeros((3, 5, 8), dtype=torch.float16)
    with pytest.raises(ValueError, match="inconsistent batch"):
        gs._batched_inputs(q, torch.zeros((2, 7, 8), dtype=torch.float16), torch.zeros((3, 7, 2)))
    with pytest.raises(ValueError, match="k must be"):
        gs._batched_inputs(q, torch.zeros((3, 7, 9), dtype=torch.float16), torch.zeros((3, 7, 2)))
    with pytest.raises(ValueError, match="GPU tensor"):
        gs._batched_inputs(q, torch.zeros((3, 7, 8), dtype=torch.float16), torch.zeros((3, 7, 2)))
