"""The MFMA calibration launch (himuon_calib_mfma) runs and its products are
what the instruction computes: with every operand word the same, each lane's
sum is a closed form."""
import pytest

import paper_2606_27216_amd as hm

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("compute,dtype", [(hm.COMPUTE_F16, "float16"), (hm.COMPUTE_BF16, "bfloat16")])
def test_calib_mfma_products(compute, dtype):
    import torch
    dev = torch.device("cuda:0")
    print(f"[gpu-case] calib_mfma {dtype}", flush=True)
    # all operands 0.5: every product of a 32x32x16 MFMA adds 16 * 0.25 = 4 to
    # each of a lane's 16 accumulator values, so after iters rounds each of the
    # four accumulators holds 4 * iters per value and a lane's sum is
    # 4 accumulators * 16 values * 4 * iters (exact in fp32 for these sizes)
    ops = torch.full((4096 * 8,), 0.5, device=dev, dtype=getattr(torch, dtype))
    grid, iters = 8, 5
    out = torch.full((grid * 256,), -1.0, device=dev)
    st = hm.himuon_calib_mfma(compute, ops.data_ptr(), out.data_ptr(), grid, iters,
                              torch.cuda.current_stream(dev).cuda_stream)
    assert st == hm.OK, hm.himuon_status_string(st)
    torch.cuda.synchronize()
    assert torch.all(out == 4 * 16 * 4 * iters).item()
