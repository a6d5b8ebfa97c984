"""The roofline denominator checks of include/dqn_profile.h on the GPU: the
streaming copy copies, and the matrix-core loop reports the FLOP count its
launch shape implies and leaves finite values."""
import pytest
import torch

import paper_1508_04186_amd as dq

pytestmark = pytest.mark.gpu


def test_stream_copy_copies(dev):
    src = torch.randint(0, 2**31 - 1, (1 << 20,), dtype=torch.int32, device=dev)
    dst = torch.zeros_like(src)
    dq.profile_stream_copy(src, dst, 64)
    torch.cuda.synchronize()
    assert torch.equal(src, dst)


@pytest.mark.parametrize("dtype,per", [(dq.DQN_PEAK_FP32, 16 * 16 * 4 * 2), (dq.DQN_PEAK_BF16, 16 * 16 * 32 * 2)])
def test_mfma_loop_flop_count(dev, dtype, per):
    out = torch.full((32,), float("nan"), device=dev)
    flop = dq.profile_mfma_peak(dtype, 32, 10, out)
    torch.cuda.synchronize()
    assert flop == 32 * 4 * 10 * 4 * per
    assert torch.isfinite(out).all()
