"""The reference streaming kernels the benchmark measures its bandwidth ceilings with:
the copy moves every byte, the read stores its folded word only on a key match."""

import numpy as np
import pytest
import torch

import paper_2602_07721_amd as pk

pytestmark = pytest.mark.gpu


def test_stream_copy_is_exact():
    for nbytes in (16, 4096 + 48, (1 << 22) + 16 * 77):
        src = torch.from_numpy(np.random.default_rng(nbytes).integers(0, 256, nbytes, dtype=np.uint8)).cuda()
        dst = torch.zeros_like(src)
        pk.stream_copy(dst, src)
        torch.cuda.synchronize()
        assert torch.equal(dst, src), nbytes


def test_stream_read_stores_only_on_a_key_match():
    src = torch.zeros(1 << 20, dtype=torch.uint8, device="cuda")  # every thread folds to 0
    sink = torch.full((1,), 0x5A5A5A5A, dtype=torch.int32, device="cuda")
    pk.stream_read(src, sink, key=1)
    torch.cuda.synchronize()
    assert int(sink.item()) == 0x5A5A5A5A
    pk.stream_read(src, sink, key=0)
    torch.cuda.synchronize()
    assert int(sink.item()) == 0
