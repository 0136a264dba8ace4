"""The guard-band allocator of the GPU tests (CPU tensors here)."""
import pytest
import torch

from guard import GUARD, PATTERN, GuardedAllocator


def test_guard_bands_detect_writes_outside_the_buffer(monkeypatch):
    monkeypatch.setattr(torch.cuda, "synchronize", lambda: None)
    a = GuardedAllocator()
    x = a((3, 5), torch.float32, "cpu")
    assert x.shape == (3, 5) and x.is_contiguous()
    # the data keeps the raw buffer's alignment (device blocks are 512-byte aligned)
    assert GUARD % 256 == 0 and x.data_ptr() - a.buffers[0][0].data_ptr() == GUARD
    x.fill_(1.0)  # writes inside the buffer leave the guards intact
    a.check()
    raw = a.buffers[0][0]
    raw[GUARD + 60] = 0  # one byte past the end
    with pytest.raises(AssertionError, match="after"):
        a.check()
    raw[GUARD + 60] = PATTERN
    raw[GUARD - 1] = 0  # one byte before the start
    with pytest.raises(AssertionError, match="before"):
        a.check()
