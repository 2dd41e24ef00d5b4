"""The guard-band allocator of the GPU tests (conftest.GuardedAllocator),
exercised on host memory: a store one element past a tensor's end, or one
element before its start, is reported; stores inside it are not."""
import torch

from conftest import GuardedAllocator


def _raw(t):
    """The allocator's whole buffer behind tensor t."""
    return t.untyped_storage()


def test_clean_tensor_passes():
    a = GuardedAllocator()
    t = a((3, 5), torch.float32, "cpu")
    t.fill_(1.0)
    assert a.damaged() == []


def test_store_past_end_is_reported():
    a = GuardedAllocator()
    t = a((7,), torch.bfloat16, "cpu")  # 14 bytes: the band starts right after them
    whole = torch.empty(0, dtype=torch.uint8).set_(_raw(t))
    off = t.storage_offset() * t.element_size()
    whole[off + 14] = 0
    assert a.damaged() == [((7,), "torch.bfloat16", "after")]


def test_store_before_start_is_reported():
    a = GuardedAllocator()
    t = a((2, 2), torch.float32, "cpu")
    whole = torch.empty(0, dtype=torch.uint8).set_(_raw(t))
    off = t.storage_offset() * t.element_size()
    whole[off - 1] = 7
    assert a.damaged() == [((2, 2), "torch.float32", "before")]


def test_alignment_and_empty_tensor():
    a = GuardedAllocator()
    t = a((0, 4), torch.float32, "cpu")
    assert t.numel() == 0 and a.damaged() == []
    u = a((33,), torch.uint8, "cpu")
    assert (u.storage_offset() * u.element_size()) % 256 == 0
