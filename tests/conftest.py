import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# Bytes of guard band on each side of every device tensor the binding (and
# the step driver) allocates during a GPU test, filled with 0xff (a NaN in
# fp32 and bf16) and checked after the test: a kernel store past either end
# of an output, a workspace or a partial-tile buffer changes them.
GUARD = 4096


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


class GuardedAllocator:
    """Allocates each tensor inside a larger uint8 buffer: GUARD bytes of 0xff
    before it, and 0xff from its last byte to GUARD bytes past its end
    (rounded up to 256 bytes, so the tensor itself stays 256-byte aligned)."""

    def __init__(self):
        self.live = []

    def __call__(self, shape, dtype, device):
        import torch
        n = 1
        for d in shape:
            n *= int(d)
        nbytes = n * torch.empty((), dtype=dtype).element_size()
        body = (nbytes + 255) // 256 * 256
        buf = torch.empty(GUARD + body + GUARD, dtype=torch.uint8, device=device)
        buf[:GUARD].fill_(0xFF)
        buf[GUARD + nbytes:].fill_(0xFF)
        self.live.append((buf, nbytes, tuple(shape), dtype))
        return buf[GUARD:GUARD + nbytes].view(dtype).view(tuple(shape))

    def damaged(self):
        """(shape, dtype, side) of every tensor whose guard bands changed."""
        import torch
        if any(buf.is_cuda for buf, _, _, _ in self.live):
            torch.cuda.synchronize()
        bad = []
        for buf, nbytes, shape, dtype in self.live:
            if not bool((buf[:GUARD] == 0xFF).all()):
                bad.append((shape, str(dtype), "before"))
            if not bool((buf[GUARD + nbytes:] == 0xFF).all()):
                bad.append((shape, str(dtype), "after"))
        return bad


@pytest.fixture(autouse=True)
def _guard_bands(request):
    """GPU tests: every binding allocation gets guard bands, checked at the end."""
    if request.node.get_closest_marker("gpu") is None:
        yield
        return
    from paper_1603_07846_amd import singa
    alloc = GuardedAllocator()
    singa.set_allocator(alloc)
    try:
        yield alloc
    finally:
        singa.set_allocator(None)
    bad = alloc.damaged()
    alloc.live.clear()
    assert not bad, ("stores outside a tensor's bounds (guard bands changed)", bad[:10])
