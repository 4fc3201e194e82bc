"""Guarded device buffers for the GPU tests: every output and workspace is
a view into a larger allocation whose margins hold a canary pattern, and
whose interior starts poisoned, so a write past either end or an output the
library never writes is caught."""
import torch

MARGIN_BYTES = 256
CANARY_BYTE = 0xA5


class Guards:
    def __init__(self, device="cuda"):
        self.device = device
        self.bufs = []

    def empty(self, shape, dtype, poison=None):
        """A contiguous tensor of `shape` inside a canaried allocation (256-byte
        margins keep the view 256-byte aligned)."""
        if isinstance(shape, int):
            shape = (shape,)
        n = 1
        for s in shape:
            n *= int(s)
        item = torch.empty(0, dtype=dtype).element_size()
        nbytes = max(n * item, 1)
        raw = torch.full((MARGIN_BYTES + nbytes + MARGIN_BYTES,), CANARY_BYTE, dtype=torch.uint8,
                         device=self.device)
        inner = raw[MARGIN_BYTES:MARGIN_BYTES + n * item]
        view = inner.view(dtype).view(shape) if n else torch.empty(shape, dtype=dtype,
                                                                   device=self.device)
        if poison is not None and n:
            view.fill_(poison)
        self.bufs.append((raw, nbytes))
        return view

    def workspace(self, nbytes):
        return self.empty(max(int(nbytes), 1), torch.uint8)

    def check(self):
        torch.cuda.synchronize()
        for raw, nbytes in self.bufs:
            head = raw[:MARGIN_BYTES]
            tail = raw[MARGIN_BYTES + nbytes:]
            assert bool(torch.all(head == CANARY_BYTE)), "write before the start of a buffer"
            assert bool(torch.all(tail == CANARY_BYTE)), "write past the end of a buffer"
