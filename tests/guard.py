"""Guard bands around every buffer the library writes in the GPU tests.

Each output and workspace the binding allocates is carved from a larger
buffer: GUARD bytes before and after it, and the buffer itself, are filled
with a fixed byte pattern before the call.  A kernel that writes before the
start or past the end of an exactly sized output changes a guard byte;
check() finds it.  The data region starts with the pattern too, so an output
element the library never writes keeps a recognisable value instead of
whatever the allocator held."""
import torch

GUARD = 4096   # bytes on each side; a multiple of the workspace alignment
PATTERN = 0xA5


class GuardedAllocator:
    def __init__(self):
        self.buffers = []  # (raw uint8 tensor, data bytes, shape, dtype)

    def __call__(self, shape, dtype, device):
        n = 1
        for s in shape:
            n *= int(s)
        nbytes = n * torch.empty((), dtype=dtype).element_size()
        raw = torch.full((nbytes + 2 * GUARD,), PATTERN, dtype=torch.uint8, device=device)
        data = raw[GUARD:GUARD + nbytes].view(dtype).view(shape)
        self.buffers.append((raw, nbytes, tuple(shape), dtype))
        return data

    def check(self):
        """Raise if any guard byte of any buffer allocated so far changed."""
        if not self.buffers:
            return
        torch.cuda.synchronize()
        for raw, nbytes, shape, dtype in self.buffers:
            head = raw[:GUARD]
            tail = raw[GUARD + nbytes:]
            bad_head = int((head != PATTERN).sum())
            bad_tail = int((tail != PATTERN).sum())
            assert bad_head == 0 and bad_tail == 0, (
                f"guard band overwritten around a {dtype} buffer of shape {shape}: "
                f"{bad_head} bytes before it, {bad_tail} bytes after it")
