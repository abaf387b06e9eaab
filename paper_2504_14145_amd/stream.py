"""Chunked evaluation of a stream of candidate batches on two HIP streams.

Candidates that do not fit on the device at once (the 16 x 64-rank large
configuration holds about 70 KB of orders per candidate) are handed over in
chunks of host memory.  Two device buffers alternate: while the compute
stream simulates chunk k from one buffer (dip_sim_evaluate, then
dip_sim_argmin folding into one key with the chunk's global index base), the
copy stream fills the other buffer with chunk k + 1.  Events order each copy
after the simulation that last read its buffer, and each simulation after its
copy.  Only argument marshalling and stream ordering happen here; the work
runs in the library's kernels.
"""
from __future__ import annotations

from . import argmin, evaluate


class ChunkStream:
    """Double-buffered chunk evaluation for one Sim handle.

    ``chunk`` is the largest chunk size; ``keep_outputs`` copies every chunk's
    outputs back to pinned host tensors (for checking), otherwise only the
    argmin key is kept.
    """

    def __init__(self, sim, chunk: int, keep_outputs: bool = False):
        import torch
        self.torch = torch
        self.sim = sim
        self.chunk = int(chunk)
        dev = torch.device("cuda", torch.cuda.current_device())
        self.copy_stream = torch.cuda.Stream(device=dev)
        self.compute_stream = torch.cuda.Stream(device=dev)
        self.bufs = [torch.empty((self.chunk, sim.stride), dtype=torch.int16, device=dev)
                     for _ in range(2)]
        self.outs = [sim.outputs(self.chunk, dev) for _ in range(2)]
        self.copied = [torch.cuda.Event() for _ in range(2)]
        self.computed = [torch.cuda.Event() for _ in range(2)]
        self.key = torch.full((1,), -1, dtype=torch.int64, device=dev)
        self.keep_outputs = keep_outputs
        self.host_outs = []
        self.k = 0
        torch.cuda.current_stream(dev).synchronize()   # the key's fill, before any argmin

    def submit(self, host_orders, index_base: int):
        """Enqueue one chunk: ``host_orders`` is a pinned int16 CPU tensor
        [n, stride] (n <= chunk) whose first candidate has global index
        ``index_base``.  Returns immediately; the host tensor must stay
        unchanged until finish()."""
        torch = self.torch
        n = int(host_orders.shape[0])
        assert 0 < n <= self.chunk and host_orders.is_pinned()
        b = self.k % 2
        with torch.cuda.stream(self.copy_stream):
            if self.k >= 2:
                self.copy_stream.wait_event(self.computed[b])
            self.bufs[b][:n].copy_(host_orders, non_blocking=True)
            self.copied[b].record(self.copy_stream)
        cs = self.compute_stream
        cs.wait_event(self.copied[b])
        out = tuple(t[:n] for t in self.outs[b])
        send = self.sim.costs if not self.sim._costs_sent else None
        evaluate(self.sim.h, send, self.bufs[b][:n], n, *out, stream=cs)
        self.sim._costs_sent = True
        argmin(self.sim.h, out[0], out[3], n, index_base, self.key, stream=cs)
        if self.keep_outputs:
            with torch.cuda.stream(cs):
                host = tuple(torch.empty(t.shape, dtype=t.dtype, pin_memory=True) for t in out)
                for h, t in zip(host, out):
                    h.copy_(t, non_blocking=True)
            self.host_outs.append((index_base, host))
        self.computed[b].record(cs)
        self.k += 1

    def finish(self):
        """Wait for every chunk; returns the folded argmin key (device tensor)."""
        self.compute_stream.synchronize()
        self.copy_stream.synchronize()
        return self.key
