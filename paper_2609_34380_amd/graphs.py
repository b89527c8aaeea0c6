"""A captured HIP graph per (batch size, precision mode) of a decode step
(Sec. IV-C, "Granularity of the precision switch": two pre-captured graphs
per supported batch size, one with upper-byte-only kernels and one with
upper-byte + residual kernels; the dispatcher picks exactly one per forward
pass, so a mode change takes effect between passes and every layer of a pass
runs in the same mode).

PyTorch supplies the graph objects (hipStreamBeginCapture / hipGraphLaunch
underneath); every kernel in them is a libdps kernel launched by the step
function.  The step must read and write only buffers that outlive the graphs
(static inputs, outputs and workspace), as any captured work does.
"""
import torch

from . import dps


class ModeGraphs:
    """graphs[(m, mode)] for every m in batch_sizes and mode in (fast, full).

    step(m, mode) enqueues one forward pass of batch m on the current stream.
    capture() runs each pass once eagerly (loading kernels), then captures it
    on `stream`; replay(m, mode) launches the matching graph on that stream.
    """

    MODES = (dps.MODE_FAST, dps.MODE_FULL)

    def __init__(self, step, batch_sizes, stream=None):
        self.step = step
        self.batch_sizes = tuple(batch_sizes)
        self.stream = stream if stream is not None else torch.cuda.Stream()
        self.graphs = {}

    def capture(self):
        with torch.cuda.stream(self.stream):
            for m in self.batch_sizes:
                for mode in self.MODES:
                    self.step(m, mode)
        self.stream.synchronize()
        for m in self.batch_sizes:
            for mode in self.MODES:
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=self.stream):
                    self.step(m, mode)
                self.graphs[(m, mode)] = g
        torch.cuda.synchronize()
        return self

    def replay(self, m, mode):
        """Launch the pass of batch m in `mode` (dps.MODE_FAST or MODE_FULL,
        e.g. a SumManager's current mode) on this object's stream."""
        g = self.graphs.get((m, mode))
        if g is None:
            raise KeyError("no graph captured for batch %r in mode %r" % (m, mode))
        with torch.cuda.stream(self.stream):
            g.replay()
