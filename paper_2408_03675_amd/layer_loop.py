"""Layer-by-layer eviction (Algorithm 1, encoding phase: every layer's cache is
evicted once, layer after layer; Section 1 and Section 5).

Each layer ell gets its own score -> select -> compact through nacl_evict,
with the Philox layer index ell.  Consecutive layers alternate between
`streams` HIP streams of default priority, each with its own workspace, so
one layer's selection and compaction overlap the next layer's scoring.
Launch plumbing only: every step runs in the library's kernels.
"""

import torch

from . import nacl


class LayerLoop:
    """Evicts a list of layers back to back.

    prob: the nacl.Problem shared by every layer (same shapes and strides).
    data: per layer (q, k, v).  C, Cr, sampling, seed: the budget and draw.
    The outputs of layer ell are outs[ell] = (scores, keep_idx, k_out, v_out),
    allocated once here and overwritten by every run()."""

    def __init__(self, prob, data, C, Cr, sampling=nacl.SAMPLE_SOFTMAX, seed=0, streams=2, device=None):
        self.prob, self.data = prob, data
        self.C, self.Cr, self.sampling, self.seed = int(C), int(Cr), int(sampling), int(seed)
        dev = device if device is not None else data[0][1].device
        self.device = dev
        n = max(1, int(streams))
        self.streams = [torch.cuda.Stream(dev) for _ in range(n)]  # default priority
        self.workspaces = [nacl.workspace(prob, dev) for _ in range(n)]
        B, H, L, D = prob.B, prob.H, prob.L, prob.D
        dt = prob.torch_dtype
        self.outs = [(torch.empty((B, H, L), dtype=torch.float32, device=dev),
                      torch.empty((B, H, self.C), dtype=torch.int32, device=dev),
                      torch.empty((B, H, self.C, D), dtype=dt, device=dev),
                      torch.empty((B, H, self.C, D), dtype=dt, device=dev)) for _ in data]

    def run(self):
        """Enqueues every layer's eviction after the current stream's work;
        the current stream waits for all of them."""
        cur = torch.cuda.current_stream(self.device)
        for s in self.streams:
            s.wait_stream(cur)
        n = len(self.streams)
        for ell, (q, k, v) in enumerate(self.data):
            with torch.cuda.stream(self.streams[ell % n]):
                F, keep, ko, vo = self.outs[ell]
                nacl.evict(self.prob, q, k, v, self.C, self.Cr, self.sampling, self.seed, ell,
                           ws=self.workspaces[ell % n], scores=F, keep_idx=keep, k_out=ko, v_out=vo)
        for s in self.streams:
            cur.wait_stream(s)

    def health(self):
        """OR of the sticky health words of every workspace (0: every call
        since construction completed normally).  Waits for the streams."""
        h = 0
        for ws in self.workspaces:
            h |= nacl.health(ws)[1]
        return h
