"""Stacked-layer decode: L sparse-FFN layers chained by pre-norm residuals,

    u_l = bf16(RMSNorm(x_l))   (eps 1e-5, norm weight 1)
    x_{l+1} = x_l + FFN_l(u_l)  (fp32 residual stream)

as in the 32-layer LLaMA-3-8B-shaped decode workload.  This module only
allocates the buffers and enqueues the C-ABI calls (prunepath_residual_rmsnorm,
prunepath_ffn_decode) on one stream; every step of the computation runs in the
HIP library.  One step can be captured once in a HIP graph and replayed.

Buffers kept per layer (so that each layer can be checked on its own):
  xs  [L+1, T, d] fp32   residual entering layer l (xs[L] = step output)
  us  [L, T, d]   bf16   normalised layer inputs
  ys  [L, T, d]   fp32   FFN outputs
  idx [L, T, E], cnt [L, T]  selections
"""
from . import _lib as pp


class DecodeStack:
    def __init__(self, handles, d, E, T, tau, eps=1e-5):
        import torch
        self.handles = list(handles)
        self.L = len(self.handles)
        self.d, self.E, self.T, self.tau, self.eps = d, E, T, float(tau), float(eps)
        dev = "cuda"
        self.x_in = torch.zeros((T, d), dtype=torch.float32, device=dev)
        self.xs = torch.zeros((self.L + 1, T, d), dtype=torch.float32, device=dev)
        self.us = torch.zeros((self.L, T, d), dtype=torch.int16, device=dev)
        self.ys = torch.zeros((self.L, T, d), dtype=torch.float32, device=dev)
        self.idx = torch.zeros((self.L, T, E), dtype=torch.int32, device=dev)
        self.cnt = torch.zeros((self.L, T), dtype=torch.int32, device=dev)
        self.graph = None

    def set_input(self, x0):
        """x0: [T, d] fp32 tensor (any device) -> the first residual."""
        self.x_in.copy_(x0)

    def enqueue(self, stream=None):
        """Enqueue one step (all L layers) on `stream` (default: current)."""
        T, d = self.T, self.d
        pp.prunepath_residual_rmsnorm(self.x_in, None, self.xs[0], T, d, self.eps, self.us[0],
                                      stream=stream)
        for l, h in enumerate(self.handles):
            pp.prunepath_ffn_decode(h, self.us[l], T, self.tau, None, self.ys[l], self.idx[l],
                                    self.cnt[l], stream=stream)
            nxt = self.us[l + 1] if l + 1 < self.L else None
            pp.prunepath_residual_rmsnorm(self.xs[l], self.ys[l], self.xs[l + 1], T, d, self.eps,
                                          nxt, stream=stream)

    def capture(self):
        """Capture one step in a HIP graph (call after an eager warm-up step)."""
        import torch
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            self.enqueue()
        self.graph = g
        return g

    def replay(self):
        self.graph.replay()

    @property
    def output(self):
        return self.xs[self.L]
