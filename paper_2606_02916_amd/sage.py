"""The consumer of X_b: GraphSAGE with the mean aggregator over a window's
sampled blocks (Algorithm 1's forward pass on the assembled tensor; the
paper trains a GraphSAGE model, Sec. VI-A).  Buffers and argument
marshalling only; both kernels per layer run in libgg."""
from __future__ import annotations

import torch

from . import gg


class SageConsumer:
    """Forward pass of L GraphSAGE layers over the windows a fetch pipeline
    produces.  layers: list of (w_self [d_in, d_out], w_neigh, bias, relu)
    fp32 tensors on the device; layer 0's d_in is the feature width.
    geo: the pipeline's geometry (FetchPipeline.geo / LookaheadPipeline.geo)."""

    def __init__(self, geo, layers, x_dtype=gg.GG_F32, device=None):
        self.device = torch.device(device if device is not None else "cuda")
        if len(layers) != geo.L:
            raise ValueError(f"{len(layers)} layers for a sampling depth of {geo.L}")
        self.layers = [tuple(l) for l in layers]
        self.arr = gg.make_sage_layers(self.layers)
        self.geo = geo
        self.x_dtype = int(x_dtype)
        self.rows_cap = geo.win_cap
        self.d_out = int(self.layers[-1][0].shape[1])
        self.ws = torch.empty(gg.gg_ws_sage(geo.N, geo.W, self.rows_cap, self.arr),
                              dtype=torch.uint8, device=self.device)
        # seeds of a window: at most the window's frontier-0 capacity
        self.out_cap = geo.seed_cap
        self.out = torch.empty((self.out_cap, self.d_out), dtype=torch.float32, device=self.device)

    def forward(self, bufs, Wk, x, x_stride, status, stream=None):
        """Runs the layers for window buffers `bufs` (a pipeline's buffer set)
        of Wk batches on the gathered rows x; returns the rows of F_0 (every
        batch's distinct seeds, back to back) of the last layer.  Enqueued on
        `stream` (default: the current stream) after whatever wrote x."""
        gg.gg_sage_forward(bufs.wsample, self.geo.N, Wk, self.geo.fanout, x, self.x_dtype, x_stride,
                           self.rows_cap, self.arr, self.out, self.out_cap, status, self.ws,
                           stream=stream)
        return self.out
