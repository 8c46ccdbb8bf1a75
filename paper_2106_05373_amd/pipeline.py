"""A two-layer BCPNN network on the C ABI: an unsupervised hidden layer and a supervised readout.

The hidden layer learns with the unsupervised rule of Alg. 1 (support, per-HCU softmax, traces,
weights, and structural plasticity scheduled by the caller).  The readout layer takes the hidden
activities as its input (one input HCU per hidden HCU) and has one output HCU with one MCU per
class; it learns with the same rule, its activity clamped to the one-hot label (the paper trains
the output layer "similarly", Sec. 2), over a full mask and without plasticity.  Inference is the
hidden forward pass followed by the readout's argmax of the support (Sec. 2, inference).

Every step runs in the library's kernels; this module only holds the two layers and the device
buffer of hidden activities between them.
"""
from __future__ import annotations

from typing import Optional

import numpy as np

from . import bcpnn


class Network:
    """Hidden layer + readout, both on one stream.  All tensors are CUDA float32 (int32 for the
    predictions), row-major, contiguous."""

    def __init__(self, hidden_cfg: bcpnn.Config, hidden_mask: Optional[np.ndarray],
                 n_classes: int, readout_alpha: Optional[float] = None, stream=None):
        """The readout takes the hidden layer's alpha (unless readout_alpha is given) and its
        storage format, k_B = 1 and a full mask."""
        import torch
        self.torch = torch
        self.hidden = bcpnn.Layer(hidden_cfg, hidden_mask, stream=stream)
        rc = bcpnn.default_config(hidden_cfg.out_hcu, hidden_cfg.out_mcu, 1, n_classes,
                                  hidden_cfg.max_batch,
                                  alpha=hidden_cfg.alpha if readout_alpha is None else readout_alpha,
                                  seed=hidden_cfg.seed + 1, storage=hidden_cfg.storage)
        self.readout = bcpnn.Layer(rc, None, stream=stream)
        self.n_classes = n_classes
        self.max_batch = hidden_cfg.max_batch
        self._y = torch.empty((self.max_batch, self.hidden.n_out), device="cuda",
                              dtype=torch.float32)
        self._win = torch.empty((self.max_batch, 1), device="cuda", dtype=torch.int32)

    def train_hidden(self, x):
        """One unsupervised batch of the hidden layer."""
        self.hidden.train_batch(x)

    def train_readout(self, x, target):
        """One supervised batch: hidden activities of x (no learning there), then the readout
        learns with its activity clamped to target ([B][n_classes] one-hot)."""
        B = x.shape[0]
        y = self._y[:B]
        self.hidden.forward(x, y)
        self.readout.train_batch(y, target)

    def predict(self, x, out=None):
        """Class index per sample ([B] int32, any B): the readout's argmax over the hidden
        activities, max_batch samples at a time.  With out given, the indices are written there
        and nothing is allocated."""
        torch = self.torch
        B = x.shape[0]
        if out is None:
            out = torch.empty(B, device="cuda", dtype=torch.int32)
        for k in range(0, B, self.max_batch):
            n = min(self.max_batch, B - k)
            y = self._y[:n]
            win = self._win[:n]
            self.hidden.forward(x[k:k + n], y)
            self.readout.readout(y, win)
            out[k:k + n].copy_(win[:, 0])
        return out

    def close(self):
        self.hidden.close()
        self.readout.close()
