"""The fully-connected head and loss driven through the C ABI.

Section III-A: three fully-connected layers follow the convolutions, each
with leaky ReLU, the last with three outputs (the cosmological parameters
Omega_M, sigma_8 and n_s).  The first layer reads each sample's NDHWC
activation flattened in memory order.  The loss is read as the mean squared
error of the three outputs over the batch.

  forward   layer 1..3:  fc -> bias + leaky ReLU;  then the loss
  backward  loss gradient; layer 3..1: leaky-ReLU backward (+ bias grad)
            -> weight grad -> data grad (layer 1's data grad is the gradient
            of the convolution stack's output)

Every step is one ``binding`` call (a HIP kernel); PyTorch allocates the
buffers once and supplies the stream.  ``step`` runs forward, loss and
backward through one cf_fc_head call (four launches) where the widths allow
it, with the same outputs.
"""
from __future__ import annotations

import torch

from . import binding as B


def _t(dtype):
    return torch.bfloat16 if dtype == "bf16" else torch.float32


class FCHead:
    def __init__(self, batch, features, widths=(128, 64, 3), dtype="f32", alpha=0.01, device="cuda"):
        self.m = batch
        self.dims = [features, *widths]
        self.dtype = dtype
        self.alpha = alpha
        t = _t(dtype)
        dev = device
        L = len(widths)
        self.w = [torch.zeros((self.dims[i], self.dims[i + 1]), dtype=t, device=dev) for i in range(L)]
        self.b = [torch.zeros(self.dims[i + 1], dtype=torch.float32, device=dev) for i in range(L)]
        self.y = [torch.empty((batch, self.dims[i + 1]), dtype=t, device=dev) for i in range(L)]
        self.dz = [torch.empty((batch, self.dims[i + 1]), dtype=t, device=dev) for i in range(L)]
        self.dx = [torch.empty((batch, self.dims[i]), dtype=t, device=dev) for i in range(L)]
        self.dw = [torch.empty((self.dims[i], self.dims[i + 1]), dtype=torch.float32, device=dev) for i in range(L)]
        self.db = [torch.empty(self.dims[i + 1], dtype=torch.float32, device=dev) for i in range(L)]
        self.target = torch.zeros((batch, widths[-1]), dtype=torch.float32, device=dev)
        self.loss = torch.zeros(4, dtype=torch.float32, device=dev)
        ws = max(B.cf_fc_fwd_workspace_size(batch, self.dims[i], self.dims[i + 1]) for i in range(L))
        ws = max(ws, max(B.cf_bias_lrelu_bwd_workspace_size(batch, self.dims[i + 1]) for i in range(L)))
        self.fused = B.cf_fc_head_workspace_size(batch, self.dims) > 0 and self._fused_fits()
        if self.fused:
            ws = max(ws, B.cf_fc_head_workspace_size(batch, self.dims))
        self.ws = torch.empty(max(ws, 16), dtype=torch.uint8, device=dev)
        self.x = None

    def set_params(self, weights, biases, target):
        for i, (w, b) in enumerate(zip(weights, biases)):
            self.w[i].copy_(torch.as_tensor(w, dtype=torch.float32).to(self.w[i].dtype))
            self.b[i].copy_(torch.as_tensor(b, dtype=torch.float32))
        self.target.copy_(torch.as_tensor(target, dtype=torch.float32))

    def forward(self, x, stream=None):
        """x: the stack's output [batch, ...] (contiguous, dtype of the head).
        Returns the device loss tensor (one fp32 in element 0)."""
        assert x.is_contiguous() and x.numel() == self.m * self.dims[0] and x.dtype == self.w[0].dtype
        self.x = x
        h = x
        for i in range(len(self.w)):
            k, n = self.dims[i], self.dims[i + 1]
            B.cf_fc_fwd(self.m, k, n, self.dtype, h, self.w[i], self.y[i], self.ws, stream=stream)
            B.cf_bias_lrelu_fwd(self.m, n, self.dtype, self.y[i], self.b[i], self.alpha, self.y[i], stream=stream)
            h = self.y[i]
        B.cf_mse_loss(self.m, self.dims[-1], self.dtype, h, self.target, self.loss, self.dz[-1], stream=stream)
        return self.loss

    def backward(self, stream=None):
        """Gradient of the loss: fills dw, db of every layer and returns the
        gradient of the head's input (shape [batch, features])."""
        g = self.dz[-1]  # dL/d(output) from the loss call
        for i in range(len(self.w) - 1, -1, -1):
            k, n = self.dims[i], self.dims[i + 1]
            B.cf_bias_lrelu_bwd(self.m, n, self.dtype, g, self.y[i], self.alpha, self.dz[i], self.db[i], self.ws,
                                stream=stream)
            xin = self.x if i == 0 else self.y[i - 1]
            B.cf_fc_bwd_weight(self.m, k, n, self.dtype, xin, self.dz[i], self.dw[i], stream=stream)
            B.cf_fc_bwd_data(self.m, k, n, self.dtype, self.dz[i], self.w[i], self.dx[i], stream=stream)
            g = self.dx[i]
        return self.dx[0]

    def _fused_fits(self):
        """The limits of cf_fc_head (checked again by the library)."""
        d, m = self.dims, self.m
        v = 8 if self.dtype == "bf16" else 4
        g = d[1] // v
        return (2 <= len(d) - 1 <= 4 and 1 <= m <= 8 and d[0] % 8 == 0 and d[1] % v == 0 and g in (8, 16, 32, 64)
                and all(1 <= n <= 512 for n in d[1:]) and m * sum(d[1:]) <= 8192
                and sum(d[i] * (d[i + 1] + 1) for i in range(1, len(d) - 1)) <= 16384)

    def step(self, x, stream=None):
        """Forward, loss and backward in one cf_fc_head call: fills y, dz, dx,
        dw, db of every layer and the loss (dz of the last layer holds dL/dz,
        not the loss gradient); returns the gradient of the head's input.
        Falls back to forward() + backward() when the widths are outside the
        fused call's limits."""
        if not self.fused:
            self.forward(x, stream)
            return self.backward(stream)
        assert x.is_contiguous() and x.numel() == self.m * self.dims[0] and x.dtype == self.w[0].dtype
        self.x = x
        B.cf_fc_head(self.m, self.dims, self.dtype, x, self.w, self.b, self.alpha, self.target, self.y, self.dz,
                     self.dx, self.dw, self.db, self.loss, self.ws, stream=stream)
        return self.dx[0]

    def weight_bytes(self):
        """Algorithmic HBM bytes of one forward + backward: every W read twice
        (forward, backward data), every dW written once in fp32."""
        es = 2 if self.dtype == "bf16" else 4
        return sum(self.dims[i] * self.dims[i + 1] * (2 * es + 4) for i in range(len(self.w)))
