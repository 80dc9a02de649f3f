"""Torch-facing wrapper of one class shard's PFC head step.

Allocates the step's output buffers and workspace once (torch device memory)
and calls the three C-ABI entry points on torch's current stream.  It does no
arithmetic of its own: sampling, forward, backward and the update all run in
libpfc's HIP kernels.
"""

import torch

from . import pfc as abi

DTYPES = {
    "f32": (torch.float32, abi.PFC_F32),
    "bf16": (torch.bfloat16, abi.PFC_BF16),
    "f16": (torch.float16, abi.PFC_F16),
}
MARGINS = {"cosface": abi.PFC_COSFACE, "arcface": abi.PFC_ARCFACE}


def _ptr(t):
    return 0 if t is None else t.data_ptr()


def _require(t, dtype, shape, name, device):
    if t.dtype != dtype or tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError(f"{name}: expected contiguous {dtype} {tuple(shape)}, "
                         f"got {t.dtype} {tuple(t.shape)} contiguous={t.is_contiguous()}")
    if t.device != device:
        raise ValueError(f"{name}: expected device {device}, got {t.device}")


class PfcShard:
    """One GPU's class shard [class_offset, class_offset + C) of a PFC head.

    tau: threshold of the PFC* conflict filter (a negative logit whose
    unmargined cosine exceeds tau leaves the row's denominator); None, or any
    tau >= 1, is plain PFC.
    """

    def __init__(self, B, d, C, r, dtype="bf16", class_offset=0, s=64.0, m=0.5,
                 margin="arcface", lr=0.1, mu=0.9, device="cuda:0", tau=None):
        self.B, self.d, self.C, self.r = int(B), int(d), int(C), float(r)
        self.class_offset = int(class_offset)
        self.dtype_name = dtype
        self.tdtype, self.code = DTYPES[dtype]
        self.s, self.m, self.margin = float(s), float(m), MARGINS[margin]
        self.lr, self.mu = float(lr), float(mu)
        self.tau = None if tau is None else float(tau)
        self.device = torch.device(device)
        self.ws_bytes, self.cap = abi.pfc_workspace_bytes(self.B, self.d, self.C, self.r, self.code)
        dev = self.device
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=dev)
        self.active = torch.empty(self.cap, dtype=torch.int32, device=dev)
        self.n_active = torch.empty(1, dtype=torch.int32, device=dev)
        self.labels_mapped = torch.empty(self.B, dtype=torch.int32, device=dev)
        self.loss = torch.empty(1, dtype=torch.float32, device=dev)
        self.row_lse = torch.empty(self.B, dtype=torch.float32, device=dev)
        self.dX = torch.empty((self.B, self.d), dtype=torch.float32, device=dev)

    def _stream(self):
        return torch.cuda.current_stream(self.device).cuda_stream

    def sample(self, labels, seed):
        _require(labels, torch.int64, (self.B,), "labels", self.device)
        abi.pfc_sample(_ptr(labels), self.B, self.C, self.class_offset, self.r, int(seed),
                       _ptr(self.active), self.cap, _ptr(self.n_active), _ptr(self.labels_mapped),
                       _ptr(self.ws), self.ws_bytes, self._stream())

    def forward(self, X, W):
        _require(X, self.tdtype, (self.B, self.d), "X", self.device)
        _require(W, self.tdtype, (self.C, self.d), "W", self.device)
        abi.pfc_forward_loss(_ptr(X), self.code, self.B, self.d, _ptr(W), self.code, self.C,
                             _ptr(self.active), _ptr(self.n_active), self.cap,
                             _ptr(self.labels_mapped), self.code, self.s, self.m, self.margin,
                             2.0 if self.tau is None else self.tau, _ptr(self.loss),
                             _ptr(self.row_lse), _ptr(self.ws), self.ws_bytes, self._stream())

    def backward(self, X, W, M, W_master=None, row_lse=None):
        _require(X, self.tdtype, (self.B, self.d), "X", self.device)
        _require(W, self.tdtype, (self.C, self.d), "W", self.device)
        _require(M, torch.float32, (self.C, self.d), "momentum", self.device)
        if W_master is not None:
            _require(W_master, torch.float32, (self.C, self.d), "W_master", self.device)
        lse = self.row_lse if row_lse is None else row_lse
        abi.pfc_backward_update(_ptr(X), self.code, self.B, self.d, _ptr(W), self.code,
                                _ptr(W_master), _ptr(M), self.C, _ptr(self.active),
                                _ptr(self.n_active), self.cap, _ptr(self.labels_mapped),
                                self.code, self.s, self.m, self.margin, _ptr(lse), self.lr,
                                self.mu, _ptr(self.dX), _ptr(self.ws), self.ws_bytes,
                                self._stream())

    def step(self, X, labels, W, M, seed, W_master=None):
        """Sample, forward, backward and update of one mini-batch (all enqueued)."""
        self.sample(labels, seed)
        self.forward(X, W)
        self.backward(X, W, M, W_master)
