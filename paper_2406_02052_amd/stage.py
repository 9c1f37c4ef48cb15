"""Owner of one stage's device buffers (torch tensors) around the C ABI.

Marshalling only: it allocates the caller-owned buffers the library asks for,
packs parameter tensors into the library's flat layout (reported by
petra_stage_param_info) and forwards calls.  No arithmetic of the method runs
here.
"""
from __future__ import annotations

from typing import List, Sequence

import numpy as np

from . import _lib as L


class Stage:
    def __init__(self, n: int, h: int, w: int, c_half: int, num_blocks: int,
                 kind: str = "basic", dtype: str = "bf16", c_mid: int = 0,
                 bn_eps: float = 1e-5, bn_momentum: float = 0.1, device: str = "cuda"):
        import torch
        self.torch = torch
        self.shape = (n, h, w, c_half)
        self.dtype = dtype
        self.tdtype = torch.bfloat16 if dtype == "bf16" else torch.float32
        self.device = device
        desc = L.StageDesc(n, h, w, c_half, c_mid, num_blocks,
                           L.PETRA_BLOCK_BASIC if kind == "basic" else L.PETRA_BLOCK_BOTTLENECK,
                           L.PETRA_BF16 if dtype == "bf16" else L.PETRA_FP32,
                           bn_eps, bn_momentum)
        self.handle = L.petra_stage_create(desc)
        self.n_params, self.n_tensors, self.n_bn, self.ws_bytes = L.petra_stage_query(self.handle)
        self.infos = [L.petra_stage_param_info(self.handle, i) for i in range(self.n_tensors)]
        f32 = dict(dtype=torch.float32, device=device)
        self.params = torch.zeros(self.n_params, **f32)
        self.grad = torch.zeros(self.n_params, **f32)
        self.mom = torch.zeros(self.n_params, **f32)
        self.run_mean = torch.zeros(self.n_bn, **f32)
        self.run_var = torch.ones(self.n_bn, **f32)
        self.workspace = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device=device)
        ws_ptr = (self.workspace.data_ptr() + 255) // 256 * 256
        L.petra_stage_bind(self.handle, self.params, self.grad, self.mom, self.run_mean,
                           self.run_var, ws_ptr, self.ws_bytes)

    def __del__(self):
        h = getattr(self, "handle", None)
        if h:
            try:
                L.petra_stage_destroy(h)
            except Exception:
                pass
            self.handle = None

    # -- parameters in canonical order ---------------------------------------
    def shapes(self) -> List[tuple]:
        return [tuple(i.shape[:i.ndim]) for i in self.infos]

    def set_params(self, tensors: Sequence[np.ndarray], stream=None) -> None:
        flat = np.zeros(self.n_params, np.float32)
        for info, t in zip(self.infos, tensors, strict=True):
            t = np.asarray(t, np.float32)
            assert t.shape == tuple(info.shape[:info.ndim]), (t.shape, tuple(info.shape[:info.ndim]))
            flat[info.offset:info.offset + info.numel] = t.reshape(-1)
        self.params.copy_(self.torch.from_numpy(flat))
        L.petra_stage_sync_weights(self.handle, stream)

    def _unflatten(self, buf) -> List[np.ndarray]:
        host = buf.detach().cpu().numpy()
        return [host[i.offset:i.offset + i.numel].reshape(tuple(i.shape[:i.ndim])).copy()
                for i in self.infos]

    def get_params(self) -> List[np.ndarray]:
        return self._unflatten(self.params)

    def get_grads(self) -> List[np.ndarray]:
        return self._unflatten(self.grad)

    def get_momentum(self) -> List[np.ndarray]:
        return self._unflatten(self.mom)

    def set_graphs(self, enable: bool) -> None:
        L.petra_stage_set_graphs(self.handle, enable)

    def set_streams(self, n: int) -> None:
        L.petra_stage_set_streams(self.handle, n)

    def set_optimizer(self, lr=0.1, momentum=0.9, weight_decay=0.0, nesterov=True, accum_k=1):
        L.petra_stage_set_optimizer(self.handle, L.Sgd(lr, momentum, weight_decay,
                                                      1 if nesterov else 0, accum_k))

    # -- activations ----------------------------------------------------------
    def act(self, a: np.ndarray | None = None):
        """A device half-tensor of this stage's storage type ([N,H,W,C/2])."""
        if a is None:
            return self.torch.empty(self.shape, dtype=self.tdtype, device=self.device)
        t = self.torch.from_numpy(np.ascontiguousarray(a, np.float32))
        return t.to(device=self.device).to(self.tdtype).contiguous()

    def forward(self, x1, x2, y1, y2, stream=None):
        L.petra_stage_forward(self.handle, x1, x2, y1, y2, stream)

    def reconstruct_backward(self, y1, y2, dy1, dy2, x1, x2, dx1, dx2, stream=None):
        L.petra_stage_reconstruct_backward(self.handle, y1, y2, dy1, dy2, x1, x2, dx1, dx2, stream)

    def update(self, stream=None) -> bool:
        return L.petra_stage_update(self.handle, stream)

    def step(self, x1, x2, y1, y2, yb1, yb2, dyb1, dyb2, xb1, xb2, dxb1, dxb2, stream=None) -> bool:
        return L.petra_stage_step(self.handle, x1, x2, y1, y2, yb1, yb2, dyb1, dyb2, xb1, xb2,
                                  dxb1, dxb2, stream)


def to_host(t) -> np.ndarray:
    return t.detach().float().cpu().numpy()


class Net:
    """Owner of a multi-stage schedule's device buffers (marshalling only)."""

    def __init__(self, n: int, h: int, w: int, c_img: int, widths, blocks_per_stage: int,
                 classes: int, dtype: str = "bf16", bn_eps: float = 1e-5,
                 bn_momentum: float = 0.1, device: str = "cuda", input_buffer: bool = False,
                 param_buffer: bool = False, split_stages: bool = False):
        import torch
        self.torch = torch
        self.device = device
        self.dtype = dtype
        self.tdtype = torch.bfloat16 if dtype == "bf16" else torch.float32
        self.img_shape = (n, h, w, c_img)
        self.widths = tuple(widths)
        ws = (ctypes_int_array(widths))
        desc = L.NetDesc(n, h, w, c_img, len(widths), ws, blocks_per_stage, classes,
                         L.PETRA_BF16 if dtype == "bf16" else L.PETRA_FP32, bn_eps, bn_momentum,
                         int(input_buffer), int(param_buffer), int(split_stages))
        self.handle = L.petra_net_create(desc)
        self.n_stages = L.petra_net_num_stages(self.handle)
        self.n_params, self.n_tensors, self.n_bn, self.ws_bytes = L.petra_net_query(self.handle)
        self.infos = [L.petra_net_param_info(self.handle, i) for i in range(self.n_tensors)]
        f32 = dict(dtype=torch.float32, device=device)
        self.params = torch.zeros(self.n_params, **f32)
        self.grad = torch.zeros(self.n_params, **f32)
        self.mom = torch.zeros(self.n_params, **f32)
        self.run_mean = torch.zeros(self.n_bn, **f32)
        self.run_var = torch.ones(self.n_bn, **f32)
        self.workspace = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device=device)
        ws_ptr = (self.workspace.data_ptr() + 255) // 256 * 256
        L.petra_net_bind(self.handle, self.params, self.grad, self.mom, self.run_mean,
                         self.run_var, ws_ptr, self.ws_bytes)
        self.loss = torch.zeros(1, **f32)

    def __del__(self):
        h = getattr(self, "handle", None)
        if h:
            try:
                L.petra_net_destroy(h)
            except Exception:
                pass
            self.handle = None

    def set_params(self, tensors, stream=None) -> None:
        flat = np.zeros(self.n_params, np.float32)
        for info, t in zip(self.infos, tensors, strict=True):
            t = np.asarray(t, np.float32)
            assert t.shape == tuple(info.shape[:info.ndim]), (t.shape, tuple(info.shape[:info.ndim]))
            flat[info.offset:info.offset + info.numel] = t.reshape(-1)
        self.params.copy_(self.torch.from_numpy(flat))
        L.petra_net_sync_weights(self.handle, stream)

    def _unflatten(self, buf):
        host = buf.detach().cpu().numpy()
        return [host[i.offset:i.offset + i.numel].reshape(tuple(i.shape[:i.ndim])).copy()
                for i in self.infos]

    def get_params(self):
        return self._unflatten(self.params)

    def get_momentum(self):
        return self._unflatten(self.mom)

    def get_grads(self):
        return self._unflatten(self.grad)

    def set_optimizer(self, lr=0.1, momentum=0.9, weight_decay=0.0, nesterov=True, accum_k=1):
        L.petra_net_set_optimizer(self.handle, L.Sgd(lr, momentum, weight_decay,
                                                    1 if nesterov else 0, accum_k))

    def images(self, a):
        t = self.torch.from_numpy(np.ascontiguousarray(a, np.float32))
        return t.to(device=self.device).to(self.tdtype).contiguous()

    def labels(self, a):
        return self.torch.from_numpy(np.ascontiguousarray(a, np.int32)).to(self.device)

    def tick(self, images=None, labels=None, stream=None) -> bool:
        return L.petra_net_tick(self.handle, images, labels, self.loss, stream)

    def drain(self, stream=None):
        """Ticks without input until nothing is in flight.  Returns the device
        fp32 losses of the micro-batches that reached the head meanwhile."""
        out = self.torch.zeros(max(self.n_stages, 4), dtype=self.torch.float32, device=self.device)
        nl, _ = L.petra_net_drain(self.handle, out, stream)
        return out[:nl]

    def backprop_step(self, images, labels, stream=None) -> None:
        """Reversible backpropagation of one micro-batch (no pipelining); the
        loss lands in self.loss."""
        L.petra_net_backprop_step(self.handle, images, labels, self.loss, stream)

    def state(self):
        return L.petra_net_state(self.handle)

    def set_backward(self, mode: int) -> None:
        L.petra_net_set_backward(self.handle, mode)

    def stage_spans(self):
        return [L.petra_net_stage_params(self.handle, j) for j in range(self.n_stages)]

    def probe_tick(self, mode: int, stream=None):
        """Unscaled gradients the next tick's backward passes would produce in
        variant `mode` (device fp32 [n_params]); nothing else changes."""
        out = self.torch.empty(self.n_params, dtype=self.torch.float32, device=self.device)
        L.petra_net_probe_tick(self.handle, mode, out, stream)
        return out

    def probe_backprop(self, images, labels, stream=None):
        """End-to-end gradient of one micro-batch at the current parameters."""
        out = self.torch.empty(self.n_params, dtype=self.torch.float32, device=self.device)
        L.petra_net_probe_backprop(self.handle, images, labels, out, stream)
        return out


def ctypes_int_array(vals):
    import ctypes
    arr = (ctypes.c_int32 * L.MAX_STAGES)()
    for i, v in enumerate(vals):
        arr[i] = int(v)
    return arr
