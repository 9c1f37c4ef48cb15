"""ctypes binding of libpetra.so (argument marshalling only).

Every function named petra_* here calls the C entry point of the same name
declared in include/petra.h; all arithmetic runs in the library's HIP kernels.
PyTorch is used only to own device memory and to supply the current stream.
If the library is missing the import fails loudly: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libpetra.so")

PETRA_FP32, PETRA_BF16 = 0, 1
PETRA_BLOCK_BASIC, PETRA_BLOCK_BOTTLENECK = 0, 1
ROLE_CONV_WEIGHT, ROLE_BN_GAMMA, ROLE_BN_BETA, ROLE_FC_WEIGHT, ROLE_FC_BIAS = range(5)
STATUS = ["PETRA_OK", "PETRA_ERR_INVALID_ARG", "PETRA_ERR_SHAPE", "PETRA_ERR_DTYPE",
          "PETRA_ERR_ALIGN", "PETRA_ERR_WORKSPACE", "PETRA_ERR_STATE", "PETRA_ERR_HIP",
          "PETRA_ERR_ALIAS"]


class PetraError(RuntimeError):
    def __init__(self, status: int, func: str, msg: str):
        name = STATUS[status] if 0 <= status < len(STATUS) else str(status)
        super().__init__(f"{func} -> {name}: {msg}")
        self.status = status
        self.name = name


class StageDesc(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("h", ctypes.c_int32), ("w", ctypes.c_int32),
                ("c_half", ctypes.c_int32), ("c_mid", ctypes.c_int32),
                ("num_blocks", ctypes.c_int32), ("kind", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("bn_eps", ctypes.c_float),
                ("bn_momentum", ctypes.c_float)]


class Sgd(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("momentum", ctypes.c_float),
                ("weight_decay", ctypes.c_float), ("nesterov", ctypes.c_int32),
                ("accum_k", ctypes.c_int32)]


class ParamInfo(ctypes.Structure):
    _fields_ = [("offset", ctypes.c_int64), ("numel", ctypes.c_int64), ("role", ctypes.c_int32),
                ("ndim", ctypes.c_int32), ("shape", ctypes.c_int32 * 4),
                ("weight_decay", ctypes.c_int32), ("bn_index", ctypes.c_int32)]


MAX_STAGES = 8


class NetDesc(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("h", ctypes.c_int32), ("w", ctypes.c_int32),
                ("c_img", ctypes.c_int32), ("num_stages", ctypes.c_int32),
                ("widths", ctypes.c_int32 * MAX_STAGES), ("blocks_per_stage", ctypes.c_int32),
                ("classes", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("bn_eps", ctypes.c_float), ("bn_momentum", ctypes.c_float),
                ("input_buffer", ctypes.c_int32), ("param_buffer", ctypes.c_int32),
                ("split_stages", ctypes.c_int32)]


class NetMem(ctypes.Structure):
    _fields_ = [("params", ctypes.c_int64), ("weight_copies", ctypes.c_int64),
                ("activation_buffer", ctypes.c_int64), ("input_buffer", ctypes.c_int64),
                ("param_buffer", ctypes.c_int64), ("scratch", ctypes.c_int64),
                ("total", ctypes.c_int64)]


# petra_bwd_mode
BWD_RECONSTRUCT, BWD_INPUT_BUFFER, BWD_PARAM_BUFFER, BWD_DELAYED = 0, 1, 2, 3

_VP = ctypes.c_void_p
_SIGS = {
    "petra_status_str": (ctypes.c_char_p, [ctypes.c_int]),
    "petra_last_error": (ctypes.c_char_p, []),
    "petra_stage_create": (ctypes.c_int, [ctypes.POINTER(StageDesc), ctypes.POINTER(_VP)]),
    "petra_stage_destroy": (ctypes.c_int, [_VP]),
    "petra_stage_query": (ctypes.c_int, [_VP, ctypes.POINTER(ctypes.c_int64),
                                          ctypes.POINTER(ctypes.c_int32),
                                          ctypes.POINTER(ctypes.c_int64),
                                          ctypes.POINTER(ctypes.c_size_t)]),
    "petra_stage_param_info": (ctypes.c_int, [_VP, ctypes.c_int32, ctypes.POINTER(ParamInfo)]),
    "petra_stage_bind": (ctypes.c_int, [_VP, _VP, _VP, _VP, _VP, _VP, _VP, ctypes.c_size_t]),
    "petra_stage_set_optimizer": (ctypes.c_int, [_VP, ctypes.POINTER(Sgd)]),
    "petra_stage_sync_weights": (ctypes.c_int, [_VP, _VP]),
    "petra_stage_set_graphs": (ctypes.c_int, [_VP, ctypes.c_int32]),
    "petra_stage_set_streams": (ctypes.c_int, [_VP, ctypes.c_int32]),
    "petra_stage_forward": (ctypes.c_int, [_VP, _VP, _VP, _VP, _VP, _VP]),
    "petra_stage_reconstruct_backward": (ctypes.c_int, [_VP] * 10),
    "petra_stage_update": (ctypes.c_int, [_VP, _VP, ctypes.POINTER(ctypes.c_int32)]),
    "petra_stage_step": (ctypes.c_int, [_VP] * 14 + [ctypes.POINTER(ctypes.c_int32)]),
    "petra_net_create": (ctypes.c_int, [ctypes.POINTER(NetDesc), ctypes.POINTER(_VP)]),
    "petra_net_destroy": (ctypes.c_int, [_VP]),
    "petra_net_num_stages": (ctypes.c_int, [_VP, ctypes.POINTER(ctypes.c_int32)]),
    "petra_net_query": (ctypes.c_int, [_VP, ctypes.POINTER(ctypes.c_int64),
                                        ctypes.POINTER(ctypes.c_int32),
                                        ctypes.POINTER(ctypes.c_int64),
                                        ctypes.POINTER(ctypes.c_size_t)]),
    "petra_net_param_info": (ctypes.c_int, [_VP, ctypes.c_int32, ctypes.POINTER(ParamInfo)]),
    "petra_net_bind": (ctypes.c_int, [_VP, _VP, _VP, _VP, _VP, _VP, _VP, ctypes.c_size_t]),
    "petra_net_set_optimizer": (ctypes.c_int, [_VP, ctypes.POINTER(Sgd)]),
    "petra_net_sync_weights": (ctypes.c_int, [_VP, _VP]),
    "petra_net_tick": (ctypes.c_int, [_VP, _VP, _VP, _VP, _VP, ctypes.POINTER(ctypes.c_int32)]),
    "petra_net_drain": (ctypes.c_int, [_VP, _VP, _VP, ctypes.POINTER(ctypes.c_int32),
                                       ctypes.POINTER(ctypes.c_int32)]),
    "petra_net_state": (ctypes.c_int, [_VP, ctypes.POINTER(ctypes.c_int64),
                                        ctypes.POINTER(ctypes.c_int64),
                                        ctypes.POINTER(ctypes.c_int64)]),
    "petra_net_backprop_step": (ctypes.c_int, [_VP, _VP, _VP, _VP, _VP]),
    "petra_net_set_backward": (ctypes.c_int, [_VP, ctypes.c_int32]),
    "petra_net_stage_params": (ctypes.c_int, [_VP, ctypes.c_int32, ctypes.POINTER(ctypes.c_int64),
                                               ctypes.POINTER(ctypes.c_int64)]),
    "petra_net_memory": (ctypes.c_int, [_VP, ctypes.c_int32, ctypes.POINTER(NetMem)]),
    "petra_net_probe_tick": (ctypes.c_int, [_VP, ctypes.c_int32, _VP, _VP]),
    "petra_net_probe_backprop": (ctypes.c_int, [_VP, _VP, _VP, _VP, _VP]),
    "petra_stage_forward_noalloc": (ctypes.c_int, [_VP, _VP, _VP, _VP, _VP, _VP]),
    "petra_stage_profile": (ctypes.c_int, [_VP, ctypes.c_int32]),
    "petra_stage_profile_read": (ctypes.c_int, [_VP, ctypes.c_int32,
                                                 ctypes.POINTER(ctypes.c_char_p),
                                                 ctypes.POINTER(ctypes.c_int64),
                                                 ctypes.POINTER(ctypes.c_double),
                                                 ctypes.POINTER(ctypes.c_double),
                                                 ctypes.POINTER(ctypes.c_double)]),
    "petra_stage_profile_kernel": (ctypes.c_int, [_VP, ctypes.c_int32,
                                                   ctypes.POINTER(ctypes.c_char_p),
                                                   ctypes.POINTER(ctypes.c_int32),
                                                   ctypes.POINTER(ctypes.c_int64),
                                                   ctypes.POINTER(ctypes.c_double),
                                                   ctypes.POINTER(ctypes.c_double),
                                                   ctypes.POINTER(ctypes.c_double)]),
}

_lib: Optional[ctypes.CDLL] = None


def load() -> ctypes.CDLL:
    """Load libpetra.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it first "
                          "(python -c 'import __graft_entry__; __graft_entry__.build()')")
    lib = ctypes.CDLL(LIB_PATH)
    for name, (res, args) in _SIGS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status: int, func: str) -> None:
    if status != 0:
        raise PetraError(status, func, load().petra_last_error().decode())


def _ptr(t) -> int:
    """Device address of a tensor (or an int address, or None)."""
    if t is None:
        return 0
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


# ---------------------------------------------------------------------------
# One wrapper per C entry point, same names and argument order.
# ---------------------------------------------------------------------------

def petra_status_str(status: int) -> str:
    return load().petra_status_str(status).decode()


def petra_last_error() -> str:
    return load().petra_last_error().decode()


def petra_stage_create(desc: StageDesc) -> int:
    h = _VP()
    _check(load().petra_stage_create(ctypes.byref(desc), ctypes.byref(h)), "petra_stage_create")
    return h.value


def petra_stage_destroy(handle: int) -> None:
    _check(load().petra_stage_destroy(handle), "petra_stage_destroy")


def petra_stage_query(handle: int):
    n_params, n_tensors = ctypes.c_int64(), ctypes.c_int32()
    n_bn, ws = ctypes.c_int64(), ctypes.c_size_t()
    _check(load().petra_stage_query(handle, ctypes.byref(n_params), ctypes.byref(n_tensors),
                                    ctypes.byref(n_bn), ctypes.byref(ws)), "petra_stage_query")
    return n_params.value, n_tensors.value, n_bn.value, ws.value


def petra_stage_param_info(handle: int, index: int) -> ParamInfo:
    info = ParamInfo()
    _check(load().petra_stage_param_info(handle, index, ctypes.byref(info)),
           "petra_stage_param_info")
    return info


def petra_stage_bind(handle, params, grad_accum, momentum, run_mean, run_var, workspace,
                     workspace_bytes: int) -> None:
    _check(load().petra_stage_bind(handle, _ptr(params), _ptr(grad_accum), _ptr(momentum),
                                   _ptr(run_mean), _ptr(run_var), _ptr(workspace),
                                   workspace_bytes), "petra_stage_bind")


def petra_stage_set_optimizer(handle: int, opt: Sgd) -> None:
    _check(load().petra_stage_set_optimizer(handle, ctypes.byref(opt)), "petra_stage_set_optimizer")


def petra_stage_set_graphs(handle: int, enable: bool) -> None:
    _check(load().petra_stage_set_graphs(handle, 1 if enable else 0), "petra_stage_set_graphs")


def petra_stage_set_streams(handle: int, n: int) -> None:
    _check(load().petra_stage_set_streams(handle, int(n)), "petra_stage_set_streams")


def petra_stage_sync_weights(handle: int, stream=None) -> None:
    _check(load().petra_stage_sync_weights(handle, _stream(stream)), "petra_stage_sync_weights")


def petra_stage_forward(handle, x1, x2, y1, y2, stream=None) -> None:
    _check(load().petra_stage_forward(handle, _ptr(x1), _ptr(x2), _ptr(y1), _ptr(y2),
                                      _stream(stream)), "petra_stage_forward")


def petra_stage_reconstruct_backward(handle, y1, y2, dy1, dy2, x1, x2, dx1, dx2,
                                     stream=None) -> None:
    _check(load().petra_stage_reconstruct_backward(
        handle, _ptr(y1), _ptr(y2), _ptr(dy1), _ptr(dy2), _ptr(x1), _ptr(x2), _ptr(dx1),
        _ptr(dx2), _stream(stream)), "petra_stage_reconstruct_backward")


def petra_stage_update(handle, stream=None) -> bool:
    upd = ctypes.c_int32()
    _check(load().petra_stage_update(handle, _stream(stream), ctypes.byref(upd)),
           "petra_stage_update")
    return bool(upd.value)


def petra_stage_step(handle, x1, x2, y1, y2, yb1, yb2, dyb1, dyb2, xb1, xb2, dxb1, dxb2,
                     stream=None) -> bool:
    upd = ctypes.c_int32()
    _check(load().petra_stage_step(handle, _ptr(x1), _ptr(x2), _ptr(y1), _ptr(y2), _ptr(yb1),
                                   _ptr(yb2), _ptr(dyb1), _ptr(dyb2), _ptr(xb1), _ptr(xb2),
                                   _ptr(dxb1), _ptr(dxb2), _stream(stream), ctypes.byref(upd)),
           "petra_stage_step")
    return bool(upd.value)


def petra_stage_forward_noalloc(handle, x1, x2, y1, y2, stream=None) -> None:
    _check(load().petra_stage_forward_noalloc(handle, _ptr(x1), _ptr(x2), _ptr(y1), _ptr(y2),
                                              _stream(stream)), "petra_stage_forward_noalloc")


def petra_stage_profile(handle, enable: bool) -> None:
    _check(load().petra_stage_profile(handle, 1 if enable else 0), "petra_stage_profile")


def petra_stage_profile_read(handle):
    """All kernel classes: {name: (launches, total_ms, flops, bytes)}."""
    out = {}
    i = 0
    while True:
        name = ctypes.c_char_p()
        n, ms = ctypes.c_int64(), ctypes.c_double()
        fl, by = ctypes.c_double(), ctypes.c_double()
        st = load().petra_stage_profile_read(handle, i, ctypes.byref(name), ctypes.byref(n),
                                             ctypes.byref(ms), ctypes.byref(fl), ctypes.byref(by))
        if st != 0:
            if STATUS[st] == "PETRA_ERR_INVALID_ARG":
                return out
            _check(st, "petra_stage_profile_read")
        out[name.value.decode()] = (n.value, ms.value, fl.value, by.value)
        i += 1


def petra_stage_profile_kernel(handle):
    """Per kernel instance: [(name, class index, launches, total_ms, flops, bytes)]."""
    out = []
    i = 0
    while True:
        name = ctypes.c_char_p()
        k, n, ms = ctypes.c_int32(), ctypes.c_int64(), ctypes.c_double()
        fl, by = ctypes.c_double(), ctypes.c_double()
        st = load().petra_stage_profile_kernel(handle, i, ctypes.byref(name), ctypes.byref(k),
                                               ctypes.byref(n), ctypes.byref(ms), ctypes.byref(fl),
                                               ctypes.byref(by))
        if st != 0:
            if STATUS[st] == "PETRA_ERR_INVALID_ARG":
                return out
            _check(st, "petra_stage_profile_kernel")
        out.append((name.value.decode(), k.value, n.value, ms.value, fl.value, by.value))
        i += 1


# ---- multi-stage schedule ----------------------------------------------------

def petra_net_create(desc: NetDesc) -> int:
    h = _VP()
    _check(load().petra_net_create(ctypes.byref(desc), ctypes.byref(h)), "petra_net_create")
    return h.value


def petra_net_destroy(handle: int) -> None:
    _check(load().petra_net_destroy(handle), "petra_net_destroy")


def petra_net_query(handle: int):
    n_params, n_tensors = ctypes.c_int64(), ctypes.c_int32()
    n_bn, ws = ctypes.c_int64(), ctypes.c_size_t()
    _check(load().petra_net_query(handle, ctypes.byref(n_params), ctypes.byref(n_tensors),
                                  ctypes.byref(n_bn), ctypes.byref(ws)), "petra_net_query")
    return n_params.value, n_tensors.value, n_bn.value, ws.value


def petra_net_param_info(handle: int, index: int) -> ParamInfo:
    info = ParamInfo()
    _check(load().petra_net_param_info(handle, index, ctypes.byref(info)), "petra_net_param_info")
    return info


def petra_net_bind(handle, params, grad_accum, momentum, run_mean, run_var, workspace,
                   workspace_bytes: int) -> None:
    _check(load().petra_net_bind(handle, _ptr(params), _ptr(grad_accum), _ptr(momentum),
                                 _ptr(run_mean), _ptr(run_var), _ptr(workspace),
                                 workspace_bytes), "petra_net_bind")


def petra_net_set_optimizer(handle: int, opt: Sgd) -> None:
    _check(load().petra_net_set_optimizer(handle, ctypes.byref(opt)), "petra_net_set_optimizer")


def petra_net_sync_weights(handle: int, stream=None) -> None:
    _check(load().petra_net_sync_weights(handle, _stream(stream)), "petra_net_sync_weights")


def petra_net_tick(handle, images, labels, loss=None, stream=None) -> bool:
    wrote = ctypes.c_int32()
    _check(load().petra_net_tick(handle, _ptr(images), _ptr(labels), _ptr(loss), _stream(stream),
                                 ctypes.byref(wrote)), "petra_net_tick")
    return bool(wrote.value)


def petra_net_drain(handle, losses=None, stream=None):
    """Returns (losses written, ticks run)."""
    nl, nt = ctypes.c_int32(), ctypes.c_int32()
    _check(load().petra_net_drain(handle, _ptr(losses), _stream(stream), ctypes.byref(nl),
                                  ctypes.byref(nt)), "petra_net_drain")
    return nl.value, nt.value


def petra_net_backprop_step(handle, images, labels, loss=None, stream=None) -> None:
    _check(load().petra_net_backprop_step(handle, _ptr(images), _ptr(labels), _ptr(loss),
                                          _stream(stream)), "petra_net_backprop_step")


def petra_net_num_stages(handle) -> int:
    j = ctypes.c_int32()
    _check(load().petra_net_num_stages(handle, ctypes.byref(j)), "petra_net_num_stages")
    return j.value


def petra_net_set_backward(handle, mode: int) -> None:
    _check(load().petra_net_set_backward(handle, mode), "petra_net_set_backward")


def petra_net_stage_params(handle, stage: int):
    off, num = ctypes.c_int64(), ctypes.c_int64()
    _check(load().petra_net_stage_params(handle, stage, ctypes.byref(off), ctypes.byref(num)),
           "petra_net_stage_params")
    return off.value, num.value


def petra_net_memory(handle, stage: int) -> dict:
    m = NetMem()
    _check(load().petra_net_memory(handle, stage, ctypes.byref(m)), "petra_net_memory")
    return {name: getattr(m, name) for name, _ in NetMem._fields_}


def petra_net_probe_tick(handle, mode: int, grad_out, stream=None) -> None:
    _check(load().petra_net_probe_tick(handle, mode, _ptr(grad_out), _stream(stream)),
           "petra_net_probe_tick")


def petra_net_probe_backprop(handle, images, labels, grad_out, stream=None) -> None:
    _check(load().petra_net_probe_backprop(handle, _ptr(images), _ptr(labels), _ptr(grad_out),
                                           _stream(stream)), "petra_net_probe_backprop")


def petra_net_state(handle):
    t, fed, fl = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    _check(load().petra_net_state(handle, ctypes.byref(t), ctypes.byref(fed), ctypes.byref(fl)),
           "petra_net_state")
    return t.value, fed.value, fl.value
