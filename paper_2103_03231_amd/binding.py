"""ctypes binding of include/donerf.h.

Functions carry the C names and only marshal arguments: every step of the
rendering runs in libdonerf.so.  Device buffers are passed as integer device
addresses (``tensor.data_ptr()``); host arrays as numpy arrays.  A missing
library raises ``DonerfLibraryMissing``: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libdonerf.so")

OK = 0
E_INVALID_ARG = -1
E_SIZE = -2
E_NONFINITE = -3
E_DEVICE = -4
E_NOMEM = -5
E_HIP = -6
E_UNSUPPORTED = -7

FP32 = 0
BF16 = 1
FP8 = 2
SELECT_TOPN = 0
SELECT_TOPN_SOFTMAX = 1
SELECT_CDF = 2
DEPTH_ENCODED = 0
DEPTH_POSITIONS = 1
MAX_SAMPLES = 16

# Every function include/donerf.h declares.
EXPORTS = ("donerf_weight_count", "donerf_create", "donerf_destroy", "donerf_set_stream",
           "donerf_render", "donerf_render_static_scratch", "donerf_render_debug", "donerf_targets",
           "donerf_debug_topn", "donerf_debug_bins", "donerf_debug_mfma_peak", "donerf_status_str",
           "donerf_last_error")


class DonerfLibraryMissing(RuntimeError):
    pass


class DonerfError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{message} (status {status})")
        self.status = status


class donerf_cfg(ctypes.Structure):
    _fields_ = [("near_dist", ctypes.c_float), ("far_dist", ctypes.c_float),
                ("n_bins", ctypes.c_int32), ("n_max", ctypes.c_int32),
                ("fov_x_deg", ctypes.c_float), ("centre", ctypes.c_float * 3),
                ("radius", ctypes.c_float), ("precision", ctypes.c_int32),
                ("select", ctypes.c_int32), ("depth_input", ctypes.c_int32)]


@dataclass
class Config:
    near: float = 0.1
    far: float = 10.0
    n_bins: int = 128
    n_max: int = 4
    fov_x_deg: float = 60.0
    centre: tuple = (0.0, 0.0, 0.0)
    radius: float = 1.5
    precision: int = BF16
    select: int = SELECT_TOPN
    depth_input: int = DEPTH_ENCODED

    def to_c(self) -> donerf_cfg:
        c = donerf_cfg()
        c.near_dist, c.far_dist = self.near, self.far
        c.n_bins, c.n_max = self.n_bins, self.n_max
        c.fov_x_deg = self.fov_x_deg
        c.centre[:] = list(self.centre)
        c.radius = self.radius
        c.precision, c.select = self.precision, self.select
        c.depth_input = self.depth_input
        return c


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise DonerfLibraryMissing(
                f"{LIB_PATH} not built; run `python -m paper_2103_03231_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, sz, fp = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t, ctypes.POINTER(ctypes.c_float)
        L.donerf_weight_count.argtypes, L.donerf_weight_count.restype = [i32, i32], sz
        L.donerf_create.argtypes = [ctypes.POINTER(donerf_cfg), fp, sz, ctypes.POINTER(vp)]
        L.donerf_create.restype = ctypes.c_int
        L.donerf_destroy.argtypes, L.donerf_destroy.restype = [vp], None
        L.donerf_set_stream.argtypes, L.donerf_set_stream.restype = [vp, vp], ctypes.c_int
        L.donerf_render.argtypes = [vp, fp, i32, i32, i32, i32, vp, vp]
        L.donerf_render.restype = ctypes.c_int
        L.donerf_render_static_scratch.argtypes = [vp, fp, i32, i32, i32, i32, vp, vp]
        L.donerf_render_static_scratch.restype = ctypes.c_int
        L.donerf_render_debug.argtypes = [vp, fp, i32, i32, i32, i32, vp, vp, vp, vp, vp]
        L.donerf_render_debug.restype = ctypes.c_int
        L.donerf_targets.argtypes = [vp, vp, i32, i32, i32, i32, i32, vp]
        L.donerf_targets.restype = ctypes.c_int
        L.donerf_debug_topn.argtypes = [vp, vp, i32, i32, vp]
        L.donerf_debug_topn.restype = ctypes.c_int
        L.donerf_debug_bins.argtypes = [vp, fp, fp, fp]
        L.donerf_debug_bins.restype = ctypes.c_int
        L.donerf_debug_mfma_peak.argtypes = [vp, i32, i32, vp, ctypes.POINTER(ctypes.c_double)]
        L.donerf_debug_mfma_peak.restype = ctypes.c_int
        L.donerf_status_str.argtypes, L.donerf_status_str.restype = [ctypes.c_int], ctypes.c_char_p
        L.donerf_last_error.argtypes, L.donerf_last_error.restype = [], ctypes.c_char_p
        _lib = L
    return _lib


def _check(status: int):
    if status != OK:
        raise DonerfError(status, donerf_last_error() or donerf_status_str(status))


def _fptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.POINTER(ctypes.c_float))


def donerf_weight_count(n_bins: int, depth_input: int = DEPTH_ENCODED) -> int:
    return int(lib().donerf_weight_count(n_bins, depth_input))


def donerf_status_str(status: int) -> str:
    return lib().donerf_status_str(status).decode()


def donerf_last_error() -> str:
    return lib().donerf_last_error().decode()


def donerf_create(cfg: Config, weights) -> int:
    """Returns the handle (an integer address); raises DonerfError."""
    w = None if weights is None else np.ascontiguousarray(weights, dtype=np.float32)
    h = ctypes.c_void_p()
    c = cfg.to_c()
    _check(lib().donerf_create(ctypes.byref(c), _fptr(w), 0 if w is None else w.size, ctypes.byref(h)))
    return h.value


def donerf_destroy(h) -> None:
    lib().donerf_destroy(h)


def donerf_set_stream(h, stream: int) -> None:
    _check(lib().donerf_set_stream(h, stream))


def _poses(poses):
    return None if poses is None else np.ascontiguousarray(poses, dtype=np.float32).reshape(-1)


def donerf_render(h, poses, P, H, W, N, out_rgb_ptr, out_depth_ptr=None) -> None:
    p = _poses(poses)
    _check(lib().donerf_render(h, _fptr(p), P, H, W, N, out_rgb_ptr, out_depth_ptr))


def donerf_render_static_scratch(h, poses, P, H, W, N, out_rgb_ptr, out_depth_ptr=None) -> None:
    p = _poses(poses)
    _check(lib().donerf_render_static_scratch(h, _fptr(p), P, H, W, N, out_rgb_ptr, out_depth_ptr))


def donerf_render_debug(h, poses, P, H, W, N, out_rgb_ptr, out_depth_ptr=None,
                        out_bins_ptr=None, out_scores_ptr=None, out_samples_ptr=None) -> None:
    p = _poses(poses)
    _check(lib().donerf_render_debug(h, _fptr(p), P, H, W, N, out_rgb_ptr, out_depth_ptr,
                                     out_bins_ptr, out_scores_ptr, out_samples_ptr))


def donerf_targets(h, depth_ptr, P, H, W, K, Z, out_ptr) -> None:
    _check(lib().donerf_targets(h, depth_ptr, P, H, W, K, Z, out_ptr))


def donerf_debug_topn(h, scores_ptr, rays, N, out_idx_ptr) -> None:
    _check(lib().donerf_debug_topn(h, scores_ptr, rays, N, out_idx_ptr))


def donerf_debug_mfma_peak(h, workgroups, iters, sink_ptr) -> float:
    """Enqueue the register-fed MFMA loop; returns the launch's FLOP."""
    flop = ctypes.c_double(0.0)
    _check(lib().donerf_debug_mfma_peak(h, workgroups, iters, sink_ptr, ctypes.byref(flop)))
    return flop.value


def donerf_debug_bins(h, n_bins):
    bounds = np.empty(n_bins + 1, np.float32)
    centres = np.empty(n_bins, np.float32)
    widths = np.empty(n_bins, np.float32)
    _check(lib().donerf_debug_bins(h, _fptr(bounds), _fptr(centres), _fptr(widths)))
    return bounds, centres, widths


class Renderer:
    """Convenience owner of a handle; outputs are torch tensors on cuda:0
    (torch provides device memory and the stream, nothing else)."""

    def __init__(self, cfg: Config, weights):
        import torch
        self.torch = torch
        self.cfg = cfg
        self.h = donerf_create(cfg, weights)
        donerf_set_stream(self.h, torch.cuda.current_stream().cuda_stream)

    def close(self):
        if self.h:
            donerf_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def targets(self, depth, K, Z):
        """Depth-oracle targets of device depth maps (P, H, W) fp32 -> (P, H, W, B)."""
        t = self.torch
        if depth.dtype != t.float32 or not depth.is_cuda or not depth.is_contiguous() or depth.dim() != 3:
            raise ValueError("depth must be a contiguous (P, H, W) float32 CUDA tensor")
        P, H, W = depth.shape
        out = t.empty((P, H, W, self.cfg.n_bins), dtype=t.float32, device=depth.device)
        donerf_targets(self.h, depth.data_ptr(), P, H, W, K, Z, out.data_ptr())
        return out

    def mfma_peak(self, workgroups, iters):
        """Enqueue the register-fed MFMA loop in the handle's precision;
        returns (sink, FLOP of the launch)."""
        import torch
        sink = torch.empty(workgroups * 256, dtype=torch.float32, device="cuda")
        return sink, donerf_debug_mfma_peak(self.h, workgroups, iters, sink.data_ptr())

    def alloc(self, P, H, W, N, depth=False, debug=False):
        t = self.torch
        dev = "cuda"
        out = {"rgb": t.empty((P, H, W, 3), dtype=t.float32, device=dev)}
        if depth:
            out["depth"] = t.empty((P, H, W), dtype=t.float32, device=dev)
        if debug:
            out["bins"] = t.empty((P, H, W, N), dtype=t.int32, device=dev)
            out["scores"] = t.empty((P, H, W, self.cfg.n_bins), dtype=t.float32, device=dev)
            out["samples"] = t.empty((P, H, W, N, 2), dtype=t.float32, device=dev)
        return out

    def _check_out(self, P, H, W, N, out):
        """Reject output tensors the library would write out of bounds:
        each present one must be a contiguous CUDA tensor of the right dtype
        holding P x H x W x {3, 1, N, B, 2 N} values."""
        t = self.torch
        per_ray = {"rgb": 3, "depth": 1, "bins": N, "scores": self.cfg.n_bins, "samples": 2 * N}
        if "rgb" not in out:
            raise ValueError("out needs an 'rgb' tensor")
        for k, v in out.items():
            if k not in per_ray:
                raise ValueError(f"unknown output {k!r}")
            dtype = t.int32 if k == "bins" else t.float32
            if not (isinstance(v, t.Tensor) and v.is_cuda and v.is_contiguous() and v.dtype == dtype):
                raise ValueError(f"out[{k!r}] must be a contiguous CUDA {dtype} tensor")
            if v.numel() != P * H * W * per_ray[k]:
                raise ValueError(f"out[{k!r}] holds {v.numel()} values, the render writes {P * H * W * per_ray[k]}")

    def render_into(self, poses, H, W, N, out, debug=False):
        P = int(np.asarray(poses).reshape(-1, 12).shape[0])
        self._check_out(P, H, W, N, out)
        ptr = lambda k: out[k].data_ptr() if k in out else None
        if debug:
            donerf_render_debug(self.h, poses, P, H, W, N, ptr("rgb"), ptr("depth"),
                                ptr("bins"), ptr("scores"), ptr("samples"))
        else:
            donerf_render(self.h, poses, P, H, W, N, ptr("rgb"), ptr("depth"))
        return out

    def render(self, poses, H, W, N, depth=False, debug=False):
        P = int(np.asarray(poses).reshape(-1, 12).shape[0])
        out = self.alloc(P, H, W, N, depth=depth, debug=debug)
        return self.render_into(poses, H, W, N, out, debug=debug)
