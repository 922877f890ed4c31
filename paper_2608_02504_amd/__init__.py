"""Token Radius Attention hot path on MI355X (gfx950): Python binding.

Thin ctypes binding of libtra.so (C ABI declared in include/tra.h).  It only
marshals arguments: every step of the path runs in the library's HIP kernels.
torch is used for device memory and streams.  The functions keep the C names:

    tra_plan_create / tra_plan_destroy / tra_plan_dims / tra_plan_host_tables
    tra_workspace_size / tra_entropy / tra_budget_radius / tra_build_block_mask
    tra_sparse_attention / tra_token_attention / tra_dense_attention

Calls that take a workspace accept one as `workspace=` (a uint8 CUDA tensor of
at least tra_workspace_size bytes); without one, the Plan keeps a workspace per
stream, allocated through torch on its first use on that stream, so calls on
one stream reuse it and calls on different streams never share one.

There is no fallback: if libtra.so is missing or fails to load, every call
raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

__all__ = [
    "LIB_PATH", "TRA_RADIUS_FULL", "TraError", "Config", "Plan", "lib", "library_loaded",
    "tra_plan_create", "tra_plan_destroy", "tra_plan_dims", "tra_plan_host_tables",
    "tra_workspace_size", "TRA_BLOCKS_PACKED", "TRA_BLOCKS_TILES", "TRA_CALL_ENTROPY", "TRA_CALL_BLOCK_MASK", "TRA_CALL_SPARSE",
    "TRA_CALL_TOKEN", "TRA_CALL_DENSE", "tra_entropy", "tra_budget_radius", "tra_build_block_mask", "tra_build_block_mask_noalloc",
    "tra_sparse_attention", "tra_token_attention", "tra_dense_attention", "tra_version",
    "tra_kernel_timing", "tra_kernel_times", "EXPORTED_SYMBOLS",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtra.so")
TRA_RADIUS_FULL = 2 ** 31 - 1
TRA_BF16, TRA_FP32 = 0, 1
TRA_MASK_VOTE, TRA_MASK_UNION = 0, 1
TRA_BUDGET_UNIFORM, TRA_BUDGET_LOGNORMAL = 0, 1
TRA_DIST_2D, TRA_DIST_1D = 0, 1
TRA_BLOCKS_PACKED, TRA_BLOCKS_TILES = 0, 1
_LAYOUT = {"packed": TRA_BLOCKS_PACKED, "tiles": TRA_BLOCKS_TILES}
TRA_CALL_ENTROPY, TRA_CALL_BLOCK_MASK, TRA_CALL_SPARSE, TRA_CALL_TOKEN, TRA_CALL_DENSE = range(5)
_CALLS = (TRA_CALL_ENTROPY, TRA_CALL_BLOCK_MASK, TRA_CALL_SPARSE, TRA_CALL_TOKEN, TRA_CALL_DENSE)
_BUDGET = {"uniform": TRA_BUDGET_UNIFORM, "lognormal": TRA_BUDGET_LOGNORMAL}
_DIST = {"2d": TRA_DIST_2D, "1d": TRA_DIST_1D}

EXPORTED_SYMBOLS = (
    "tra_plan_create", "tra_plan_destroy", "tra_plan_dims", "tra_plan_host_tables",
    "tra_last_error", "tra_version", "tra_entropy", "tra_budget_radius",
    "tra_build_block_mask", "tra_sparse_attention", "tra_token_attention", "tra_dense_attention",
    "tra_build_block_mask_noalloc", "tra_workspace_size", "tra_kernel_timing", "tra_kernel_times",
)

_STATUS = {0: "TRA_OK", 1: "TRA_ERR_INVALID_ARG", 2: "TRA_ERR_UNSUPPORTED",
           3: "TRA_ERR_DEVICE", 4: "TRA_ERR_ALLOC"}


class TraError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{_STATUS.get(status, status)}: {message}")
        self.status = status


class _Config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "batch", "heads", "frames", "height", "width", "head_dim", "block",
        "tile_h", "tile_w", "dtype", "rule", "budget_map", "distance", "text_tokens",
        "block_layout")] + [
        ("tau", ctypes.c_double), ("gamma", ctypes.c_double)]


@dataclass(frozen=True)
class Config:
    """Shape and policy of one attention call (mirrors struct tra_config)."""
    batch: int
    heads: int
    frames: int
    height: int
    width: int
    head_dim: int
    block: int = 128
    tile_h: int = 8
    tile_w: int = 16
    dtype: str = "bf16"       # "bf16" or "fp32"
    rule: str = "vote"        # "vote" (Alg. 1) or "union"
    tau: float = 0.9
    gamma: float = 0.6
    budget: str = "uniform"   # "uniform" (Eq. 8) or "lognormal" (App. A.2)
    distance: str = "2d"      # "2d" (Eq. 15) or "1d" (sequence-distance ablation)
    text_tokens: int = 0      # text tokens after the video tokens (joint attention)
    block_layout: str = "packed"  # "packed" or "tiles" (tile-aligned padded blocks)

    @property
    def n_video(self) -> int:
        return self.frames * self.height * self.width

    @property
    def n_tokens(self) -> int:
        return self.n_video + self.text_tokens

    @property
    def n_blocks(self) -> int:
        if self.block_layout == "tiles":
            return (self.frames * -(-self.height // self.tile_h) * -(-self.width // self.tile_w)
                    + -(-self.text_tokens // self.block))
        return -(-self.n_tokens // self.block)

    @property
    def n_positions(self) -> int:
        """Positions of the block layout's order (the length of the plan's perm)."""
        return self.n_blocks * self.block if self.block_layout == "tiles" else self.n_tokens

    def to_c(self) -> _Config:
        return _Config(self.batch, self.heads, self.frames, self.height, self.width,
                       self.head_dim, self.block, self.tile_h, self.tile_w,
                       TRA_BF16 if self.dtype == "bf16" else TRA_FP32 if self.dtype == "fp32" else 99,
                       TRA_MASK_VOTE if self.rule == "vote" else TRA_MASK_UNION if self.rule == "union" else 99,
                       _BUDGET.get(self.budget, 99), _DIST.get(self.distance, 99), self.text_tokens,
                       _LAYOUT.get(self.block_layout, 99), self.tau, self.gamma)

    @classmethod
    def from_workload(cls, w, **kw) -> "Config":
        base = dict(batch=w.batch, heads=w.heads, frames=w.frames, height=w.height,
                    width=w.width, head_dim=w.head_dim, block=w.block, tile_h=w.tile_h,
                    tile_w=w.tile_w, dtype=w.dtype, tau=w.tau, gamma=w.gamma,
                    text_tokens=getattr(w, "text_tokens", 0))
        base.update(kw)
        return cls(**base)


_lib = None


def lib() -> ctypes.CDLL:
    """Load libtra.so (once).  Raises if it is not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run python -m paper_2608_02504_amd.build")
    L = ctypes.CDLL(LIB_PATH)
    P, I, V, Z = ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_size_t
    cfgp = ctypes.POINTER(_Config)
    L.tra_plan_create.argtypes = [cfgp, ctypes.POINTER(P)]
    L.tra_plan_destroy.argtypes = [P]
    L.tra_plan_dims.argtypes = [P, P, P, P]
    L.tra_plan_host_tables.argtypes = [cfgp, P, P, P, P, P]
    L.tra_last_error.restype = ctypes.c_char_p
    L.tra_version.restype = ctypes.c_char_p
    L.tra_workspace_size.argtypes = [P, ctypes.c_int32, ctypes.POINTER(Z)]
    L.tra_entropy.argtypes = [P, V, V, V, V, V, V, Z, V]
    L.tra_budget_radius.argtypes = [P, V, V, V, V]
    L.tra_build_block_mask.argtypes = [P, V, V, V, V, V, V, Z, V]
    L.tra_build_block_mask_noalloc.argtypes = [P, V, V, V, V, V, V]
    L.tra_sparse_attention.argtypes = [P, V, V, V, V, V, V, V, V, V, Z, V]
    L.tra_token_attention.argtypes = [P, V, V, V, V, V, V, V, V, V, V, Z, V]
    L.tra_dense_attention.argtypes = [P, V, V, V, V, V, V, Z, V]
    L.tra_kernel_timing.argtypes = [ctypes.c_int32, ctypes.c_int32]
    L.tra_kernel_times.argtypes = [V, ctypes.c_int32, V]
    for name in ("tra_plan_create", "tra_plan_destroy", "tra_plan_dims", "tra_plan_host_tables",
                 "tra_workspace_size", "tra_kernel_timing", "tra_kernel_times",
                 "tra_entropy", "tra_budget_radius", "tra_build_block_mask", "tra_build_block_mask_noalloc",
                 "tra_sparse_attention", "tra_token_attention", "tra_dense_attention"):
        getattr(L, name).restype = I
    _lib = L
    return L


def library_loaded() -> bool:
    return _lib is not None


def _check(status: int):
    if status != 0:
        raise TraError(status, lib().tra_last_error().decode())


def tra_version() -> str:
    return lib().tra_version().decode()


# ------------------------------------------------------------------ plans
class Plan:
    """Owns a tra_plan (device tables for one shape)."""

    def __init__(self, cfg: Config):
        self.cfg = cfg
        self._c = cfg.to_c()
        h = ctypes.c_void_p()
        _check(lib().tra_plan_create(ctypes.byref(self._c), ctypes.byref(h)))
        self.handle = h
        n, nb, cap = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
        _check(lib().tra_plan_dims(h, ctypes.byref(n), ctypes.byref(nb), ctypes.byref(cap)))
        self.n_tokens, self.n_blocks, self.n_cap = n.value, nb.value, cap.value
        self._ws = {}  # stream handle -> workspace tensor of ws_bytes
        self.ws_bytes = max(tra_workspace_size(self, c) for c in _CALLS)

    @property
    def rows(self) -> int:
        return self.cfg.batch * self.cfg.heads * self.n_blocks

    def close(self):
        self._ws = {}
        if getattr(self, "handle", None) is not None and self.handle.value:
            lib().tra_plan_destroy(self.handle)
            self.handle = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def tra_plan_create(cfg: Config) -> Plan:
    return Plan(cfg)


def tra_plan_destroy(plan: Plan):
    plan.close()


def tra_workspace_size(plan: Plan, call: int) -> int:
    """Bytes of workspace `call` (a TRA_CALL_* value) needs on this plan."""
    n = ctypes.c_size_t()
    _check(lib().tra_workspace_size(plan.handle, call, ctypes.byref(n)))
    return n.value


def tra_kernel_timing(call: int, n: int) -> None:
    """Time the attention kernel of the calling thread's next n calls of kind
    `call` (a TRA_CALL_* value) with HIP events; n = 0 stops."""
    _check(lib().tra_kernel_timing(call, n))


def tra_kernel_times(n: int):
    """Kernel times (ms, call order) of up to n timed calls, after waiting for them."""
    ms = (ctypes.c_float * max(n, 1))()
    got = ctypes.c_int32()
    _check(lib().tra_kernel_times(ms if n > 0 else None, n, ctypes.byref(got)))
    return [float(ms[i]) for i in range(min(n, got.value))]


def tra_plan_dims(plan: Plan):
    return plan.n_tokens, plan.n_blocks, plan.n_cap


def tra_plan_host_tables(cfg: Config):
    """Host-only tables of cfg: (perm[P], thr[(n_cap+1), F], thr1[(n_cap+1), F],
    blocks[NB, 10], n_cap); P = cfg.n_positions, perm -1 at padding positions."""
    c = cfg.to_c()
    cap = ctypes.c_int32()
    _check(lib().tra_plan_host_tables(ctypes.byref(c), None, None, None, None, ctypes.byref(cap)))
    perm = np.empty(cfg.n_positions, dtype=np.int32)
    thr = np.empty((cap.value + 1, cfg.frames), dtype=np.int32)
    thr1 = np.empty((cap.value + 1, cfg.frames), dtype=np.int32)
    blocks = np.empty((cfg.n_blocks, 10), dtype=np.int32)
    _check(lib().tra_plan_host_tables(ctypes.byref(c), perm.ctypes.data, thr.ctypes.data,
                                      thr1.ctypes.data, blocks.ctypes.data, ctypes.byref(cap)))
    return perm, thr, thr1, blocks, cap.value


# ------------------------------------------------------------------ marshalling
def _ptr(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensor must be on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        import torch
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _workspace(plan: Plan, stream, workspace):
    """(pointer, bytes, tensor) of the workspace for a call on `stream`: the
    caller's, or the plan's own for that stream (created on first use)."""
    import torch
    if workspace is not None:
        if workspace.dtype != torch.uint8:
            raise ValueError("workspace must be a uint8 tensor")
        return _ptr(workspace), workspace.numel(), workspace
    if plan.ws_bytes == 0:
        return None, 0, None
    handle = _stream(stream).value or 0
    ws = plan._ws.get(handle)
    if ws is None:
        ws = torch.empty(plan.ws_bytes, dtype=torch.uint8, device="cuda")
        if handle != (torch.cuda.current_stream().cuda_stream or 0):
            # freed only when the plan closes: keep it until that stream's work is done
            ws.record_stream(torch.cuda.ExternalStream(handle))
        plan._ws[handle] = ws
    return ctypes.c_void_p(ws.data_ptr()), ws.numel(), ws


def _want(t, shape, dtype, name):
    if t is None:
        return
    if tuple(t.shape) != tuple(shape) or t.dtype != dtype:
        raise ValueError(f"{name}: expected {tuple(shape)} {dtype}, got {tuple(t.shape)} {t.dtype}")


def _qkv_dtype(plan: Plan):
    import torch
    return torch.bfloat16 if plan.cfg.dtype == "bf16" else torch.float32


def _shapes(plan: Plan):
    c = plan.cfg
    return ((c.batch, c.heads, plan.n_tokens, c.head_dim), (c.batch, c.heads, plan.n_tokens),
            (c.batch, c.heads, plan.n_blocks), (c.batch, c.heads, plan.n_blocks, plan.n_blocks))


def tra_entropy(plan: Plan, q, k, v, o, entropy, stream=None, workspace=None):
    import torch
    tok, per, _, _ = _shapes(plan)
    dt = _qkv_dtype(plan)
    for t, n in ((q, "q"), (k, "k"), (v, "v"), (o, "o")):
        _want(t, tok, dt, n)
    _want(entropy, per, torch.float32, "entropy")
    wp, wn, _ = _workspace(plan, stream, workspace)
    _check(lib().tra_entropy(plan.handle, _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(entropy),
                             wp, wn, _stream(stream)))


def tra_budget_radius(plan: Plan, entropy, budget, radius_sq, stream=None):
    import torch
    _, per, _, _ = _shapes(plan)
    _want(entropy, per, torch.float32, "entropy")
    _want(budget, per, torch.int32, "budget")
    _want(radius_sq, per, torch.int32, "radius_sq")
    _check(lib().tra_budget_radius(plan.handle, _ptr(entropy), _ptr(budget), _ptr(radius_sq),
                                   _stream(stream)))


def tra_build_block_mask(plan: Plan, radius_sq, mask, cnt, cols, order=None, stream=None, workspace=None):
    import torch
    _, per, rowsh, sq = _shapes(plan)
    _want(radius_sq, per, torch.int32, "radius_sq")
    _want(mask, sq, torch.uint8, "mask")
    _want(cnt, rowsh, torch.int32, "cnt")
    _want(cols, sq, torch.int32, "cols")
    _want(order, (plan.rows,), torch.int32, "order")
    wp, wn, _ = _workspace(plan, stream, workspace) if order is not None else (None, 0, None)
    _check(lib().tra_build_block_mask(plan.handle, _ptr(radius_sq), _ptr(mask), _ptr(cnt),
                                      _ptr(cols), _ptr(order), wp, wn, _stream(stream)))


def tra_build_block_mask_noalloc(plan: Plan, radius_sq, mask, cnt, cols, order=None, stream=None):
    import torch
    _, per, rowsh, sq = _shapes(plan)
    _want(radius_sq, per, torch.int32, "radius_sq")
    _want(mask, sq, torch.uint8, "mask")
    _want(cnt, rowsh, torch.int32, "cnt")
    _want(cols, sq, torch.int32, "cols")
    _want(order, (plan.rows,), torch.int32, "order")
    _check(lib().tra_build_block_mask_noalloc(plan.handle, _ptr(radius_sq), _ptr(mask), _ptr(cnt),
                                              _ptr(cols), _ptr(order), _stream(stream)))


def tra_sparse_attention(plan: Plan, q, k, v, cnt, cols, order, o, lse=None, stream=None, workspace=None):
    import torch
    tok, per, rowsh, sq = _shapes(plan)
    dt = _qkv_dtype(plan)
    for t, n in ((q, "q"), (k, "k"), (v, "v"), (o, "o")):
        _want(t, tok, dt, n)
    _want(cnt, rowsh, torch.int32, "cnt")
    _want(cols, sq, torch.int32, "cols")
    _want(order, (plan.rows,), torch.int32, "order")
    _want(lse, per, torch.float32, "lse")
    wp, wn, _ = _workspace(plan, stream, workspace)
    _check(lib().tra_sparse_attention(plan.handle, _ptr(q), _ptr(k), _ptr(v), _ptr(cnt),
                                      _ptr(cols), _ptr(order), _ptr(o), _ptr(lse), wp, wn,
                                      _stream(stream)))


def tra_token_attention(plan: Plan, q, k, v, radius_sq, cnt, cols, order, o, lse=None, stream=None,
                        workspace=None):
    import torch
    tok, per, rowsh, sq = _shapes(plan)
    dt = _qkv_dtype(plan)
    for t, n in ((q, "q"), (k, "k"), (v, "v"), (o, "o")):
        _want(t, tok, dt, n)
    _want(radius_sq, per, torch.int32, "radius_sq")
    _want(cnt, rowsh, torch.int32, "cnt")
    _want(cols, sq, torch.int32, "cols")
    _want(order, (plan.rows,), torch.int32, "order")
    _want(lse, per, torch.float32, "lse")
    wp, wn, _ = _workspace(plan, stream, workspace)
    _check(lib().tra_token_attention(plan.handle, _ptr(q), _ptr(k), _ptr(v), _ptr(radius_sq),
                                     _ptr(cnt), _ptr(cols), _ptr(order), _ptr(o), _ptr(lse), wp, wn,
                                     _stream(stream)))


def tra_dense_attention(plan: Plan, q, k, v, o, lse=None, stream=None, workspace=None):
    import torch
    tok, per, _, _ = _shapes(plan)
    dt = _qkv_dtype(plan)
    for t, n in ((q, "q"), (k, "k"), (v, "v"), (o, "o")):
        _want(t, tok, dt, n)
    _want(lse, per, torch.float32, "lse")
    wp, wn, _ = _workspace(plan, stream, workspace)
    _check(lib().tra_dense_attention(plan.handle, _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse),
                                     wp, wn, _stream(stream)))
