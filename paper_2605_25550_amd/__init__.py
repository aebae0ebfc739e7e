"""Python binding of libditmi (the gfx950 DiT denoising-step library).

Argument marshalling only: torch tensors are checked (device, dtype,
contiguity) and their device pointers, together with the current HIP stream,
are handed to the C ABI declared in include/ditmi.h.  Every step of the
computation runs in the library's HIP kernels; there is no fallback path, and
a missing library raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# DITMI_LIB names another build of the same library (a sanitizer build, or a
# variant being measured); the default is the in-tree build.
LIB_PATH = os.environ.get("DITMI_LIB") or os.path.join(_HERE, "libditmi.so")

DIT_OK, DIT_ERR_INVALID_ARG, DIT_ERR_UNSUPPORTED, DIT_ERR_WORKSPACE, DIT_ERR_HIP = 0, -1, -2, -3, -4
DIT_F32, DIT_BF16 = 0, 1
DIT_WS_BLOCK, DIT_WS_STEP, DIT_WS_COND, DIT_WS_SAMPLE, DIT_WS_SERVE = 0, 1, 2, 3, 4
NOALLOC_SCRATCH_BYTES = 128 << 20  # DIT_NOALLOC_SCRATCH_BYTES of include/ditmi.h
KERNEL_CLASSES = {"gemm_qkv": 0, "attention": 1, "gemm_out": 2, "gemm_fc1": 3, "gemm_fc2": 4,
                  "ln_mod": 5, "adaln": 6, "other": 7}

STREAM_FIELDS = ("w_ada", "b_ada", "w_qkv", "b_qkv", "w_o", "b_o", "w_fc1", "b_fc1", "w_fc2", "b_fc2")
C_API = ("dit_workspace_bytes", "dit_block_forward", "dit_block_forward_noalloc", "dit_step_forward", "dit_sample_euler", "dit_serve", "dit_cond_embed", "dit_pos_embed_2d",
         "dit_timing_enable", "dit_timing_read", "dit_timing_disable", "dit_status_string", "dit_last_error",
         "dit_version")


class DitError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"ditmi status {status}: {msg}")
        self.status = status


class Shape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("tokens", ctypes.c_int32), ("text_tokens", ctypes.c_int32),
                ("hidden", ctypes.c_int32), ("heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("mlp_hidden", ctypes.c_int32), ("n_blocks", ctypes.c_int32), ("patch_in", ctypes.c_int32),
                ("patch_out", ctypes.c_int32), ("dtype", ctypes.c_int32), ("ln_eps", ctypes.c_float)]


class StreamWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in STREAM_FIELDS]


class BlockWeights(ctypes.Structure):
    _fields_ = [("img", StreamWeights), ("txt", StreamWeights)]


class StepWeights(ctypes.Structure):
    _fields_ = [("w_patch", ctypes.c_void_p), ("b_patch", ctypes.c_void_p), ("pos", ctypes.c_void_p),
                ("blocks", ctypes.POINTER(BlockWeights)), ("w_ada_final", ctypes.c_void_p),
                ("b_ada_final", ctypes.c_void_p), ("w_final", ctypes.c_void_p), ("b_final", ctypes.c_void_p)]


_LIB: Optional[ctypes.CDLL] = None


class CondWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("w_t1", "b_t1", "w_t2", "b_t2", "class_table")]


class Request(ctypes.Structure):
    _fields_ = [("z_in", ctypes.c_void_p), ("z_out", ctypes.c_void_p), ("y", ctypes.c_void_p), ("cond", ctypes.c_void_p)]


def lib() -> ctypes.CDLL:
    """Load libditmi.so (raises if it has not been built)."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built: run paper_2605_25550_amd/build.py (or __graft_entry__.build())")
    L = ctypes.CDLL(LIB_PATH)
    vp, sz, i32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32
    P = ctypes.POINTER
    L.dit_workspace_bytes.argtypes = [P(Shape), ctypes.c_int]
    L.dit_workspace_bytes.restype = sz
    L.dit_block_forward.argtypes = [P(Shape), P(BlockWeights), vp, vp, vp, vp, sz, vp]
    L.dit_block_forward_noalloc.argtypes = [P(Shape), P(BlockWeights), vp, vp, vp, vp]
    L.dit_step_forward.argtypes = [P(Shape), P(StepWeights), vp, vp, vp, vp, vp, sz, vp]
    L.dit_cond_embed.argtypes = [P(Shape), vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    L.dit_sample_euler.argtypes = [P(Shape), P(StepWeights), P(CondWeights), vp, vp, P(ctypes.c_float), i32,
                                   ctypes.c_float, vp, vp, vp, sz, vp]
    L.dit_serve.argtypes = [P(Shape), P(StepWeights), P(CondWeights), P(Request), i32, P(ctypes.c_float), i32,
                            ctypes.c_float, i32, ctypes.c_uint32, ctypes.c_uint32, vp, sz, vp, vp]
    L.dit_pos_embed_2d.argtypes = [i32, i32, i32, vp, vp]
    L.dit_timing_enable.argtypes = [ctypes.c_int, ctypes.c_int]
    L.dit_timing_read.argtypes = [P(ctypes.c_double), P(ctypes.c_int), P(ctypes.c_double), P(ctypes.c_double)]
    L.dit_timing_disable.argtypes = []
    for fn in ("dit_block_forward", "dit_block_forward_noalloc", "dit_step_forward", "dit_cond_embed", "dit_pos_embed_2d", "dit_timing_enable",
               "dit_timing_read", "dit_timing_disable"):
        getattr(L, fn).restype = ctypes.c_int
    L.dit_status_string.argtypes = [ctypes.c_int]
    L.dit_status_string.restype = ctypes.c_char_p
    L.dit_last_error.argtypes = []
    L.dit_last_error.restype = ctypes.c_char_p
    L.dit_version.restype = ctypes.c_int
    _LIB = L
    return L


def _check(st: int) -> None:
    if st != DIT_OK:
        raise DitError(st, lib().dit_last_error().decode())


def last_error() -> str:
    return lib().dit_last_error().decode()


# ---------------------------------------------------------------- marshalling
def make_shape(batch, tokens, hidden, heads, head_dim, mlp_hidden, n_blocks=1, text_tokens=0, patch_in=16,
               patch_out=16, dtype="bf16", ln_eps=1e-6) -> Shape:
    return Shape(batch, tokens, text_tokens, hidden, heads, head_dim, mlp_hidden, n_blocks, patch_in, patch_out,
                 DIT_BF16 if dtype == "bf16" else DIT_F32, ln_eps)


def shape_of(cfg) -> Shape:
    """Shape struct of a workload description with the DiT shape attributes
    (batch, tokens, text_tokens, hidden, heads, head_dim, mlp_hidden, n_blocks,
    patch_in, patch_out, dtype, ln_eps)."""
    return make_shape(cfg.batch, cfg.tokens, cfg.hidden, cfg.heads, cfg.head_dim, cfg.mlp_hidden, cfg.n_blocks,
                      cfg.text_tokens, cfg.patch_in, cfg.patch_out, cfg.dtype, cfg.ln_eps)


def weight_dtype(shape: Shape) -> torch.dtype:
    return torch.bfloat16 if shape.dtype == DIT_BF16 else torch.float32


def _ptr(t: Optional[torch.Tensor], dtype: Optional[torch.dtype] = None, name: str = "tensor"):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device tensor (got {t.device})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype} (got {t.dtype})")
    return t.data_ptr()


def _stream(stream=None) -> int:
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def stream_struct(w: Dict[str, torch.Tensor], dtype: torch.dtype) -> StreamWeights:
    return StreamWeights(*[_ptr(w[n], dtype, n) for n in STREAM_FIELDS])


def block_struct(img: Dict[str, torch.Tensor], txt: Optional[Dict[str, torch.Tensor]], dtype: torch.dtype) -> BlockWeights:
    bw = BlockWeights()
    bw.img = stream_struct(img, dtype)
    if txt is not None:
        bw.txt = stream_struct(txt, dtype)
    return bw


class StepWeightTable:
    """Holds the ctypes step-weight struct and the host array of block structs it points to."""

    def __init__(self, step_w: Dict[str, torch.Tensor], blocks: Sequence[BlockWeights], dtype: torch.dtype,
                 pos: Optional[torch.Tensor] = None):
        self.block_array = (BlockWeights * len(blocks))(*blocks)
        self.struct = StepWeights(
            _ptr(step_w["w_patch"], dtype, "w_patch"), _ptr(step_w["b_patch"], dtype, "b_patch"),
            _ptr(pos, torch.float32, "pos"), ctypes.cast(self.block_array, ctypes.POINTER(BlockWeights)),
            _ptr(step_w["w_ada_final"], dtype, "w_ada_final"), _ptr(step_w["b_ada_final"], dtype, "b_ada_final"),
            _ptr(step_w["w_final"], dtype, "w_final"), _ptr(step_w["b_final"], dtype, "b_final"))
        self._keep = (step_w, blocks, pos)


def _check_pos(shape: Shape, pos: Optional[torch.Tensor]) -> None:
    """The step reads the position table as [tokens, hidden] fp32 rows; the C
    ABI cannot see the size of a device buffer, so a short table is refused
    here rather than read past its end on the device."""
    if pos is None:
        return
    if pos.dim() != 2 or pos.shape[0] < shape.tokens or pos.shape[1] != shape.hidden:
        raise ValueError(f"pos is {tuple(pos.shape)}; the step reads [{shape.tokens}, {shape.hidden}] "
                         "(one row per image token)")


# ---------------------------------------------------------------- entry points
def workspace_bytes(shape: Shape, kind: int = DIT_WS_BLOCK) -> int:
    n = lib().dit_workspace_bytes(ctypes.byref(shape), kind)
    if n == 0:
        raise DitError(DIT_ERR_INVALID_ARG, last_error())
    return n


def alloc_workspace(shape: Shape, kind: int, device="cuda") -> torch.Tensor:
    return torch.empty(workspace_bytes(shape, kind), dtype=torch.uint8, device=device)


def block_forward(shape: Shape, weights: BlockWeights, x: torch.Tensor, cond: torch.Tensor, workspace: torch.Tensor,
                  x_txt: Optional[torch.Tensor] = None, stream=None) -> None:
    """One DiT block in place on x (and x_txt for the joint block)."""
    _check(lib().dit_block_forward(ctypes.byref(shape), ctypes.byref(weights), _ptr(x, torch.float32, "x"),
                                   _ptr(x_txt, torch.float32, "x_txt"), _ptr(cond, torch.float32, "cond"),
                                   _ptr(workspace, None, "workspace"), workspace.numel() * workspace.element_size(),
                                   _stream(stream)))


def block_forward_noalloc(shape: Shape, weights: BlockWeights, x: torch.Tensor, cond: torch.Tensor,
                          x_txt: Optional[torch.Tensor] = None, stream=None) -> None:
    """One DiT block in place on x, with the library's static per-GPU scratch
    as workspace (no device allocation)."""
    _check(lib().dit_block_forward_noalloc(ctypes.byref(shape), ctypes.byref(weights), _ptr(x, torch.float32, "x"),
                                           _ptr(x_txt, torch.float32, "x_txt"), _ptr(cond, torch.float32, "cond"),
                                           _stream(stream)))


def step_forward(shape: Shape, table: StepWeightTable, patches: torch.Tensor, cond: torch.Tensor, out: torch.Tensor,
                 workspace: torch.Tensor, x_txt: Optional[torch.Tensor] = None, stream=None) -> None:
    """One denoising step (patch embed, blocks, final layer) into out."""
    _check_pos(shape, table._keep[2])
    _check(lib().dit_step_forward(ctypes.byref(shape), ctypes.byref(table.struct),
                                  _ptr(patches, torch.float32, "patches"), _ptr(x_txt, torch.float32, "x_txt"),
                                  _ptr(cond, torch.float32, "cond"), _ptr(out, torch.float32, "out"),
                                  _ptr(workspace, None, "workspace"), workspace.numel() * workspace.element_size(),
                                  _stream(stream)))


def sample_euler(shape: Shape, table: StepWeightTable, z: torch.Tensor, sigmas, workspace: torch.Tensor,
                 cond_w: Optional[Dict[str, torch.Tensor]] = None, y: Optional[torch.Tensor] = None,
                 cond: Optional[torch.Tensor] = None, t_scale: float = 1000.0,
                 x_txt: Optional[torch.Tensor] = None, stream=None) -> None:
    """Multi-step Euler loop over the step (z updated in place): with cond_w and
    y the conditioning is recomputed per step at t_i = sigmas[i] * t_scale;
    otherwise cond is used for every step.  sigmas: n_steps + 1 floats (host)."""
    _check_pos(shape, table._keep[2])
    sig = [float(v) for v in sigmas]
    if len(sig) < 1:
        raise ValueError("sigmas needs at least one value")
    arr = (ctypes.c_float * len(sig))(*sig)
    cw = None
    if cond_w is not None:
        dt = weight_dtype(shape)
        cw = CondWeights(*[_ptr(cond_w[k], dt, k) for k in ("w_t1", "b_t1", "w_t2", "b_t2", "class_table")])
    _check(lib().dit_sample_euler(ctypes.byref(shape), ctypes.byref(table.struct),
                                  ctypes.byref(cw) if cw is not None else None,
                                  _ptr(y, torch.int32, "y"), _ptr(cond, torch.float32, "cond"), arr, len(sig) - 1,
                                  float(t_scale), _ptr(z, torch.float32, "z"), _ptr(x_txt, torch.float32, "x_txt"),
                                  _ptr(workspace, None, "workspace"), workspace.numel() * workspace.element_size(),
                                  _stream(stream)))


def _host_ptr(t: Optional[torch.Tensor], dtype: torch.dtype, name: str):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or t.device.type != "cpu" or not t.is_contiguous() or t.dtype != dtype:
        raise ValueError(f"{name} must be a contiguous host {dtype} tensor")
    return t.data_ptr()


def serve(shape: Shape, table: StepWeightTable, requests, sigmas, workspace: torch.Tensor,
          cond_w: Optional[Dict[str, torch.Tensor]] = None, t_scale: float = 1000.0, overlap: bool = True,
          jitter_us: int = 0, jitter_seed: int = 0, stream=None, copy_stream=None) -> None:
    """Run requests through the DiT stage with copy/compute overlap.  requests:
    list of dicts with host tensors z_in, z_out ([B,T,P] fp32, ideally pinned)
    and y ([B] int32, with cond_w) or cond ([B,D] fp32).  Returns after
    enqueueing; synchronise the stream before reading z_out."""
    _check_pos(shape, table._keep[2])
    sig = [float(v) for v in sigmas]
    arr = (ctypes.c_float * len(sig))(*sig)
    reqs = (Request * max(1, len(requests)))()
    for i, r in enumerate(requests):
        reqs[i] = Request(_host_ptr(r["z_in"], torch.float32, "z_in"), _host_ptr(r["z_out"], torch.float32, "z_out"),
                          _host_ptr(r.get("y"), torch.int32, "y"), _host_ptr(r.get("cond"), torch.float32, "cond"))
    cw = None
    if cond_w is not None:
        dt = weight_dtype(shape)
        cw = CondWeights(*[_ptr(cond_w[k], dt, k) for k in ("w_t1", "b_t1", "w_t2", "b_t2", "class_table")])
    cs = copy_stream.cuda_stream if copy_stream is not None else None
    _check(lib().dit_serve(ctypes.byref(shape), ctypes.byref(table.struct), ctypes.byref(cw) if cw is not None else None,
                           reqs, len(requests), arr, len(sig) - 1, float(t_scale), 1 if overlap else 0, int(jitter_us),
                           int(jitter_seed), _ptr(workspace, None, "workspace"),
                           workspace.numel() * workspace.element_size(), _stream(stream), cs))


def cond_embed(shape: Shape, t: torch.Tensor, y: torch.Tensor, w: Dict[str, torch.Tensor], cond: torch.Tensor,
               workspace: torch.Tensor, stream=None) -> None:
    """Timestep + class conditioning into cond [B, D]."""
    dt = weight_dtype(shape)
    _check(lib().dit_cond_embed(ctypes.byref(shape), _ptr(t, torch.float32, "t"), _ptr(y, torch.int32, "y"),
                                _ptr(w["w_t1"], dt, "w_t1"), _ptr(w["b_t1"], dt, "b_t1"), _ptr(w["w_t2"], dt, "w_t2"),
                                _ptr(w["b_t2"], dt, "b_t2"), _ptr(w["class_table"], dt, "class_table"),
                                _ptr(cond, torch.float32, "cond"), _ptr(workspace, None, "workspace"),
                                workspace.numel() * workspace.element_size(), _stream(stream)))


def pos_embed_2d(grid_h: int, grid_w: int, hidden: int, pos: torch.Tensor, stream=None) -> None:
    _check(lib().dit_pos_embed_2d(grid_h, grid_w, hidden, _ptr(pos, torch.float32, "pos"), _stream(stream)))


def timing_enable(kclass: str, max_launches: int) -> None:
    _check(lib().dit_timing_enable(KERNEL_CLASSES[kclass], max_launches))


def timing_read():
    """(total_ms, launches, flops, bytes) of the launches recorded since timing_enable."""
    ms, n, fl, by = ctypes.c_double(), ctypes.c_int(), ctypes.c_double(), ctypes.c_double()
    _check(lib().dit_timing_read(ctypes.byref(ms), ctypes.byref(n), ctypes.byref(fl), ctypes.byref(by)))
    return ms.value, n.value, fl.value, by.value


def timing_disable() -> None:
    _check(lib().dit_timing_disable())
