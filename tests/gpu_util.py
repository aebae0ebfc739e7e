"""Helpers for the GPU tests: upload seeded synthetic weights, call the C ABI
through the binding, download results.  Imports torch.cuda lazily so the CPU
suite can import this module."""
from __future__ import annotations

import numpy as np
import torch

import paper_2605_25550_amd as dm
import synth


def dev(a, dtype=torch.float32) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).to(device="cuda", dtype=dtype)


def host(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def upload_stream(w, dt):
    return {k: dev(v, dt) for k, v in w.items()}


class DeviceBlock:
    """One block's weights on the device plus the ctypes struct pointing at them."""

    def __init__(self, cfg, w_np):
        self.shape = dm.shape_of(cfg.with_(n_blocks=1))
        self.dt = dm.weight_dtype(self.shape)
        self.img = upload_stream(w_np["img"], self.dt)
        self.txt = upload_stream(w_np["txt"], self.dt) if cfg.joint else None
        self.struct = dm.block_struct(self.img, self.txt, self.dt)


def run_block(cfg, w_np, x, cond, x_txt=None, repeat=1):
    """Runs dit_block_forward; returns (y, y_txt) as float64 numpy arrays."""
    db = DeviceBlock(cfg, w_np)
    ws = dm.alloc_workspace(db.shape, dm.DIT_WS_BLOCK)
    outs = []
    for _ in range(repeat):
        xd = dev(x)
        xtd = dev(x_txt) if x_txt is not None else None
        dm.block_forward(db.shape, db.struct, xd, dev(cond), ws, x_txt=xtd)
        torch.cuda.synchronize()
        outs.append((host(xd), host(xtd) if xtd is not None else None))
    return outs[0] if repeat == 1 else outs


class DeviceStep:
    """All step weights of a config on the device."""

    def __init__(self, cfg, blocks_np=None, step_np=None):
        self.cfg = cfg
        self.shape = dm.shape_of(cfg)
        self.dt = dm.weight_dtype(self.shape)
        step_np = step_np if step_np is not None else synth.step_weights(cfg)
        self.step = {k: dev(v, self.dt) for k, v in step_np.items()}
        self.blocks = []
        structs = []
        for l in range(cfg.n_blocks):
            bw = blocks_np[l] if blocks_np is not None else synth.block_weights(cfg, l)
            img = upload_stream(bw["img"], self.dt)
            txt = upload_stream(bw["txt"], self.dt) if cfg.joint else None
            self.blocks.append((img, txt))
            structs.append(dm.block_struct(img, txt, self.dt))
        self.pos = None
        if cfg.grid is not None:  # fixed 2-D sin-cos table, computed on the device
            self.pos = torch.empty((cfg.grid[0] * cfg.grid[1], cfg.hidden), dtype=torch.float32, device="cuda")
            dm.pos_embed_2d(cfg.grid[0], cfg.grid[1], cfg.hidden, self.pos)
        self.table = dm.StepWeightTable(self.step, structs, self.dt, self.pos)
        self.ws = dm.alloc_workspace(self.shape, dm.DIT_WS_STEP)

    def run(self, patches, cond, x_txt=None):
        c = self.cfg
        out = torch.empty((c.batch, c.tokens, c.patch_out), dtype=torch.float32, device="cuda")
        xtd = dev(x_txt) if x_txt is not None else None
        dm.step_forward(self.shape, self.table, dev(patches), dev(cond), out, self.ws, x_txt=xtd)
        torch.cuda.synchronize()
        return host(out), (host(xtd) if xtd is not None else None)


def zero_gates(w, D):
    """Copy of stream weights with the two gate chunks of adaLN zeroed."""
    w = {k: v.copy() for k, v in w.items()}
    for ch in (2, 5):
        w["w_ada"][ch * D:(ch + 1) * D] = 0.0
        w["b_ada"][ch * D:(ch + 1) * D] = 0.0
    return w
