"""Seeded synthetic inputs for the DiT denoising step.

This module is shared by the fp64 oracle and by the GPU harness (tests,
bench, smoke).  It holds shapes and random draws only: none of the
denoising step's arithmetic lives here.

The shapes stand in for the paper's workloads (DiT-stage forward of the
Encoder-Transformer-Decoder pipeline, Background: Diffusion Model
Architecture; Workload Characteristics), whose trained weights and prompts
are not available: every tensor is drawn from a fixed distribution under a
seed derived from (config, block, tensor).
"""
from __future__ import annotations

import concurrent.futures as cf
import dataclasses
import os
from typing import Dict, Optional

import numpy as np

SEED_ROOT = 2605


@dataclasses.dataclass(frozen=True)
class DiTConfig:
    """Shape of one DiT workload.

    tokens       image/latent patch tokens per sample (T)
    text_tokens  text tokens of the joint two-stream block (0: single stream)
    patch_in     channels of one flattened latent patch (p*p*C)
    patch_out    channels predicted per token by the final layer
    cond         'class': timestep + class-label embedding computes c;
                 'given': the pooled conditioning vector c is an input
    grid         (h, w) patch grid for the fixed 2-D sin-cos position table,
                 or None when the model adds no position table
    """
    key: str
    index: int
    name: str
    batch: int
    tokens: int
    text_tokens: int
    hidden: int
    heads: int
    head_dim: int
    mlp_hidden: int
    n_blocks: int
    patch_in: int
    patch_out: int
    dtype: str            # 'f32' or 'bf16' (weights and GEMM operands)
    cond: str             # 'class' or 'given'
    grid: Optional[tuple]
    ln_eps: float = 1e-6
    n_classes: int = 1000
    freq_dim: int = 256

    def with_(self, **kw) -> "DiTConfig":
        return dataclasses.replace(self, **kw)

    @property
    def joint(self) -> bool:
        return self.text_tokens > 0


CONFIGS: Dict[str, DiTConfig] = {
    # 32x32x4 latent, patch 2 -> 16x16 = 256 tokens; one block in fp32.
    "c0": DiTConfig("c0", 0, "dit_block_fp32_t256_d384", batch=1, tokens=256, text_tokens=0,
                    hidden=384, heads=6, head_dim=64, mlp_hidden=1536, n_blocks=1,
                    patch_in=16, patch_out=16, dtype="f32", cond="given", grid=(16, 16)),
    # DiT-XL/2 at a 32x32x4 latent: 256 tokens, batch 8.
    "c1": DiTConfig("c1", 1, "dit_xl2_256px_b8", batch=8, tokens=256, text_tokens=0,
                    hidden=1152, heads=16, head_dim=72, mlp_hidden=4608, n_blocks=28,
                    patch_in=16, patch_out=16, dtype="bf16", cond="class", grid=(16, 16)),
    # DiT-XL/2 at a 64x64x4 latent: 1024 tokens, batch 4.
    "c2": DiTConfig("c2", 2, "dit_xl2_512px_b4", batch=4, tokens=1024, text_tokens=0,
                    hidden=1152, heads=16, head_dim=72, mlp_hidden=4608, n_blocks=28,
                    patch_in=16, patch_out=16, dtype="bf16", cond="class", grid=(32, 32)),
    # Joint text-image DiT: 128x128x16 latent, patch 2 -> 4096 image tokens + 256 text tokens.
    "c3": DiTConfig("c3", 3, "joint_dit_4096img_256txt", batch=1, tokens=4096, text_tokens=256,
                    hidden=3072, heads=24, head_dim=128, mlp_hidden=12288, n_blocks=24,
                    patch_in=64, patch_out=64, dtype="bf16", cond="given", grid=None),
    # Video DiT: 13 latent frames x 30x45 patches = 17550 tokens.
    "c4": DiTConfig("c4", 4, "video_dit_17550tok", batch=1, tokens=17550, text_tokens=0,
                    hidden=3072, heads=24, head_dim=128, mlp_hidden=12288, n_blocks=30,
                    patch_in=64, patch_out=64, dtype="bf16", cond="given", grid=None),
}

# Tensor ids inside one (config, block) seed stream.
_T = {name: i for i, name in enumerate([
    "w_ada", "b_ada", "w_qkv", "b_qkv", "w_o", "b_o", "w_fc1", "b_fc1", "w_fc2", "b_fc2",
])}
_STEP_T = {name: 100 + i for i, name in enumerate([
    "w_patch", "b_patch", "w_ada_final", "b_ada_final", "w_final", "b_final",
    "w_t1", "b_t1", "w_t2", "b_t2", "class_table",
])}
_INPUT_T = {name: 200 + i for i, name in enumerate([
    "x", "x_txt", "cond", "patches", "t", "y",
])}
WEIGHT_STD = 0.02
STREAM_IMG, STREAM_TXT = 0, 1


def _rng(cfg: DiTConfig, block: int, tensor_id: int, salt: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([SEED_ROOT, cfg.index, block + 2, tensor_id, salt]))


def _bf16_round_inplace(a: np.ndarray) -> None:
    """Rounds a float32 array to the nearest bfloat16 (ties to even) in place."""
    nan = np.isnan(a)
    u = a.view(np.uint32)
    r = u >> 16
    r &= 1
    r += 0x7FFF
    u += r
    u &= np.uint32(0xFFFF0000)
    if nan.any():
        a[nan] = np.nan


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32.

    Input preparation only: the bf16 path consumes bf16 weights, and the oracle
    consumes the same values upcast exactly.  NaN stays NaN.
    """
    out = np.array(a, dtype=np.float32, copy=True, order="C")
    _bf16_round_inplace(out.reshape(-1))
    return out


# Large tensors are drawn in chunks of _CHUNK values, chunk i from its own
# seed stream (the tensor's seed plus i), so the chunks can be drawn on
# several threads and the values do not depend on how many run.
_CHUNK = 1 << 22
_POOL: Optional[cf.ThreadPoolExecutor] = None


def _pool() -> cf.ThreadPoolExecutor:
    global _POOL
    if _POOL is None:
        _POOL = cf.ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1))
    return _POOL


def _normal(cfg, block, tid, shape, std, salt=0, weight=True):
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.float32)
    rnd = weight and cfg.dtype == "bf16"

    def fill(i):
        seg = out[i * _CHUNK:(i + 1) * _CHUNK]
        np.random.default_rng(np.random.SeedSequence([SEED_ROOT, cfg.index, block + 2, tid, salt, i])) \
            .standard_normal(out=seg, dtype=np.float32)
        if std != 1.0:
            seg *= np.float32(std)
        if rnd:
            _bf16_round_inplace(seg)

    nch = (n + _CHUNK - 1) // _CHUNK
    if nch <= 1:
        for i in range(nch):
            fill(i)
    else:
        list(_pool().map(fill, range(nch)))
    return out.reshape(shape)


def stream_weights(cfg: DiTConfig, block: int, stream: int = STREAM_IMG) -> Dict[str, np.ndarray]:
    """Weights of one stream of one block, [out, in] row-major, float32 values
    (bf16-representable when cfg.dtype == 'bf16'). Gate rows are drawn like the
    rest (not zero)."""
    D, F = cfg.hidden, cfg.mlp_hidden
    shapes = {"w_ada": (6 * D, D), "b_ada": (6 * D,), "w_qkv": (3 * D, D), "b_qkv": (3 * D,),
              "w_o": (D, D), "b_o": (D,), "w_fc1": (F, D), "b_fc1": (F,), "w_fc2": (D, F), "b_fc2": (D,)}
    return {k: _normal(cfg, block, _T[k], s, WEIGHT_STD, salt=stream) for k, s in shapes.items()}


def block_weights(cfg: DiTConfig, block: int) -> Dict[str, Dict[str, np.ndarray]]:
    w = {"img": stream_weights(cfg, block, STREAM_IMG)}
    if cfg.joint:
        w["txt"] = stream_weights(cfg, block, STREAM_TXT)
    return w


def step_weights(cfg: DiTConfig) -> Dict[str, np.ndarray]:
    """Patch embedding, final layer and (class-conditioned configs) the
    timestep/class conditioning weights."""
    D, Pi, Po = cfg.hidden, cfg.patch_in, cfg.patch_out
    shapes = {"w_patch": (D, Pi), "b_patch": (D,), "w_ada_final": (2 * D, D), "b_ada_final": (2 * D,),
              "w_final": (Po, D), "b_final": (Po,)}
    if cfg.cond == "class":
        shapes.update({"w_t1": (D, cfg.freq_dim), "b_t1": (D,), "w_t2": (D, D), "b_t2": (D,),
                       "class_table": (cfg.n_classes + 1, D)})
    return {k: _normal(cfg, -1, _STEP_T[k], s, WEIGHT_STD) for k, s in shapes.items()}


def inputs(cfg: DiTConfig, salt: int = 0) -> Dict[str, np.ndarray]:
    """Block/step inputs: residual tokens x [B,T,D], text tokens x_txt [B,Tt,D],
    conditioning c [B,D], latent patches [B,T,patch_in] (all N(0,1) fp32), and
    for class-conditioned configs integer timesteps t in [0,999] and labels y in
    [0,999]."""
    B, T, Tt, D = cfg.batch, cfg.tokens, cfg.text_tokens, cfg.hidden
    out = {
        "x": _normal(cfg, -2, _INPUT_T["x"], (B, T, D), 1.0, salt, weight=False),
        "cond": _normal(cfg, -2, _INPUT_T["cond"], (B, D), 1.0, salt, weight=False),
        "patches": _normal(cfg, -2, _INPUT_T["patches"], (B, T, cfg.patch_in), 1.0, salt, weight=False),
    }
    if Tt:
        out["x_txt"] = _normal(cfg, -2, _INPUT_T["x_txt"], (B, Tt, D), 1.0, salt, weight=False)
    if cfg.cond == "class":
        out["t"] = _rng(cfg, -2, _INPUT_T["t"], salt).integers(0, 1000, size=(B,)).astype(np.float32)
        out["y"] = _rng(cfg, -2, _INPUT_T["y"], salt).integers(0, cfg.n_classes, size=(B,)).astype(np.int32)
    return out


def small(cfg: DiTConfig, **kw) -> DiTConfig:
    """A reduced copy of a config (fewer tokens/blocks/batch) for oracle-speed tests."""
    return cfg.with_(**kw)
