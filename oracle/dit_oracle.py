"""fp64 CPU oracle of the DiT denoising step.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU
baseline leg of the benchmark may import this module.  The product path
(the HIP library and its binding) never calls it, and this module never
imports the product package: the two share only the seeded input generator
in ``synth``, which holds no arithmetic of the method.

What is computed.  The paper (Background and Motivation: Diffusion Model
Architecture; Workload Characteristics) names the Diffusion Transformer as
the stage that iteratively denoises the latent and dominates run time, with
attention cost growing as O(T^2 D); it does not write the block out.  The
block followed here is the adaLN-Zero DiT block of the work the paper cites
for that stage (Peebles & Xie, "Scalable Diffusion Models with
Transformers", arXiv:2212.09748): conditioning-dependent shift/scale/gate
vectors, LayerNorm without affine, multi-head self-attention and a tanh-GELU
MLP, each branch added back through its gate.  Every function below is the
plain definition, written in float64 with numpy; contractions use np.matmul.
There is no blocking, fusion or online softmax: the score matrix is
materialised per (sample, head), in slices of query rows for long sequences
(each slice is still the exact row-wise softmax).

Readings taken where the paper is silent (each is also listed in the
design notes):
  * modulation chunk order (shift, scale, gate) for attention then MLP;
    modulate(z) = z * (1 + scale) + shift; SiLU before the adaLN linear;
  * LayerNorm: biased variance, eps = 1e-6, no affine;
  * every linear layer has a bias;
  * GELU is the tanh approximation;
  * attention: full, bidirectional, scale 1/sqrt(head_dim), no mask, no
    positional terms inside the block;
  * joint (two-stream) block: each stream has its own weights and the same
    conditioning; attention runs over the concatenation [image; text];
  * step = patch embedding (+ fixed 2-D sin-cos table when the model has a
    patch grid) -> blocks -> final layer;
  * the multi-step loop (sample_euler) is the first-order Euler method on the
    flow-matching ODE in the patchified latent space, z += (s_{i+1} - s_i) v,
    with the timestep t_i = s_i * t_scale rounded to float32.

Parity status: every function here is pinned by a CPU test against facts of
the mathematics (identity under zero gates, softmax normalisation, the
single-token closed form, brute-force attention, permutation equivariance,
library routines of torch in float64, closed forms of the embeddings).  The
end-to-end step composition is pinned only as the composition of pinned
parts plus the zero-gate closed form of the whole step.
"""
from __future__ import annotations

import concurrent.futures as cf
import math
import os
from typing import Dict, Optional, Sequence, Tuple

import numpy as np
from threadpoolctl import threadpool_limits

F64 = np.float64


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=F64)


# Execution only, no arithmetic: independent pieces of work (the heads of
# attention, slices of token rows for row-wise functions) are evaluated on
# several host threads, each with exactly the arithmetic it has when run
# alone, so that full-size configurations finish in test time.
_POOL: Optional[cf.ThreadPoolExecutor] = None


def _pool() -> cf.ThreadPoolExecutor:
    global _POOL
    if _POOL is None:
        _POOL = cf.ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1))
    return _POOL


def _token_slices(T: int, n: int):
    step = max(1, -(-T // n))
    return [slice(t, min(T, t + step)) for t in range(0, T, step)]


def _rowwise(fn, x: np.ndarray, *per_sample) -> np.ndarray:
    """fn applied to slices of the token axis (axis 1 of [B, T, ...]) of x,
    with any per-sample arguments passed whole: for functions whose result at
    a token depends only on that token's row."""
    x = _f64(x)
    T = x.shape[1] if x.ndim == 3 else 0
    if x.size < (1 << 20) or T < 2:
        return fn(x, *per_sample)
    sl = _token_slices(T, 4 * _pool()._max_workers)
    parts = list(_pool().map(lambda s_: fn(x[:, s_], *per_sample), sl))
    return np.concatenate(parts, axis=1)


# ---------------------------------------------------------------- elementwise
def silu(z: np.ndarray) -> np.ndarray:
    """SiLU(z) = z * sigmoid(z), applied to the conditioning vector before every
    adaLN linear (adaLN-Zero block of the cited DiT work)."""
    z = _f64(z)
    return z / (1.0 + np.exp(-z))


def gelu_tanh(u: np.ndarray) -> np.ndarray:
    """tanh-approximated GELU: 0.5 u (1 + tanh(sqrt(2/pi) (u + 0.044715 u^3)))."""
    u = _f64(u)
    return 0.5 * u * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (u + 0.044715 * u * u * u)))


def layer_norm(x: np.ndarray, eps: float) -> np.ndarray:
    """LayerNorm over the last axis without affine: (x - mean) / sqrt(var + eps),
    var the biased (population) variance."""
    x = _f64(x)
    mu = x.mean(axis=-1, keepdims=True)
    d = x - mu
    var = (d * d).mean(axis=-1, keepdims=True)
    return d / np.sqrt(var + eps)


def modulate(xn: np.ndarray, shift: np.ndarray, scale: np.ndarray) -> np.ndarray:
    """xn * (1 + scale) + shift with per-sample shift/scale [B, D] broadcast over tokens."""
    return _f64(xn) * (1.0 + _f64(scale)[:, None, :]) + _f64(shift)[:, None, :]


def linear(x: np.ndarray, w: np.ndarray, b: Optional[np.ndarray]) -> np.ndarray:
    """y = x W^T + b with W stored [out, in]."""
    y = np.matmul(_f64(x), _f64(w).T)
    if b is not None:
        y = y + _f64(b)
    return y


# ---------------------------------------------------------------- adaLN-Zero
MOD_NAMES = ("shift_msa", "scale_msa", "gate_msa", "shift_mlp", "scale_mlp", "gate_mlp")


def adaln_modulation(c: np.ndarray, w_ada: np.ndarray, b_ada: np.ndarray, n_chunks: int = 6) -> Tuple[np.ndarray, ...]:
    """m = SiLU(c) W_ada^T + b_ada, split along features into n_chunks vectors of
    width D: (shift_msa, scale_msa, gate_msa, shift_mlp, scale_mlp, gate_mlp) for a
    block, (shift, scale) for the final layer."""
    m = linear(silu(c), w_ada, b_ada)
    D = m.shape[-1] // n_chunks
    return tuple(m[:, i * D:(i + 1) * D] for i in range(n_chunks))


# ---------------------------------------------------------------- attention
def attention_heads(q: np.ndarray, k: np.ndarray, v: np.ndarray, rows: Optional[Sequence[int]] = None,
                    chunk: int = 2048) -> np.ndarray:
    """Scaled dot-product attention per head, plain definition.

    q: [B, H, Tq, dh], k, v: [B, H, Tk, dh].  For each (b, h):
    S = q k^T / sqrt(dh); P = row-softmax(S) (row max subtracted, exact exp);
    O = P v.  ``rows`` restricts the query rows computed (all keys are used).
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, H, Tq, dh = q.shape
    if rows is not None:
        q = q[:, :, np.asarray(rows), :]
        Tq = q.shape[2]
    out = np.empty((B, H, Tq, dh), dtype=F64)
    scale = 1.0 / math.sqrt(dh)

    def one_head(bh):
        b, h = bh
        kt = k[b, h].T
        for r0 in range(0, Tq, chunk):
            s = np.matmul(q[b, h, r0:r0 + chunk], kt) * scale
            s = s - s.max(axis=-1, keepdims=True)
            p = np.exp(s)
            p /= p.sum(axis=-1, keepdims=True)
            out[b, h, r0:r0 + chunk] = np.matmul(p, v[b, h])

    pairs = [(b, h) for b in range(B) for h in range(H)]
    if len(pairs) > 1 and Tq * k.shape[2] >= (1 << 20):
        with threadpool_limits(limits=1, user_api="blas"):  # one BLAS thread per head
            list(_pool().map(one_head, pairs))
    else:
        for bh in pairs:
            one_head(bh)
    return out


def split_heads(t: np.ndarray, heads: int) -> np.ndarray:
    """[B, T, H*dh] -> [B, H, T, dh] (column = head*dh + d)."""
    B, T, D = t.shape
    return t.reshape(B, T, heads, D // heads).transpose(0, 2, 1, 3)


def merge_heads(t: np.ndarray) -> np.ndarray:
    """[B, H, T, dh] -> [B, T, H*dh]."""
    B, H, T, dh = t.shape
    return t.transpose(0, 2, 1, 3).reshape(B, T, H * dh)


def qkv_project(h: np.ndarray, w_qkv: np.ndarray, b_qkv: np.ndarray, heads: int):
    """qkv = h W_qkv^T + b; column j = s*D + head*dh + d with s in (q, k, v)."""
    D = h.shape[-1]
    qkv = linear(h, w_qkv, b_qkv)
    return tuple(split_heads(qkv[..., s * D:(s + 1) * D], heads) for s in range(3))


# ---------------------------------------------------------------- blocks
def dit_block(x: np.ndarray, c: np.ndarray, w: Dict[str, np.ndarray], heads: int, eps: float = 1e-6,
              rows: Optional[Sequence[int]] = None) -> np.ndarray:
    """One adaLN-Zero DiT block (the DiT-stage unit of work; attention part of
    the O(T^2 D) cost the paper attributes to this stage).

    x: [B, T, D] residual stream, c: [B, D] conditioning, w: stream weights.
      (shift1, scale1, gate1, shift2, scale2, gate2) = adaLN(c)
      x1 = x  + gate1 * Attn(modulate(LN(x),  shift1, scale1)) W_o^T + b_o
      y  = x1 + gate2 * (GELU(modulate(LN(x1), shift2, scale2) W_1^T + b_1) W_2^T + b_2)
    ``rows`` returns only those token rows (every token still feeds K and V).
    """
    x = _f64(x)
    sh1, sc1, g1, sh2, sc2, g2 = adaln_modulation(c, w["w_ada"], w["b_ada"])
    h = _ln_modulate(x, sh1, sc1, eps)
    q, k, v = qkv_project(h, w["w_qkv"], w["b_qkv"], heads)
    o = merge_heads(attention_heads(q, k, v, rows=rows))
    xs = x if rows is None else x[:, np.asarray(rows), :]
    x1 = xs + g1[:, None, :] * linear(o, w["w_o"], w["b_o"])
    return _mlp_branch(x1, sh2, sc2, g2, w, eps)


def _ln_modulate(x, shift, scale, eps):
    """modulate(LN(x), shift, scale), evaluated over slices of tokens."""
    return _rowwise(lambda xs, sh, sc: modulate(layer_norm(xs, eps), sh, sc), x, shift, scale)


def _mlp_branch(x1, sh2, sc2, g2, w, eps):
    h2 = _ln_modulate(x1, sh2, sc2, eps)
    g = _rowwise(gelu_tanh, linear(h2, w["w_fc1"], w["b_fc1"]))
    return x1 + g2[:, None, :] * linear(g, w["w_fc2"], w["b_fc2"])


def joint_block(x_img: np.ndarray, x_txt: np.ndarray, c: np.ndarray, w_img: Dict[str, np.ndarray],
                w_txt: Dict[str, np.ndarray], heads: int, eps: float = 1e-6,
                rows_img: Optional[Sequence[int]] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Two-stream (joint text-image) block: each stream modulates, projects and
    runs its MLP with its own weights under the same conditioning c; attention is
    one softmax over the concatenated tokens [image; text].  Returns
    (y_img, y_txt); ``rows_img`` restricts the image rows returned (text rows are
    then still all returned)."""
    x_img, x_txt = _f64(x_img), _f64(x_txt)
    Ti = x_img.shape[1]
    mi = adaln_modulation(c, w_img["w_ada"], w_img["b_ada"])
    mt = adaln_modulation(c, w_txt["w_ada"], w_txt["b_ada"])
    hi = _ln_modulate(x_img, mi[0], mi[1], eps)
    ht = _ln_modulate(x_txt, mt[0], mt[1], eps)
    qi, ki, vi = qkv_project(hi, w_img["w_qkv"], w_img["b_qkv"], heads)
    qt, kt, vt = qkv_project(ht, w_txt["w_qkv"], w_txt["b_qkv"], heads)
    q = np.concatenate([qi, qt], axis=2)
    k = np.concatenate([ki, kt], axis=2)
    v = np.concatenate([vi, vt], axis=2)
    Tt = x_txt.shape[1]
    if rows_img is None:
        rows = None
        sel_img = np.arange(Ti)
    else:
        sel_img = np.asarray(rows_img)
        rows = np.concatenate([sel_img, Ti + np.arange(Tt)])
    o = merge_heads(attention_heads(q, k, v, rows=rows))
    n_img = len(sel_img)
    o_img, o_txt = o[:, :n_img], o[:, n_img:]
    x1i = x_img[:, sel_img] + mi[2][:, None, :] * linear(o_img, w_img["w_o"], w_img["b_o"])
    x1t = x_txt + mt[2][:, None, :] * linear(o_txt, w_txt["w_o"], w_txt["b_o"])
    yi = _mlp_branch(x1i, mi[3], mi[4], mi[5], w_img, eps)
    yt = _mlp_branch(x1t, mt[3], mt[4], mt[5], w_txt, eps)
    return yi, yt


# ---------------------------------------------------------------- step pieces
def timestep_embedding(t: np.ndarray, dim: int = 256, max_period: float = 10000.0) -> np.ndarray:
    """Sinusoidal timestep features of the cited DiT work: f_i = exp(-ln(max_period) i / (dim/2)),
    i = 0..dim/2-1; e = [cos(t f), sin(t f)]."""
    half = dim // 2
    f = np.exp(-math.log(max_period) * np.arange(half, dtype=F64) / half)
    a = _f64(t)[:, None] * f[None, :]
    return np.concatenate([np.cos(a), np.sin(a)], axis=-1)


def class_conditioning(t, y, w_t1, b_t1, w_t2, b_t2, class_table, freq_dim: int = 256) -> np.ndarray:
    """Conditioning of class-conditional DiT: c = MLP(timestep_embedding(t)) + E[y],
    MLP = Linear(freq_dim -> D), SiLU, Linear(D -> D)."""
    e = timestep_embedding(t, freq_dim)
    h = silu(linear(e, w_t1, b_t1))
    return linear(h, w_t2, b_t2) + _f64(class_table)[np.asarray(y, dtype=np.int64)]


def pos_embed_2d(grid_h: int, grid_w: int, dim: int) -> np.ndarray:
    """Fixed 2-D sin-cos position table [grid_h*grid_w, dim] of the cited DiT work,
    token n = r*grid_w + c.  The first dim/2 features encode the column c, the last
    dim/2 the row r; each half is [sin(p w_i), cos(p w_i)], w_i = 10000^(-i/(dim/4)),
    i = 0..dim/4-1."""
    assert dim % 4 == 0
    q = dim // 4
    omega = 1.0 / (10000.0 ** (np.arange(q, dtype=F64) / q))
    r, cidx = np.meshgrid(np.arange(grid_h, dtype=F64), np.arange(grid_w, dtype=F64), indexing="ij")
    def one(p):
        a = p.reshape(-1)[:, None] * omega[None, :]
        return np.concatenate([np.sin(a), np.cos(a)], axis=1)
    return np.concatenate([one(cidx), one(r)], axis=1)


def patch_embed(patches: np.ndarray, w_patch, b_patch, pos: Optional[np.ndarray]) -> np.ndarray:
    """x0 = z W_p^T + b_p (+ pos): patches [B, T, p*p*C] -> tokens [B, T, D]."""
    x = linear(patches, w_patch, b_patch)
    if pos is not None:
        x = x + _f64(pos)[None]
    return x


def final_layer(x: np.ndarray, c: np.ndarray, w_ada_final, b_ada_final, w_final, b_final, eps: float = 1e-6) -> np.ndarray:
    """Final layer: (shift, scale) = adaLN(c); out = modulate(LN(x), shift, scale) W_f^T + b_f."""
    sh, sc = adaln_modulation(c, w_ada_final, b_ada_final, n_chunks=2)
    return linear(modulate(layer_norm(x, eps), sh, sc), w_final, b_final)


def dit_step(cfg, patches: np.ndarray, cond: np.ndarray, step_w: Dict[str, np.ndarray], blocks,
             x_txt: Optional[np.ndarray] = None, pos: Optional[np.ndarray] = None):
    """One DiT denoising step (one full DiT-stage forward, the unit the paper's
    per-stage times are built from, Table: per-stage execution time):
    patch embed (+pos) -> n_blocks blocks -> final layer.  ``blocks`` is a
    sequence (or generator) of per-block weight dicts {'img': ..., 'txt': ...}.
    Returns (out [B,T,patch_out], x_txt after the last block or None)."""
    x = patch_embed(patches, step_w["w_patch"], step_w["b_patch"], pos)
    xt = None if x_txt is None else _f64(x_txt)
    for bw in blocks:
        if xt is not None:
            x, xt = joint_block(x, xt, cond, bw["img"], bw["txt"], cfg.heads, cfg.ln_eps)
        else:
            x = dit_block(x, cond, bw["img"], cfg.heads, cfg.ln_eps)
    out = final_layer(x, cond, step_w["w_ada_final"], step_w["b_ada_final"], step_w["w_final"],
                      step_w["b_final"], cfg.ln_eps)
    return out, xt


# ---------------------------------------------------------------- multi-step loop
def sample_euler(cfg, z0: np.ndarray, sigmas: Sequence[float], step_w: Dict[str, np.ndarray], blocks, *,
                 t_scale: float = 1000.0, y: Optional[np.ndarray] = None, cond: Optional[np.ndarray] = None,
                 x_txt: Optional[np.ndarray] = None, pos: Optional[np.ndarray] = None) -> np.ndarray:
    """The DiT stage's iterative denoising loop.  The paper (Background and
    Motivation, Workload Characteristics) has the DiT run many iterations per
    request (40-50 for standard samplers, 4 or 8 for distilled ones), and its
    Transformer service runs the backbone over the diffusion timesteps and
    updates the latent (System Design); it names no sampler.  The reading
    taken: first-order Euler on the flow-matching ODE dz/dsigma = v(z, sigma)
    in the patchified latent space [B, T, P] (P = patch_in = patch_out):

        v_i     = dit_step(z_i, c_i)
        z_{i+1} = z_i + (sigma_{i+1} - sigma_i) * v_i,   i = 0 .. n-1,

    with c_i = class_conditioning(t_i, y), t_i = float32(float32(sigma_i) *
    float32(t_scale)), for class-conditioned models, and the given cond
    otherwise.  Joint models restart every step from the given text states
    x_txt.  sigma differences are taken in float32, as the schedule is given
    in float32.  Returns z_n."""
    sig = np.asarray(sigmas, dtype=np.float32)
    z = _f64(z0)
    blocks = list(blocks)
    for i in range(len(sig) - 1):
        if y is not None:
            t = np.full(z.shape[0], np.float32(sig[i] * np.float32(t_scale)), dtype=np.float64)
            c = class_conditioning(t, y, step_w["w_t1"], step_w["b_t1"], step_w["w_t2"], step_w["b_t2"],
                                   step_w["class_table"])
        else:
            c = _f64(cond)
        v, _ = dit_step(cfg, z, c, step_w, blocks, x_txt=x_txt, pos=pos)
        z = z + F64(np.float32(sig[i + 1] - sig[i])) * v
    return z


# ---------------------------------------------------------------- error metric
def rel_err(got: np.ndarray, ref: np.ndarray) -> float:
    """max|got - ref| / max|ref| over the whole tensor (the parity metric)."""
    got, ref = _f64(got), _f64(ref)
    den = float(np.max(np.abs(ref))) if ref.size else 0.0
    num = float(np.max(np.abs(got - ref))) if ref.size else 0.0
    if den == 0.0:
        return num
    return num / den
