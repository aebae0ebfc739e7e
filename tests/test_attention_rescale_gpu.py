"""GPU parity of attention's lazy max against the fp64 oracle.

The kernels keep the softmax's running max m_run fixed after the first key
tile and move it (rescaling O, l and the tile's scores) only when a tile's
scores lead it by more than 2^64 in the exp2 domain.  Ordinary inputs never
take that branch after the first tile, and their first tile's max sits near
zero; both cases are forced here:

- a move mid-sequence: the tokens of the first key tiles and those after a
  boundary lie along two different directions, the k projection is set equal
  to the q projection (so a query scores highest against keys of its own
  direction) and both are scaled by a power of two, so queries after the
  boundary see a later tile lead the first tiles' max by about a hundred or
  more (log2 units).  At 150 tokens the boundary at 64 or 128 tokens puts
  the move in the second or third key tile; at 600 tokens, boundaries at
  320 and 448 put it inside the second trip of the pipelined kernel's
  four-tile loop (its second and fourth ring slot).
- a first tile far below zero: the first tokens point the opposite way, so
  for queries after the boundary every score of the first tile is below
  -128, where the first max, taken as the new m_run, would overflow a
  rescale factor 2^-delta of the still-zero accumulators.

Each case checks with the oracle's own projections that the condition
really occurs before comparing the block output with the oracle.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import dit_oracle as O

pytestmark = pytest.mark.gpu

TOL = 2e-2


def _case(cfg, boundary, scale, amp, sign):
    """Block weights and inputs: tokens before `boundary` along sign * v
    (v = -u for sign -1), tokens after it along u; k projection = q
    projection, both times `scale` (a power of two: still exact bf16)."""
    w = {k: v.copy() for k, v in synth.block_weights(cfg, 0)["img"].items()}
    inp = synth.inputs(cfg)
    x, c = inp["x"].copy(), inp["cond"]
    D = cfg.hidden
    rng = np.random.default_rng([2605, 77, boundary])
    u = rng.standard_normal(D).astype(np.float32)
    v = rng.standard_normal(D).astype(np.float32) if sign > 0 else -u
    x[:, :boundary, :] += amp * v
    x[:, boundary:, :] += amp * u
    w["w_qkv"][D:2 * D] = w["w_qkv"][:D]
    w["b_qkv"][D:2 * D] = w["b_qkv"][:D]
    w["w_qkv"][:2 * D] *= scale
    w["b_qkv"][:2 * D] *= scale
    return w, x, c


def _scores(cfg, w, x, c):
    """Scores in the exp2 domain, [B, H, T, T], from the oracle's projections."""
    w = {k: a.astype(np.float64) for k, a in w.items()}
    sh, sc, *_ = O.adaln_modulation(c.astype(np.float64), w["w_ada"], w["b_ada"])
    h = O.modulate(O.layer_norm(x.astype(np.float64), cfg.ln_eps), sh, sc)
    q, k, _ = O.qkv_project(h, w["w_qkv"], w["b_qkv"], cfg.heads)
    return np.matmul(q, np.swapaxes(k, -1, -2)) / np.sqrt(cfg.head_dim) * np.log2(np.e)


def _compare(name, cfg, w, x, c):
    from tests import gpu_util
    y, _ = gpu_util.run_block(cfg, {"img": w}, x, c)
    ref = O.dit_block(x, c, {k: a.astype(np.float64) for k, a in w.items()}, cfg.heads, cfg.ln_eps)
    e_y = O.rel_err(y, ref)
    e_d = O.rel_err(y - x, ref - x)
    print(f"[rescale] {name}: err_y={e_y:.3e} err_delta={e_d:.3e}", flush=True)
    assert np.all(np.isfinite(y)), name
    assert e_y <= TOL and e_d <= TOL, (name, e_y, e_d)


def _cfg(kind):
    return {
        # >= 256 (sample, head, 256-query) items: the software-pipelined kernel
        "pipe_dh128": synth.CONFIGS["c1"].with_(batch=32, tokens=150, hidden=1024, heads=8, head_dim=128,
                                                mlp_hidden=512, n_blocks=1),
        "pipe_dh72_fold": synth.CONFIGS["c1"].with_(batch=16, tokens=150, n_blocks=1),
        "pipe_dh64": synth.CONFIGS["c1"].with_(batch=16, tokens=150, hidden=1024, heads=16, head_dim=64,
                                               mlp_hidden=512, n_blocks=1),
        # ten key tiles: two four-tile trips of the pipelined kernel's loop and two after them
        "pipe_dh128_long": synth.CONFIGS["c1"].with_(batch=12, tokens=600, hidden=1024, heads=8, head_dim=128,
                                                     mlp_hidden=512, n_blocks=1),
        "pipe_dh72_fold_long": synth.CONFIGS["c1"].with_(batch=6, tokens=600, n_blocks=1),
        "pipe_dh64_long": synth.CONFIGS["c1"].with_(batch=6, tokens=600, hidden=1024, heads=16, head_dim=64,
                                                    mlp_hidden=512, n_blocks=1),
        # small grids: the four-wave kernel
        "small_dh128": synth.CONFIGS["c1"].with_(batch=2, tokens=150, hidden=256, heads=2, head_dim=128,
                                                 mlp_hidden=512, n_blocks=1),
        "small_dh72_fold": synth.CONFIGS["c1"].with_(batch=2, tokens=150, hidden=576, heads=8, head_dim=72,
                                                     mlp_hidden=256, n_blocks=1),
    }[kind]


# (case, q/k scale): the least power of two that moves the max for most later queries
MOVE = [("pipe_dh128", 4.0), ("pipe_dh72_fold", 4.0), ("pipe_dh64", 8.0), ("small_dh128", 8.0),
        ("small_dh72_fold", 8.0)]
# (case, q/k scale, amplitude): first tiles far below zero for some later queries
LOW = [("pipe_dh128", 4.0, 20.0), ("pipe_dh72_fold", 4.0, 20.0), ("pipe_dh64", 8.0, 6.0),
       ("small_dh72_fold", 8.0, 6.0)]


MOVE_LONG = [("pipe_dh128_long", 4.0), ("pipe_dh72_fold_long", 4.0), ("pipe_dh64_long", 8.0)]


@pytest.mark.parametrize("boundary", [320, 448])
@pytest.mark.parametrize("name,scale", MOVE_LONG, ids=[m[0] for m in MOVE_LONG])
def test_lazy_max_moves_inside_a_loop_trip(name, scale, boundary):
    test_lazy_max_moves_mid_sequence(name, scale, boundary)


@pytest.mark.parametrize("boundary", [64, 128])
@pytest.mark.parametrize("name,scale", MOVE, ids=[m[0] for m in MOVE])
def test_lazy_max_moves_mid_sequence(name, scale, boundary):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cfg = _cfg(name)
    w, x, c = _case(cfg, boundary, scale, amp=6.0, sign=+1)
    s = _scores(cfg, w, x, c)
    lead = s[..., boundary:, boundary:].max(-1) - s[..., boundary:, :boundary].max(-1)
    frac = float((lead > 64.0).mean())
    print(f"[rescale] {name} boundary={boundary}: {frac:.2f} of the later queries move the max", flush=True)
    assert frac > 0.8, (name, boundary, frac)  # the branch is really exercised
    _compare(f"{name}/move{boundary}", cfg, w, x, c)


@pytest.mark.parametrize("boundary", [64, 128])
@pytest.mark.parametrize("name,scale,amp", LOW, ids=[m[0] for m in LOW])
def test_first_tile_far_below_zero(name, scale, amp, boundary):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cfg = _cfg(name)
    w, x, c = _case(cfg, boundary, scale, amp=amp, sign=-1)
    s = _scores(cfg, w, x, c)
    first = s[..., boundary:, :64].max(-1)
    n_low = int((first < -128.0).sum())
    print(f"[rescale] {name} boundary={boundary}: {n_low} (sample, head, query) with a first-tile max "
          f"below -128", flush=True)
    assert n_low >= 8, (name, boundary, n_low)
    _compare(f"{name}/low{boundary}", cfg, w, x, c)


def test_split_key_ranges_lazy_max():
    """The pipelined kernel's last, partial round of work items runs as key
    ranges merged afterwards (33 query blocks x 8 heads = 264 items: the last
    8, queries 6400.. of head 7, as 8 ranges of 16-17 key tiles).  Tokens
    before 1280 point against those after it, so for every split query the
    first tile of ranges 0 and 1 lies below -128 and, inside range 1, tile 20
    leads tiles 16-19 by more than 64 (log2 units)."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cfg = synth.CONFIGS["c4"].with_(tokens=8448, hidden=1024, heads=8, head_dim=128, mlp_hidden=1024, n_blocks=1)
    w, x, c = _case(cfg, 1280, 8.0, amp=6.0, sign=-1)
    s = _scores(cfg, w, x, c)[0, 7, 6400:]
    low0 = int((s[:, :64].max(-1) < -128.0).sum())
    low1 = int((s[:, 16 * 64:17 * 64].max(-1) < -128.0).sum())
    lead = s[:, 20 * 64:21 * 64].max(-1) - s[:, 16 * 64:20 * 64].max(-1)
    frac = float((lead > 64.0).mean())
    print(f"[rescale] split ranges: {low0} / {low1} split queries with range 0 / 1 starting below -128, "
          f"{frac:.2f} moving the max inside range 1", flush=True)
    assert low0 >= 1000 and low1 >= 1000 and frac > 0.8, (low0, low1, frac)
    _compare("split_ranges", cfg, w, x, c)
