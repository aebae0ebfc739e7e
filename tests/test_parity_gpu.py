"""GPU parity of the HIP path (through the C ABI) against the fp64 oracle on
the same seeded inputs.

Metric: err = max|gpu - oracle| / max|oracle| over the compared tensor,
applied to the block output y AND to the branch increment y - x (the exact
pass-through of x would otherwise hide branch errors).  Bars: 2e-2 for the
bf16 path, 1e-4 for the fp32 path.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import dit_oracle as O

pytestmark = pytest.mark.gpu

TOL = {"bf16": 2e-2, "f32": 1e-4}


def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests import gpu_util
    return gpu_util


def f64(w):
    return {k: v.astype(np.float64) for k, v in w.items()}


def check(name, got, ref, base, tol):
    e_y = O.rel_err(got, ref)
    e_d = O.rel_err(got - base, ref - base) if base is not None else e_y
    print(f"[parity] {name}: err_y={e_y:.3e} err_delta={e_d:.3e} tol={tol:g}", flush=True)
    assert np.all(np.isfinite(got)), name
    assert e_y <= tol and e_d <= tol, (name, e_y, e_d)


def block_case(cfg, salt=0, rows=None, block=0):
    g = _gpu()
    w = synth.block_weights(cfg, block)
    inp = synth.inputs(cfg, salt)
    x, c = inp["x"], inp["cond"]
    xt = inp.get("x_txt")
    y, yt = g.run_block(cfg, w, x, c, xt)
    tol = TOL[cfg.dtype]
    if cfg.joint:
        ry, ryt = O.joint_block(x, xt, c, f64(w["img"]), f64(w["txt"]), cfg.heads, cfg.ln_eps, rows_img=rows)
        sel = slice(None) if rows is None else rows
        check(f"{cfg.key}/img", y[:, sel], ry, x[:, sel], tol)
        check(f"{cfg.key}/txt", yt, ryt, xt, tol)
    else:
        ry = O.dit_block(x, c, f64(w["img"]), cfg.heads, cfg.ln_eps, rows=rows)
        sel = slice(None) if rows is None else rows
        check(cfg.key, y[:, sel], ry, x[:, sel], tol)


# ------------------------------------------------------------------ small (oracle-fast) shapes
SMALL = [
    ("c0_full_fp32", synth.CONFIGS["c0"]),
    ("fp32_dh72_ragged", synth.CONFIGS["c0"].with_(tokens=77, hidden=576, heads=8, head_dim=72, mlp_hidden=256, batch=2)),
    ("fp32_dh128_joint", synth.CONFIGS["c0"].with_(tokens=40, text_tokens=9, hidden=256, heads=2, head_dim=128,
                                                   mlp_hidden=512, batch=2)),
    ("bf16_dh72_t200_b2", synth.CONFIGS["c1"].with_(batch=2, tokens=200, n_blocks=1)),
    ("bf16_dh64_t130", synth.CONFIGS["c1"].with_(batch=1, tokens=130, hidden=256, heads=4, head_dim=64,
                                                 mlp_hidden=1024, n_blocks=1)),
    ("bf16_dh128_t150_b2", synth.CONFIGS["c1"].with_(batch=2, tokens=150, hidden=256, heads=2, head_dim=128,
                                                     mlp_hidden=1024, n_blocks=1)),
    ("bf16_t1", synth.CONFIGS["c1"].with_(batch=3, tokens=1, hidden=256, heads=2, head_dim=128, mlp_hidden=512, n_blocks=1)),
    ("bf16_t17", synth.CONFIGS["c1"].with_(batch=2, tokens=17, hidden=576, heads=8, head_dim=72, mlp_hidden=256, n_blocks=1)),
    ("bf16_t65_m_tail", synth.CONFIGS["c1"].with_(batch=1, tokens=65, hidden=192, heads=3, head_dim=64, mlp_hidden=320, n_blocks=1)),
    ("bf16_t257", synth.CONFIGS["c1"].with_(batch=1, tokens=257, hidden=256, heads=2, head_dim=128, mlp_hidden=512, n_blocks=1)),
    ("bf16_joint_t130_tt21_b2", synth.CONFIGS["c3"].with_(batch=2, tokens=130, text_tokens=21, hidden=256, heads=2,
                                                          head_dim=128, mlp_hidden=1024, n_blocks=1)),
    ("bf16_joint_dh72_tt5", synth.CONFIGS["c3"].with_(batch=1, tokens=64, text_tokens=5, hidden=576, heads=8,
                                                      head_dim=72, mlp_hidden=256, n_blocks=1)),
    # DiT-XL widths with ragged row counts that select the 256-row GEMM tiles:
    # 2000 rows -> QKV 256x128, fc1 256x256, out/fc2 64x144 (last M tile ragged)
    ("bf16_xl_t250_b8_tiles", synth.CONFIGS["c1"].with_(batch=8, tokens=250, n_blocks=1)),
    # 4096 rows at hidden 576 and MLP 1728 (both multiples of 144, 9 and 27
    # k-slices): the output projection and fc2 take the 64x144 tiles with a
    # single k-group (odd slice count)
    ("bf16_144_one_kgroup", synth.CONFIGS["c1"].with_(batch=4, tokens=1024, hidden=576, heads=8, head_dim=72,
                                                      mlp_hidden=1728, n_blocks=1)),
    # DiT-XL widths at one or two samples: the output projection and fc2 run
    # too few 64x128 tiles to fill the GPU and are split into k-ranges
    # (fc2 at 256 rows: 36 tiles x 6 ranges; 250 rows: a ragged row tile)
    ("bf16_xl_b1_split", synth.CONFIGS["c1"].with_(batch=1, n_blocks=1)),
    ("bf16_xl_b1_t250_split", synth.CONFIGS["c1"].with_(batch=1, tokens=250, n_blocks=1)),
    ("bf16_xl_b2_split", synth.CONFIGS["c1"].with_(batch=2, n_blocks=1)),
    ("bf16_xl_b4_split", synth.CONFIGS["c1"].with_(batch=4, n_blocks=1)),
    # 2340 rows -> QKV (incl. the v^T columns) and fc1 on 256x256 tiles
    ("bf16_xl_t260_b9_tiles", synth.CONFIGS["c1"].with_(batch=9, tokens=260, n_blocks=1)),
    # 600 rows (and 512 + 64 joint rows) at widths that are multiples of 144:
    # the QKV projection takes the 64x144 tiles, whose 48-column wave strips
    # give each lane three column groups (q/k heads, head_dim 72 padding,
    # v^T columns, text rows after the image rows)
    ("bf16_qkv_144_dh72", synth.CONFIGS["c1"].with_(batch=2, tokens=300, n_blocks=1)),
    ("bf16_joint_qkv_144", synth.CONFIGS["c3"].with_(batch=1, tokens=512, text_tokens=64, hidden=1152, heads=9,
                                                     head_dim=128, mlp_hidden=1024, n_blocks=1)),
    # >= 256 (sample, head, 256-query) items select the software-pipelined
    # attention kernel: one, two and three key tiles, ragged last tiles
    ("bf16_pipe_dh64_t17_b16", synth.CONFIGS["c1"].with_(batch=16, tokens=17, hidden=1024, heads=16, head_dim=64,
                                                         mlp_hidden=512, n_blocks=1)),
    ("bf16_pipe_dh128_t100_b32", synth.CONFIGS["c1"].with_(batch=32, tokens=100, hidden=1024, heads=8, head_dim=128,
                                                           mlp_hidden=512, n_blocks=1)),
    ("bf16_pipe_dh72_t150_b16", synth.CONFIGS["c1"].with_(batch=16, tokens=150, n_blocks=1)),
    ("bf16_pipe_joint_dh128", synth.CONFIGS["c3"].with_(batch=32, tokens=120, text_tokens=9, hidden=1024, heads=8,
                                                        head_dim=128, mlp_hidden=512, n_blocks=1)),
    # the key loop runs four tiles per trip (one per ring slot): five, eight
    # and seven key tiles leave one, none and three tiles after the trips
    ("bf16_pipe_dh128_t300_b16", synth.CONFIGS["c1"].with_(batch=16, tokens=300, hidden=1024, heads=8, head_dim=128,
                                                           mlp_hidden=512, n_blocks=1)),
    ("bf16_pipe_dh72_t450_b8", synth.CONFIGS["c1"].with_(batch=8, tokens=450, n_blocks=1)),
    ("bf16_pipe_dh64_t420_b16", synth.CONFIGS["c1"].with_(batch=16, tokens=420, hidden=1024, heads=16, head_dim=64,
                                                          mlp_hidden=512, n_blocks=1)),
]


@pytest.mark.parametrize("name,cfg", SMALL, ids=[s[0] for s in SMALL])
def test_block_small(name, cfg):
    print(f"[case] block {name} B={cfg.batch} T={cfg.tokens} Tt={cfg.text_tokens} D={cfg.hidden} "
          f"dh={cfg.head_dim} {cfg.dtype}", flush=True)
    block_case(cfg)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_zero_gates_identity_bitwise(dtype):
    g = _gpu()
    cfg = synth.CONFIGS["c1"].with_(batch=2, tokens=70, text_tokens=6, hidden=256, heads=2, head_dim=128,
                                    mlp_hidden=512, n_blocks=1, dtype=dtype)
    w = synth.block_weights(cfg, 0)
    w = {"img": g.zero_gates(w["img"], cfg.hidden), "txt": g.zero_gates(w["txt"], cfg.hidden)}
    inp = synth.inputs(cfg)
    y, yt = g.run_block(cfg, w, inp["x"], inp["cond"], inp["x_txt"])
    assert np.array_equal(y, inp["x"].astype(np.float64))
    assert np.array_equal(yt, inp["x_txt"].astype(np.float64))


def test_determinism_bitwise():
    g = _gpu()
    cfg = synth.CONFIGS["c1"].with_(batch=2, tokens=300, n_blocks=1)
    w = synth.block_weights(cfg, 0)
    inp = synth.inputs(cfg)
    (y1, _), (y2, _) = g.run_block(cfg, w, inp["x"], inp["cond"], repeat=2)
    assert np.array_equal(y1, y2)


def test_cond_embed_and_pos_table():
    g = _gpu()
    import paper_2605_25550_amd as dm
    cfg = synth.CONFIGS["c1"]
    sw = synth.step_weights(cfg)
    inp = synth.inputs(cfg)
    shape = dm.shape_of(cfg)
    dt = dm.weight_dtype(shape)
    wd = {k: g.dev(sw[k], dt) for k in ("w_t1", "b_t1", "w_t2", "b_t2", "class_table")}
    cond = torch.empty((cfg.batch, cfg.hidden), dtype=torch.float32, device="cuda")
    ws = dm.alloc_workspace(shape, dm.DIT_WS_COND)
    dm.cond_embed(shape, g.dev(inp["t"]), g.dev(inp["y"], torch.int32), wd, cond, ws)
    ref = O.class_conditioning(inp["t"], inp["y"], *[sw[k].astype(np.float64) for k in
                                                      ("w_t1", "b_t1", "w_t2", "b_t2", "class_table")])
    check("cond_embed", g.host(cond), ref, None, 2e-3)
    for gh, gw, D in ((16, 16, 1152), (32, 32, 1152), (3, 5, 8)):
        pos = torch.empty((gh * gw, D), dtype=torch.float32, device="cuda")
        dm.pos_embed_2d(gh, gw, D, pos)
        torch.cuda.synchronize()
        assert np.max(np.abs(g.host(pos) - O.pos_embed_2d(gh, gw, D))) < 1e-6


# ------------------------------------------------------------------ step (small)
STEP_SMALL = [
    ("fp32_step_l2", synth.CONFIGS["c0"].with_(n_blocks=2, batch=2, tokens=64, grid=(8, 8))),
    # patch embeddings of 80 and 150 channels: the tiled patch kernel's full
    # 64-channel chunks plus a partial one, and a ragged last row block
    ("bf16_step_patch80", synth.CONFIGS["c4"].with_(n_blocks=1, batch=1, tokens=100, hidden=256, heads=2, head_dim=128,
                                                    mlp_hidden=512, patch_in=80, patch_out=80)),
    ("bf16_step_patch150_b2", synth.CONFIGS["c4"].with_(n_blocks=1, batch=2, tokens=45, hidden=512, heads=4,
                                                        head_dim=128, mlp_hidden=512, patch_in=150, patch_out=16)),
    ("fp32_step_patch33", synth.CONFIGS["c0"].with_(n_blocks=1, batch=1, tokens=40, grid=(5, 8), patch_in=33,
                                                    patch_out=8)),
    ("bf16_step_class_l3", synth.CONFIGS["c1"].with_(n_blocks=3, batch=2, tokens=64, hidden=256, heads=2,
                                                     head_dim=128, mlp_hidden=512, grid=(8, 8))),
    ("bf16_step_joint_l2", synth.CONFIGS["c3"].with_(n_blocks=2, batch=1, tokens=96, text_tokens=7, hidden=256,
                                                     heads=2, head_dim=128, mlp_hidden=512)),
]


def step_ref(cfg, sw, blocks, inp, pos, c):
    out, xt = O.dit_step(cfg, inp["patches"], c, {k: v.astype(np.float64) for k, v in sw.items()},
                         [{k: f64(v) for k, v in b.items()} for b in blocks], x_txt=inp.get("x_txt"), pos=pos)
    return out, xt


@pytest.mark.parametrize("name,cfg", STEP_SMALL, ids=[s[0] for s in STEP_SMALL])
def test_step_small(name, cfg):
    g = _gpu()
    print(f"[case] step {name}", flush=True)
    sw = synth.step_weights(cfg)
    blocks = [synth.block_weights(cfg, l) for l in range(cfg.n_blocks)]
    inp = synth.inputs(cfg)
    pos = O.pos_embed_2d(*cfg.grid, cfg.hidden) if cfg.grid else None
    c = inp["cond"]
    ds = g.DeviceStep(cfg, blocks, sw)
    out, xt = ds.run(inp["patches"], c, inp.get("x_txt"))
    rout, rxt = step_ref(cfg, sw, blocks, inp, pos, c)
    check(f"step/{name}", out, rout, None, TOL[cfg.dtype])
    if cfg.joint:
        check(f"step/{name}/txt", xt, rxt, inp["x_txt"], TOL[cfg.dtype])


# ------------------------------------------------------------------ full-size shapes
def test_block_max_hidden():
    """The largest hidden size the library accepts (4096 = 32 heads x 128),
    MLP 16384, a ragged 70 tokens x 2."""
    block_case(synth.CONFIGS["c1"].with_(batch=2, tokens=70, hidden=4096, heads=32, head_dim=128, mlp_hidden=16384,
                                         n_blocks=1))


def test_block_c1_full():
    block_case(synth.CONFIGS["c1"].with_(n_blocks=1))


def test_block_c1_ragged_rows():
    """B=7, T=250: 1750 rows, a ragged last row tile; the out and fc2 GEMMs
    (N = 1152) take the 64x144 tile path at this size (224 tiles)."""
    block_case(synth.CONFIGS["c1"].with_(batch=7, tokens=250, n_blocks=1))


def test_block_c2_full():
    block_case(synth.CONFIGS["c2"].with_(n_blocks=1))


def test_block_c3_full():
    """The joint text-image block at full size: all 4096 image rows and all
    256 text rows against the oracle."""
    print("[case] block c3 full (4096 + 256 tokens, D 3072)", flush=True)
    block_case(synth.CONFIGS["c3"].with_(n_blocks=1))


def test_block_joint_split_text_fc1():
    """Joint block whose text-stream fc1 runs as k-range units in the last
    round (image fc1 2048 x 8192 fills whole rounds of 256-row tiles; the 40
    text rows are split into 4 k-ranges and reduced with bias and GELU after
    the GEMM).  The text stream is compared in full."""
    cfg = synth.CONFIGS["c3"].with_(batch=1, tokens=2048, text_tokens=40, hidden=1024, heads=8, head_dim=128,
                                    mlp_hidden=8192, n_blocks=1)
    block_case(cfg, rows=[0, 1, 1000, 2047])


def test_block_row_tail_split():
    """One sample of 8200 tokens at hidden 2048: the output projection and
    fc2 are 528 tiles of 256 x 128, two whole rounds plus 16 tiles; rows from
    8192 on run as k-range units in the last round and their partials are
    reduced with the bias, gate and residual update.  Compared in full, and
    bitwise between two runs."""
    cfg = synth.CONFIGS["c4"].with_(tokens=8200, hidden=2048, heads=16, head_dim=128, mlp_hidden=8192, n_blocks=1)
    print("[case] row tail split, 8200 tokens, hidden 2048", flush=True)
    block_case(cfg)
    g = _gpu()
    inp = synth.inputs(cfg)
    (y1, _), (y2, _) = g.run_block(cfg, synth.block_weights(cfg, 0), inp["x"], inp["cond"], repeat=2)
    assert np.array_equal(y1, y2)


ATTN_SPLIT = [
    # 33 query blocks x 8 heads = 264 items: 256 run whole, the last 8 run as
    # 8 key ranges each, merged afterwards
    ("attn_split_dh128", synth.CONFIGS["c4"].with_(tokens=8448, hidden=1024, heads=8, head_dim=128,
                                                   mlp_hidden=1024, n_blocks=1)),
    # head_dim 72 (softmax bookkeeping in the MFMA padding): 17 x 16 = 272
    # items, a ragged last query block
    ("attn_split_dh72", synth.CONFIGS["c1"].with_(batch=1, tokens=4300, n_blocks=1)),
]


@pytest.mark.parametrize("name,cfg", ATTN_SPLIT, ids=[c[0] for c in ATTN_SPLIT])
def test_block_attention_split_tail(name, cfg):
    """The pipelined attention's last, partial round split into key ranges
    whose partial results are merged: compared in full, and bitwise between
    two runs (the ranges are merged in a fixed order)."""
    print(f"[case] attention split tail {name}", flush=True)
    block_case(cfg)
    g = _gpu()
    inp = synth.inputs(cfg)
    (y1, _), (y2, _) = g.run_block(cfg, synth.block_weights(cfg, 0), inp["x"], inp["cond"], repeat=2)
    assert np.array_equal(y1, y2)


def test_block_joint_split_text_fc1_deterministic():
    """The split ranges are added in a fixed order: two runs agree bitwise."""
    g = _gpu()
    cfg = synth.CONFIGS["c3"].with_(batch=1, tokens=2048, text_tokens=40, hidden=1024, heads=8, head_dim=128,
                                    mlp_hidden=8192, n_blocks=1)
    inp = synth.inputs(cfg)
    (y1, t1), (y2, t2) = g.run_block(cfg, synth.block_weights(cfg, 0), inp["x"], inp["cond"], inp["x_txt"], repeat=2)
    assert np.array_equal(y1, y2) and np.array_equal(t1, t2)


@pytest.mark.slow
@pytest.mark.timeout(900)
@pytest.mark.parametrize("block", [0, 14, 29])
def test_block_c4_full(block):
    """The video DiT block at full size (17550 tokens, all rows compared),
    with the weights of blocks 0, 14 and 29 of the 30-block model."""
    print(f"[case] block c4 full, weights of block {block}", flush=True)
    block_case(synth.CONFIGS["c4"].with_(n_blocks=1), block=block)


def test_block_c4_sp8_token_share():
    """One GPU's token share of an 8-way sequence-parallel video DiT step:
    ceil(17550 / 8) = 2194 tokens with all 24 heads (a ragged last row tile)."""
    block_case(synth.CONFIGS["c4"].with_(tokens=2194, n_blocks=1), rows=[0, 1, 1000, 2193])


def test_block_c4_sp8_head_share():
    """One GPU's head share of an 8-way sequence-parallel video DiT step:
    attention of 3 heads x 128 over all 17550 tokens (hidden 384)."""
    block_case(synth.CONFIGS["c4"].with_(hidden=384, heads=3, mlp_hidden=1536, n_blocks=1),
               rows=[0, 5, 9000, 17549])


@pytest.mark.parametrize("key", ["c1", "c2"])
def test_step_full_end_to_end(key):
    """Conditioning + the full 28-block step: DiT-XL/2 at 256 tokens x 8 (the
    benchmarked workload) and at 1024 tokens x 4."""
    g = _gpu()
    import paper_2605_25550_amd as dm
    cfg = synth.CONFIGS[key]
    print(f"[case] step {key} full", flush=True)
    sw = synth.step_weights(cfg)
    inp = synth.inputs(cfg)
    blocks = [synth.block_weights(cfg, l) for l in range(cfg.n_blocks)]
    pos = O.pos_embed_2d(*cfg.grid, cfg.hidden)
    ds = g.DeviceStep(cfg, blocks, sw)
    shape = ds.shape
    cond = torch.empty((cfg.batch, cfg.hidden), dtype=torch.float32, device="cuda")
    wsc = dm.alloc_workspace(shape, dm.DIT_WS_COND)
    dm.cond_embed(shape, g.dev(inp["t"]), g.dev(inp["y"], torch.int32),
                  {k: ds.step[k] for k in ("w_t1", "b_t1", "w_t2", "b_t2", "class_table")}, cond, wsc)
    out, _ = ds.run(inp["patches"], g.host(cond).astype(np.float32))
    c = O.class_conditioning(inp["t"], inp["y"], *[sw[k].astype(np.float64) for k in
                                                    ("w_t1", "b_t1", "w_t2", "b_t2", "class_table")])
    rout, _ = step_ref(cfg, sw, blocks, inp, pos, c)
    check(f"step/{key}_full", out, rout, None, TOL["bf16"])


def _oracle_blocks(cfg, blocks_np):
    """Per-block float64 weights for the oracle, converted one block at a
    time, with a progress line per block."""
    for l, b in enumerate(blocks_np):
        print(f"[oracle] block {l + 1}/{len(blocks_np)}", flush=True)
        yield {k: f64(v) for k, v in b.items()}


def _step_full(cfg):
    g = _gpu()
    sw = synth.step_weights(cfg)
    inp = synth.inputs(cfg)
    blocks = [synth.block_weights(cfg, l) for l in range(cfg.n_blocks)]
    ds = g.DeviceStep(cfg, blocks, sw)
    out, xt = ds.run(inp["patches"], inp["cond"], inp.get("x_txt"))
    del ds
    torch.cuda.empty_cache()
    print("[case] device step done, oracle running", flush=True)
    rout, rxt = O.dit_step(cfg, inp["patches"], inp["cond"], {k: v.astype(np.float64) for k, v in sw.items()},
                           _oracle_blocks(cfg, blocks), x_txt=inp.get("x_txt"))
    check(f"step/{cfg.key}_L{cfg.n_blocks}", out, rout, None, TOL["bf16"])
    if cfg.joint:
        check(f"step/{cfg.key}_L{cfg.n_blocks}/txt", xt, rxt, inp["x_txt"], TOL["bf16"])


@pytest.mark.slow
@pytest.mark.timeout(900)
def test_step_c3_full_end_to_end():
    """The joint text-image step end to end: patch embedding, 24 two-stream
    blocks with their own weights, final layer; output and the text stream's
    final state against the oracle."""
    print("[case] step c3 full, 24 joint blocks", flush=True)
    _step_full(synth.CONFIGS["c3"])


@pytest.mark.slow
@pytest.mark.timeout(900)
def test_step_c4_two_blocks_end_to_end():
    """The video DiT step at full sequence length with its first two blocks:
    patch embedding, blocks 0 and 1, final layer."""
    print("[case] step c4, 17550 tokens, 2 blocks", flush=True)
    _step_full(synth.CONFIGS["c4"].with_(n_blocks=2))


# ------------------------------------------------------------------ multi-step sampler loop
SAMPLE_CASES = [
    ("fp32_given_l2_s3", synth.CONFIGS["c0"].with_(n_blocks=2, batch=2, tokens=64, grid=(8, 8)), [1.0, 0.7, 0.35, 0.0]),
    ("bf16_class_l2_s4", synth.CONFIGS["c1"].with_(n_blocks=2, batch=2, tokens=64, hidden=256, heads=2, head_dim=128,
                                                   mlp_hidden=512, grid=(8, 8)), [1.0, 0.8, 0.55, 0.25, 0.0]),
    ("bf16_joint_l2_s3", synth.CONFIGS["c3"].with_(n_blocks=2, batch=1, tokens=96, text_tokens=7, hidden=256, heads=2,
                                                   head_dim=128, mlp_hidden=512), [1.0, 0.6, 0.3, 0.0]),
]


def _sample_setup(cfg):
    g = _gpu()
    sw = synth.step_weights(cfg)
    blocks = [synth.block_weights(cfg, l) for l in range(cfg.n_blocks)]
    inp = synth.inputs(cfg)
    ds = g.DeviceStep(cfg, blocks, sw)
    import paper_2605_25550_amd as dm
    ws = dm.alloc_workspace(ds.shape, dm.DIT_WS_SAMPLE)
    kw = {}
    if cfg.cond == "class":
        kw["cond_w"] = {k: ds.step[k] for k in ("w_t1", "b_t1", "w_t2", "b_t2", "class_table")}
        kw["y"] = g.dev(inp["y"], torch.int32)
    else:
        kw["cond"] = g.dev(inp["cond"])
    if cfg.joint:
        kw["x_txt"] = g.dev(inp["x_txt"])
    return g, dm, sw, blocks, inp, ds, ws, kw


@pytest.mark.parametrize("name,cfg,sigmas", SAMPLE_CASES, ids=[s[0] for s in SAMPLE_CASES])
def test_sample_euler(name, cfg, sigmas):
    print(f"[case] sampler {name} steps={len(sigmas) - 1}", flush=True)
    g, dm, sw, blocks, inp, ds, ws, kw = _sample_setup(cfg)
    z = g.dev(inp["patches"])
    dm.sample_euler(ds.shape, ds.table, z, sigmas, ws, **kw)
    torch.cuda.synchronize()
    if cfg.joint:  # the given text states are read only
        assert np.array_equal(g.host(kw["x_txt"]), inp["x_txt"].astype(np.float32))
    pos = O.pos_embed_2d(*cfg.grid, cfg.hidden) if cfg.grid else None
    ref = O.sample_euler(cfg, inp["patches"], sigmas, {k: v.astype(np.float64) for k, v in sw.items()},
                         [{k: f64(v) for k, v in b.items()} for b in blocks],
                         y=inp["y"] if cfg.cond == "class" else None,
                         cond=None if cfg.cond == "class" else inp["cond"], x_txt=inp.get("x_txt"), pos=pos)
    check(f"sample/{name}", g.host(z), ref, inp["patches"], TOL[cfg.dtype])


def test_sample_euler_graph_replay():
    """The loop captured into a graph and replayed three times (with eager
    work between replays) gives the eager result each time, bitwise."""
    name, cfg, sigmas = SAMPLE_CASES[1]
    g, dm, sw, blocks, inp, ds, ws, kw = _sample_setup(cfg)
    z0 = g.dev(inp["patches"])
    z_eager = z0.clone()
    dm.sample_euler(ds.shape, ds.table, z_eager, sigmas, ws, **kw)
    torch.cuda.synchronize()
    z_static = z0.clone()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        dm.sample_euler(ds.shape, ds.table, z_static, sigmas, ws, **kw)
    for r in range(3):
        z_static.copy_(z0)
        junk = torch.randn(1 << 16, device="cuda").sum()  # eager work between replays
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(z_static, z_eager), f"replay {r} differs from the eager loop"
        del junk


# ------------------------------------------------------------------ serving with copy/compute overlap
def test_serve_overlap_and_jitter_do_not_change_results():
    """Five requests through dit_serve: in order on one stream, with the
    copies overlapped on a second stream, and with host-side arrival jitter,
    the outputs are bitwise identical, each equals dit_sample_euler run on
    that request alone, and each matches the oracle's Euler loop on that
    request's latent and labels."""
    name, cfg, sigmas = SAMPLE_CASES[1]
    g, dm, sw, blocks, inp, ds, ws_sample, kw = _sample_setup(cfg)
    ws = dm.alloc_workspace(ds.shape, dm.DIT_WS_SERVE)
    cond_w = kw["cond_w"]
    reqs = []
    for i in range(5):
        r = synth.inputs(cfg, salt=i + 1)
        reqs.append({"z_in": torch.from_numpy(r["patches"].astype(np.float32)).pin_memory(),
                     "y": torch.from_numpy(r["y"].astype(np.int32)),
                     "z_out": torch.empty(r["patches"].shape, dtype=torch.float32).pin_memory()})
    outs = {}
    copy_stream = torch.cuda.Stream()
    for mode, (overlap, jitter) in {"serial": (False, 0), "overlap": (True, 0), "overlap_jitter": (True, 400)}.items():
        for r in reqs:
            r["z_out"].fill_(float("nan"))
        dm.serve(ds.shape, ds.table, reqs, sigmas, ws, cond_w=cond_w, overlap=overlap, jitter_us=jitter, jitter_seed=7,
                 copy_stream=copy_stream)
        torch.cuda.synchronize()
        outs[mode] = [r["z_out"].clone() for r in reqs]
        print(f"[serve] {mode}: done", flush=True)
    for mode in ("overlap", "overlap_jitter"):
        for i in range(5):
            assert torch.equal(outs[mode][i], outs["serial"][i]), (mode, i)
    for i, r in enumerate(reqs):
        z = r["z_in"].cuda()
        dm.sample_euler(ds.shape, ds.table, z, sigmas, ws_sample, cond_w=cond_w, y=r["y"].cuda())
        torch.cuda.synchronize()
        assert torch.equal(z.cpu(), outs["serial"][i]), i
    # and each request's denoised latent against the oracle's Euler loop
    pos = O.pos_embed_2d(*cfg.grid, cfg.hidden)
    sw64 = {k: v.astype(np.float64) for k, v in sw.items()}
    bl64 = [{k: f64(v) for k, v in b.items()} for b in blocks]
    for i, r in enumerate(reqs):
        ref = O.sample_euler(cfg, r["z_in"].numpy().astype(np.float64), sigmas, sw64, bl64, y=r["y"].numpy(), pos=pos)
        check(f"serve/request{i}", outs["overlap_jitter"][i].numpy().astype(np.float64), ref,
              r["z_in"].numpy().astype(np.float64), TOL["bf16"])
