"""Pins of the fp64 oracle against facts fixed by the mathematics of the DiT
block (no paper-printed worked example exists for this stage).

Each test is chosen so that a plausible slip in the oracle (wrong modulation
chunk, dropped bias, transposed weight, wrong softmax axis or scale, wrong
GELU form, wrong LayerNorm variance, swapped sin/cos) fails at least one.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth
from oracle import dit_oracle as O

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")


def tiny_cfg(**kw):
    base = synth.CONFIGS["c0"].with_(tokens=12, hidden=32, heads=4, head_dim=8, mlp_hidden=64, batch=2)
    return base.with_(**kw)


def weights(cfg, block=0, stream=0):
    return {k: v.astype(np.float64) for k, v in synth.stream_weights(cfg, block, stream).items()}


def rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


# ------------------------------------------------------------ torch float64 re-derivation
def torch_block(x, c, w, heads, eps=1e-6):
    """Independent composition from torch library routines (float64)."""
    t = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64))
    x, c = t(x), t(c)
    m = F.linear(F.silu(c), t(w["w_ada"]), t(w["b_ada"]))
    sh1, sc1, g1, sh2, sc2, g2 = m.chunk(6, dim=-1)
    B, T, D = x.shape
    h = F.layer_norm(x, (D,), eps=eps) * (1 + sc1[:, None]) + sh1[:, None]
    qkv = F.linear(h, t(w["w_qkv"]), t(w["b_qkv"])).reshape(B, T, 3, heads, D // heads).permute(2, 0, 3, 1, 4)
    o = F.scaled_dot_product_attention(qkv[0], qkv[1], qkv[2])
    o = o.transpose(1, 2).reshape(B, T, D)
    x = x + g1[:, None] * F.linear(o, t(w["w_o"]), t(w["b_o"]))
    h2 = F.layer_norm(x, (D,), eps=eps) * (1 + sc2[:, None]) + sh2[:, None]
    u = F.gelu(F.linear(h2, t(w["w_fc1"]), t(w["b_fc1"])), approximate="tanh")
    return (x + g2[:, None] * F.linear(u, t(w["w_fc2"]), t(w["b_fc2"]))).numpy()


def brute_attention(q, k, v):
    """Scalar triple loop, pure Python floats."""
    B, H, T, dh = q.shape
    Tk = k.shape[2]
    out = np.zeros((B, H, T, dh))
    for b in range(B):
        for h in range(H):
            for i in range(T):
                s = [sum(float(q[b, h, i, d]) * float(k[b, h, j, d]) for d in range(dh)) / math.sqrt(dh) for j in range(Tk)]
                mx = max(s)
                e = [math.exp(z - mx) for z in s]
                tot = sum(e)
                for d in range(dh):
                    out[b, h, i, d] = sum(e[j] * float(v[b, h, j, d]) for j in range(Tk)) / tot
    return out


# ------------------------------------------------------------ gates / residual
def test_zero_gates_make_block_identity_bitwise():
    cfg = tiny_cfg()
    w = weights(cfg)
    D = cfg.hidden
    for chunk in (2, 5):                      # gate_msa, gate_mlp
        w["w_ada"][chunk * D:(chunk + 1) * D] = 0.0
        w["b_ada"][chunk * D:(chunk + 1) * D] = 0.0
    x = rand((cfg.batch, cfg.tokens, D), 1)
    c = rand((cfg.batch, D), 2)
    y = O.dit_block(x, c, w, cfg.heads)
    assert np.array_equal(y, x)


def test_other_zero_chunks_do_not_give_identity():
    """Zeroing a non-gate chunk (shift/scale) must not give the identity: pins the chunk order."""
    cfg = tiny_cfg()
    D = cfg.hidden
    x = rand((cfg.batch, cfg.tokens, D), 1)
    c = rand((cfg.batch, D), 2)
    for chunks in ((0, 3), (1, 4)):
        w = weights(cfg)
        for ch in chunks:
            w["w_ada"][ch * D:(ch + 1) * D] = 0.0
            w["b_ada"][ch * D:(ch + 1) * D] = 0.0
        assert not np.allclose(O.dit_block(x, c, w, cfg.heads), x)


def test_mlp_increment_is_linear_in_gate():
    cfg = tiny_cfg()
    D = cfg.hidden
    x = rand((cfg.batch, cfg.tokens, D), 3)
    c = rand((cfg.batch, D), 4)
    w = weights(cfg)
    w["w_ada"][5 * D:6 * D] = 0.0            # gate_mlp = b only
    w["b_ada"][5 * D:6 * D] = 0.0
    y0 = O.dit_block(x, c, w, cfg.heads)     # = x1 (MLP branch gated off)
    w["b_ada"][5 * D:6 * D] = 1.0
    y1 = O.dit_block(x, c, w, cfg.heads)
    w["b_ada"][5 * D:6 * D] = 3.0
    y3 = O.dit_block(x, c, w, cfg.heads)
    np.testing.assert_allclose(y3 - y0, 3.0 * (y1 - y0), rtol=1e-12, atol=1e-12)


# ------------------------------------------------------------ softmax / attention
def test_softmax_rows_sum_to_one_and_nonnegative():
    rng = np.random.default_rng(5)
    Tk = 16
    q = rng.standard_normal((2, 3, 7, Tk)) * 4
    k = rng.standard_normal((2, 3, Tk, Tk)) * 4
    v = np.broadcast_to(np.eye(Tk), (2, 3, Tk, Tk)).copy()   # O = P
    p = O.attention_heads(q, k, v)
    assert np.all(p >= 0)
    assert np.max(np.abs(p.sum(-1) - 1.0)) <= 1e-13


def test_equal_keys_give_uniform_weights():
    rng = np.random.default_rng(6)
    q = rng.standard_normal((1, 2, 5, 8))
    k = np.broadcast_to(rng.standard_normal((1, 2, 1, 8)), (1, 2, 9, 8)).copy()
    v = rng.standard_normal((1, 2, 9, 8))
    o = O.attention_heads(q, k, v)
    np.testing.assert_allclose(o, np.broadcast_to(v.mean(axis=2, keepdims=True), o.shape), rtol=0, atol=1e-14)


def test_attention_matches_brute_force():
    rng = np.random.default_rng(7)
    q = rng.standard_normal((2, 2, 5, 4)) * 2
    k = rng.standard_normal((2, 2, 6, 4)) * 2
    v = rng.standard_normal((2, 2, 6, 4))
    assert np.max(np.abs(O.attention_heads(q, k, v) - brute_attention(q, k, v))) <= 1e-12


def test_attention_scale_closed_form():
    """Two keys, one query: weights are the logistic of the scaled score gap."""
    q = np.array([[[[1.0, 0.0]]]])
    k = np.array([[[[1.0, 0.0], [0.0, 1.0]]]])
    v = np.array([[[[2.0, -1.0], [0.5, 4.0]]]])
    a = 1.0 / math.sqrt(2.0)
    p0 = math.exp(a) / (math.exp(a) + 1.0)
    want = p0 * v[0, 0, 0] + (1 - p0) * v[0, 0, 1]
    np.testing.assert_allclose(O.attention_heads(q, k, v)[0, 0, 0], want, rtol=0, atol=1e-15)


def test_attention_row_subset_and_chunking():
    rng = np.random.default_rng(8)
    q = rng.standard_normal((1, 2, 37, 8))
    k = rng.standard_normal((1, 2, 37, 8))
    v = rng.standard_normal((1, 2, 37, 8))
    full = O.attention_heads(q, k, v)
    np.testing.assert_allclose(O.attention_heads(q, k, v, chunk=5), full, rtol=0, atol=1e-14)
    rows = [0, 3, 36, 17]
    np.testing.assert_allclose(O.attention_heads(q, k, v, rows=rows), full[:, :, rows], rtol=0, atol=1e-14)


def test_single_token_closed_form():
    """T = 1: softmax over one key is 1, so attention returns v and the block is
    x + g1*((h W_v^T + b_v) W_o^T + b_o) followed by the MLP branch."""
    cfg = tiny_cfg(tokens=1)
    D = cfg.hidden
    w = weights(cfg)
    x = rand((cfg.batch, 1, D), 9)
    c = rand((cfg.batch, D), 10)
    t = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64))
    m = F.linear(F.silu(t(c)), t(w["w_ada"]), t(w["b_ada"])).numpy()
    sh1, sc1, g1, sh2, sc2, g2 = np.split(m, 6, axis=-1)
    xt = t(x)
    h = F.layer_norm(xt, (D,), eps=1e-6).numpy() * (1 + sc1[:, None]) + sh1[:, None]
    v = h @ w["w_qkv"][2 * D:].T + w["b_qkv"][2 * D:]
    x1 = x + g1[:, None] * (v @ w["w_o"].T + w["b_o"])
    h2 = F.layer_norm(t(x1), (D,), eps=1e-6).numpy() * (1 + sc2[:, None]) + sh2[:, None]
    u = F.gelu(t(h2 @ w["w_fc1"].T + w["b_fc1"]), approximate="tanh").numpy()
    want = x1 + g2[:, None] * (u @ w["w_fc2"].T + w["b_fc2"])
    np.testing.assert_allclose(O.dit_block(x, c, w, cfg.heads), want, rtol=1e-12, atol=1e-12)


# ------------------------------------------------------------ whole block
def test_block_matches_torch_float64_library_routines():
    cfg = tiny_cfg()
    w = weights(cfg)
    x = rand((cfg.batch, cfg.tokens, cfg.hidden), 11)
    c = rand((cfg.batch, cfg.hidden), 12)
    np.testing.assert_allclose(O.dit_block(x, c, w, cfg.heads), torch_block(x, c, w, cfg.heads), rtol=0, atol=1e-10)


def test_block_token_permutation_equivariance():
    cfg = tiny_cfg()
    w = weights(cfg)
    x = rand((cfg.batch, cfg.tokens, cfg.hidden), 13)
    c = rand((cfg.batch, cfg.hidden), 14)
    perm = np.random.default_rng(15).permutation(cfg.tokens)
    np.testing.assert_allclose(O.dit_block(x[:, perm], c, w, cfg.heads), O.dit_block(x, c, w, cfg.heads)[:, perm],
                               rtol=0, atol=1e-12)


def test_block_batch_independence():
    cfg = tiny_cfg()
    w = weights(cfg)
    x = rand((cfg.batch, cfg.tokens, cfg.hidden), 16)
    c = rand((cfg.batch, cfg.hidden), 17)
    y = O.dit_block(x, c, w, cfg.heads)
    for b in range(cfg.batch):
        np.testing.assert_allclose(O.dit_block(x[b:b + 1], c[b:b + 1], w, cfg.heads), y[b:b + 1], rtol=0, atol=1e-12)


def test_block_row_subset():
    cfg = tiny_cfg()
    w = weights(cfg)
    x = rand((cfg.batch, cfg.tokens, cfg.hidden), 18)
    c = rand((cfg.batch, cfg.hidden), 19)
    rows = [11, 0, 5]
    np.testing.assert_allclose(O.dit_block(x, c, w, cfg.heads, rows=rows), O.dit_block(x, c, w, cfg.heads)[:, rows],
                               rtol=0, atol=1e-13)


# ------------------------------------------------------------ joint block
def test_joint_with_shared_weights_equals_block_on_concatenation():
    cfg = tiny_cfg(text_tokens=5)
    w = weights(cfg)
    xi = rand((cfg.batch, cfg.tokens, cfg.hidden), 20)
    xt = rand((cfg.batch, 5, cfg.hidden), 21)
    c = rand((cfg.batch, cfg.hidden), 22)
    yi, yt = O.joint_block(xi, xt, c, w, w, cfg.heads)
    y = O.dit_block(np.concatenate([xi, xt], axis=1), c, w, cfg.heads)
    np.testing.assert_allclose(yi, y[:, :cfg.tokens], rtol=0, atol=1e-12)
    np.testing.assert_allclose(yt, y[:, cfg.tokens:], rtol=0, atol=1e-12)


def test_joint_with_no_text_equals_plain_block():
    cfg = tiny_cfg(text_tokens=3)
    wi = weights(cfg, stream=0)
    wt = weights(cfg, stream=1)
    xi = rand((cfg.batch, cfg.tokens, cfg.hidden), 23)
    c = rand((cfg.batch, cfg.hidden), 24)
    yi, yt = O.joint_block(xi, np.zeros((cfg.batch, 0, cfg.hidden)), c, wi, wt, cfg.heads)
    np.testing.assert_allclose(yi, O.dit_block(xi, c, wi, cfg.heads), rtol=0, atol=1e-13)
    assert yt.shape == (cfg.batch, 0, cfg.hidden)


def test_joint_text_stream_uses_its_own_weights():
    cfg = tiny_cfg(text_tokens=4)
    wi, wt = weights(cfg, stream=0), weights(cfg, stream=1)
    xi = rand((cfg.batch, cfg.tokens, cfg.hidden), 25)
    xt = rand((cfg.batch, 4, cfg.hidden), 26)
    c = rand((cfg.batch, cfg.hidden), 27)
    yi_a, yt_a = O.joint_block(xi, xt, c, wi, wt, cfg.heads)
    yi_b, yt_b = O.joint_block(xi, xt, c, wi, wi, cfg.heads)
    assert not np.allclose(yt_a, yt_b)
    rows = [1, 7]
    yi_r, yt_r = O.joint_block(xi, xt, c, wi, wt, cfg.heads, rows_img=rows)
    np.testing.assert_allclose(yi_r, yi_a[:, rows], rtol=0, atol=1e-13)
    np.testing.assert_allclose(yt_r, yt_a, rtol=0, atol=1e-13)


def torch_joint_block(xi, xt, c, wi, wt, heads, eps=1e-6):
    """Independent two-stream composition from torch float64 library routines:
    each stream's adaLN, LayerNorm, modulation, QKV, output projection and MLP
    use that stream's own weights; one scaled_dot_product_attention runs over
    the concatenated [image; text] q, k and v."""
    t = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64))
    c = t(c)
    xs = [t(xi), t(xt)]
    ws = [wi, wt]
    B, D = c.shape
    mods = [F.linear(F.silu(c), t(w["w_ada"]), t(w["b_ada"])).chunk(6, dim=-1) for w in ws]
    qkvs = []
    for x, w, m in zip(xs, ws, mods):
        h = F.layer_norm(x, (D,), eps=eps) * (1 + m[1][:, None]) + m[0][:, None]
        T = x.shape[1]
        qkvs.append(F.linear(h, t(w["w_qkv"]), t(w["b_qkv"])).reshape(B, T, 3, heads, D // heads).permute(2, 0, 3, 1, 4))
    qkv = torch.cat(qkvs, dim=3)
    o = F.scaled_dot_product_attention(qkv[0], qkv[1], qkv[2]).transpose(1, 2).reshape(B, -1, D)
    Ti = xs[0].shape[1]
    outs = []
    for x, w, m, oo in zip(xs, ws, mods, (o[:, :Ti], o[:, Ti:])):
        x = x + m[2][:, None] * F.linear(oo, t(w["w_o"]), t(w["b_o"]))
        h2 = F.layer_norm(x, (D,), eps=eps) * (1 + m[4][:, None]) + m[3][:, None]
        u = F.gelu(F.linear(h2, t(w["w_fc1"]), t(w["b_fc1"])), approximate="tanh")
        outs.append((x + m[5][:, None] * F.linear(u, t(w["w_fc2"]), t(w["b_fc2"]))).numpy())
    return outs[0], outs[1]


def _distinct_stream_weights(cfg):
    """Image and text weights that differ in every tensor, with the text set's
    values scaled up so that routing an image tensor into the text stream (or
    the reverse) moves the result far beyond rounding."""
    wi = weights(cfg, stream=0)
    wt = {k: v * 3.0 for k, v in weights(cfg, stream=1).items()}
    return wi, wt


def test_joint_matches_torch_two_stream_composition():
    """Pins the per-stream routing of every weight of the joint block."""
    cfg = tiny_cfg(text_tokens=6)
    wi, wt = _distinct_stream_weights(cfg)
    xi = rand((cfg.batch, cfg.tokens, cfg.hidden), 35)
    xt = rand((cfg.batch, 6, cfg.hidden), 36)
    c = rand((cfg.batch, cfg.hidden), 37)
    yi, yt = O.joint_block(xi, xt, c, wi, wt, cfg.heads)
    ri, rt = torch_joint_block(xi, xt, c, wi, wt, cfg.heads)
    np.testing.assert_allclose(yi, ri, rtol=0, atol=1e-10)
    np.testing.assert_allclose(yt, rt, rtol=0, atol=1e-10)


@pytest.mark.parametrize("name", ["w_ada", "b_ada", "w_qkv", "b_qkv", "w_o", "b_o", "w_fc1", "b_fc1", "w_fc2", "b_fc2"])
def test_joint_each_text_weight_routes_to_text_stream(name):
    """Replacing one text-stream tensor changes the result exactly as the
    torch composition predicts (and for the tensors after attention, only
    the text rows)."""
    cfg = tiny_cfg(text_tokens=5)
    wi, wt = _distinct_stream_weights(cfg)
    xi = rand((cfg.batch, cfg.tokens, cfg.hidden), 38)
    xt = rand((cfg.batch, 5, cfg.hidden), 39)
    c = rand((cfg.batch, cfg.hidden), 40)
    wt2 = dict(wt)
    wt2[name] = wt[name] + rand(wt[name].shape, 41) * 0.05
    yi, yt = O.joint_block(xi, xt, c, wi, wt2, cfg.heads)
    ri, rt = torch_joint_block(xi, xt, c, wi, wt2, cfg.heads)
    np.testing.assert_allclose(yi, ri, rtol=0, atol=1e-10)
    np.testing.assert_allclose(yt, rt, rtol=0, atol=1e-10)
    yi0, yt0 = O.joint_block(xi, xt, c, wi, wt, cfg.heads)
    assert not np.allclose(yt, yt0)
    if name in ("w_o", "b_o", "w_fc1", "b_fc1", "w_fc2", "b_fc2"):
        assert np.array_equal(yi, yi0)


def _zero_gate_rows(w, D):
    w = dict(w)
    for k in ("w_ada", "b_ada"):
        a = w[k].copy()
        a[2 * D:3 * D] = 0.0
        a[5 * D:6 * D] = 0.0
        w[k] = a
    return w


def test_joint_zero_gates_per_stream():
    """Zero gates in one stream make that stream the identity (bitwise) and
    leave the other stream's branches active."""
    cfg = tiny_cfg(text_tokens=5)
    wi, wt = _distinct_stream_weights(cfg)
    D = cfg.hidden
    xi = rand((cfg.batch, cfg.tokens, D), 42)
    xt = rand((cfg.batch, 5, D), 43)
    c = rand((cfg.batch, D), 44)
    yi, yt = O.joint_block(xi, xt, c, wi, _zero_gate_rows(wt, D), cfg.heads)
    assert np.array_equal(yt, xt)
    assert not np.allclose(yi, xi)
    ri, _ = torch_joint_block(xi, xt, c, wi, _zero_gate_rows(wt, D), cfg.heads)
    np.testing.assert_allclose(yi, ri, rtol=0, atol=1e-10)
    yi, yt = O.joint_block(xi, xt, c, _zero_gate_rows(wi, D), wt, cfg.heads)
    assert np.array_equal(yi, xi)
    assert not np.allclose(yt, xt)
    _, rt = torch_joint_block(xi, xt, c, _zero_gate_rows(wi, D), wt, cfg.heads)
    np.testing.assert_allclose(yt, rt, rtol=0, atol=1e-10)


# ------------------------------------------------------------ elementwise pieces
def test_gelu_tanh_identities_and_library():
    u = np.linspace(-7, 7, 1001)
    g = O.gelu_tanh(u)
    assert O.gelu_tanh(np.array([0.0]))[0] == 0.0
    np.testing.assert_allclose(g - O.gelu_tanh(-u), u, rtol=0, atol=1e-14)
    np.testing.assert_allclose(g, F.gelu(torch.from_numpy(u), approximate="tanh").numpy(), rtol=0, atol=1e-14)
    # differs from the erf form by more than the fp32 tolerance somewhere
    assert np.max(np.abs(g - F.gelu(torch.from_numpy(u)).numpy())) > 1e-4


def test_layer_norm_moments():
    x = rand((3, 17, 40), 28) * 3 + 5
    eps = 1e-6
    y = O.layer_norm(x, eps)
    var = x.var(axis=-1, keepdims=True)
    np.testing.assert_allclose(y.mean(-1), 0.0, atol=1e-13)
    np.testing.assert_allclose(y.var(-1, keepdims=True), var / (var + eps), rtol=1e-12)
    np.testing.assert_allclose(y, F.layer_norm(torch.from_numpy(x), (40,), eps=eps).numpy(), rtol=0, atol=1e-12)


def test_silu_and_modulate():
    z = np.linspace(-30, 30, 601)
    np.testing.assert_allclose(O.silu(z), F.silu(torch.from_numpy(z)).numpy(), rtol=1e-14, atol=1e-300)
    xn = rand((2, 3, 4), 29)
    sh, sc = rand((2, 4), 30), rand((2, 4), 31)
    np.testing.assert_allclose(O.modulate(xn, np.zeros((2, 4)), np.zeros((2, 4))), xn, rtol=0, atol=0)
    np.testing.assert_allclose(O.modulate(xn, sh, -np.ones((2, 4))), np.broadcast_to(sh[:, None], xn.shape), atol=0)


def test_adaln_chunks_library():
    c = rand((2, 8), 32)
    w, b = rand((48, 8), 33), rand((48,), 34)
    chunks = O.adaln_modulation(c, w, b)
    ref = F.linear(F.silu(torch.from_numpy(c)), torch.from_numpy(w), torch.from_numpy(b)).chunk(6, dim=-1)
    for a, r in zip(chunks, ref):
        np.testing.assert_allclose(a, r.numpy(), rtol=0, atol=1e-14)


# ------------------------------------------------------------ step pieces
def test_timestep_embedding_closed_forms():
    e0 = O.timestep_embedding(np.array([0.0]), 256)
    np.testing.assert_array_equal(e0[0, :128], 1.0)
    np.testing.assert_array_equal(e0[0, 128:], 0.0)
    t = np.array([3.0, 517.0])
    e = O.timestep_embedding(t, 256)
    np.testing.assert_allclose(e[:, 0], np.cos(t), atol=1e-15)          # f_0 = 1
    np.testing.assert_allclose(e[:, 128], np.sin(t), atol=1e-15)
    np.testing.assert_allclose((e * e).sum(-1), 128.0, rtol=1e-14)      # cos^2 + sin^2 per frequency
    # f_{64} = 10000^(-1/2) = 1/100
    np.testing.assert_allclose(e[:, 64], np.cos(t / 100.0), atol=1e-13)


def test_class_conditioning_reduces_to_table_row():
    D = 16
    rng = np.random.default_rng(35)
    table = rng.standard_normal((11, D))
    y = np.array([3, 10])
    c = O.class_conditioning(np.array([5.0, 9.0]), y, rng.standard_normal((D, 256)), rng.standard_normal(D),
                             np.zeros((D, D)), np.zeros(D), table)
    np.testing.assert_allclose(c, table[y], atol=0)
    # t = 0, identity second layer: c = SiLU(W1 e0 + b1) + E[y], e0 = [1..1, 0..0]
    w1, b1 = rng.standard_normal((D, 256)), rng.standard_normal(D)
    c2 = O.class_conditioning(np.array([0.0]), np.array([1]), w1, b1, np.eye(D), np.zeros(D), table)
    z = w1[:, :128].sum(1) + b1
    np.testing.assert_allclose(c2[0], z / (1 + np.exp(-z)) + table[1], rtol=1e-13)


def test_pos_embed_2d_closed_forms():
    gh, gw, D = 4, 6, 16
    p = O.pos_embed_2d(gh, gw, D)
    assert p.shape == (gh * gw, D)
    np.testing.assert_allclose((p * p).sum(-1), D / 2, rtol=1e-14)
    for r in range(gh):
        for c in range(gw):
            n = r * gw + c
            assert abs(p[n, 0] - math.sin(c)) < 1e-15           # omega_0 = 1, column half, sin first
            assert abs(p[n, D // 4] - math.cos(c)) < 1e-15
            assert abs(p[n, D // 2] - math.sin(r)) < 1e-15      # row half
            assert abs(p[n, 3 * D // 4] - math.cos(r)) < 1e-15
            assert abs(p[n, 2] - math.sin(c * 10000.0 ** (-0.5))) < 1e-15   # i = 2 of D/4 = 4


def test_final_layer_library():
    rng = np.random.default_rng(36)
    B, T, D, P = 2, 5, 12, 7
    x, c = rng.standard_normal((B, T, D)), rng.standard_normal((B, D))
    wa, ba, wf, bf = rng.standard_normal((2 * D, D)), rng.standard_normal(2 * D), rng.standard_normal((P, D)), rng.standard_normal(P)
    t = torch.from_numpy
    sh, sc = F.linear(F.silu(t(c)), t(wa), t(ba)).chunk(2, dim=-1)
    want = F.linear(F.layer_norm(t(x), (D,), eps=1e-6) * (1 + sc[:, None]) + sh[:, None], t(wf), t(bf)).numpy()
    np.testing.assert_allclose(O.final_layer(x, c, wa, ba, wf, bf), want, rtol=0, atol=1e-12)


def test_step_with_zero_gates_is_embed_then_final_layer():
    cfg = tiny_cfg(n_blocks=3, patch_in=8, patch_out=6, batch=2)
    D = cfg.hidden
    sw = {k: v.astype(np.float64) for k, v in synth.step_weights(cfg).items()}
    blocks = []
    for l in range(cfg.n_blocks):
        w = weights(cfg, block=l)
        for ch in (2, 5):
            w["w_ada"][ch * D:(ch + 1) * D] = 0.0
            w["b_ada"][ch * D:(ch + 1) * D] = 0.0
        blocks.append({"img": w})
    z = rand((cfg.batch, cfg.tokens, cfg.patch_in), 37)
    c = rand((cfg.batch, D), 38)
    pos = rand((cfg.tokens, D), 39)
    out, _ = O.dit_step(cfg, z, c, sw, blocks, pos=pos)
    t = torch.from_numpy
    x0 = F.linear(t(z), t(sw["w_patch"]), t(sw["b_patch"])) + t(pos)[None]
    sh, sc = F.linear(F.silu(t(c)), t(sw["w_ada_final"]), t(sw["b_ada_final"])).chunk(2, dim=-1)
    want = F.linear(F.layer_norm(x0, (D,), eps=1e-6) * (1 + sc[:, None]) + sh[:, None], t(sw["w_final"]), t(sw["b_final"]))
    np.testing.assert_allclose(out, want.numpy(), rtol=0, atol=1e-12)


def test_step_matches_torch_composition():
    cfg = tiny_cfg(n_blocks=2, patch_in=8, patch_out=6, batch=2)
    sw = {k: v.astype(np.float64) for k, v in synth.step_weights(cfg).items()}
    blocks = [{"img": weights(cfg, block=l)} for l in range(cfg.n_blocks)]
    z = rand((cfg.batch, cfg.tokens, cfg.patch_in), 40)
    c = rand((cfg.batch, cfg.hidden), 41)
    out, _ = O.dit_step(cfg, z, c, sw, blocks)
    x = z @ sw["w_patch"].T + sw["b_patch"]
    for bw in blocks:
        x = torch_block(x, c, bw["img"], cfg.heads)
    t = torch.from_numpy
    sh, sc = F.linear(F.silu(t(c)), t(sw["w_ada_final"]), t(sw["b_ada_final"])).chunk(2, dim=-1)
    want = F.linear(F.layer_norm(t(x), (cfg.hidden,), eps=1e-6) * (1 + sc[:, None]) + sh[:, None],
                    t(sw["w_final"]), t(sw["b_final"]))
    np.testing.assert_allclose(out, want.numpy(), rtol=0, atol=1e-10)


def test_rel_err_metric():
    ref = np.array([1.0, -4.0, 2.0])
    assert O.rel_err(ref, ref) == 0.0
    assert O.rel_err(ref + np.array([0, 0.4, 0]), ref) == pytest.approx(0.1)


# ------------------------------------------------------------ generator sanity
def test_generator_is_deterministic_and_bf16_representable():
    cfg = synth.CONFIGS["c1"].with_(hidden=64, mlp_hidden=256, heads=2, head_dim=32)
    a = synth.stream_weights(cfg, 3)
    b = synth.stream_weights(cfg, 3)
    for k in a:
        np.testing.assert_array_equal(a[k], b[k])
        bits = a[k].view(np.uint32)
        assert np.all((bits & 0xFFFF) == 0), k
    c = synth.stream_weights(cfg, 4)
    assert not np.array_equal(a["w_qkv"], c["w_qkv"])
    assert abs(float(a["w_fc1"].std()) - 0.02) < 0.002


def test_generator_inputs_all_configs():
    for key, cfg in synth.CONFIGS.items():
        small = cfg.with_(tokens=min(cfg.tokens, 32))
        inp = synth.inputs(small)
        assert inp["x"].shape == (small.batch, small.tokens, small.hidden)
        assert inp["cond"].shape == (small.batch, small.hidden)
        assert ("x_txt" in inp) == small.joint
        if small.cond == "class":
            assert np.all((inp["t"] >= 0) & (inp["t"] < 1000)) and np.all((inp["y"] >= 0) & (inp["y"] < 1000))
        np.testing.assert_array_equal(synth.inputs(small)["x"], inp["x"])
        assert not np.array_equal(synth.inputs(small, salt=1)["x"], inp["x"])


# ------------------------------------------------------------ multi-step sampler loop
def _zero_network(cfg, seed=50):
    """Step weights and blocks whose velocity is the constant b_final: every
    block has zero gates (identity) and the final projection is zero."""
    D = cfg.hidden
    sw = {k: v.astype(np.float64) for k, v in synth.step_weights(cfg).items()}
    sw["w_final"] = np.zeros_like(sw["w_final"])
    sw["b_final"] = rand(sw["b_final"].shape, seed)
    blocks = []
    for l in range(cfg.n_blocks):
        w = weights(cfg, block=l)
        for ch in (2, 5):
            w["w_ada"][ch * D:(ch + 1) * D] = 0.0
            w["b_ada"][ch * D:(ch + 1) * D] = 0.0
        blocks.append({"img": w})
    return sw, blocks


@pytest.mark.parametrize("sigmas", [[1.0, 0.75, 0.5, 0.25, 0.0], [1.0, 0.875, 0.5, 0.125, 0.0], [0.0, 0.5, 1.0]])
@pytest.mark.parametrize("class_cond", [False, True])
def test_sampler_constant_velocity_closed_form(sigmas, class_cond):
    """Constant velocity b: the Euler loop integrates dz/dsigma = b exactly,
    z_n = z_0 + (sigma_n - sigma_0) b (dyadic schedules: float32 differences are exact)."""
    cfg = tiny_cfg(n_blocks=2, patch_in=6, patch_out=6, batch=2, cond="class" if class_cond else "given")
    sw, blocks = _zero_network(cfg)
    z0 = rand((cfg.batch, cfg.tokens, 6), 51)
    kw = {"y": np.array([3, 7])} if class_cond else {"cond": rand((cfg.batch, cfg.hidden), 52)}
    z = O.sample_euler(cfg, z0, sigmas, sw, blocks, **kw)
    want = z0 + (sigmas[-1] - sigmas[0]) * sw["b_final"][None, None, :]
    np.testing.assert_allclose(z, want, rtol=0, atol=1e-12)


def test_sampler_zero_steps_is_identity():
    cfg = tiny_cfg(n_blocks=1, patch_in=6, patch_out=6)
    sw = {k: v.astype(np.float64) for k, v in synth.step_weights(cfg).items()}
    z0 = rand((cfg.batch, cfg.tokens, 6), 53)
    z = O.sample_euler(cfg, z0, [0.7], sw, [{"img": weights(cfg)}], cond=rand((cfg.batch, cfg.hidden), 54))
    assert np.array_equal(z, z0)


def test_sampler_splits_into_consecutive_runs():
    """The loop is a sequence of independent steps: running [a, b, c] equals
    running [a, b] and then [b, c] from its result, bitwise."""
    cfg = tiny_cfg(n_blocks=2, patch_in=6, patch_out=6, batch=2, cond="class")
    sw = {k: v.astype(np.float64) for k, v in synth.step_weights(cfg).items()}
    blocks = [{"img": weights(cfg, block=l)} for l in range(2)]
    z0 = rand((cfg.batch, cfg.tokens, 6), 55)
    y = np.array([1, 900])
    whole = O.sample_euler(cfg, z0, [1.0, 0.6, 0.3, 0.0], sw, blocks, y=y)
    part = O.sample_euler(cfg, z0, [1.0, 0.6], sw, blocks, y=y)
    rest = O.sample_euler(cfg, part, [0.6, 0.3, 0.0], sw, blocks, y=y)
    assert np.array_equal(whole, rest)


def test_sampler_step_uses_left_endpoint_conditioning():
    """One step: z1 = z0 + (s1 - s0) v(z0, c(t0)), t0 = s0 * 1000 in float32;
    the conditioning at the other endpoint gives a different result."""
    cfg = tiny_cfg(n_blocks=2, patch_in=6, patch_out=6, batch=2, cond="class")
    sw = {k: v.astype(np.float64) for k, v in synth.step_weights(cfg).items()}
    blocks = [{"img": weights(cfg, block=l)} for l in range(2)]
    z0 = rand((cfg.batch, cfg.tokens, 6), 56)
    y = np.array([4, 5])
    s0, s1 = 0.8, 0.3
    z1 = O.sample_euler(cfg, z0, [s0, s1], sw, blocks, y=y)
    cw = [sw[k] for k in ("w_t1", "b_t1", "w_t2", "b_t2", "class_table")]
    t0 = np.full(2, np.float32(np.float32(s0) * np.float32(1000.0)), dtype=np.float64)
    v0, _ = O.dit_step(cfg, z0, O.class_conditioning(t0, y, *cw), sw, blocks)
    np.testing.assert_allclose(z1, z0 + float(np.float32(s1) - np.float32(s0)) * v0, rtol=0, atol=1e-12)
    v1, _ = O.dit_step(cfg, z0, O.class_conditioning(np.full(2, 300.0), y, *cw), sw, blocks)
    assert np.max(np.abs(v1 - v0)) > 1e-6


def test_sampler_joint_restarts_text_stream():
    """Joint models: every step starts from the given text states, so a
    two-step run equals two one-step runs that both use the original x_txt."""
    cfg = tiny_cfg(n_blocks=1, patch_in=6, patch_out=6, batch=1, text_tokens=5)
    sw = {k: v.astype(np.float64) for k, v in synth.step_weights(cfg).items()}
    blocks = [{"img": weights(cfg, block=0, stream=0), "txt": weights(cfg, block=0, stream=1)}]
    z0 = rand((1, cfg.tokens, 6), 57)
    xt = rand((1, 5, cfg.hidden), 58)
    c = rand((1, cfg.hidden), 59)
    whole = O.sample_euler(cfg, z0, [1.0, 0.5, 0.0], sw, blocks, cond=c, x_txt=xt)
    a = O.sample_euler(cfg, z0, [1.0, 0.5], sw, blocks, cond=c, x_txt=xt)
    b = O.sample_euler(cfg, a, [0.5, 0.0], sw, blocks, cond=c, x_txt=xt)
    assert np.array_equal(whole, b)
