"""CPU tests of the C ABI: every function declared in include/ditmi.h is
exported by the library, and the validation paths return the documented
status codes without launching anything (no GPU needed: a rejected call
returns before any HIP call, so the pointers below are never dereferenced)."""
import ctypes
import os
import re

import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ditmi.h")


@pytest.fixture(scope="module")
def dm():
    import paper_2605_25550_amd as dm
    if not os.path.exists(dm.LIB_PATH):
        from paper_2605_25550_amd.build import build
        build()
    dm.lib()
    return dm


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dit_[a-z0-9_]+)\s*\(", text)))


def test_header_functions_are_exported(dm):
    names = declared_functions()
    assert len(names) >= 11, names
    lib = dm.lib()
    for n in names:
        assert hasattr(lib, n), f"{n} declared in ditmi.h but not exported"
    assert set(names) == set(dm.C_API)


def test_version_and_status_strings(dm):
    lib = dm.lib()
    assert lib.dit_version() == 1
    for st, word in ((0, b"ok"), (-1, b"invalid"), (-2, b"unsupported"), (-3, b"workspace"), (-4, b"HIP")):
        assert word in lib.dit_status_string(st)


def shape(dm, key="c1", **kw):
    return dm.shape_of(synth.CONFIGS[key].with_(**kw))


def test_workspace_sizes(dm):
    for key in synth.CONFIGS:
        s = shape(dm, key)
        blk = dm.workspace_bytes(s, dm.DIT_WS_BLOCK)
        stp = dm.workspace_bytes(s, dm.DIT_WS_STEP)
        cnd = dm.workspace_bytes(s, dm.DIT_WS_COND)
        assert 0 < cnd < blk < stp
        assert blk % 256 == 0 and stp % 256 == 0
    # C4's step workspace (activations for 17550 tokens + modulation for 30 blocks)
    s4 = shape(dm, "c4")
    assert 1.0e9 < dm.workspace_bytes(s4, dm.DIT_WS_STEP) < 1.6e9


@pytest.mark.parametrize("field,value,status", [
    ("head_dim", 80, -2), ("heads", 7, -1), ("hidden", 1000, -1), ("hidden", 8192, -2), ("tokens", 0, -1),
    ("batch", 0, -1), ("mlp_hidden", 100, -1), ("dtype", 5, -1), ("ln_eps", 0.0, -1), ("text_tokens", -1, -1),
])
def test_workspace_rejects_bad_shapes(dm, field, value, status):
    s = shape(dm)
    setattr(s, field, value)
    lib = dm.lib()
    assert lib.dit_workspace_bytes(ctypes.byref(s), 0) == 0
    assert dm.last_error()


def test_weight_matrix_size_limit(dm):
    """A weight matrix of 2^31 or more elements (F * D) is rejected before any
    launch: the kernels address one operand with 32-bit byte offsets.  Hidden
    4096 with MLP width 524288 is a 4 GiB fc1 weight, which the HBM could
    hold; one width step below the limit is accepted."""
    s = shape(dm, "c1", batch=1, tokens=16, hidden=4096, heads=32, head_dim=128, mlp_hidden=524288)
    lib = dm.lib()
    assert lib.dit_workspace_bytes(ctypes.byref(s), 0) == 0
    assert "mlp_hidden" in dm.last_error()
    bw = fake_block(dm)
    assert block_call(dm, s, bw) == -2
    s.mlp_hidden = 524288 - 64
    assert lib.dit_workspace_bytes(ctypes.byref(s), 0) > 0


def test_noalloc_rejects_blocks_beyond_its_scratch(dm):
    """dit_block_forward_noalloc refuses, before any HIP call, a block whose
    workspace exceeds the static scratch (the video DiT block needs ~0.9 GB);
    the header's size constant matches the binding's."""
    text = open(HEADER).read()
    assert "#define DIT_NOALLOC_SCRATCH_BYTES (128u << 20)" in text
    assert dm.NOALLOC_SCRATCH_BYTES == 128 << 20
    s = shape(dm, "c4", n_blocks=1)
    assert dm.workspace_bytes(s, dm.DIT_WS_BLOCK) > dm.NOALLOC_SCRATCH_BYTES
    bw = fake_block(dm)
    assert dm.lib().dit_block_forward_noalloc(ctypes.byref(s), ctypes.byref(bw), FAKE, None, FAKE, None) == -2
    assert "scratch" in dm.last_error()
    # argument errors come first, as for dit_block_forward
    s1 = shape(dm, n_blocks=1)
    assert dm.lib().dit_block_forward_noalloc(ctypes.byref(s1), ctypes.byref(bw), None, None, FAKE, None) == -1
    assert dm.workspace_bytes(s1, dm.DIT_WS_BLOCK) <= dm.NOALLOC_SCRATCH_BYTES


FAKE = 0x100000  # 1 MiB-aligned fake device address; never dereferenced


def fake_block(dm, joint=False):
    sw = dm.StreamWeights(*[FAKE + 4096 * i for i in range(10)])
    bw = dm.BlockWeights()
    bw.img = sw
    if joint:
        bw.txt = dm.StreamWeights(*[FAKE + 65536 + 4096 * i for i in range(10)])
    return bw


def block_call(dm, s, bw, x=FAKE, x_txt=None, cond=FAKE, ws=FAKE, ws_bytes=None):
    if ws_bytes is None:
        ws_bytes = 1 << 40
    return dm.lib().dit_block_forward(ctypes.byref(s), ctypes.byref(bw), x, x_txt, cond, ws, ws_bytes, None)


def test_block_forward_validation(dm):
    s = shape(dm)
    bw = fake_block(dm)
    assert block_call(dm, s, dm.BlockWeights()) == -1                # NULL weights
    assert block_call(dm, s, bw, x=None) == -1
    assert block_call(dm, s, bw, x=FAKE + 4) == -1                     # misaligned x
    assert block_call(dm, s, bw, x_txt=FAKE) == -1                     # x_txt without text tokens
    assert block_call(dm, s, bw, cond=None) == -1
    assert block_call(dm, s, bw, ws=FAKE + 16) == -1                   # workspace not 256-aligned
    need = dm.workspace_bytes(s, dm.DIT_WS_BLOCK)
    assert block_call(dm, s, bw, ws_bytes=need - 1) == -3
    assert "workspace" in dm.last_error()
    bad = fake_block(dm)
    bad.img.b_qkv = FAKE + 2                                           # misaligned bias
    assert block_call(dm, s, bad) == -1
    s2 = shape(dm, head_dim=80, heads=16, hidden=1280)
    assert block_call(dm, s2, bw) == -2


def test_joint_block_needs_text_stream(dm):
    s = shape(dm, "c3")
    assert block_call(dm, s, fake_block(dm, joint=False), x_txt=FAKE) == -1   # txt weights NULL
    assert block_call(dm, s, fake_block(dm, joint=True), x_txt=None) == -1    # x_txt NULL
    need = dm.workspace_bytes(s, dm.DIT_WS_BLOCK)
    assert block_call(dm, s, fake_block(dm, joint=True), x_txt=FAKE, ws_bytes=need - 256) == -3


def test_step_forward_validation(dm):
    lib = dm.lib()
    s = shape(dm, n_blocks=2)
    blocks = (dm.BlockWeights * 2)(fake_block(dm), fake_block(dm))
    sw = dm.StepWeights(FAKE, FAKE, None, ctypes.cast(blocks, ctypes.POINTER(dm.BlockWeights)), FAKE, FAKE, FAKE, FAKE)
    call = lambda s_, w_, **kw: lib.dit_step_forward(ctypes.byref(s_), ctypes.byref(w_), kw.get("patches", FAKE),
                                                    kw.get("x_txt"), FAKE, kw.get("out", FAKE), FAKE,
                                                    kw.get("ws_bytes", 1 << 40), None)
    need = dm.workspace_bytes(s, dm.DIT_WS_STEP)
    assert call(s, sw, ws_bytes=need - 1) == -3
    assert call(s, sw, out=FAKE + 4) == -1                       # out must be 16-byte aligned
    s_bad = shape(dm, n_blocks=2, patch_out=6)
    assert call(s_bad, sw) == -1                                 # patch_out not a multiple of 4
    s_bad = shape(dm, n_blocks=0)
    assert call(s_bad, sw) == -1
    nob = dm.StepWeights(FAKE, FAKE, None, None, FAKE, FAKE, FAKE, FAKE)
    assert call(s, nob) == -1                                    # no block array


def test_sample_euler_validation(dm):
    lib = dm.lib()
    s = shape(dm, n_blocks=2)
    blocks = (dm.BlockWeights * 2)(fake_block(dm), fake_block(dm))
    sw = dm.StepWeights(FAKE, FAKE, None, ctypes.cast(blocks, ctypes.POINTER(dm.BlockWeights)), FAKE, FAKE, FAKE, FAKE)
    cw = dm.CondWeights(FAKE, FAKE, FAKE, FAKE, FAKE)
    sig = (ctypes.c_float * 3)(1.0, 0.5, 0.0)
    need = dm.workspace_bytes(s, dm.DIT_WS_SAMPLE)
    assert need > dm.workspace_bytes(s, dm.DIT_WS_STEP)

    def call(s_=s, cw_=cw, y=FAKE, cond=None, sigmas=sig, n=2, z=FAKE, xt=None, ws_bytes=None):
        return lib.dit_sample_euler(ctypes.byref(s_), ctypes.byref(sw), ctypes.byref(cw_) if cw_ is not None else None,
                                    y, cond, sigmas, n, 1000.0, z, xt, FAKE, need if ws_bytes is None else ws_bytes,
                                    None)

    assert call(ws_bytes=need - 1) == -3
    assert call(n=-1) == -1
    assert call(sigmas=None) == -1
    assert call(z=FAKE + 4) == -1                       # z must be 16-byte aligned
    assert call(y=None) == -1                           # class conditioning needs labels
    assert call(cw_=None) == -1                         # neither conditioning weights nor cond
    assert call(cw_=dm.CondWeights(FAKE + 8, FAKE, FAKE, FAKE, FAKE)) == -1  # w_t1 misaligned
    assert call(s_=shape(dm, n_blocks=2, patch_out=8)) == -1  # patch_in != patch_out
    assert call(xt=FAKE) == -1                          # text states without text tokens


def test_serve_validation(dm):
    lib = dm.lib()
    s = shape(dm, n_blocks=2)
    blocks = (dm.BlockWeights * 2)(fake_block(dm), fake_block(dm))
    sw = dm.StepWeights(FAKE, FAKE, None, ctypes.cast(blocks, ctypes.POINTER(dm.BlockWeights)), FAKE, FAKE, FAKE, FAKE)
    cw = dm.CondWeights(FAKE, FAKE, FAKE, FAKE, FAKE)
    sig = (ctypes.c_float * 2)(1.0, 0.0)
    reqs = (dm.Request * 2)(dm.Request(FAKE, FAKE, FAKE, None), dm.Request(FAKE, FAKE, FAKE, None))
    need = dm.workspace_bytes(s, dm.DIT_WS_SERVE)
    assert need > dm.workspace_bytes(s, dm.DIT_WS_SAMPLE)

    def call(s_=s, cw_=cw, r=reqs, n=2, overlap=1, cs=FAKE, ws_bytes=None):
        return lib.dit_serve(ctypes.byref(s_), ctypes.byref(sw), ctypes.byref(cw_) if cw_ is not None else None, r, n,
                             sig, 1, 1000.0, overlap, 0, 0, FAKE, need if ws_bytes is None else ws_bytes, None, cs)

    assert call(ws_bytes=need - 1) == -3
    assert call(cs=None) == -1                                          # overlap needs a copy stream
    assert call(cw_=None) == -1                                         # requests carry y but no cond
    assert call(r=None) == -1
    assert call(n=-1) == -1
    assert call(n=0, r=None, overlap=0, cs=None) == 0                   # nothing to do, nothing enqueued
    joint = shape(dm, "c3", n_blocks=2)
    assert lib.dit_serve(ctypes.byref(joint), ctypes.byref(sw), None, reqs, 2, sig, 1, 1000.0, 0, 0, 0, FAKE, 1 << 40,
                         None, None) == -2                              # image-only models


def test_cond_pos_and_timing_validation(dm):
    lib = dm.lib()
    s = shape(dm)
    z = [FAKE] * 8
    assert lib.dit_cond_embed(ctypes.byref(s), *z, FAKE, 4, None) == -3
    assert lib.dit_cond_embed(ctypes.byref(s), None, *z[1:], FAKE, 1 << 30, None) == -1
    assert lib.dit_cond_embed(ctypes.byref(s), FAKE, FAKE, FAKE + 8, *z[3:], FAKE, 1 << 30, None) == -1  # w_t1 misaligned
    assert lib.dit_pos_embed_2d(0, 4, 8, FAKE, None) == -1
    assert lib.dit_pos_embed_2d(4, 4, 6, FAKE, None) == -1
    assert lib.dit_pos_embed_2d(4, 4, 8, None, None) == -1
    assert lib.dit_timing_enable(99, 10) == -1
    assert lib.dit_timing_enable(0, 0) == -1
    assert lib.dit_timing_disable() == 0


def test_binding_rejects_host_tensors(dm):
    import torch
    s = shape(dm)
    with pytest.raises(ValueError):
        dm.block_forward(s, fake_block(dm), torch.zeros(4), torch.zeros(4), torch.zeros(4, dtype=torch.uint8))
