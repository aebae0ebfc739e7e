"""GPU robustness of the C ABI: every write stays inside the caller's
buffers, const inputs come back unchanged, and NaN in the input propagates
the way the oracle's arithmetic does, with the call returning normally.

Guard bands: x, x_txt, out and the workspace are carved out of larger
device buffers whose margins hold a NaN byte pattern; after the call the
margins must be byte-identical.  Const inputs (weights, cond, patches) are
hashed before and after the call; this is the tensor-hash consistency check
the paper applies to data moved between stages, used here to show the
library never writes what it only reads.
"""
import hashlib

import numpy as np
import pytest
import torch

import synth
from oracle import dit_oracle as O

pytestmark = pytest.mark.gpu

GUARD = 4096             # bytes of margin on each side (a multiple of 256)
PATTERN = 0x7FBADBAD     # a NaN as fp32, repeated over the margins


def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests import gpu_util
    import paper_2605_25550_amd as dm
    return gpu_util, dm


class Guarded:
    """A device region of nbytes with GUARD bytes of PATTERN on each side."""

    def __init__(self, nbytes):
        self.n = nbytes
        span = (nbytes + 255) // 256 * 256
        self.buf = torch.empty(GUARD + span + GUARD, dtype=torch.uint8, device="cuda")
        self.buf.view(torch.int32).fill_(PATTERN)
        self.inner = self.buf[GUARD:GUARD + nbytes]
        self.ref_lo = self.buf[:GUARD].clone()
        self.ref_hi = self.buf[GUARD + nbytes:].clone()

    def f32(self, shape, init=None):
        t = self.inner.view(torch.float32).view(*shape)
        if init is not None:
            t.copy_(torch.from_numpy(np.ascontiguousarray(init, dtype=np.float32)))
        return t

    def intact(self):
        torch.cuda.synchronize()
        return torch.equal(self.buf[:GUARD], self.ref_lo) and torch.equal(self.buf[GUARD + self.n:], self.ref_hi)


def digest(tensors):
    h = hashlib.sha256()
    for t in tensors:
        h.update(t.detach().cpu().contiguous().view(torch.uint8).numpy().tobytes())
    return h.hexdigest()


def _stream_tensors(streams):
    out = []
    for s in streams:
        if s is not None:
            out += [s[k] for k in sorted(s)]
    return out


BLOCK_CASES = [
    ("c1_block", synth.CONFIGS["c1"].with_(n_blocks=1)),
    # one sample: the output projection and fc2 run as k-range units whose
    # fp32 partials live in a workspace region
    ("c1_block_b1_split", synth.CONFIGS["c1"].with_(batch=1, n_blocks=1)),
    ("joint_block", synth.CONFIGS["c3"].with_(batch=2, tokens=130, text_tokens=21, hidden=256, heads=2, head_dim=128,
                                              mlp_hidden=1024, n_blocks=1)),
]


@pytest.mark.parametrize("name,cfg", BLOCK_CASES, ids=[c[0] for c in BLOCK_CASES])
def test_block_writes_stay_in_bounds_and_inputs_are_unchanged(name, cfg):
    g, dm = _gpu()
    print(f"[case] guard bands, block {name}", flush=True)
    db = g.DeviceBlock(cfg, synth.block_weights(cfg, 0))
    inp = synth.inputs(cfg)
    B, T, Tt, D = cfg.batch, cfg.tokens, cfg.text_tokens, cfg.hidden
    gx = Guarded(B * T * D * 4)
    x = gx.f32((B, T, D), inp["x"])
    gxt, xt = None, None
    if cfg.joint:
        gxt = Guarded(B * Tt * D * 4)
        xt = gxt.f32((B, Tt, D), inp["x_txt"])
    gws = Guarded(dm.workspace_bytes(db.shape, dm.DIT_WS_BLOCK))
    cond = g.dev(inp["cond"])
    consts = _stream_tensors([db.img, db.txt]) + [cond]
    before = digest(consts)
    dm.block_forward(db.shape, db.struct, x, cond, gws.inner, x_txt=xt)
    torch.cuda.synchronize()
    assert gx.intact(), "write outside x"
    assert gxt is None or gxt.intact(), "write outside x_txt"
    assert gws.intact(), "write outside the workspace"
    assert digest(consts) == before, "a const input changed"
    assert torch.isfinite(x).all()


def test_step_writes_stay_in_bounds_and_inputs_are_unchanged():
    g, dm = _gpu()
    cfg = synth.CONFIGS["c1"].with_(n_blocks=2)
    print("[case] guard bands, c1 step with 2 blocks", flush=True)
    ds = g.DeviceStep(cfg)
    inp = synth.inputs(cfg)
    B, T = cfg.batch, cfg.tokens
    gout = Guarded(B * T * cfg.patch_out * 4)
    out = gout.f32((B, T, cfg.patch_out))
    gws = Guarded(dm.workspace_bytes(ds.shape, dm.DIT_WS_STEP))
    patches, cond = g.dev(inp["patches"]), g.dev(inp["cond"])
    consts = [patches, cond, ds.pos] + [ds.step[k] for k in sorted(ds.step)]
    for img, txt in ds.blocks:
        consts += _stream_tensors([img, txt])
    before = digest(consts)
    dm.step_forward(ds.shape, ds.table, patches, cond, out, gws.inner)
    torch.cuda.synchronize()
    assert gout.intact(), "write outside out"
    assert gws.intact(), "write outside the workspace"
    assert digest(consts) == before, "a const input changed"
    assert torch.isfinite(out).all()


NAN_CASES = [
    ("dh128", synth.CONFIGS["c1"].with_(batch=2, tokens=40, hidden=256, heads=2, head_dim=128, mlp_hidden=512,
                                        n_blocks=1)),
    # head_dim 72: the attention kernel carries the softmax bookkeeping in the
    # MFMA padding column
    ("dh72", synth.CONFIGS["c1"].with_(batch=2, tokens=40, n_blocks=1)),
]


@pytest.mark.parametrize("name,cfg", NAN_CASES, ids=[c[0] for c in NAN_CASES])
def test_nan_in_x_propagates_like_the_oracle(name, cfg):
    """A NaN in one token of sample 0: the call returns normally, the NaN
    positions of the result are those of the oracle (every output of sample
    0: the poisoned key reaches every query through attention), and sample 1
    is bitwise what a clean run gives."""
    g, dm = _gpu()
    print(f"[case] NaN propagation {name}", flush=True)
    w = synth.block_weights(cfg, 0)
    inp = synth.inputs(cfg)
    x_bad = inp["x"].copy()
    x_bad[0, 3, 5] = np.nan
    y_bad, _ = g.run_block(cfg, w, x_bad, inp["cond"])
    y_ok, _ = g.run_block(cfg, w, inp["x"], inp["cond"])
    ref = O.dit_block(x_bad, inp["cond"], {k: v.astype(np.float64) for k, v in w["img"].items()}, cfg.heads,
                      cfg.ln_eps)
    assert np.isnan(ref[0]).all() and np.isfinite(ref[1]).all()
    assert np.array_equal(np.isnan(y_bad), np.isnan(ref))
    assert np.array_equal(y_bad[1], y_ok[1])
