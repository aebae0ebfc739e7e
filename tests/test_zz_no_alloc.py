"""dit_block_forward_noalloc (the block call for callers that cannot
allocate device memory) against dit_block_forward, through the C ABI: two
calls in a row on the library's static per-GPU scratch, the second with a
smaller input, each bitwise equal to the workspace entry point's result on
the same inputs (the same kernels run on the same data)."""
import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu

CASES = [
    ("c1_block", synth.CONFIGS["c1"].with_(n_blocks=1)),
    ("joint_small", synth.CONFIGS["c3"].with_(batch=2, tokens=130, text_tokens=21, hidden=256, heads=2, head_dim=128,
                                              mlp_hidden=1024, n_blocks=1)),
]


def test_noalloc_matches_workspace_entry_point_twice():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests import gpu_util as g
    import paper_2605_25550_amd as dm
    for name, cfg in CASES:
        print(f"[case] noalloc {name} B={cfg.batch} T={cfg.tokens} Tt={cfg.text_tokens} D={cfg.hidden}", flush=True)
        db = g.DeviceBlock(cfg, synth.block_weights(cfg, 0))
        assert dm.workspace_bytes(db.shape, dm.DIT_WS_BLOCK) <= dm.NOALLOC_SCRATCH_BYTES
        inp = synth.inputs(cfg)
        cond = g.dev(inp["cond"])
        # reference: the workspace entry point
        ws = dm.alloc_workspace(db.shape, dm.DIT_WS_BLOCK)
        x_ref = g.dev(inp["x"])
        xt_ref = g.dev(inp["x_txt"]) if cfg.joint else None
        dm.block_forward(db.shape, db.struct, x_ref, cond, ws, x_txt=xt_ref)
        # the no-allocation entry point on the same inputs
        x = g.dev(inp["x"])
        xt = g.dev(inp["x_txt"]) if cfg.joint else None
        dm.block_forward_noalloc(db.shape, db.struct, x, cond, x_txt=xt)
        torch.cuda.synchronize()
        assert torch.isfinite(x).all()
        assert torch.equal(x, x_ref), name
        if cfg.joint:
            assert torch.equal(xt, xt_ref), name
        assert not np.array_equal(g.host(x), inp["x"].astype(np.float64))
        del ws
