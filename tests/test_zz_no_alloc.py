"""fc_select_noalloc (no device allocation, static scratch) against fc_select.

The two entry points run the same kernels; the no-alloc one takes its workspace
from the library's static device array.  Two calls in a row, the second on a
smaller input, must each give exactly the outputs of fc_select on the same
inputs; the smaller one is also checked against the oracle.
"""
import numpy as np
import pytest
import torch

import fcdata
from oracle import select as osel
from tests import fcutil

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fc():
    import paper_2604_24391_amd as fc
    return fc


def _run(fc, fn, prm, prev, cur, N):
    out = fc.SelectOut.alloc(cur.shape[0], N)
    # poison the outputs so that a field the call leaves unwritten cannot match by luck
    for k in ("sim", "energy", "reuse_mask", "recompute_idx", "n_recompute", "shift", "scalars",
              "counts", "flags"):
        getattr(out, k).fill_(7)
    fn(prm, prev, cur, out)
    torch.cuda.synchronize()
    return fcutil.select_out_np(out)


def test_noalloc_matches_fc_select_twice_then_smaller(fc):
    torch.cuda.set_device(0)
    ctx = fc.Context(fc.Caps(max_batch=8, max_height=448, max_width=448, max_tokens=1024,
                             max_seq=64, max_d_model=64, max_ffn=64, max_qkv=64))
    try:
        cases = []
        prev, cur, _ = fcdata.sel_pairs(1, batch=6)                 # 6 pairs of 448x448
        cases.append((fc.SelectParams(), prev, cur))
        tp, tc, _ = fcdata.tiny_pair(0)                             # then one 224x224 pair
        cases.append((fc.SelectParams(adaptive=False, alpha_fixed=0.5), tp, tc))
        for prm, p_np, c_np in cases:
            print(f"[no-alloc] B={c_np.shape[0]} {c_np.shape[2]}x{c_np.shape[3]}", flush=True)
            p = torch.from_numpy(np.ascontiguousarray(p_np)).cuda()
            c = torch.from_numpy(np.ascontiguousarray(c_np)).cuda()
            gh, gw = fc.token_grid(c.shape[2], c.shape[3], prm)
            ref = _run(fc, lambda *a: fc.fc_select(ctx, *a), prm, p, c, gh * gw)
            got = _run(fc, fc.fc_select_noalloc, prm, p, c, gh * gw)
            for k, v in ref.items():
                np.testing.assert_array_equal(got[k], v, err_msg=k)
        # the smaller call against the oracle as well
        op = fcutil.oracle_select_params(cases[1][0])
        res = osel.select_item(tp[0], tc[0], op)
        mg, esc = fcutil.check_select(got, res, op, 0)
        assert not esc
    finally:
        ctx.close()


def test_noalloc_rejects_oversize_batch(fc):
    """64 pairs of 448x448 need about 55 MB of workspace: refused, nothing launched."""
    prm = fc.SelectParams()
    cur = torch.zeros(64, 3, 448, 448, device="cuda")
    out = fc.SelectOut.alloc(64, 1024)
    with pytest.raises(fc.FcError) as e:
        fc.fc_select_noalloc(prm, None, cur, out)
    assert e.value.status == 3
