"""dard_confidence_noalloc (the confidence reduction with the library's
preallocated scratch) against dard_confidence with a caller workspace: the
same kernels on the same inputs, so every output must be identical.  Two
calls in a row, the second smaller, so that the second reads nothing left
over from the first; and a size beyond the scratch is refused."""
import sys

import numpy as np
import pytest
import torch

from paper_2608_26574_amd import dard

pytestmark = pytest.mark.gpu


def announce(*a):
    print("[case]", *a, file=sys.stderr, flush=True)


def run_both(rows, V, mixed, stats, pcur, seed):
    g = torch.Generator(device="cuda").manual_seed(seed)
    ls = torch.randn(rows, V, generator=g, device="cuda") * 4.0
    lx = torch.randn(rows, V, generator=g, device="cuda") * 4.0 if mixed else None
    w = torch.rand(rows, generator=g, device="cuda") if mixed else None
    cur = torch.randint(0, V, (rows,), generator=g, device="cuda", dtype=torch.int32) if pcur else None
    outs = []
    for noalloc in (False, True):
        o = dict(argmax=torch.full((rows,), -7, dtype=torch.int32, device="cuda"),
                 maxprob=torch.full((rows,), -1.0, device="cuda"))
        if pcur:
            o["pcur"] = torch.full((rows,), -1.0, device="cuda")
        if stats:
            o["entropy"] = torch.full((rows,), -1.0, device="cuda")
            o["margin"] = torch.full((rows,), -1.0, device="cuda")
        kw = dict(logits_x=lx, w=w, cur_tok=cur, pcur=o.get("pcur"), entropy=o.get("entropy"),
                  margin=o.get("margin"))
        if noalloc:
            dard.dard_confidence_noalloc(ls, o["argmax"], o["maxprob"], **kw)
        else:
            ws = torch.empty(dard.dard_confidence_workspace_bytes(rows, V), dtype=torch.uint8, device="cuda")
            dard.dard_confidence(ls, o["argmax"], o["maxprob"], ws=ws, **kw)
        torch.cuda.synchronize()
        outs.append({k: v.cpu().numpy() for k, v in o.items()})
    return outs


def test_noalloc_confidence_matches_workspace_entry():
    # a large call (the 7B GQA batch-8 step's 696 rows, vocab 152064, mixed
    # rows with the entropy / margin statistics), then a smaller one (the 8B
    # step's 44 rows, vocab 126464, plain rows with the current token's
    # probability)
    for rows, V, mixed, stats, pcur, seed in ((696, 152064, True, True, False, 1),
                                             (44, 126464, False, False, True, 2)):
        announce("confidence noalloc", rows, V, mixed, stats, pcur)
        ref, got = run_both(rows, V, mixed, stats, pcur, seed)
        for k in ref:
            assert np.array_equal(ref[k], got[k]), k
        assert np.all(got["argmax"] >= 0) and np.all(got["maxprob"] > 0)


def test_noalloc_confidence_refuses_sizes_beyond_the_scratch():
    announce("confidence noalloc size limit")
    V = 152064                                  # 19 chunks of 8192
    rows = (1 << 20) // (19 * 5) + 1            # one row more than the scratch holds with statistics
    ls = torch.zeros(1, 8, device="cuda")       # never read: the call is refused on the host
    am = torch.zeros(1, dtype=torch.int32, device="cuda")
    mp = torch.zeros(1, device="cuda")
    L = dard.lib()
    rc = L.dard_confidence_noalloc(ls.data_ptr(), None, None, None, rows, V, V, am.data_ptr(), mp.data_ptr(), None,
                                   mp.data_ptr(), None, None)
    assert rc == -2, rc
    assert b"scratch" in L.dard_last_error()
