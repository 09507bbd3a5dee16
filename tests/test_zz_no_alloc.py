"""wino_epilogue_noalloc (partials in the library's per-GPU scratch array, no
workspace argument) against wino_epilogue (caller workspace) on the same
inputs: the same kernels run, so tokens, mask bitmap, flags and statistics
must be bit-identical.  Two calls in a row, the second with a smaller input,
so the second call runs on scratch the first one left behind."""
import numpy as np
import pytest
import torch

import wino_inputs as wi

pytestmark = pytest.mark.gpu

STATS_BYTES = 24


@pytest.fixture(scope="module")
def P():
    import paper_2605_16941_amd as pkg
    return pkg


def run_both(P, B, lb, V, heights, seed):
    mask = V - 1
    logits, cur, _ = wi.epilogue_inputs(B, lb, V, mask, seed=seed, heights=heights, device="cuda")
    prm = P.make_params(B, 1, lb, lb, mask, 0.7, 0.9)
    outs = []
    for noalloc in (True, False):
        c = cur.clone()
        bitmap = torch.full((B, lb), 9, dtype=torch.uint8, device="cuda")
        flags = torch.full((B, lb), 9, dtype=torch.uint8, device="cuda")
        stats = torch.full((B * lb * STATS_BYTES,), 7, dtype=torch.uint8, device="cuda")
        if noalloc:
            P.wino_epilogue_noalloc(prm, V, logits, c, bitmap, flags, stats)
        else:
            ws = torch.zeros(P.wino_epilogue_workspace_bytes(B, lb, V), dtype=torch.uint8, device="cuda")
            P.wino_epilogue(prm, V, logits, c, bitmap, flags, stats, ws)
        torch.cuda.synchronize()
        outs.append((c.cpu(), bitmap.cpu(), flags.cpu(), stats.cpu()))
    (ct, cb, cf, cs), (wt, wb, wf, wsx) = outs
    assert torch.equal(ct, wt) and torch.equal(cb, wb) and torch.equal(cf, wf) and torch.equal(cs, wsx)
    # the call decided something: tokens changed and the bitmap marks masks
    assert not torch.equal(ct, cur.cpu())
    assert torch.equal(cb, (ct == mask).to(torch.uint8))
    return int((cf > 0).sum())


def test_noalloc_epilogue_matches_workspace_entry_point(P):
    # the standalone-epilogue shape (logits [8, 64, 126464]), then a smaller call
    n1 = run_both(P, 8, 32, 126464, (10.0, 16.0), seed=2)
    n2 = run_both(P, 3, 5, 1000, (0.0, 14.0), seed=3)
    print(f"decisions other than keep: {n1} (8x32 positions), {n2} (3x5 positions)")
    assert n1 > 0 and n2 > 0


def test_noalloc_epilogue_rejects_inputs_beyond_its_scratch(P):
    # 128 x 128 positions at vocab 126464 need 5.2 MB of partials > 2 MiB:
    # rejected on the host before any device work
    B, lb, V = 128, 128, 126464
    assert P.wino_epilogue_workspace_bytes(B, lb, V) > P._abi.EPILOGUE_NOALLOC_MAX_BYTES
    prm = P.make_params(B, 1, lb, lb, V - 1, 0.7, 0.9)
    dummy = torch.zeros(8, dtype=torch.bfloat16, device="cuda")
    cur = torch.zeros(8, dtype=torch.int32, device="cuda")
    bm = torch.zeros(8, dtype=torch.uint8, device="cuda")
    with pytest.raises(P.WinoError) as e:
        P.wino_epilogue_noalloc(prm, V, dummy, cur, bm)
    assert e.value.status == -2
    torch.cuda.synchronize()
    assert torch.equal(cur.cpu(), torch.zeros(8, dtype=torch.int32))
