"""The allocation-free selection (sphinx_select_mask_static, scratch in a
static device array of the library) against sphinx_select_mask with a
caller workspace, through the C ABI: two calls in a row, the second with a
smaller input, then the headline input; masks, indices and cu_sel
bit-identical to the workspace call and to the oracle."""
import numpy as np
import pytest

import oracle as O
import workloads as W
from pins import MICRO_BF16

torch = pytest.importorskip("torch")
S = pytest.importorskip("paper_2511_18672_amd")

pytestmark = pytest.mark.gpu


def _run(fn, wl, ws=None):
    N = wl.N
    reqs = S.make_requests(wl.requests)
    mask = torch.full((N,), 7, dtype=torch.uint8, device="cuda")
    idx = torch.full((N,), -7, dtype=torch.int32, device="cuda")
    cu = torch.full((wl.R + 1,), -7, dtype=torch.int32, device="cuda")
    u = torch.from_numpy(wl.u).cuda()
    thr = torch.from_numpy(wl.thr).cuda()
    if ws is None:
        host = fn(reqs, u, thr, None, mask, idx, cu)
    else:
        host = fn(reqs, u, thr, None, mask, idx, cu, ws)
    n = int(host[-1])
    return mask.cpu().numpy(), idx[:n].cpu().numpy(), host, cu.cpu().numpy()


def test_select_static_matches_workspace_call():
    big = W.custom("static_big", MICRO_BF16, [W.Request(150, 128, 128), W.Request(2, 6, 4)], [0.3, 0.6],
                   [0.5, 0.5], [1, 1], u_recipe="uniform", with_weights=False)
    small = W.custom("static_small", MICRO_BF16, [W.Request(3, 6, 10), W.Request(1, 64, 66)], [0.5, 0.2],
                     [0.5, 0.5], [1, 1], u_recipe="uniform", with_weights=False)
    head = W.headline(with_weights=False)
    for wl in (big, small, head):
        print(f"[select_static] {wl.name} N={wl.N} chunks={(wl.N + 4095) // 4096}", flush=True)
        ws = torch.full((S.sphinx_select_workspace_bytes(wl.N),), 0xAB, dtype=torch.uint8, device="cuda")
        ref = _run(S.sphinx_select_mask, wl, ws)
        got = _run(S.sphinx_select_mask_static, wl)
        for a, b in zip(ref, got):
            assert np.array_equal(a, b)
        info = O.token_info(wl.requests)
        mask, idx, cu, n = O.select(wl.u, wl.thr[info.gframe], np.ones(wl.N, bool), wl.tok_offset[:-1])
        assert np.array_equal(got[0].astype(bool), mask)
        assert np.array_equal(got[1], idx)
        assert list(got[2]) == list(cu) + [n]
        print(f"[select_static] {wl.name} n_sel={n} bit-identical", flush=True)
