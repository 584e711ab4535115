"""GPU parity of the varlen attention step (sphinx_varlen_attention, the
attention of the denoiser blocks on its own) against the oracle's attention
in fp64 on the same bf16 inputs, through the C ABI.

The kernels take q already multiplied by log2(e)/sqrt(d) and run a base-2
softmax, i.e. softmax(ln(2) q k^T) in the oracle's terms.  Covered: ragged
segments around the 64-key tile and 128-query tile edges, queries and keys of
different lengths (the latent-cache layout), strided rows as in the QKV
buffer, both bf16 head dims, the fp32 path, inputs whose scores rise by
far more than 2^64 above the first tile's maximum, so that the kernel's rare
rebase path runs: once, in the last (partial) tile, and repeatedly, and
inputs whose first-tile maxima lie far above or below zero (at head_dim 64
the running max starts at zero only for maxima in [-64, 32]; these waves
start shifted, in some cases next to unshifted waves of the same tile).

Bound for bf16: every probability is rounded to bf16 (relative 2^-9), which
moves an output by at most 2^-8 max|v|; o itself is rounded to bf16
(relative 2^-9); accumulation is fp32.  The test allows 1.2e-2 max|v|.
"""
import math

import numpy as np
import pytest

import oracle as O

torch = pytest.importorskip("torch")
S = pytest.importorskip("paper_2511_18672_amd")

pytestmark = pytest.mark.gpu

LN2 = math.log(2.0)


def bf16(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16)


def run(q, k, v, heads, hd, cu_q, cu_kv, dtype="bf16", ldq=None, ldkv=None):
    """q, k, v: float arrays [rows][heads*hd] (bf16 values for bf16).  Rows are
    placed in buffers of stride ldq / ldkv.  Returns o (float64) and the exact
    inputs used."""
    D = heads * hd
    ldq, ldkv = ldq or D, ldkv or D
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    code = S.BF16 if dtype == "bf16" else S.F32

    def place(a, ld):
        buf = torch.zeros((a.shape[0], ld), dtype=tdt)
        buf[:, :D] = torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(tdt)
        return buf

    qb, kb, vb = place(q, ldq), place(k, ldkv), place(v, ldkv)
    o = torch.full((q.shape[0], D), float("nan"), dtype=tdt, device="cuda")
    print(f"[attention] {dtype} heads={heads} hd={hd} cu_q={list(cu_q)} cu_kv={list(cu_kv)}", flush=True)
    S.sphinx_varlen_attention(code, heads, hd, qb.cuda(), ldq, kb.cuda(), vb.cuda(), ldkv, o, cu_q, cu_kv)
    torch.cuda.synchronize()
    exact = lambda b: b[:, :D].double().numpy()
    return o.double().cpu().numpy(), exact(qb), exact(kb), exact(vb)


def check(q, k, v, heads, hd, cu_q, cu_kv, dtype="bf16", tag="", **kw):
    got, qe, ke, ve = run(q, k, v, heads, hd, cu_q, cu_kv, dtype, **kw)
    ref = O.attention(qe, ke, ve, heads, np.asarray(cu_q), kv_seg=np.asarray(cu_kv), scale=LN2)
    rows = np.concatenate([np.arange(cu_q[i], cu_q[i + 1]) for i in range(len(cu_q) - 1)])
    err = float(np.abs(got[rows] - ref[rows]).max())
    tol = 1.2e-2 * float(np.abs(ve).max()) if dtype == "bf16" else 1e-5
    print(f"[attention {tag}] max_abs = {err:.3e} (tol {tol:.3e})", flush=True)
    assert np.isfinite(got[rows]).all()
    assert err <= tol
    return err


def rand(rng, n, D, scale=1.0):
    return (rng.standard_normal((n, D)) * scale).astype(np.float32)


@pytest.mark.parametrize("hd", [64, 72])
def test_ragged_self_attention(hd):
    rng = np.random.default_rng(1)
    heads = 4
    lens = [1, 63, 64, 65, 127, 128, 129, 200, 700]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    n = int(cu[-1])
    q, k, v = rand(rng, n, heads * hd, 0.3), rand(rng, n, heads * hd), rand(rng, n, heads * hd)
    check(q, k, v, heads, hd, cu, cu, tag=f"ragged hd{hd}")


@pytest.mark.parametrize("hd", [64, 72])
def test_queries_and_keys_differ(hd):
    """Query and key segments of different lengths (the latent-cache layout),
    rows strided as in the QKV buffer (q stride 3D, k/v stride 2D)."""
    rng = np.random.default_rng(2)
    heads = 2
    D = heads * hd
    cu_q = np.array([0, 5, 5, 150, 420], np.int32)
    cu_kv = np.array([0, 300, 301, 1301, 1350], np.int32)
    q = rand(rng, int(cu_q[-1]), D, 0.3)
    k, v = rand(rng, int(cu_kv[-1]), D), rand(rng, int(cu_kv[-1]), D)
    check(q, k, v, heads, hd, cu_q, cu_kv, tag=f"q!=kv hd{hd}", ldq=3 * D, ldkv=2 * D)


def _first_tile_gap(q, k, cu_q, cu_kv, heads, hd):
    """Largest (max score over the segment) - (max score over its first 64 keys),
    in log2 units, over the queries and heads: > 64 means a rebase must happen."""
    worst = 0.0
    for i in range(len(cu_q) - 1):
        for h in range(heads):
            c = slice(h * hd, (h + 1) * hd)
            s = q[cu_q[i]:cu_q[i + 1], c].astype(np.float64) @ k[cu_kv[i]:cu_kv[i + 1], c].astype(np.float64).T
            worst = max(worst, float((s.max(axis=1) - s[:, :64].max(axis=1)).max()))
    return worst


@pytest.mark.parametrize("hd", [64, 72])
@pytest.mark.parametrize("case", ["later_tiles", "last_partial_tile", "rising"])
def test_rebase_path(hd, case):
    """Scores that climb far above the first tile's maximum force the kernel's
    rare rebase (running max moved, O and l rescaled, probabilities remade)."""
    rng = np.random.default_rng(3)
    heads = 2
    D = heads * hd
    n = 200 if case == "last_partial_tile" else 700
    q = rand(rng, n, D, 0.5)
    k = rand(rng, n, D, 0.5)
    v = rand(rng, n, D)
    if case == "later_tiles":
        k[128:] *= 40.0
    elif case == "last_partial_tile":
        k[192:] *= 40.0  # keys 192..199: the last tile holds 8 keys
    else:
        for t in range(n // 64 + 1):
            k[64 * t:64 * (t + 1)] *= 1.0 + 12.0 * t
    cu = np.array([0, n], np.int32)
    qe = bf16(q).double().numpy()
    ke = bf16(k).double().numpy()
    gap = _first_tile_gap(qe, ke, cu, cu, heads, hd)
    print(f"[attention rebase {case} hd{hd}] scores rise {gap:.0f} above the first tile's max (log2 units)")
    assert gap > 128
    check(q, k, v, heads, hd, cu, cu, tag=f"rebase {case} hd{hd}")


@pytest.mark.parametrize("hd", [64, 72])
@pytest.mark.parametrize("case", ["high", "low", "mixed"])
def test_shifted_from_start(hd, case):
    """Every score near +512 ("high": exp2 overflows without the shift), near
    -512 ("low": the row sum underflows to zero without it), or the queries
    32..63 of every 128-query tile near -512 and the rest moderate ("mixed":
    one shifted wave per workgroup)."""
    rng = np.random.default_rng(6)
    heads = 2
    D = heads * hd
    n = 300
    e = np.ones((1, D), np.float32)
    k = rand(rng, n, D, 0.3) + 4.0 * e
    q = rand(rng, n, D, 0.3) + (2.0 if case == "high" else -2.0) * e
    if case == "mixed":
        moderate = (np.arange(n) % 128 < 32) | (np.arange(n) % 128 >= 64)
        q[moderate] = rand(rng, int(moderate.sum()), D, 0.3)
    v = rand(rng, n, D)
    cu = np.array([0, n], np.int32)
    qe, ke = bf16(q).double().numpy(), bf16(k).double().numpy()
    m0 = np.stack([qe[:, h * hd:(h + 1) * hd] @ ke[:64, h * hd:(h + 1) * hd].T for h in range(heads)]).max(axis=2)
    print(f"[attention shifted {case} hd{hd}] first-tile maxima in [{m0.min():.0f}, {m0.max():.0f}]")
    assert (m0.max() > 256) if case == "high" else (m0.min() < -256)
    check(q, k, v, heads, hd, cu, cu, tag=f"shifted {case} hd{hd}")


def test_fp32_path():
    rng = np.random.default_rng(4)
    heads, hd = 4, 16
    cu = np.array([0, 1, 40, 170], np.int32)
    n = int(cu[-1])
    q, k, v = rand(rng, n, heads * hd, 0.5), rand(rng, n, heads * hd), rand(rng, n, heads * hd)
    check(q, k, v, heads, hd, cu, cu, dtype="f32", tag="fp32")


def test_zero_query_is_mean_of_values():
    """q = 0: every key has weight 2^0, the output is the mean of the segment's values."""
    rng = np.random.default_rng(5)
    heads, hd = 1, 64
    cu = np.array([0, 300], np.int32)
    v = rand(rng, 300, hd)
    got, _, _, ve = run(np.zeros((300, hd), np.float32), rand(rng, 300, hd), v, heads, hd, cu, cu)
    err = float(np.abs(got - ve.mean(axis=0)[None, :]).max())
    print(f"[attention q=0] max_abs vs mean of values = {err:.3e}")
    assert err <= 1.2e-2 * float(np.abs(ve).max())
