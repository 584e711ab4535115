"""ctypes binding of ``libsphinx.so`` (include/sphinx.h).

Argument marshalling only: torch tensors provide device memory and streams,
every computation runs in the library's HIP kernels.  Each C entry point has a
Python function of the same name (``sphinx_select_mask`` ...) and a short alias
(``select_mask`` ...).  A non-OK status raises ``SphinxError``.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_char_p, c_float, c_int32, c_int64, c_size_t, c_uint8, c_void_p
from typing import Dict, Optional, Sequence

import numpy as np

# SPHINX_LIBRARY names another build of the same library (the host-only
# sanitizer build of the CPU tests); by default the in-tree gfx950 build.
LIB_PATH = os.environ.get("SPHINX_LIBRARY") or os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsphinx.so")

F32, BF16 = 0, 1
NCHW, TOKENS = 0, 1  # sphinx_layout
ATTN_JOINT, ATTN_FACTORISED = 0, 1  # sphinx_attention
GRID_SHARED, GRID_PER_FRAME = 0, 1  # sphinx_grid
MAX_REQUESTS = 64
STATUS_NAMES = {0: "SPHINX_OK", 1: "SPHINX_E_INVALID", 2: "SPHINX_E_UNSUPPORTED", 3: "SPHINX_E_WORKSPACE",
                4: "SPHINX_E_HIP"}
PARAMS = ["PE_W", "PE_B", "T1_W", "T1_B", "T2_W", "T2_B", "COND_W", "COND_B", "QKV_W", "QKV_B", "O_W", "O_B",
          "FC1_W", "FC1_B", "FC2_W", "FC2_B", "OUT_W", "OUT_B"]
PARAM_ID = {n: i for i, n in enumerate(PARAMS)}
EXPORTED = ["sphinx_status_string", "sphinx_model_blob_bytes", "sphinx_model_param", "sphinx_plan_step",
            "sphinx_plan_step_grid",
            "sphinx_select_workspace_bytes", "sphinx_select_mask", "sphinx_gather", "sphinx_refine_workspace_bytes",
            "sphinx_refine_step", "sphinx_scatter_blend", "sphinx_timing_enable", "sphinx_timing_read",
            "sphinx_peak_mfma", "sphinx_plan_cache", "sphinx_kv_cache_bytes", "sphinx_gather_ctx",
            "sphinx_refine_step_cached", "sphinx_scatter_masked", "sphinx_mask_frontend_workspace_bytes",
            "sphinx_mask_frontend", "sphinx_adaptive_start", "sphinx_select_mask_static", "sphinx_varlen_attention"]
PEAK_BLOCKS = 2048
PEAK_CONSTANT, PEAK_RANDOM = 0, 1
KERNEL_CLASSES = ["select", "gather", "cond", "embed", "ln", "gemm_qkv", "attention", "gemm_out", "gemm_mlp1",
                  "gemm_mlp2", "final", "scatter", "kv_store", "frontend"]


class SphinxError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn} returned {STATUS_NAMES.get(status, status)}")


class Request(ctypes.Structure):
    _fields_ = [("frames", c_int32), ("h", c_int32), ("w", c_int32), ("frame_offset", c_int32),
                ("tok_offset", c_int64)]


class KLogic(ctypes.Structure):
    _fields_ = [("n", c_int32), ("ratio", ctypes.c_float * 15), ("k", c_int32 * 16)]


def make_klogic(ratio: Sequence[float], k: Sequence[int]) -> KLogic:
    """C k-decision table: len(ratio) breakpoints, len(ratio)+1 start steps."""
    t = KLogic()
    t.n = len(ratio)
    for i, v in enumerate(ratio):
        t.ratio[i] = v
    for i, v in enumerate(k):
        t.k[i] = v
    return t


class ModelDesc(ctypes.Structure):
    _fields_ = [("D", c_int32), ("heads", c_int32), ("head_dim", c_int32), ("mlp", c_int32), ("L", c_int32),
                ("dtype", c_int32), ("attention", c_int32), ("weights", c_void_p)]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libsphinx.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built: run __graft_entry__.build() first")
    L = ctypes.CDLL(LIB_PATH)
    P = c_void_p
    sig = {
        "sphinx_status_string": (c_char_p, [c_int32]),
        "sphinx_model_blob_bytes": (c_int32, [POINTER(ModelDesc), POINTER(c_size_t)]),
        "sphinx_model_param": (c_int32, [POINTER(ModelDesc), c_int32, c_int32, POINTER(c_size_t),
                                         POINTER(c_size_t)]),
        "sphinx_plan_step": (c_int32, [POINTER(Request), c_int32, P, P, c_int32, P, P, P, P, P, P, P]),
        "sphinx_plan_step_grid": (c_int32, [POINTER(Request), c_int32, P, P, c_int32, c_int32, P, P, P, P, P, P, P]),
        "sphinx_select_workspace_bytes": (c_int32, [c_int64, POINTER(c_size_t)]),
        "sphinx_select_mask": (c_int32, [POINTER(Request), c_int32, P, P, P, P, P, P, P, P, c_size_t, P]),
        "sphinx_select_mask_static": (c_int32, [POINTER(Request), c_int32, P, P, P, P, P, P, P, P]),
        "sphinx_varlen_attention": (c_int32, [c_int32, c_int32, c_int32, P, c_int32, P, P, c_int32, P, P, P, c_int32,
                                              P]),
        "sphinx_gather": (c_int32, [POINTER(Request), c_int32, c_int32, P, c_int32, P, c_int32, P, c_int32, P, P, P,
                                    P]),
        "sphinx_refine_workspace_bytes": (c_int32, [POINTER(ModelDesc), POINTER(Request), c_int32, c_int64,
                                                    POINTER(c_size_t)]),
        "sphinx_refine_step": (c_int32, [POINTER(ModelDesc), POINTER(Request), c_int32, P, c_int32, P, P, P, P,
                                         P, P, c_size_t, P]),
        "sphinx_scatter_blend": (c_int32, [POINTER(Request), c_int32, P, P, c_int32, P, c_int32, c_int32, P, c_int32,
                                           c_int32, P]),
        "sphinx_timing_enable": (c_int32, [c_int32]),
        "sphinx_timing_read": (c_int32, [c_int32, POINTER(c_int64), POINTER(ctypes.c_double)]),
        "sphinx_peak_mfma": (c_int32, [c_int32, c_int32, P, P]),
        "sphinx_plan_cache": (c_int32, [POINTER(Request), c_int32, P, P, c_int32, c_int32, c_int32, P, P, P, P]),
        "sphinx_kv_cache_bytes": (c_int32, [POINTER(ModelDesc), POINTER(Request), c_int32, POINTER(c_size_t)]),
        "sphinx_gather_ctx": (c_int32, [POINTER(Request), c_int32, c_int32, P, c_int32, P, c_int32, P, c_int32, P, P,
                                        P, P, P, P, P]),
        "sphinx_refine_step_cached": (c_int32, [POINTER(ModelDesc), POINTER(Request), c_int32, P, c_int32, P, P, P,
                                                P, P, P, P, c_size_t, P]),
        "sphinx_scatter_masked": (c_int32, [POINTER(Request), c_int32, P, P, c_int32, P, P, c_int32, c_int32, P]),
        "sphinx_mask_frontend_workspace_bytes": (c_int32, [POINTER(Request), c_int32, POINTER(c_size_t)]),
        "sphinx_adaptive_start": (c_int32, [POINTER(Request), c_int32, P, P, ctypes.c_float, POINTER(KLogic), c_int32,
                                            P, c_int32, P, P, P, P]),
        "sphinx_mask_frontend": (c_int32, [POINTER(Request), c_int32, P, P, ctypes.c_float, P, P, P, P, c_size_t,
                                           P]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def _check(fn: str, status: int):
    if status != 0:
        raise SphinxError(fn, status)


def _ptr(t) -> Optional[int]:
    """Device/host address of a torch tensor or numpy array (None passes NULL)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch

        return torch.cuda.current_stream().cuda_stream
    return stream if isinstance(stream, int) else stream.cuda_stream


def make_requests(shapes: Sequence) -> ctypes.Array:
    """C request table from objects with .frames/.h/.w (offsets are running sums)."""
    arr = (Request * len(shapes))()
    tok = fr = 0
    for i, q in enumerate(shapes):
        arr[i] = Request(q.frames, q.h, q.w, fr, tok)
        tok += q.frames * (q.h // 2) * (q.w // 2)
        fr += q.frames
    return arr


def dtype_code(name: str) -> int:
    return {"f32": F32, "bf16": BF16}[name]


def model_desc(cfg, weights_ptr: Optional[int] = None) -> ModelDesc:
    attn = ATTN_FACTORISED if getattr(cfg, "attention", "joint") == "factorised" else ATTN_JOINT
    return ModelDesc(cfg.D, cfg.heads, cfg.head_dim, cfg.mlp, cfg.L, dtype_code(cfg.dtype), attn, weights_ptr)


# ----------------------------------------------------------------------------
# entry points
# ----------------------------------------------------------------------------
def sphinx_status_string(status: int) -> str:
    return lib().sphinx_status_string(status).decode()


def sphinx_model_blob_bytes(desc: ModelDesc) -> int:
    out = c_size_t()
    _check("sphinx_model_blob_bytes", lib().sphinx_model_blob_bytes(ctypes.byref(desc), ctypes.byref(out)))
    return out.value


def sphinx_model_param(desc: ModelDesc, param: str, block: int = 0):
    off, cnt = c_size_t(), c_size_t()
    _check("sphinx_model_param", lib().sphinx_model_param(ctypes.byref(desc), PARAM_ID[param], block,
                                                          ctypes.byref(off), ctypes.byref(cnt)))
    return off.value, cnt.value


def sphinx_plan_step(reqs, s_start: np.ndarray, nsteps: np.ndarray, step: int, grid: int = GRID_SHARED
                     ) -> Dict[str, np.ndarray]:
    """Step schedule of all frames (sphinx_plan_step_grid; the shared grid is sphinx_plan_step)."""
    G = sum(r.frames for r in reqs)
    s_start = np.ascontiguousarray(s_start, dtype=np.int32)
    nsteps = np.ascontiguousarray(nsteps, dtype=np.int32)
    out = {"active": np.zeros(G, np.uint8), "newly": np.zeros(G, np.uint8), "tau": np.zeros(G, np.int32),
           "a": np.zeros(G, np.float32), "b": np.zeros(G, np.float32), "c1": np.zeros(G, np.float32),
           "c2": np.zeros(G, np.float32)}
    if grid == GRID_SHARED:
        _check("sphinx_plan_step", lib().sphinx_plan_step(
            reqs, len(reqs), _ptr(s_start), _ptr(nsteps), step, _ptr(out["active"]), _ptr(out["newly"]),
            _ptr(out["tau"]), _ptr(out["a"]), _ptr(out["b"]), _ptr(out["c1"]), _ptr(out["c2"])))
    else:
        _check("sphinx_plan_step_grid", lib().sphinx_plan_step_grid(
            reqs, len(reqs), _ptr(s_start), _ptr(nsteps), step, grid, _ptr(out["active"]), _ptr(out["newly"]),
            _ptr(out["tau"]), _ptr(out["a"]), _ptr(out["b"]), _ptr(out["c1"]), _ptr(out["c2"])))
    return out


def sphinx_plan_step_grid(reqs, s_start: np.ndarray, nsteps: np.ndarray, step: int, grid: int) -> Dict[str, np.ndarray]:
    return sphinx_plan_step(reqs, s_start, nsteps, step, grid)


def sphinx_select_workspace_bytes(N: int) -> int:
    out = c_size_t()
    _check("sphinx_select_workspace_bytes", lib().sphinx_select_workspace_bytes(N, ctypes.byref(out)))
    return out.value


def sphinx_select_mask(reqs, uncert, thr, active, mask, idx, cu_sel, ws, readback: bool = True, stream=None):
    """Mask + stable compaction.  With readback=True returns cu_sel as a host
    numpy array (the call then synchronizes the stream once)."""
    host = np.zeros(len(reqs) + 1, np.int32) if readback else None
    _check("sphinx_select_mask", lib().sphinx_select_mask(
        reqs, len(reqs), _ptr(uncert), _ptr(thr), _ptr(active), _ptr(mask), _ptr(idx), _ptr(cu_sel),
        _ptr(host), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))
    return host


def sphinx_select_mask_static(reqs, uncert, thr, active, mask, idx, cu_sel, readback: bool = True, stream=None):
    """sphinx_select_mask on the library's static scratch (no workspace, no
    device allocation).  With readback=True returns cu_sel on the host."""
    host = np.zeros(len(reqs) + 1, np.int32) if readback else None
    _check("sphinx_select_mask_static", lib().sphinx_select_mask_static(
        reqs, len(reqs), _ptr(uncert), _ptr(thr), _ptr(active), _ptr(mask), _ptr(idx), _ptr(cu_sel),
        _ptr(host), _stream(stream)))
    return host


def sphinx_varlen_attention(dtype: int, heads: int, head_dim: int, q, ldq: int, k, v, ldkv: int, o, cu_q, cu_kv,
                            stream=None):
    """Varlen attention (base-2 softmax; q already scaled by log2(e)/sqrt(d)).
    cu_q, cu_kv: host int sequences of segment bounds."""
    cq = np.ascontiguousarray(cu_q, dtype=np.int32)
    ck = np.ascontiguousarray(cu_kv, dtype=np.int32)
    assert cq.size == ck.size and cq.size >= 2
    _check("sphinx_varlen_attention", lib().sphinx_varlen_attention(
        dtype, heads, head_dim, _ptr(q), ldq, _ptr(k), _ptr(v), ldkv, _ptr(o), _ptr(cq), _ptr(ck), cq.size - 1,
        _stream(stream)))


def sphinx_gather(reqs, layout: int, state, state_dtype: int, eps, eps_dtype: int, idx, n_sel: int, a, b, x_sel,
                  stream=None):
    _check("sphinx_gather", lib().sphinx_gather(
        reqs, len(reqs), layout, _ptr(state), state_dtype, _ptr(eps), eps_dtype, _ptr(idx), n_sel, _ptr(a),
        _ptr(b), _ptr(x_sel), _stream(stream)))


def sphinx_refine_workspace_bytes(desc: ModelDesc, reqs, max_sel: int) -> int:
    out = c_size_t()
    _check("sphinx_refine_workspace_bytes", lib().sphinx_refine_workspace_bytes(
        ctypes.byref(desc), reqs, len(reqs), max_sel, ctypes.byref(out)))
    return out.value


def sphinx_refine_step(desc: ModelDesc, reqs, idx, n_sel: int, cu_sel_host: np.ndarray, tau, c1, c2, x_sel, ws,
                       stream=None):
    cu = np.ascontiguousarray(cu_sel_host, dtype=np.int32)
    _check("sphinx_refine_step", lib().sphinx_refine_step(
        ctypes.byref(desc), reqs, len(reqs), _ptr(idx), n_sel, _ptr(cu), _ptr(tau), _ptr(c1), _ptr(c2),
        _ptr(x_sel), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def sphinx_scatter_blend(reqs, x_sel, idx, n_sel: int, z_in, in_dtype: int, in_layout: int, z_out, out_dtype: int,
                         out_layout: int, stream=None):
    _check("sphinx_scatter_blend", lib().sphinx_scatter_blend(
        reqs, len(reqs), _ptr(x_sel), _ptr(idx), n_sel, _ptr(z_in), in_dtype, in_layout, _ptr(z_out), out_dtype,
        out_layout, _stream(stream)))


def sphinx_timing_enable(on=True, classes: Optional[Sequence[str]] = None):
    """Bracket the launches of the given kernel classes (all when None) with HIP
    events on their stream (profiling aid); on=False turns timing off."""
    if not on:
        mask = 0
    elif classes is None:
        mask = (1 << len(KERNEL_CLASSES)) - 1
    else:
        mask = 0
        for c in classes:
            mask |= 1 << KERNEL_CLASSES.index(c)
    _check("sphinx_timing_enable", lib().sphinx_timing_enable(mask))


def sphinx_timing_read() -> Dict[str, tuple]:
    """{kernel class: (launches, summed GPU ms)} since timing was last enabled."""
    out = {}
    for i, name in enumerate(KERNEL_CLASSES):
        n, ms = c_int64(), ctypes.c_double()
        _check("sphinx_timing_read", lib().sphinx_timing_read(i, ctypes.byref(n), ctypes.byref(ms)))
        out[name] = (n.value, ms.value)
    return out


def sphinx_peak_mfma(iters: int, out, operands: int = PEAK_CONSTANT, stream=None):
    """MFMA calibration loop (outside the method): SPHINX_PEAK_BLOCKS * 4 * iters * 4 * 32768 FLOP
    on constant (PEAK_CONSTANT) or random (PEAK_RANDOM) bf16 operands."""
    _check("sphinx_peak_mfma", lib().sphinx_peak_mfma(iters, operands, _ptr(out), _stream(stream)))


def sphinx_plan_cache(reqs, s_start: np.ndarray, nsteps: np.ndarray, step: int, period: int,
                      grid: int = GRID_SHARED) -> Dict[str, np.ndarray]:
    G = sum(r.frames for r in reqs)
    s_start = np.ascontiguousarray(s_start, dtype=np.int32)
    nsteps = np.ascontiguousarray(nsteps, dtype=np.int32)
    out = {"full": np.zeros(len(reqs), np.uint8), "forward_all": np.zeros(G, np.uint8),
           "a_ctx": np.zeros(G, np.float32), "b_ctx": np.zeros(G, np.float32)}
    _check("sphinx_plan_cache", lib().sphinx_plan_cache(
        reqs, len(reqs), _ptr(s_start), _ptr(nsteps), step, period, grid, _ptr(out["full"]), _ptr(out["forward_all"]),
        _ptr(out["a_ctx"]), _ptr(out["b_ctx"])))
    return out


def sphinx_kv_cache_bytes(desc: ModelDesc, reqs) -> int:
    out = c_size_t()
    _check("sphinx_kv_cache_bytes", lib().sphinx_kv_cache_bytes(ctypes.byref(desc), reqs, len(reqs),
                                                                ctypes.byref(out)))
    return out.value


def sphinx_gather_ctx(reqs, layout: int, state, state_dtype: int, eps, eps_dtype: int, idx, n: int, wmask, a, b,
                      a_ctx, b_ctx, x, stream=None):
    _check("sphinx_gather_ctx", lib().sphinx_gather_ctx(
        reqs, len(reqs), layout, _ptr(state), state_dtype, _ptr(eps), eps_dtype, _ptr(idx), n, _ptr(wmask), _ptr(a),
        _ptr(b), _ptr(a_ctx), _ptr(b_ctx), _ptr(x), _stream(stream)))


def sphinx_refine_step_cached(desc: ModelDesc, reqs, idx, n: int, cu_host: np.ndarray, tau, c1, c2, x, kv_cache, ws,
                              stream=None):
    cu = np.ascontiguousarray(cu_host, dtype=np.int32)
    _check("sphinx_refine_step_cached", lib().sphinx_refine_step_cached(
        ctypes.byref(desc), reqs, len(reqs), _ptr(idx), n, _ptr(cu), _ptr(tau), _ptr(c1), _ptr(c2), _ptr(x),
        _ptr(kv_cache), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def sphinx_scatter_masked(reqs, x, idx, n: int, wmask, z, dtype: int, layout: int, stream=None):
    _check("sphinx_scatter_masked", lib().sphinx_scatter_masked(
        reqs, len(reqs), _ptr(x), _ptr(idx), n, _ptr(wmask), _ptr(z), dtype, layout, _stream(stream)))


def sphinx_mask_frontend_workspace_bytes(reqs) -> int:
    out = c_size_t()
    _check("sphinx_mask_frontend_workspace_bytes", lib().sphinx_mask_frontend_workspace_bytes(
        reqs, len(reqs), ctypes.byref(out)))
    return out.value


def sphinx_mask_frontend(reqs, rgb, opacity, tau_o: float, token_mask, uncert, otsu_t, ws, stream=None):
    _check("sphinx_mask_frontend", lib().sphinx_mask_frontend(
        reqs, len(reqs), _ptr(rgb), _ptr(opacity), tau_o, _ptr(token_mask), _ptr(uncert), _ptr(otsu_t), _ptr(ws),
        ws.numel() * ws.element_size(), _stream(stream)))


def sphinx_adaptive_start(reqs, q_in: np.ndarray, q_reg: np.ndarray, gamma: float, tables: Sequence[KLogic],
                          cluster: np.ndarray, S: int = 50) -> Dict[str, np.ndarray]:
    """Per-frame start steps k and start indices, per-request step counts, ratios."""
    G = sum(r.frames for r in reqs)
    q_in = np.ascontiguousarray(q_in, dtype=np.float32).ravel()
    q_reg = np.ascontiguousarray(q_reg, dtype=np.float32)
    cluster = np.ascontiguousarray(cluster, dtype=np.int32)
    arr = (KLogic * len(tables))(*tables)
    out = {"k": np.zeros(G, np.int32), "s_start": np.zeros(G, np.int32), "nsteps": np.zeros(len(reqs), np.int32),
           "ratio": np.zeros(G, np.float64)}
    _check("sphinx_adaptive_start", lib().sphinx_adaptive_start(
        reqs, len(reqs), _ptr(q_in), _ptr(q_reg), gamma, arr, len(tables), _ptr(cluster), S, _ptr(out["k"]),
        _ptr(out["s_start"]), _ptr(out["nsteps"]), _ptr(out["ratio"])))
    return out


select_mask = sphinx_select_mask
gather = sphinx_gather
refine_step = sphinx_refine_step
scatter_blend = sphinx_scatter_blend
plan_step = sphinx_plan_step
