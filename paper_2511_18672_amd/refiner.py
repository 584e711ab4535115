"""Driver of the partial-denoising loop on one GPU (Alg. 1 loop with per-frame
start steps and the selective mask of Sec. 5.3).

``Refiner`` owns the device buffers of one batch of packed requests and runs,
for each step: ``sphinx_select_mask`` (whenever the set of active frames
changes, or every step when asked), ``sphinx_gather``, ``sphinx_refine_step``
and ``sphinx_scatter_blend``.  Python only sequences the calls; every value is
computed by libsphinx.so.  The per-step schedule comes from
``sphinx_plan_step`` (library host code) and is uploaded once.

With ``cache_period`` T > 0 the latent cache of Sec. 5.2 is on: every T-th
step is a full step that forwards every token of the live requests (a second
``sphinx_select_mask`` with threshold -inf over the frames of full requests),
and every step runs ``sphinx_gather_ctx``, ``sphinx_refine_step_cached`` and
``sphinx_scatter_masked`` so that only the write set (the mask) is updated.

The fp32 state of record and the noise live token-major by default (token t's
16 values contiguous at 16*t), so each gathered or scattered token is one
contiguous row; the NCHW latents are converted once at ``reset`` and back in
``output``.  ``layout=B.NCHW`` keeps them NCHW throughout (same arithmetic).
"""
from __future__ import annotations

from typing import Dict, Optional, Sequence

import numpy as np
import torch

from . import binding as B


def _torch_dtype(name: str):
    return torch.bfloat16 if name == "bf16" else torch.float32


def pack_weights(cfg, weights: Dict[str, np.ndarray], device="cuda") -> torch.Tensor:
    """Place named parameters into the library's blob layout and upload it.

    ``weights`` uses the names ``pe_w, pe_b, t1_w, t1_b, t2_w, t2_b,
    b{l}.{ada_w, ada_b, qkv_w, qkv_b, o_w, o_b, fc1_w, fc1_b, fc2_w, fc2_b},
    fada_w, fada_b, out_w, out_b`` with matrices [out][in]."""
    desc = B.model_desc(cfg)
    tdt = _torch_dtype(cfg.dtype)
    esz = 2 if cfg.dtype == "bf16" else 4
    blob = torch.zeros(B.sphinx_model_blob_bytes(desc) // esz, dtype=tdt)

    def put(param: str, block: int, arr: np.ndarray, elem0: int = 0):
        off, cnt = B.sphinx_model_param(desc, param, block)
        flat = torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32).ravel()).to(tdt)
        assert elem0 + flat.numel() <= cnt, (param, block)
        start = off // esz + elem0
        blob[start:start + flat.numel()] = flat

    D, L = cfg.D, cfg.L
    for p in ("pe_w", "pe_b", "t1_w", "t1_b", "t2_w", "t2_b", "out_w", "out_b"):
        put(p.upper(), 0, weights[p])
    for l in range(L):
        put("COND_W", 0, weights[f"b{l}.ada_w"], 6 * D * l * D)
        put("COND_B", 0, weights[f"b{l}.ada_b"], 6 * D * l)
        for p in ("qkv_w", "qkv_b", "o_w", "o_b", "fc1_w", "fc1_b", "fc2_w", "fc2_b"):
            put(p.upper(), l, weights[f"b{l}.{p}"])
    put("COND_W", 0, weights["fada_w"], 6 * D * L * D)
    put("COND_B", 0, weights["fada_b"], 6 * D * L)
    return blob.to(device)


class Refiner:
    """Selective partial denoising of one batch of packed requests on one GPU."""

    def __init__(self, requests: Sequence, cfg, blob: torch.Tensor, s_start: np.ndarray, nsteps: np.ndarray,
                 u: np.ndarray, thr: np.ndarray, z0: np.ndarray, eps: np.ndarray, device="cuda",
                 max_sel: Optional[int] = None, layout: int = B.TOKENS, cache_period: int = 0,
                 per_frame_grid: bool = False):
        if not torch.cuda.is_available():
            raise RuntimeError("Refiner needs a GPU: the selective-refinement step has no CPU path")
        B.lib()
        self.shapes = list(requests)
        self.reqs = B.make_requests(self.shapes)
        self.cfg = cfg
        self.blob = blob
        self.desc = B.model_desc(cfg, blob.data_ptr())
        self.N = sum(r.frames * (r.h // 2) * (r.w // 2) for r in self.shapes)
        self.G = sum(r.frames for r in self.shapes)
        self.R = len(self.shapes)
        self.dt = B.dtype_code(cfg.dtype)
        tdt = _torch_dtype(cfg.dtype)
        dev = torch.device(device)
        self.layout = int(layout)
        self.z0 = torch.from_numpy(np.ascontiguousarray(z0, np.float32)).to(tdt).to(dev)
        eps_nchw = torch.from_numpy(np.ascontiguousarray(eps, np.float32)).to(tdt).to(dev)
        if self.layout == B.NCHW:
            self.eps = eps_nchw
        else:  # noise in the state's layout, converted once
            self.eps = torch.empty_like(eps_nchw)
            B.sphinx_scatter_blend(self.reqs, None, None, 0, eps_nchw, self.dt, B.NCHW, self.eps, self.dt,
                                   self.layout)
        self.u = torch.from_numpy(np.ascontiguousarray(u, np.float32)).to(dev)
        self.thr = torch.from_numpy(np.ascontiguousarray(thr, np.float32)).to(dev)
        self.z = torch.empty(16 * self.N, dtype=torch.float32, device=dev)  # state of record, in self.layout
        # two selection slots: the selection of the next step is computed (and its
        # cu_sel copied to pinned host memory) while the current step runs
        self._mask = [torch.empty(self.N, dtype=torch.uint8, device=dev) for _ in range(2)]
        self._idx = [torch.empty(self.N, dtype=torch.int32, device=dev) for _ in range(2)]
        self._cu = [torch.empty(self.R + 1, dtype=torch.int32, device=dev) for _ in range(2)]
        self._cu_pinned = [torch.empty(self.R + 1, dtype=torch.int32, pin_memory=True) for _ in range(2)]
        self._cu_ready = [torch.cuda.Event() for _ in range(2)]
        self._slot_key = [None, None]  # active-frame flags each slot was selected for
        self.mask, self.idx, self.cu_sel = self._mask[0], self._idx[0], self._cu[0]
        self.max_sel = self.N if max_sel is None else int(max_sel)
        self.x_sel = torch.empty(16 * self.max_sel, dtype=torch.float32, device=dev)
        self.ws_sel = torch.empty(B.sphinx_select_workspace_bytes(self.N), dtype=torch.uint8, device=dev)
        self.ws = torch.empty(B.sphinx_refine_workspace_bytes(self.desc, self.reqs, self.max_sel),
                              dtype=torch.uint8, device=dev)
        self.total_steps = int(np.max(nsteps))
        self.grid = B.GRID_PER_FRAME if per_frame_grid else B.GRID_SHARED
        plans = [B.sphinx_plan_step(self.reqs, s_start, nsteps, i, self.grid) for i in range(self.total_steps)]
        self.plan_host = {k: np.stack([p[k] for p in plans]) for k in plans[0]}
        self.plan = {k: torch.from_numpy(v).to(dev) for k, v in self.plan_host.items()}
        self._pending = None  # (step index, slot) of a selection already enqueued
        self.n_sel = 0
        self.n_fwd = 0
        self.cu_fwd = None
        self.cu_host = None
        self.cache_period = int(cache_period)
        self.kv_cache = None
        if self.cache_period > 0:
            if self.max_sel != self.N:
                raise ValueError("the latent cache forwards every token on full steps: max_sel must be N")
            self.kv_cache = torch.zeros(B.sphinx_kv_cache_bytes(self.desc, self.reqs), dtype=torch.uint8, device=dev)
            cplans = [B.sphinx_plan_cache(self.reqs, s_start, nsteps, i, self.cache_period, self.grid)
                      for i in range(self.total_steps)]
            self.cache_host = {k: np.stack([p[k] for p in cplans]) for k in cplans[0]}
            self.cache_plan = {k: torch.from_numpy(v).to(dev) for k, v in self.cache_host.items()}
            self.thr_all = torch.full((self.G,), -float("inf"), dtype=torch.float32, device=dev)
            self._fmask = torch.empty(self.N, dtype=torch.uint8, device=dev)
            self._fidx = torch.empty(self.N, dtype=torch.int32, device=dev)
            self._fcu = torch.empty(self.R + 1, dtype=torch.int32, device=dev)

    def reset(self, stream=None):
        """state <- fp32(z0) (a converting copy through scatter_blend with no tokens)."""
        B.sphinx_scatter_blend(self.reqs, None, None, 0, self.z0, self.dt, B.NCHW, self.z, B.F32, self.layout,
                               stream)
        self._pending = None
        self._slot_key = [None, None]

    def load_state(self, state_nchw, stream=None):
        """state <- the given fp32 NCHW latents of all requests (host array or
        tensor), converted into the state's layout by the library."""
        src = torch.as_tensor(np.ascontiguousarray(state_nchw, dtype=np.float32)
                              if not isinstance(state_nchw, torch.Tensor) else state_nchw)
        src = src.to(device=self.z.device, dtype=torch.float32).contiguous()
        if src.numel() != self.z.numel():
            raise ValueError(f"state has {src.numel()} values, expected {self.z.numel()}")
        B.sphinx_scatter_blend(self.reqs, None, None, 0, src, B.F32, B.NCHW, self.z, B.F32, self.layout, stream)
        self._pending = None
        self._slot_key = [None, None]

    def _enqueue_select(self, k: int, slot: int, stream=None):
        """Selection of schedule step k into `slot`; cu_sel reaches pinned host
        memory asynchronously (no host synchronization)."""
        B.sphinx_select_mask(self.reqs, self.u, self.thr, self.plan["active"][k], self._mask[slot], self._idx[slot],
                             self._cu[slot], self.ws_sel, False, stream)
        s = torch.cuda.current_stream() if stream is None else stream
        with torch.cuda.stream(s):
            self._cu_pinned[slot].copy_(self._cu[slot], non_blocking=True)
            self._cu_ready[slot].record(s)
        self._slot_key[slot] = self.plan_host["active"][k].copy()

    def select(self, k: int, stream=None) -> int:
        """Selection of schedule step k, waited for (it becomes the current one)."""
        slot = 0 if self._pending is None else 1 - self._pending[1]
        self._enqueue_select(k, slot, stream)
        return self._use_slot(slot)

    def _use_slot(self, slot: int) -> int:
        self._cu_ready[slot].synchronize()
        self.cu_host = self._cu_pinned[slot].numpy().copy()
        self.n_sel = int(self.cu_host[-1])
        if self.n_sel > self.max_sel:
            raise RuntimeError(f"{self.n_sel} selected tokens exceed the buffers sized for {self.max_sel}")
        self.mask, self.idx, self.cu_sel = self._mask[slot], self._idx[slot], self._cu[slot]
        self._cur_slot = slot
        return self.n_sel

    def step(self, i: int, force_select: bool = False, stream=None) -> int:
        """One partial-denoising step (schedule index i modulo the schedule length).

        The selection (mask and compaction) runs whenever the set of active
        frames changes, or every step with force_select.  The selection of step
        i+1 is enqueued before this step's work, so its cu_sel read-back never
        stalls the stream."""
        k = i % self.total_steps
        if self._pending is not None and self._pending[0] == i:
            slot = self._pending[1]
        else:
            slot = 0 if self._pending is None else 1 - self._pending[1]
            self._enqueue_select(k, slot, stream)
        # selection of the next step: a fresh one when asked or when the active
        # frames change, otherwise the current one is reused
        k1 = (i + 1) % self.total_steps
        if force_select or not np.array_equal(self.plan_host["active"][k1], self._slot_key[slot]):
            self._enqueue_select(k1, 1 - slot, stream)
            self._pending = (i + 1, 1 - slot)
        else:
            self._pending = (i + 1, slot)
        n = self._use_slot(slot)
        if self.kv_cache is not None:
            return self._step_cached(k, n, stream)
        if n == 0:
            return 0
        P = self.plan
        B.sphinx_gather(self.reqs, self.layout, self.z, B.F32, self.eps, self.dt, self.idx, n, P["a"][k],
                        P["b"][k], self.x_sel, stream)
        B.sphinx_refine_step(self.desc, self.reqs, self.idx, n, self.cu_host, P["tau"][k], P["c1"][k],
                             P["c2"][k], self.x_sel, self.ws, stream)
        B.sphinx_scatter_blend(self.reqs, self.x_sel, self.idx, n, self.z, B.F32, self.layout, self.z, B.F32,
                               self.layout, stream)
        return n

    def _step_cached(self, k: int, n: int, stream=None) -> int:
        """Step k with the latent cache; the write-set selection is current."""
        P, C = self.plan, self.cache_plan
        if self.cache_host["full"][k].any():
            cu_f = B.sphinx_select_mask(self.reqs, self.u, self.thr_all, C["forward_all"][k], self._fmask,
                                        self._fidx, self._fcu, self.ws_sel, True, stream)
            idx_f, n_f = self._fidx, int(cu_f[-1])
        else:
            cu_f, idx_f, n_f = self.cu_host, self.idx, n
        self.n_fwd = n_f
        self.cu_fwd = np.asarray(cu_f).copy()
        if n_f == 0:
            return 0
        B.sphinx_gather_ctx(self.reqs, self.layout, self.z, B.F32, self.eps, self.dt, idx_f, n_f, self.mask,
                            P["a"][k], P["b"][k], C["a_ctx"][k], C["b_ctx"][k], self.x_sel, stream)
        B.sphinx_refine_step_cached(self.desc, self.reqs, idx_f, n_f, cu_f, P["tau"][k], P["c1"][k], P["c2"][k],
                                    self.x_sel, self.kv_cache, self.ws, stream)
        B.sphinx_scatter_masked(self.reqs, self.x_sel, idx_f, n_f, self.mask, self.z, B.F32, self.layout, stream)
        return n

    def run(self, stream=None) -> torch.Tensor:
        """The whole schedule from z0; returns the fp32 state (NCHW of all requests)."""
        self.reset(stream)
        for i in range(self.total_steps):
            self.step(i, stream=stream)
        return self.state

    def output(self, dtype: str = "bf16", stream=None) -> torch.Tensor:
        """The state as NCHW latents of the given dtype (bf16 rounds to nearest even)."""
        out = torch.empty(16 * self.N, dtype=_torch_dtype(dtype), device=self.z.device)
        B.sphinx_scatter_blend(self.reqs, None, None, 0, self.z, B.F32, self.layout, out, B.dtype_code(dtype),
                               B.NCHW, stream)
        return out

    @property
    def state(self) -> torch.Tensor:
        """A fp32 NCHW copy of the state of record (a new tensor on every access)."""
        return self.output("f32")


def from_workload(wl, device="cuda", **kw) -> Refiner:
    """Refiner for a ``workloads.Workload`` (seeded inputs and weights)."""
    blob = pack_weights(wl.model, wl.weights, device)
    return Refiner(wl.requests, wl.model, blob, wl.s_start, wl.nsteps, wl.u, wl.thr, wl.z0, wl.eps, device, **kw)
