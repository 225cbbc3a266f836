"""Device-memory plumbing around libfe.so: torch tensors hold weights, caches,
inputs, outputs and the workspace; every step of the pass runs in the
library's HIP kernels through the C ABI (paper_2509_20416_amd.fe)."""
from __future__ import annotations

import ctypes as C
import dataclasses
from typing import Dict, List, Optional

import numpy as np

from . import fe


def _torch():
    import torch
    return torch


def to_device(a: np.ndarray, dtype: str, device):
    """Host array (bf16 bit patterns as uint16, or float32/int32) -> device tensor."""
    torch = _torch()
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(a).to(device)


@dataclasses.dataclass
class DeviceInputs:
    batch: int
    features: object
    next_tokens: object
    prefix_lens: object
    cu_prefix: object
    kcache: List[object]
    vcache: List[object]
    max_prefix: int


class Drafter:
    """One drafter (weights + workspace + library handle) on one GPU."""

    def __init__(self, cfg, weights, device="cuda:0", max_batch: Optional[int] = None,
                 max_prefix: Optional[int] = None, max_topk: Optional[int] = None,
                 graph: bool = False):
        torch = _torch()
        self.cfg = cfg
        self.device = torch.device(device)
        dev = self.device
        dt = cfg.dtype
        # host arrays are copied in; device tensors (already in the storage
        # dtype) are used as they are
        up = lambda a: a.to(dev) if isinstance(a, torch.Tensor) else to_device(a, dt, dev)
        self.w = {n: up(getattr(weights, n)) for n in ("w_fuse", "w_in", "embed", "final_norm",
                                                       "lm_head")}
        self.w["d2t"] = to_device(np.asarray(weights.d2t, dtype=np.int32), "i32", dev)
        self.layers = [{f: up(getattr(lw, f)) for f in lw.FIELDS} for lw in weights.layers]
        self._cl = (fe.fe_layer_weights * cfg.n_layers)()
        for i, lw in enumerate(self.layers):
            for f in lw:
                setattr(self._cl[i], f, lw[f].data_ptr())
        self._cw = fe.fe_weights(self.w["w_fuse"].data_ptr(), self.w["w_in"].data_ptr(),
                                 self.w["embed"].data_ptr(), self.w["final_norm"].data_ptr(),
                                 self.w["lm_head"].data_ptr(), self.w["d2t"].data_ptr(),
                                 C.cast(self._cl, C.POINTER(fe.fe_layer_weights)))
        lo_hi = cfg.prefix if isinstance(cfg.prefix, tuple) else (cfg.prefix, cfg.prefix)
        self.ccfg = fe.fe_config(
            cfg.hidden, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.intermediate,
            cfg.n_layers, cfg.draft_vocab, cfg.target_vocab, cfg.n_feat_levels,
            max_batch or cfg.batch, max_topk or max(cfg.topk, 1),
            int(max_prefix if max_prefix is not None else lo_hi[1]),
            float(cfg.rope_theta), float(cfg.rms_eps),
            fe.FE_BF16 if dt == "bf16" else fe.FE_F32,
            {"cascade": fe.FE_CTX_CASCADE, "self": fe.FE_CTX_SELF,
             "parallel": fe.FE_CTX_PARALLEL}[cfg.cascade_ctx])
        self.ws_bytes = fe.fe_workspace_bytes(self.ccfg)
        if self.ws_bytes == 0:
            raise fe.FeError(fe.FE_E_UNSUPPORTED, fe.fe_last_error())
        self.workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=dev)
        self.handle = fe.fe_drafter_create(self.ccfg, self._cw, self.workspace.data_ptr(),
                                           self.ws_bytes, self.stream())
        if graph:
            fe.fe_set_graph_mode(self.handle, True)

    def stream(self) -> int:
        return _torch().cuda.current_stream(self.device).cuda_stream

    def set_graph_mode(self, on: bool) -> None:
        fe.fe_set_graph_mode(self.handle, on)

    def set_attention_split(self, chunks_per_workgroup: int) -> None:
        """64-key prefix chunks per attention work unit; 0 = automatic."""
        fe.fe_set_attention_split(self.handle, chunks_per_workgroup)

    def set_pass_mode(self, mode: int) -> None:
        """0: persistent launches for batch-1 passes when the shape allows; 1: one launch per stage."""
        fe.fe_set_pass_mode(self.handle, mode)

    def pass_status(self) -> int:
        """Waits for the stream; bit 0: a persistent pass gave up waiting (outputs
        unspecified), bit 16: the last pass ran as persistent launches."""
        return fe.fe_pass_status(self.handle, self.stream())

    def upload_inputs(self, inp, max_prefix: Optional[int] = None) -> DeviceInputs:
        torch = _torch()
        dev, dt = self.device, self.cfg.dtype
        plens = np.asarray(inp.prefix_lens, dtype=np.int32)
        return DeviceInputs(
            batch=len(plens), features=to_device(inp.features, dt, dev),
            next_tokens=to_device(np.asarray(inp.next_tokens, np.int32), "i32", dev),
            prefix_lens=to_device(plens, "i32", dev),
            cu_prefix=to_device(inp.cu_prefix, "i32", dev),
            kcache=[to_device(k, dt, dev) for k in inp.kcache],
            vcache=[to_device(v, dt, dev) for v in inp.vcache],
            max_prefix=int(plens.max()) if max_prefix is None and len(plens) else int(max_prefix or 0))

    def kv_view(self, di: DeviceInputs) -> fe.fe_kv_view:
        N = self.cfg.n_layers
        self._kp = (C.c_void_p * N)(*[k.data_ptr() for k in di.kcache])
        self._vp = (C.c_void_p * N)(*[v.data_ptr() for v in di.vcache])
        return fe.fe_kv_view(C.cast(self._kp, C.POINTER(C.c_void_p)),
                             C.cast(self._vp, C.POINTER(C.c_void_p)),
                             di.cu_prefix.data_ptr(), di.max_prefix)

    def alloc_outputs(self, batch: int, topk: int, logits=False, hidden=False,
                      draft=True) -> Dict[str, object]:
        torch = _torch()
        N, d, V, dev = self.cfg.n_layers, self.cfg.hidden, self.cfg.draft_vocab, self.device
        o = dict(topk_ids=torch.empty((batch, N, topk), dtype=torch.int32, device=dev),
                 topk_probs=torch.empty((batch, N, topk), dtype=torch.float32, device=dev))
        if draft:
            o["topk_draft"] = torch.empty((batch, N, topk), dtype=torch.int32, device=dev)
        if logits:
            o["logits"] = torch.empty((batch, N, V), dtype=torch.float32, device=dev)
        if hidden:
            o["hidden"] = torch.empty((batch, N + 1, d), dtype=torch.float32, device=dev)
        return o

    def forward(self, di: DeviceInputs, topk: Optional[int] = None, logits=False, hidden=False,
                out: Optional[Dict[str, object]] = None,
                tree: Optional[Dict[str, object]] = None, temperature: Optional[float] = None,
                uniforms=None, seed_offset=None) -> Dict[str, object]:
        """One drafting pass; with `tree` (from alloc_tree) the Backbone Expansion
        tree of the pass is built in the same launch sequence.  With a
        temperature and/or `uniforms` ([B, N, V] float32 on the device) the pass
        runs through fe_draft_sample (candidates sampled without replacement);
        with `seed_offset` (a device int64/uint64 tensor [2]: seed, offset) through
        fe_draft_sample_seeded, the uniforms drawn in the pass."""
        k = int(topk or self.cfg.topk)
        if out is None:
            out = self.alloc_outputs(di.batch, k, logits, hidden)
        p = lambda n: out[n].data_ptr() if n in out else None
        self._out = fe.fe_draft_out(p("topk_ids"), p("topk_probs"), p("topk_draft"),
                                    p("logits"), p("hidden"))
        if tree is not None:
            self._fwd_tree = fe.fe_tree_out(*[tree[n].data_ptr() for n in
                                              ("tokens", "parents", "depth", "positions", "mask",
                                               "retrieve")])
            self._out.tree = fe.C.pointer(self._fwd_tree)
        if seed_offset is not None:
            fe.fe_draft_sample_seeded(self.handle, di.batch, di.features.data_ptr(),
                                      di.next_tokens.data_ptr(), self.kv_view(di), k,
                                      float(1.0 if temperature is None else temperature),
                                      seed_offset.data_ptr(), self._out, self.stream())
        elif temperature is None and uniforms is None:
            fe.fe_draft_forward(self.handle, di.batch, di.features.data_ptr(),
                                di.next_tokens.data_ptr(), self.kv_view(di), k, self._out,
                                self.stream())
        else:
            fe.fe_draft_sample(self.handle, di.batch, di.features.data_ptr(),
                               di.next_tokens.data_ptr(), self.kv_view(di), k,
                               float(1.0 if temperature is None else temperature),
                               uniforms.data_ptr() if uniforms is not None else None, self._out,
                               self.stream())
        return out

    def alloc_tree(self, batch: int, topk: int) -> Dict[str, object]:
        torch = _torch()
        N, dev = self.cfg.n_layers, self.device
        T, NL = 1 + N * topk, N * (topk - 1) + 1
        i32 = dict(dtype=torch.int32, device=dev)
        return dict(tokens=torch.empty((batch, T), **i32), parents=torch.empty((batch, T), **i32),
                    depth=torch.empty((batch, T), **i32), positions=torch.empty((batch, T), **i32),
                    mask=torch.empty((batch, T, T), dtype=torch.uint8, device=dev),
                    retrieve=torch.empty((batch, NL, N + 1), **i32))

    def build_tree(self, di: DeviceInputs, topk_ids, topk: Optional[int] = None,
                   out: Optional[Dict[str, object]] = None) -> Dict[str, object]:
        k = int(topk or self.cfg.topk)
        if out is None:
            out = self.alloc_tree(di.batch, k)
        self._tout = fe.fe_tree_out(*[out[n].data_ptr() for n in
                                      ("tokens", "parents", "depth", "positions", "mask",
                                       "retrieve")])
        fe.fe_build_tree(self.handle, di.batch, k, di.next_tokens.data_ptr(),
                         topk_ids.data_ptr(), di.prefix_lens.data_ptr(), self._tout,
                         self.stream())
        return out

    def accept_greedy(self, tree: Dict[str, object], target_next, topk: Optional[int] = None,
                      batch: Optional[int] = None,
                      out: Optional[Dict[str, object]] = None) -> Dict[str, object]:
        """Greedy acceptance of one cycle (fe_accept_greedy): tree as returned by
        build_tree, target_next [B, T] int32 on the device."""
        import torch
        k = int(topk or self.cfg.topk)
        B = int(batch if batch is not None else tree["tokens"].shape[0])
        N = self.cfg.n_layers
        dev = tree["tokens"].device
        if out is None:
            out = {"accept_len": torch.empty(B, dtype=torch.int32, device=dev),
                   "accept_path": torch.empty(B, dtype=torch.int32, device=dev),
                   "accepted": torch.empty(B, N + 1, dtype=torch.int32, device=dev)}
        fe.fe_accept_greedy(self.handle, B, k, tree["tokens"].data_ptr(),
                            tree["retrieve"].data_ptr(), target_next.data_ptr(),
                            out["accept_len"].data_ptr(), out["accept_path"].data_ptr(),
                            out["accepted"].data_ptr(), self.stream())
        return out

    def accept_sample(self, tree: Dict[str, object], topk_draft, draft_logits, target_probs,
                      uniforms, temperature: float = 1.0, draft_uniforms=None,
                      topk: Optional[int] = None, batch: Optional[int] = None,
                      out: Optional[Dict[str, object]] = None,
                      draft_seed_offset=None) -> Dict[str, object]:
        """Speculative-sampling acceptance of one cycle (fe_accept_sample, or
        fe_accept_sample_seeded with `draft_seed_offset`, the device (seed,
        offset) pair the pass drew with); all arrays on the device (see
        include/fe.h for shapes)."""
        import torch
        k = int(topk or self.cfg.topk)
        B = int(batch if batch is not None else tree["tokens"].shape[0])
        N = self.cfg.n_layers
        dev = tree["tokens"].device
        if out is None:
            out = {"accept_len": torch.empty(B, dtype=torch.int32, device=dev),
                   "accept_path": torch.empty(B, dtype=torch.int32, device=dev),
                   "accepted": torch.empty(B, N + 1, dtype=torch.int32, device=dev)}
        if draft_seed_offset is not None:
            fe.fe_accept_sample_seeded(self.handle, B, k, tree["tokens"].data_ptr(),
                                       tree["retrieve"].data_ptr(), topk_draft.data_ptr(),
                                       draft_logits.data_ptr(), float(temperature),
                                       draft_seed_offset.data_ptr(), target_probs.data_ptr(),
                                       uniforms.data_ptr(), out["accept_len"].data_ptr(),
                                       out["accept_path"].data_ptr(), out["accepted"].data_ptr(),
                                       self.stream())
            return out
        fe.fe_accept_sample(self.handle, B, k, tree["tokens"].data_ptr(),
                            tree["retrieve"].data_ptr(), topk_draft.data_ptr(),
                            draft_logits.data_ptr(), float(temperature),
                            draft_uniforms.data_ptr() if draft_uniforms is not None else None,
                            target_probs.data_ptr(), uniforms.data_ptr(),
                            out["accept_len"].data_ptr(), out["accept_path"].data_ptr(),
                            out["accepted"].data_ptr(), self.stream())
        return out

    def kv_update(self, features, tokens, positions, dst_rows, kcache, vcache,
                  chunk_rows: int = 1024, n_rows: Optional[int] = None) -> None:
        """Write the drafter cache rows of verified positions (fe_kv_update):
        features [M, 3d], tokens / positions / dst_rows [M] int32 and the
        per-layer caches kcache / vcache ([rows, H_kv, D]), all on the device.
        The workspace for `chunk_rows`-row chunks is allocated once and kept."""
        torch = _torch()
        N = self.cfg.n_layers
        M = int(n_rows if n_rows is not None else tokens.shape[0])
        need = fe.fe_kv_update_workspace_bytes(self.ccfg, int(chunk_rows))
        if need == 0:
            raise fe.FeError(fe.FE_E_INVALID, fe.fe_last_error())
        if getattr(self, "_upd_ws", None) is None or self._upd_ws.numel() < need:
            self._upd_ws = torch.empty(need, dtype=torch.uint8, device=self.device)
        self._ukp = (C.c_void_p * N)(*[k.data_ptr() for k in kcache])
        self._uvp = (C.c_void_p * N)(*[v.data_ptr() for v in vcache])
        rows = int(kcache[0].shape[0])
        cache = fe.fe_kv_cache(C.cast(self._ukp, C.POINTER(C.c_void_p)),
                               C.cast(self._uvp, C.POINTER(C.c_void_p)), rows)
        fe.fe_kv_update(self.handle, M, features.data_ptr(), tokens.data_ptr(),
                        positions.data_ptr(), dst_rows.data_ptr(), cache,
                        self._upd_ws.data_ptr(), need, self.stream())

    def close(self) -> None:
        if getattr(self, "handle", None):
            fe.fe_drafter_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
