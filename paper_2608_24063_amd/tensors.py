"""PyTorch-side marshalling for libviscache: allocates the outputs and the
workspace that the C ABI asks for and passes device addresses and the current
stream.  No computation happens here."""
from __future__ import annotations

import torch

from . import (VC_PRUNE_EVENTS, VC_RANK_GLOBAL, make_params, make_prune_io, make_shape, prune_with_io, vc_cache,
               vc_decode_shape, vc_qcache, viscache_append_kv, viscache_budget, viscache_decode_attn,
               viscache_decode_plan, viscache_decode_step, viscache_decode_step_noalloc,
               viscache_decode_step_planned, viscache_decode_step_q4,
               viscache_decode_step_workspace_bytes,
               viscache_decode_workspace_bytes, viscache_out_rows, viscache_prune_workspace_bytes,
               viscache_quantize_rows)


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _addr(t: torch.Tensor | None) -> int:
    return 0 if t is None or t.numel() == 0 else t.data_ptr()


class PruneCall:
    """One PruneKV problem: shape, parameters, per-layer outputs, workspace.

    k_in / v_in: per-layer bf16 tensors [sum_b Hkv*n_b, d]; q_win: per-layer
    fp32 tensors [B, Hq, W, d] (window scores) or [sum_b Hq*(n_b+W), d]
    (prefill scores); k_text: per-layer bf16 [B, Hkv, W, d] (prefill scores
    only).  `run()` enqueues viscache_prune on the current stream."""

    def __init__(self, B, L, Hq, Hkv, d, W, n_vis, params, k_in, v_in, q_win, with_drop=False, k_text=None):
        self.B, self.L, self.Hq, self.Hkv, self.d, self.W = B, L, Hq, Hkv, d, W
        self.n_vis = [int(x) for x in n_vis]
        self.params = params
        self.shape = make_shape(B, L, Hq, Hkv, d, W, self.n_vis)
        self.k, self.n_surv, self.h = viscache_budget(self.shape, params)
        self.rows = viscache_out_rows(self.shape, params)
        dev = k_in[0].device
        vdt = torch.float32 if params.v_out_fp32 else torch.bfloat16
        self.k_in, self.v_in, self.q_win = list(k_in), list(v_in), list(q_win)
        self.k_text = list(k_text) if k_text is not None else None
        self.k_out, self.v_out, self.idx_out, self.drop_out = [], [], [], []
        for l in range(L):
            nrow = self.rows[l * (B + 1) + B]
            self.k_out.append(torch.empty((nrow, d), dtype=torch.bfloat16, device=dev))
            self.v_out.append(torch.empty((nrow, d), dtype=vdt, device=dev))
            self.idx_out.append(torch.empty((nrow,), dtype=torch.int32, device=dev))
            if with_drop:
                ndrop = sum(Hkv * (self.n_surv[b * L + l] - self.k[b * L + l]) for b in range(B)) if l < self.h else 0
                self.drop_out.append(torch.empty((ndrop,), dtype=torch.int32, device=dev))
        self.ws_bytes = viscache_prune_workspace_bytes(self.shape, params)
        self.ws = torch.empty((self.ws_bytes,), dtype=torch.uint8, device=dev)
        self._io = None

    @property
    def global_rank(self) -> bool:
        return self.params.rank_mode == VC_RANK_GLOBAL

    def _prune_io(self):
        """The call's vc_prune_io, built once (the buffers never move)."""
        if self._io is None:
            a = lambda ts: [_addr(t) for t in ts]
            self._io = make_prune_io(a(self.k_in), a(self.v_in), a(self.q_win), a(self.k_out), a(self.v_out),
                                     a(self.idx_out), a(self.drop_out) if self.drop_out else None,
                                     a(self.k_text) if self.k_text is not None else None)
        return self._io

    def run(self, events=None) -> None:
        """Enqueue viscache_prune on the current stream; with `events`
        (VC_PRUNE_EVENTS torch.cuda.Event objects created with
        enable_timing=True, or raw hipEvent_t handles as ints) the stages are
        bracketed (viscache_prune_staged)."""
        handles = None
        if events is not None:
            assert len(events) == VC_PRUNE_EVENTS
            handles = []
            for e in events:
                if isinstance(e, int):
                    handles.append(e)
                    continue
                if e.cuda_event == 0:
                    e.record()  # materialise the handle
                handles.append(e.cuda_event)
        prune_with_io(self.shape, self.params, self._prune_io(), self.ws.data_ptr(), self.ws_bytes, _stream(),
                      handles)

    def unit_rows(self, l: int, b: int, g: int):
        """Row range of (layer, sequence, kv head) in layer l's outputs."""
        k = self.k[b * self.L + l]
        r0 = self.rows[l * (self.B + 1) + b] + g * k
        return r0, r0 + k

    def unit_drop_rows(self, l: int, b: int, g: int):
        r = self.n_surv[b * self.L + l] - self.k[b * self.L + l]
        base = sum(self.Hkv * (self.n_surv[bb * self.L + l] - self.k[bb * self.L + l]) for bb in range(b))
        return base + g * r, base + (g + 1) * r


class DecodeCache:
    """A decode cache pool over L layers x B sequences x Hkv heads.  Unit
    u = (l*B + b)*Hkv + g owns `cap[u]` rows starting at row_off[u]."""

    def __init__(self, L, B, Hq, Hkv, d, caps, device):
        self.shape = vc_decode_shape(B, L, Hq, Hkv, d)
        self.L, self.B, self.Hq, self.Hkv, self.d = L, B, Hq, Hkv, d
        caps = [int(c) for c in caps]
        offs, o = [], 0
        for c in caps:
            offs.append(o)
            o += c
        self.total_rows = o
        self.max_cap = max(caps) if caps else 0
        self.k_pool = torch.zeros((max(o, 1), d), dtype=torch.bfloat16, device=device)
        self.v_pool = torch.zeros((max(o, 1), d), dtype=torch.bfloat16, device=device)
        self.row_off = torch.tensor(offs, dtype=torch.int64, device=device)
        self.cap = torch.tensor(caps, dtype=torch.int32, device=device)
        self.len = torch.zeros(len(caps), dtype=torch.int32, device=device)
        self.offs_host, self.caps_host = offs, caps
        self.ws_bytes = viscache_decode_workspace_bytes(self.shape, self.max_cap)
        self.ws = torch.empty((max(self.ws_bytes, 256),), dtype=torch.uint8, device=device)
        # The fused step keeps arrival counters in its workspace: zero-filled once.
        self.step_ws_bytes = viscache_decode_step_workspace_bytes(self.shape, self.max_cap)
        self.step_ws = torch.zeros((max(self.step_ws_bytes, 256),), dtype=torch.uint8, device=device)
        self.c = vc_cache(self.k_pool.data_ptr(), self.v_pool.data_ptr(), self.row_off.data_ptr(),
                          self.cap.data_ptr(), self.len.data_ptr())

    def append(self, k_new: torch.Tensor, v_new: torch.Tensor) -> None:
        viscache_append_kv(self.shape, self.c, k_new.data_ptr(), v_new.data_ptr(), _stream())

    def attend(self, q: torch.Tensor, out: torch.Tensor, scale: float) -> None:
        viscache_decode_attn(self.shape, self.c, q.data_ptr(), out.data_ptr(), scale, self.max_cap,
                             self.ws.data_ptr(), self.ws_bytes, _stream())

    def step(self, k_new: torch.Tensor, v_new: torch.Tensor, q: torch.Tensor, out: torch.Tensor,
             scale: float) -> None:
        """append + attend in one launch (viscache_decode_step)."""
        viscache_decode_step(self.shape, self.c, k_new.data_ptr(), v_new.data_ptr(), q.data_ptr(),
                             out.data_ptr(), scale, self.max_cap, self.step_ws.data_ptr(), self.step_ws_bytes,
                             _stream())

    def step_noalloc(self, k_new: torch.Tensor, v_new: torch.Tensor, q: torch.Tensor, out: torch.Tensor,
                     scale: float) -> None:
        """step() through viscache_decode_step_noalloc: no workspace, the
        library's own scratch."""
        viscache_decode_step_noalloc(self.shape, self.c, k_new.data_ptr(), v_new.data_ptr(), q.data_ptr(),
                                     out.data_ptr(), scale, self.max_cap, _stream())

    def step_layers(self, k_new: torch.Tensor, v_new: torch.Tensor, q: torch.Tensor, out: torch.Tensor,
                    scale: float) -> None:
        """The same decode step as L launches, one per layer (the loop of a
        model that attends layer by layer): viscache_decode_step on each
        layer's units, with the layer's slices of the pool tables, inputs and
        outputs.  The launches are ordered on one stream, so they share one
        step workspace."""
        if not hasattr(self, "_layer_caches"):
            per = self.B * self.Hkv
            self.layer_shape = vc_decode_shape(self.B, 1, self.Hq, self.Hkv, self.d)
            self._layer_caches = [
                vc_cache(self.k_pool.data_ptr(), self.v_pool.data_ptr(), self.row_off[l * per:].data_ptr(),
                         self.cap[l * per:].data_ptr(), self.len[l * per:].data_ptr()) for l in range(self.L)]
            self.layer_caps = [max(self.caps_host[l * per:(l + 1) * per]) for l in range(self.L)]
            nb = max(viscache_decode_step_workspace_bytes(self.layer_shape, c) for c in self.layer_caps)
            self.layer_ws_bytes = max(nb, 256)
            self.layer_ws = torch.zeros((self.layer_ws_bytes,), dtype=torch.uint8, device=self.k_pool.device)
        for l in range(self.L):
            viscache_decode_step(self.layer_shape, self._layer_caches[l], k_new[l].data_ptr(), v_new[l].data_ptr(),
                                 q[l].data_ptr(), out[l].data_ptr(), scale, self.layer_caps[l],
                                 self.layer_ws.data_ptr(), self.layer_ws_bytes, _stream())

    def quantize(self, nq) -> None:
        """Quantise every pool row to 4 bits (viscache_quantize_rows) and let
        unit u read its first nq[u] rows (rounded down to the 32-row tile)
        from the codes in later q4 steps; the rows stay in the bf16 pools."""
        dev = self.k_pool.device
        rows, d = self.k_pool.shape
        self.qk = torch.empty((rows, d // 2), dtype=torch.uint8, device=dev)
        self.qv = torch.empty((rows, d // 2), dtype=torch.uint8, device=dev)
        self.qkm = torch.empty((rows, d // 32, 2), dtype=torch.float32, device=dev)
        self.qvm = torch.empty((rows, d // 32, 2), dtype=torch.float32, device=dev)
        viscache_quantize_rows(d, rows, self.k_pool.data_ptr(), self.qk.data_ptr(), self.qkm.data_ptr(), _stream())
        viscache_quantize_rows(d, rows, self.v_pool.data_ptr(), self.qv.data_ptr(), self.qvm.data_ptr(), _stream())
        self.nq = torch.as_tensor([int(x) for x in nq], dtype=torch.int32).to(dev)
        self.qc = vc_qcache(self.qk.data_ptr(), self.qkm.data_ptr(), self.qv.data_ptr(), self.qvm.data_ptr(),
                            self.row_off.data_ptr(), self.nq.data_ptr())

    def plan(self, max_rows=None, hint=True) -> None:
        """Builds the piece table of this cache on the host
        (viscache_decode_plan) and keeps a device copy for step_planned.  The
        length hint: the current lengths (hint True), none (False), or the
        given sequence."""
        self.plan_rows = self.max_cap if max_rows is None else int(max_rows)
        if hint is True:
            lens = self.len.cpu().tolist()
        elif hint is False or hint is None:
            lens = None
        else:
            lens = [int(x) for x in hint]
        blob = viscache_decode_plan(self.shape, self.caps_host, self.offs_host, self.plan_rows, lens)
        host = torch.frombuffer(bytearray(blob), dtype=torch.uint8)
        self.plan_dev = host.to(self.k_pool.device)
        self.plan_bytes = len(blob)

    def step_planned(self, k_new: torch.Tensor, v_new: torch.Tensor, q: torch.Tensor, out: torch.Tensor,
                     scale: float, q4: bool = False, max_rows=None) -> None:
        """step() (or step_q4() with q4) over the piece table of plan()
        (viscache_decode_step_planned)."""
        rows = self.plan_rows if max_rows is None else int(max_rows)
        viscache_decode_step_planned(self.shape, self.c, self.qc if q4 else None, self.plan_dev.data_ptr(),
                                     self.plan_bytes, k_new.data_ptr(), v_new.data_ptr(), q.data_ptr(),
                                     out.data_ptr(), scale, rows, self.step_ws.data_ptr(), self.step_ws_bytes,
                                     _stream())

    def step_q4(self, k_new: torch.Tensor, v_new: torch.Tensor, q: torch.Tensor, out: torch.Tensor,
                scale: float) -> None:
        """step() with each unit's quantised rows read from the 4-bit codes
        (viscache_decode_step_q4); quantize() first."""
        viscache_decode_step_q4(self.shape, self.c, self.qc, k_new.data_ptr(), v_new.data_ptr(), q.data_ptr(),
                                out.data_ptr(), scale, self.max_cap, self.step_ws.data_ptr(), self.step_ws_bytes,
                                _stream())


__all__ = ["PruneCall", "DecodeCache", "make_params"]
