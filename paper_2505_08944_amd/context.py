"""Python surface of libaep: torch tensors in, raw pointers to the C ABI.

torch provides device memory (the workspace, outputs) and the current HIP
stream; every computation happens in libaep's kernels.  The context keeps a
reference to every tensor the library borrows (fragment rows until their
layer is drained, expert weights while registered).
"""

from __future__ import annotations

import ctypes
from typing import Dict, List, Optional, Tuple

import numpy as np
import torch

from . import _lib as L

_ACT = {"f32": (L.AEP_F32, torch.float32), "bf16": (L.AEP_BF16, torch.bfloat16)}
_WDT = {"f32": L.AEP_F32, "bf16": L.AEP_BF16, "fp8": L.AEP_FP8_E4M3}
_POLICY = {"mtfs": L.AEP_POLICY_MTFS, "flfs": L.AEP_POLICY_FLFS, "defrag": L.AEP_POLICY_DEFRAG}


def _stream() -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _need(t: torch.Tensor, name: str, dtype=None, shape=None) -> None:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a CUDA (HIP) tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype not in (dtype if isinstance(dtype, tuple) else (dtype,)):
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")


class BatchView:
    """A drained layer (host handle + device views into the workspace)."""

    def __init__(self, ctx: "Context", b: L.Batch):
        self.ctx, self.c = ctx, b

    layer = property(lambda self: self.c.layer)
    n_tokens = property(lambda self: self.c.n_tokens)
    n_routed = property(lambda self: self.c.n_routed)
    n_rows = property(lambda self: self.c.n_rows)

    def _view(self, ptr: int, dtype: torch.dtype, shape: Tuple[int, ...]) -> torch.Tensor:
        ws = self.ctx.workspace
        if ws is None:
            raise RuntimeError("batch views need a torch-allocated workspace (this context uses the static one)")
        off = ptr - ws.data_ptr()
        n = int(np.prod(shape)) if shape else 1
        nbytes = n * torch.empty((), dtype=dtype).element_size()
        assert 0 <= off and off + nbytes <= ws.numel()
        return ws[off:off + nbytes].view(dtype).view(shape)

    def counts(self) -> torch.Tensor:
        return self._view(self.c.counts, torch.int32, (self.ctx.G,))

    def offsets(self) -> torch.Tensor:
        return self._view(self.c.offsets, torch.int32, (self.ctx.G + 1,))

    def x_perm(self) -> torch.Tensor:
        rows = self.n_routed + (self.n_tokens if self.ctx.n_shared else 0)
        return self._view(self.c.x_perm, self.ctx.act_torch, (rows, self.ctx.d_model))

    def row_token(self) -> torch.Tensor:
        return self._view(self.c.row_token, torch.int32, (self.n_routed,))

    def row_weight(self) -> torch.Tensor:
        return self._view(self.c.row_weight, torch.float32, (self.n_routed,))

    def token_pos(self) -> torch.Tensor:
        return self._view(self.c.token_pos, torch.int32, (self.n_tokens, self.ctx.top_k))

    def token_weight(self) -> torch.Tensor:
        return self._view(self.c.token_weight, torch.float32, (self.n_tokens, self.ctx.top_k))


class Context:
    """One libaep context: the mu-queues of n_layers MoE layers on one GPU."""

    def __init__(self, n_layers: int, n_experts: int, d_model: int, d_ffn: int, top_k: int, *,
                 n_shared: int = 0, renorm: bool = True, act: str = "bf16", wdt: str = "bf16",
                 max_tokens_per_layer: int, token_pool: bool = False, device: Optional[torch.device] = None,
                 static_workspace: bool = False):
        self.lib = L.lib()
        self.n_layers, self.n_experts, self.n_shared = n_layers, n_experts, n_shared
        self.d_model, self.d_ffn, self.top_k = d_model, d_ffn, top_k
        self.G = n_experts + n_shared
        self.act, self.wdt = act, wdt
        act_code, self.act_torch = _ACT[act]
        cfg = L.Config(n_layers, n_experts, n_shared, d_model, d_ffn, top_k, int(bool(renorm)), act_code,
                       _WDT[wdt], max_tokens_per_layer, int(bool(token_pool)))
        self.max_tokens = max_tokens_per_layer
        h = ctypes.c_void_p()
        L.check(self.lib.aep_create(ctypes.byref(cfg), ctypes.byref(h)), "aep_create")
        self.h = h
        nbytes = ctypes.c_size_t()
        L.check(self.lib.aep_workspace_size(self.h, ctypes.byref(nbytes)), "aep_workspace_size")
        dev = device or torch.device("cuda", torch.cuda.current_device())
        self.device = dev
        if static_workspace:
            # the library's own workspace: nothing is allocated here (batch
            # internals then have no tensor views; outputs are caller tensors)
            self._raw = self.workspace = None
            with torch.cuda.device(dev):
                L.check(self.lib.aep_bind_static_workspace(self.h, _stream()), "aep_bind_static_workspace")
        else:
            # 256-byte alignment: over-allocate and slice
            raw = torch.empty(nbytes.value + 256, dtype=torch.uint8, device=dev)
            pad = (-raw.data_ptr()) % 256
            self._raw = raw
            self.workspace = raw[pad:pad + nbytes.value]
            L.check(self.lib.aep_bind_workspace(self.h, self.workspace.data_ptr(), nbytes.value, _stream()),
                    "aep_bind_workspace")
        self.workspace_need = nbytes.value
        self._frag_refs: Dict[int, List[torch.Tensor]] = {l: [] for l in range(n_layers)}
        self._w_refs: Dict[Tuple[int, int], Tuple[torch.Tensor, ...]] = {}

    def __del__(self):
        h = getattr(self, "h", None)
        if h is not None and h.value:
            self.lib.aep_destroy(h)
            self.h = ctypes.c_void_p()

    @property
    def workspace_bytes(self) -> int:
        return self.workspace_need

    # ------------------------------------------------------------- weights
    def set_expert_weights(self, layer: int, expert: int, gate: torch.Tensor, up: torch.Tensor,
                           down: torch.Tensor, scale_gate_up: Optional[torch.Tensor] = None,
                           scale_down: Optional[torch.Tensor] = None) -> None:
        f, d = self.d_ffn, self.d_model
        wt = {"f32": torch.float32, "bf16": torch.bfloat16, "fp8": (torch.uint8, torch.float8_e4m3fn)}[self.wdt]
        _need(gate, "gate", wt, (f, d))
        _need(up, "up", wt, (f, d))
        _need(down, "down", wt, (d, f))
        if self.wdt == "fp8":
            _need(scale_gate_up, "scale_gate_up", (torch.bfloat16, torch.int16, torch.uint16), (2 * f,))
            _need(scale_down, "scale_down", (torch.bfloat16, torch.int16, torch.uint16), (d,))
        L.check(self.lib.aep_set_expert_weights(self.h, layer, expert, gate.data_ptr(), up.data_ptr(),
                                                down.data_ptr(), _ptr(scale_gate_up), _ptr(scale_down),
                                                _stream()), "aep_set_expert_weights")
        self._w_refs[(layer, expert)] = (gate, up, down, scale_gate_up, scale_down)

    # ------------------------------------------------------------- receptor
    def route_enqueue(self, layer: int, x: torch.Tensor, logits: torch.Tensor,
                      routing_out: bool = False) -> Optional[Tuple[torch.Tensor, torch.Tensor]]:
        T = x.shape[0]
        _need(x, "x", self.act_torch, (T, self.d_model))
        _need(logits, "logits", torch.float32, (T, self.n_experts))
        idx = w = None
        if routing_out:
            idx = torch.empty((T, self.top_k), dtype=torch.int32, device=x.device)
            w = torch.empty((T, self.top_k), dtype=torch.float32, device=x.device)
        L.check(self.lib.aep_route_enqueue(self.h, layer, x.data_ptr(), logits.data_ptr(), T, _ptr(idx),
                                           _ptr(w), _stream()), "aep_route_enqueue")
        if T:
            self._frag_refs[layer].append(x)
            self._frag_refs[layer].append(logits)
        return (idx, w) if routing_out else None

    def route_enqueue_ids(self, layer: int, x: torch.Tensor, logits: torch.Tensor, token_ids: torch.Tensor,
                          routing_out: bool = False) -> Optional[Tuple[torch.Tensor, torch.Tensor]]:
        """Route a fragment whose tokens carry caller ids (token-pool mode)."""
        T = x.shape[0]
        _need(x, "x", self.act_torch, (T, self.d_model))
        _need(logits, "logits", torch.float32, (T, self.n_experts))
        _need(token_ids, "token_ids", torch.int32, (T,))
        idx = w = None
        if routing_out:
            idx = torch.empty((T, self.top_k), dtype=torch.int32, device=x.device)
            w = torch.empty((T, self.top_k), dtype=torch.float32, device=x.device)
        L.check(self.lib.aep_route_enqueue_ids(self.h, layer, x.data_ptr(), logits.data_ptr(), T,
                                               token_ids.data_ptr(), _ptr(idx), _ptr(w), _stream()),
                "aep_route_enqueue_ids")
        if T:
            self._frag_refs[layer].extend([x, logits, token_ids])
        return (idx, w) if routing_out else None

    def enqueue_rows(self, layer: int, expert: int, rows: torch.Tensor, token_ids: torch.Tensor,
                     gate_w: torch.Tensor, n_tokens: int, slots: Optional[torch.Tensor] = None) -> None:
        n = rows.shape[0]
        _need(rows, "rows", self.act_torch, (n, self.d_model))
        _need(token_ids, "token_ids", torch.int32, (n,))
        _need(gate_w, "gate_w", torch.float32, (n,))
        if slots is not None:
            _need(slots, "slots", torch.int32, (n,))
        L.check(self.lib.aep_enqueue_rows(self.h, layer, expert, rows.data_ptr(), token_ids.data_ptr(),
                                          _ptr(slots), gate_w.data_ptr(), n, n_tokens, _stream()),
                "aep_enqueue_rows")
        if n:
            self._frag_refs[layer].extend([rows, token_ids, gate_w] + ([slots] if slots is not None else []))

    def enqueue_rows_grouped(self, layer: int, counts, rows: torch.Tensor, token_ids: torch.Tensor,
                             gate_w: torch.Tensor, n_tokens: int, slots: Optional[torch.Tensor] = None) -> None:
        """Rows of several experts in one call: rows grouped by expert in
        ascending order, counts[e] of them for expert e (host sequence)."""
        h = np.ascontiguousarray(np.asarray(counts, dtype=np.int32))
        if h.shape != (self.n_experts,):
            raise ValueError(f"counts: expected {self.n_experts} entries, got {h.shape}")
        n = rows.shape[0]
        _need(rows, "rows", self.act_torch, (n, self.d_model))
        _need(token_ids, "token_ids", torch.int32, (n,))
        _need(gate_w, "gate_w", torch.float32, (n,))
        if slots is not None:
            _need(slots, "slots", torch.int32, (n,))
        if int(h.sum()) != n:
            raise ValueError(f"counts sum to {int(h.sum())}, rows has {n}")
        L.check(self.lib.aep_enqueue_rows_grouped(self.h, layer, h.ctypes.data, rows.data_ptr(),
                                                  token_ids.data_ptr(), _ptr(slots), gate_w.data_ptr(), n_tokens,
                                                  _stream()), "aep_enqueue_rows_grouped")
        if n:
            self._frag_refs[layer].extend([rows, token_ids, gate_w] + ([slots] if slots is not None else []))

    def queue_depth(self, layer: int) -> Tuple[int, int]:
        t, r = ctypes.c_int64(), ctypes.c_int64()
        L.check(self.lib.aep_queue_depth(self.h, layer, ctypes.byref(t), ctypes.byref(r)), "aep_queue_depth")
        return t.value, r.value

    def expert_counts(self, layer: int) -> np.ndarray:
        out = np.zeros(self.n_experts, dtype=np.int32)
        L.check(self.lib.aep_expert_counts(self.h, layer, out.ctypes.data, _stream()), "aep_expert_counts")
        return out

    # ------------------------------------------------------------- scheduler
    def pick_layer(self, policy: str = "mtfs", delta: float = 0.5, lookahead: int = 2) -> Optional[int]:
        b = ctypes.c_int32(-1)
        st = self.lib.aep_pick_layer(self.h, _POLICY[policy], float(delta), int(lookahead), ctypes.byref(b))
        if st == L.AEP_ERR_EMPTY:
            return None
        L.check(st, "aep_pick_layer")
        return b.value

    # ------------------------------------------------------------- executor
    def rebatch(self, layer: int) -> BatchView:
        b = L.Batch()
        L.check(self.lib.aep_rebatch(self.h, layer, ctypes.byref(b), _stream()), "aep_rebatch")
        bv = BatchView(self, b)
        bv._frags = self._frag_refs[layer]   # rows stay referenced until the batch is released
        self._frag_refs[layer] = []
        return bv

    def rebatch_expert(self, layer: int, expert: int) -> BatchView:
        """Drain one expert's queue of a token-pool layer."""
        b = L.Batch()
        L.check(self.lib.aep_rebatch_expert(self.h, layer, expert, ctypes.byref(b), _stream()),
                "aep_rebatch_expert")
        bv = BatchView(self, b)
        if self.queue_depth(layer)[1] == 0:   # the last queued row of these fragments is in this batch
            bv._frags = self._frag_refs[layer]
            self._frag_refs[layer] = []
        return bv

    def pool_accumulate(self, batch: BatchView, y: torch.Tensor) -> None:
        _need(y, "y", self.act_torch, (batch.n_rows, self.d_model))
        L.check(self.lib.aep_pool_accumulate(self.h, ctypes.byref(batch.c), y.data_ptr(), _stream()),
                "aep_pool_accumulate")

    def pool_release(self, layer: int, out: torch.Tensor, ready: Optional[torch.Tensor] = None) -> None:
        """Write every completed token of the layer's pool to out[id]; ready[id] = 1 for those."""
        _need(out, "out", self.act_torch, (self.max_tokens, self.d_model))
        if ready is not None:
            _need(ready, "ready", torch.int32, (self.max_tokens,))
        L.check(self.lib.aep_pool_release(self.h, layer, out.data_ptr(), _ptr(ready), _stream()),
                "aep_pool_release")

    def expert_ffn(self, batch: BatchView, y: Optional[torch.Tensor] = None) -> torch.Tensor:
        if y is None:
            y = torch.empty((batch.n_rows, self.d_model), dtype=self.act_torch, device=self.device)
        _need(y, "y", self.act_torch, (batch.n_rows, self.d_model))
        L.check(self.lib.aep_expert_ffn(self.h, ctypes.byref(batch.c), y.data_ptr(), _stream()), "aep_expert_ffn")
        return y

    def expert_gate_up(self, batch: BatchView) -> None:
        L.check(self.lib.aep_expert_gate_up(self.h, ctypes.byref(batch.c), _stream()), "aep_expert_gate_up")

    def expert_down(self, batch: BatchView, y: Optional[torch.Tensor] = None) -> torch.Tensor:
        if y is None:
            y = torch.empty((batch.n_rows, self.d_model), dtype=self.act_torch, device=self.device)
        _need(y, "y", self.act_torch, (batch.n_rows, self.d_model))
        L.check(self.lib.aep_expert_down(self.h, ctypes.byref(batch.c), y.data_ptr(), _stream()), "aep_expert_down")
        return y

    def combine(self, batch: BatchView, y: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
        _need(y, "y", self.act_torch, (batch.n_rows, self.d_model))
        if out is None:
            out = torch.empty((batch.n_tokens, self.d_model), dtype=self.act_torch, device=y.device)
        _need(out, "out", self.act_torch, (batch.n_tokens, self.d_model))
        L.check(self.lib.aep_combine(self.h, ctypes.byref(batch.c), y.data_ptr(), out.data_ptr(), _stream()),
                "aep_combine")
        return out

    def release(self, batch: BatchView) -> None:
        L.check(self.lib.aep_release_batch(self.h, ctypes.byref(batch.c)), "aep_release_batch")

    def sync(self) -> None:
        L.check(self.lib.aep_sync(self.h, _stream()), "aep_sync")

    def set_clock_probe(self, buf: Optional[torch.Tensor]) -> None:
        """Record per-workgroup (shader-clock cycles, 100 MHz ticks) of later
        FFN launches into buf (device int64 [n, 2]); None turns it off."""
        if buf is None:
            L.check(self.lib.aep_set_clock_probe(self.h, None, 0), "aep_set_clock_probe")
            return
        if buf.device.type != "cuda" or buf.dtype != torch.int64 or buf.dim() != 2 or buf.shape[1] != 2 \
                or not buf.is_contiguous():
            raise ValueError("clock probe buffer: contiguous device int64 [n, 2]")
        self._clock_buf = buf
        L.check(self.lib.aep_set_clock_probe(self.h, buf.data_ptr(), buf.shape[0]), "aep_set_clock_probe")

    def run_layer(self, layer: int, y: Optional[torch.Tensor] = None,
                  out: Optional[torch.Tensor] = None) -> torch.Tensor:
        """Drain one layer: re-batch, expert FFN, combine; returns out [n_tokens, d]."""
        b = self.rebatch(layer)
        try:
            y = self.expert_ffn(b, y if y is not None and y.shape[0] == b.n_rows else None)
            return self.combine(b, y, out if out is not None and out.shape[0] == b.n_tokens else None)
        finally:
            self.release(b)


def fp8_e4m3_to_bf16(codes: torch.Tensor) -> torch.Tensor:
    """Exact OCP e4m3fn -> bf16 decode on the GPU."""
    _need(codes, "codes", (torch.uint8, torch.float8_e4m3fn))
    out = torch.empty(codes.shape, dtype=torch.bfloat16, device=codes.device)
    L.check(L.lib().aep_fp8_e4m3_to_bf16(codes.data_ptr(), out.data_ptr(), codes.numel(), _stream()),
            "aep_fp8_e4m3_to_bf16")
    return out
