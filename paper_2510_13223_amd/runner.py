"""One decode-attention step of a workload on the GPU: every partition, then the merge.

Marshalling and orchestration only: uploads a ``workloads.Workload`` to
device tensors once, pre-builds the ctypes argument lists, and issues the
library calls (``bana_decode_attn_partial`` once per partition, then
``bana_merge_partials``; or the single ``bana_decode_attn_fused``) on one
stream.  No arithmetic happens here.
"""

from __future__ import annotations

import ctypes
from typing import List, Optional

import numpy as np
import torch

from . import bana


def _bf16(a: np.ndarray, device) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(device)


def _i32(a: np.ndarray, device) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(device)


class DeviceWorkload:
    """Device-resident inputs and outputs of one workload, plus prepared call arguments."""

    def __init__(self, w, device="cuda", waves_hint: int = 0, chunks_hint: int = 0, use_workspace: bool = True,
                 range_hints: bool = True, order_hints: bool = True, plan_hint: int = 0):
        self.w = w
        self.device = torch.device(device)
        self.q = _bf16(w.q, self.device)
        self.k_cache = _bf16(w.k_cache, self.device)
        self.v_cache = _bf16(w.v_cache, self.device)
        self.block_table = _i32(w.block_table, self.device)
        self.seq_lens = _i32(w.seq_lens, self.device)
        self.kv_begin = _i32(w.kv_begin, self.device)  # [P, B]; row p is contiguous
        self.kv_end = _i32(w.kv_end, self.device)
        P, B, Hq = w.n_parts, w.batch, w.num_q_heads
        self.out_partials = torch.empty((P, B, Hq, bana.HEAD_DIM), dtype=torch.float32, device=self.device)
        self.lses = torch.empty((P, B, Hq), dtype=torch.float32, device=self.device)
        self.out = torch.empty((B, Hq, bana.HEAD_DIM), dtype=torch.float32, device=self.device)
        self.lse_out = torch.empty((B, Hq), dtype=torch.float32, device=self.device)

        # Dispatch order hints: sequences with the longest range first (stable), so short ones fill
        # the end of each launch.  Results do not depend on the order.
        def order(lens):
            if not order_hints:
                return None
            return torch.from_numpy(np.argsort(-lens, kind="stable").astype(np.int32)).to(self.device)

        self.dims: List[bana.bana_dims] = []
        self._orders = []
        for p in range(P):
            lens = w.kv_end[p].astype(np.int64) - w.kv_begin[p]
            self._orders.append(order(lens))
            self.dims.append(bana.make_dims(B, Hq, w.num_kv_heads, w.max_blocks_per_seq, w.num_blocks,
                                            max_range_tokens=int(lens.max()) if range_hints else 0,
                                            waves_hint=waves_hint, chunks_hint=chunks_hint,
                                            total_range_tokens=int(lens.sum()) if range_hints else 0,
                                            seq_order=self._orders[-1], plan_hint=plan_hint,
                                            nonempty_ranges=int(np.count_nonzero(lens)) if range_hints else 0))
        # The fused call sees each sequence's ranges as one concatenated range.
        lens_all = (w.kv_end.astype(np.int64) - w.kv_begin).sum(axis=0)
        self._orders.append(order(lens_all))
        self.fused_dims = bana.make_dims(B, Hq, w.num_kv_heads, w.max_blocks_per_seq, w.num_blocks,
                                         max_range_tokens=int(lens_all.max()) if range_hints else 0,
                                         waves_hint=waves_hint, chunks_hint=chunks_hint,
                                         total_range_tokens=int(lens_all.sum()) if range_hints else 0,
                                         seq_order=self._orders[-1], plan_hint=plan_hint,
                                         nonempty_ranges=int(np.count_nonzero(lens_all)) if range_hints else 0)
        self.fused_out = torch.empty((B, Hq, bana.HEAD_DIM), dtype=torch.float32, device=self.device)
        self.fused_lse = torch.empty((B, Hq), dtype=torch.float32, device=self.device)
        ws = max(bana.bana_decode_attn_workspace_bytes(d) for d in self.dims + [self.fused_dims]) if use_workspace else 0
        self.workspace: Optional[torch.Tensor] = (
            torch.empty(max(ws, 256), dtype=torch.uint8, device=self.device) if ws > 0 else None)
        # Validate every argument once through the checked binding (this also runs the step once), and
        # wait for it: calls on other streams must not overlap it, since they share the workspace.
        self.run_checked()
        torch.cuda.synchronize(self.device)
        self._prepare_fast_args()

    def run_checked(self, stream=None) -> None:
        for p in range(self.w.n_parts):
            bana.bana_decode_attn_partial(self.q, self.k_cache, self.v_cache, self.block_table, self.seq_lens,
                                          self.kv_begin[p], self.kv_end[p], self.out_partials[p], self.lses[p],
                                          workspace=self.workspace, stream=stream, dims=self.dims[p])
        bana.bana_merge_partials(self.out_partials, self.lses, self.out, self.lse_out, stream=stream)
        bana.bana_decode_attn_fused(self.q, self.k_cache, self.v_cache, self.block_table, self.seq_lens,
                                    self.kv_begin, self.kv_end, self.fused_out, self.fused_lse,
                                    workspace=self.workspace, stream=stream, dims=self.fused_dims)

    def _prepare_fast_args(self) -> None:
        vp = lambda t: ctypes.c_void_p(t.data_ptr())
        ws_ptr = vp(self.workspace) if self.workspace is not None else None
        ws_bytes = self.workspace.numel() if self.workspace is not None else 0
        self._partial_args = []
        for p in range(self.w.n_parts):
            self._partial_args.append([
                ctypes.byref(self.dims[p]), vp(self.q), vp(self.k_cache), vp(self.v_cache), vp(self.block_table),
                vp(self.seq_lens), vp(self.kv_begin[p]), vp(self.kv_end[p]), vp(self.out_partials[p]),
                vp(self.lses[p]), ws_ptr, ws_bytes])
        B, Hq = self.w.batch, self.w.num_q_heads
        self._merge_dims = bana.bana_dims(B, Hq, 1, bana.HEAD_DIM, bana.BLOCK_SIZE, 1, 1, 0, 0, 0, 0, 0, None, 0)
        self._merge_args = [ctypes.byref(self._merge_dims), vp(self.out_partials), vp(self.lses), self.w.n_parts,
                            vp(self.out), vp(self.lse_out)]
        self._fused_args = [ctypes.byref(self.fused_dims), vp(self.q), vp(self.k_cache), vp(self.v_cache),
                            vp(self.block_table), vp(self.seq_lens), vp(self.kv_begin), vp(self.kv_end),
                            self.w.n_parts, vp(self.fused_out), vp(self.fused_lse), ws_ptr, ws_bytes]

    def partial(self, p: int, stream_handle: ctypes.c_void_p) -> None:
        st = bana.lib().bana_decode_attn_partial(*self._partial_args[p], stream_handle)
        if st != bana.BANA_OK:
            raise bana.BanaError(st, "bana_decode_attn_partial")

    def merge(self, stream_handle: ctypes.c_void_p) -> None:
        st = bana.lib().bana_merge_partials(*self._merge_args, stream_handle)
        if st != bana.BANA_OK:
            raise bana.BanaError(st, "bana_merge_partials")

    def fused(self, stream_handle: ctypes.c_void_p) -> None:
        """All partitions and their merge in one call (into fused_out / fused_lse)."""
        st = bana.lib().bana_decode_attn_fused(*self._fused_args, stream_handle)
        if st != bana.BANA_OK:
            raise bana.BanaError(st, "bana_decode_attn_fused")

    def step(self, stream: Optional[torch.cuda.Stream] = None) -> None:
        """All partitions, then the merge, on ``stream`` (default: torch's current stream)."""
        self.step_on(ctypes.c_void_p((stream or torch.cuda.current_stream()).cuda_stream))

    def step_on(self, stream_handle: ctypes.c_void_p) -> None:
        """All partitions, then the merge, on a raw HIP stream handle."""
        for p in range(self.w.n_parts):
            self.partial(p, stream_handle)
        self.merge(stream_handle)

    def results(self):
        """(out_partials, lses, out, lse_out) as host float32 arrays."""
        torch.cuda.synchronize(self.device)
        return (self.out_partials.cpu().numpy(), self.lses.cpu().numpy(), self.out.cpu().numpy(),
                self.lse_out.cpu().numpy())

    def fused_results(self):
        """(out, lse_out) of the fused call as host float32 arrays."""
        torch.cuda.synchronize(self.device)
        return self.fused_out.cpu().numpy(), self.fused_lse.cpu().numpy()
