"""Layer-wise three-stage KV pipeline around the attention call.

Paper Sec. 4.2 (Global KV Cache Store): the KV of a request's cached prefix
lives in a host-side store; layer by layer, while the GPU computes layer i,
the host-to-device channel fetches the KV of layer i+1 and the device-to-host
channel stores the newly computed KV of layer i-1, so the per-layer transfer
T_KV = S_kv * L * r / B hides under the per-layer compute when it is shorter.

Here the compute stage of layer i is the split paged decode attention of that
layer (``bana_decode_attn_fused`` over all partitions).  Layers rotate through
a ring of three device pools.  Two overlapped schedules:

* ``run_fused``: one launch per layer on one stream.  The attention launch of
  layer i carries the fetch of layer i+1 and the store of layer i-1 as side
  copies in workgroups of its own (``bana_decode_attn_fused_copies``), so the
  three stages overlap inside the launch and the stream alone orders them
  against the neighbouring layers (the fetch into a ring slot follows, in an
  earlier launch, the store that last read it).
* ``run_pipelined``: three HIP streams at default priority (compute, and one
  copy stream shared by fetches and stores unless asked for two) ordered by
  events; transfers are the library's stream-ordered copy kernel
  (``bana_copy_async``).  Each layer's attention waits on an event of the copy
  stream, which costs a gap between consecutive attention launches.

Every schedule runs the same launch plan (4 wavefronts per workgroup, chunked
launch: the copy workgroups of the fused schedule need free CU slots beside a
plan that would otherwise fill one dispatch round), so all give the same
results bit for bit.  Orchestration only: the arithmetic and the copies are
the library's kernels.
"""

from __future__ import annotations

import ctypes
from typing import List, Optional

import numpy as np
import torch

from . import bana


def _bf16(a: np.ndarray, device=None, pin: bool = False) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
    if pin:
        return t.pin_memory()
    return t.to(device) if device is not None else t


class LayerPipeline:
    """Runs `store.num_layers` layers of fetch -> attention -> store on one GPU."""

    def __init__(self, store, device="cuda", ring: int = 3, compute_stream: Optional[torch.cuda.Stream] = None,
                 separate_copy_streams: bool = False):
        self.store = store
        w = store.w
        self.w = w
        self.device = torch.device(device)
        self.ring = ring
        self.L = store.num_layers
        fb, sb = store.fetch_blocks, store.store_blocks
        self.fb, self.sb = fb, sb
        # Device pools: a ring of full copies of the layer's KV pools.
        k = _bf16(w.k_cache, self.device)
        v = _bf16(w.v_cache, self.device)
        self.pool_k = [k] + [k.clone() for _ in range(ring - 1)]
        self.pool_v = [v] + [v.clone() for _ in range(ring - 1)]
        # Host store (pinned): fetched prefix blocks per layer, stored blocks per layer.
        self.host_fetch_k = [_bf16(store.fetch_k[i], pin=True) for i in range(self.L)]
        self.host_fetch_v = [_bf16(store.fetch_v[i], pin=True) for i in range(self.L)]
        self.host_store_k = [torch.empty((sb,) + tuple(k.shape[1:]), dtype=torch.bfloat16).pin_memory()
                             for _ in range(self.L)]
        self.host_store_v = [torch.empty((sb,) + tuple(v.shape[1:]), dtype=torch.bfloat16).pin_memory()
                             for _ in range(self.L)]
        i32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(self.device)
        self.q = _bf16(w.q, self.device)
        self.block_table = i32(w.block_table)
        self.seq_lens = i32(w.seq_lens)
        self.kv_begin = i32(w.kv_begin)
        self.kv_end = i32(w.kv_end)
        B, Hq = w.batch, w.num_q_heads
        lens_all = (w.kv_end.astype(np.int64) - w.kv_begin).sum(axis=0)
        self.dims = bana.make_dims(B, Hq, w.num_kv_heads, w.max_blocks_per_seq, w.num_blocks,
                                   max_range_tokens=int(lens_all.max()), total_range_tokens=int(lens_all.sum()),
                                   nonempty_ranges=int(np.count_nonzero(lens_all)), waves_hint=4, plan_hint=1)
        ws = bana.bana_decode_attn_workspace_bytes(self.dims)
        self.workspace = torch.empty(max(ws, 256), dtype=torch.uint8, device=self.device) if ws else None
        self.out = torch.empty((self.L, B, Hq, bana.HEAD_DIM), dtype=torch.float32, device=self.device)
        self.lse = torch.empty((self.L, B, Hq), dtype=torch.float32, device=self.device)
        # Fetches and stores share one copy stream by default: measured on MI355X (llama3_8b layer),
        # giving the two channels streams of their own took 0.26 ms per layer against 0.23 ms.
        self.s_comp = compute_stream or torch.cuda.current_stream(self.device)
        self.s_h2d = torch.cuda.Stream(device=self.device)
        self.s_d2h = torch.cuda.Stream(device=self.device) if separate_copy_streams else self.s_h2d
        self.stage_ms = None

        # Validate the attention arguments once through the checked binding, then keep raw
        # argument lists so the per-layer host work stays far below the per-layer GPU work.
        for slot in range(ring):
            bana.bana_decode_attn_fused(self.q, self.pool_k[slot], self.pool_v[slot], self.block_table,
                                        self.seq_lens, self.kv_begin, self.kv_end, self.out[0], self.lse[0],
                                        workspace=self.workspace, stream=self.s_comp, dims=self.dims)
        torch.cuda.synchronize(self.device)
        vp = lambda t: ctypes.c_void_p(t.data_ptr())
        ws = vp(self.workspace) if self.workspace is not None else None
        ws_bytes = self.workspace.numel() if self.workspace is not None else 0
        self._attn_args = [[ctypes.byref(self.dims), vp(self.q), vp(self.pool_k[s]), vp(self.pool_v[s]),
                            vp(self.block_table), vp(self.seq_lens), vp(self.kv_begin), vp(self.kv_end),
                            w.n_parts, vp(self.out[i]), vp(self.lse[i]), ws, ws_bytes]
                           for i, s in ((i, i % ring) for i in range(self.L))]
        kb = self.pool_k[0][:1].numel() * 2  # bytes per block, all kv heads (same for V)
        self._fetch_bytes = fb * kb
        self._store_bytes = sb * kb
        self._kb = kb
        # Side copies of each layer's launch in the fused schedule: fetch of layer i+1, store of i-1.
        self._side = []
        for i in range(self.L):
            c = []
            if i + 1 < self.L:
                c += self._fetch_copies(i + 1)
            if i >= 1:
                c += self._store_copies(i - 1)
            arr = (bana.bana_copy * max(1, len(c)))(*[bana.bana_copy(d, s_, n) for d, s_, n in c])
            self._side.append((arr, len(c)))

    def _fetch_copies(self, layer: int):
        s = layer % self.ring
        return [(self.pool_k[s].data_ptr(), self.host_fetch_k[layer].data_ptr(), self._fetch_bytes),
                (self.pool_v[s].data_ptr(), self.host_fetch_v[layer].data_ptr(), self._fetch_bytes)]

    def _store_copies(self, layer: int):
        s = layer % self.ring
        off = self.fb * self._kb
        return [(self.host_store_k[layer].data_ptr(), self.pool_k[s].data_ptr() + off, self._store_bytes),
                (self.host_store_v[layer].data_ptr(), self.pool_v[s].data_ptr() + off, self._store_bytes)]

    # -- stages ------------------------------------------------------------------------------------
    def _copy(self, dst: int, src: int, nbytes: int, stream) -> None:
        # A copy kernel, not the DMA engines: measured on MI355X, DMA copies ordered behind
        # cross-stream waits held the issuing thread until the wait resolved, which starved
        # the compute stream; kernels order on device-side events only.
        st = bana.lib().bana_copy_async(ctypes.c_void_p(dst), ctypes.c_void_p(src), nbytes,
                                        ctypes.c_void_p(stream.cuda_stream))
        if st != bana.BANA_OK:
            raise bana.BanaError(st, "bana_copy_async")

    def _fetch(self, layer: int, stream) -> None:
        for dst, src, n in self._fetch_copies(layer):
            self._copy(dst, src, n, stream)

    def _attend(self, layer: int, stream) -> None:
        st = bana.lib().bana_decode_attn_fused(*self._attn_args[layer], ctypes.c_void_p(stream.cuda_stream))
        if st != bana.BANA_OK:
            raise bana.BanaError(st, "bana_decode_attn_fused")

    def _store(self, layer: int, stream) -> None:
        for dst, src, n in self._store_copies(layer):
            self._copy(dst, src, n, stream)

    def _attend_with_copies(self, layer: int, stream) -> None:
        arr, n = self._side[layer]
        st = bana.lib().bana_decode_attn_fused_copies(*self._attn_args[layer], arr, n,
                                                      ctypes.c_void_p(stream.cuda_stream))
        if st != bana.BANA_OK:
            raise bana.BanaError(st, "bana_decode_attn_fused_copies")

    # -- schedules ---------------------------------------------------------------------------------
    def run_serial(self) -> None:
        """All stages of all layers on one stream, one after the other."""
        st = self.s_comp
        for i in range(self.L):
            self._fetch(i, st)
            self._attend(i, st)
            self._store(i, st)

    def run_fused(self, marks=None) -> None:
        """One launch per layer on the compute stream: the attention of layer i with the fetch of
        layer i+1 and the store of layer i-1 as side copies of the same launch.  The fetch of the
        first layer and the store of the last (the pipeline's fill and drain) are copy launches of
        their own; ``marks`` (two events) are recorded around the layer launches."""
        st = self.s_comp
        self._fetch(0, st)
        if marks is not None:
            marks[0].record(st)
        for i in range(self.L):
            self._attend_with_copies(i, st)
        if marks is not None:
            marks[1].record(st)
        self._store(self.L - 1, st)

    def run_attention_only(self) -> None:
        """The attention launches alone (no transfers), for comparison."""
        for i in range(self.L):
            self._attend(i, self.s_comp)

    def run_pipelined(self, timing: bool = False) -> None:
        """Fetch of layer i+1 and store of layer i-1 overlap the attention of layer i."""
        L, R = self.L, self.ring
        ev = lambda: torch.cuda.Event(enable_timing=timing)
        fetched = [ev() for _ in range(L)]
        attended = [ev() for _ in range(L)]
        stored = [ev() for _ in range(L)]
        marks = [[ev() for _ in range(6)] for _ in range(L)] if timing else None
        start = torch.cuda.Event()
        start.record(self.s_comp)
        for s in (self.s_h2d, self.s_d2h):
            s.wait_event(start)

        def fetch(i):
            if i >= R:  # the ring slot was last used by layer i - R; wait until its store is done
                self.s_h2d.wait_event(stored[i - R])
            if timing:
                marks[i][0].record(self.s_h2d)
            self._fetch(i, self.s_h2d)
            if timing:
                marks[i][1].record(self.s_h2d)
            fetched[i].record(self.s_h2d)

        def attend(i):
            self.s_comp.wait_event(fetched[i])
            if timing:
                marks[i][2].record(self.s_comp)
            self._attend(i, self.s_comp)
            if timing:
                marks[i][3].record(self.s_comp)
            attended[i].record(self.s_comp)

        def store(i):
            self.s_d2h.wait_event(attended[i])
            if timing:
                marks[i][4].record(self.s_d2h)
            self._store(i, self.s_d2h)
            if timing:
                marks[i][5].record(self.s_d2h)
            stored[i].record(self.s_d2h)

        # Issue order keeps the next layer's attention queued before the store that waits for the
        # current one: a copy behind a cross-stream wait can hold the issuing thread until that
        # wait resolves, and the compute stream must not run dry meanwhile.
        for i in range(min(2, L)):
            fetch(i)
        attend(0)
        for i in range(L):
            if i + 1 < L:
                attend(i + 1)
            store(i)
            if i + 2 < L:
                fetch(i + 2)
        self.s_comp.wait_event(stored[-1])
        if timing:
            torch.cuda.synchronize(self.device)
            self.stage_ms = np.array([[m[0].elapsed_time(m[1]), m[2].elapsed_time(m[3]), m[4].elapsed_time(m[5])]
                                      for m in marks])

    def outputs(self):
        torch.cuda.synchronize(self.device)
        return self.out.cpu().numpy(), self.lse.cpu().numpy()

    def stored(self) -> List[np.ndarray]:
        torch.cuda.synchronize(self.device)
        return [(self.host_store_k[i].view(torch.int16).numpy().view(np.uint16),
                 self.host_store_v[i].view(torch.int16).numpy().view(np.uint16)) for i in range(self.L)]


def t_kv_ms(s_kv_bytes: float, tokens: int, hit_rate: float, link_gbps: float) -> float:
    """Per-layer KV transfer time of the store (Sec. 4.2): S_kv x L x r over the link bandwidth, in ms."""
    return s_kv_bytes * tokens * hit_rate * 8 / (link_gbps * 1e9) * 1e3


def t_f_layer_ms(t_f_ms: float, hit_rate: float, layers: int) -> float:
    """Per-layer forward time of the same example (Sec. 4.2): T_F x r / N, in ms."""
    return t_f_ms * hit_rate / layers


def measure(workload: str = "llama3_8b", layers: int = 8, fetch_tokens: int = 500, store_tokens: int = 500,
            reps: int = 5) -> dict:
    """Per-layer times of the serial, three-stream and fused schedules (the fused one also in steady
    state, without the pipeline's fill and drain), of the attention alone, and the measured T_KV.

    Defaults follow the paper's worked example for the store (Sec. 4.2): a 1000-token request with a
    50 % prefix-cache hit fetches 500 tokens of KV per layer (S_kv = 4 KiB per token per layer for
    the Llama-3.1-8B shape) and stores the 500 new ones; the analytic T_KV at 200 Gbps is 0.082 ms.
    """
    import time

    from . import workloads

    w = workloads.make_config(workload, 0)
    pipe = LayerPipeline(workloads.make_layer_store(w, layers, fetch_tokens, store_tokens, seed=1),
                         compute_stream=torch.cuda.Stream())

    def timed(fn):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        t = time.perf_counter()
        for _ in range(reps):
            fn()
        torch.cuda.synchronize()
        return (time.perf_counter() - t) * 1e3 / reps / layers

    serial = timed(pipe.run_serial)
    pipelined = timed(pipe.run_pipelined)
    fused = timed(pipe.run_fused)
    alone = timed(pipe.run_attention_only)
    # Steady state of the fused schedule: events around the layer launches only (the fill and
    # drain copies outside), median over repetitions.
    steady = []
    for _ in range(reps):
        marks = [torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)]
        pipe.run_fused(marks)
        torch.cuda.synchronize()
        steady.append(marks[0].elapsed_time(marks[1]) / layers)
    fused_steady = float(np.median(steady))
    pipe.run_pipelined(timing=True)
    stage = pipe.stage_ms.mean(axis=0)
    s_kv = w.num_kv_heads * HEAD_DIM_BYTES_PER_TOKEN
    fetch_bytes = pipe.fb * w.num_kv_heads * 8192
    return {
        "workload": workload,
        "layers": layers,
        "fetch_tokens_per_layer": fetch_tokens,
        "store_tokens_per_layer": store_tokens,
        "fetch_bytes_per_layer": fetch_bytes,
        "ms_per_layer_serial": round(serial, 5),
        "ms_per_layer_pipelined": round(pipelined, 5),
        "ms_per_layer_fused_copies": round(fused, 5),
        "ms_per_layer_fused_copies_steady": round(fused_steady, 5),
        "ms_per_layer_attention_alone": round(alone, 5),
        "fused_over_attention_alone": round(fused / alone, 4),
        "fused_steady_over_attention_alone": round(fused_steady / alone, 4),
        "stage_ms_fetch_attend_store": [round(float(x), 5) for x in stage],
        "t_kv_measured_ms": round(float(stage[0]), 5),
        "h2d_gbs": round(fetch_bytes / (float(stage[0]) / 1e3) / 1e9, 2),
        "t_kv_formula_ms_at_200gbps": round(t_kv_ms(s_kv, fetch_tokens, 1.0, 200.0), 5),
    }


HEAD_DIM_BYTES_PER_TOKEN = bana.HEAD_DIM * 2 * 2  # K and V, bf16, per kv head


if __name__ == "__main__":
    import json
    import sys

    print(json.dumps(measure(*(sys.argv[1:2] or ["llama3_8b"]))))
