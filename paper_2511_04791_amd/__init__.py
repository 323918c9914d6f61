"""Mixed-batch paged attention for MI355X: the iteration hot path of adaptive prefill/decode
multiplexing (DuetServe, arXiv 2511.04791), as a C-ABI HIP library with a thin Python binding.

    attn_mixed_batch(q, k_cache, v_cache, page_table, seq_meta, cu_split) -> out
    predict_iter_latency(batch, cu_split, shape) -> microseconds
    choose_cu_split(batch, tbt_slo_us, shape) -> (CuSplit, predicted_us, rho, flags)

Every step of the path runs in libduet.so; this module only marshals arguments.  PyTorch
supplies device memory and streams.
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass

import numpy as np

from . import _native as N
from ._native import (AGG, BF16, CONCURRENT, CU_STEP, F32, KIND_DECODE, KIND_PREFILL, SPLIT, STATUS_SLO_INFEASIBLE,
                      STATUS_UNCALIBRATED, TOTAL_CUS, DuetError)
from .workloads import AttnShape

__all__ = ["AGG", "SPLIT", "CONCURRENT", "CuSplit", "Context", "Model", "DuetError", "attn_mixed_batch", "predict_iter_latency",
           "choose_cu_split", "default_context", "AttnShape", "STATUS_SLO_INFEASIBLE", "STATUS_UNCALIBRATED"]


@dataclass(frozen=True)
class CuSplit:
    mode: int = AGG
    cus_prefill: int = TOTAL_CUS
    cus_decode: int = 0
    k_decode_steps: int = 1

    @staticmethod
    def agg(k: int = 1) -> "CuSplit":
        """Aggregated execution; k > 1 only matters to duet_attn_lookahead (k decode steps)."""
        return CuSplit(AGG, TOTAL_CUS, 0, k)

    @staticmethod
    def split(cus_prefill: int, cus_decode: int, k: int = 1) -> "CuSplit":
        return CuSplit(SPLIT, cus_prefill, cus_decode, k)

    @staticmethod
    def concurrent(k: int = 1) -> "CuSplit":
        """Control for measurements: both halves at once on two unpartitioned streams."""
        return CuSplit(CONCURRENT, TOTAL_CUS, TOTAL_CUS, k)

    def to_c(self) -> N.CuSplit:
        return N.CuSplit(self.mode, self.cus_prefill, self.cus_decode, self.k_decode_steps)

    def __str__(self):
        if self.mode == AGG:
            return "AGG" if self.k_decode_steps == 1 else f"AGG(k={self.k_decode_steps})"
        if self.mode == CONCURRENT:
            return "CONCURRENT" if self.k_decode_steps == 1 else f"CONCURRENT(k={self.k_decode_steps})"
        return f"SPLIT(Sp={self.cus_prefill},Sd={self.cus_decode},k={self.k_decode_steps})"


def _shape_c(shape: AttnShape) -> N.Shape:
    return N.Shape(shape.num_q_heads, shape.num_kv_heads, shape.head_dim, shape.page_size,
                   BF16 if shape.dtype == "bf16" else F32, shape.num_layers)


def _meta_rows(seq_meta):
    """Accepts an int array [R, 4] of (kind, q_start, q_len, cached_len) or a list of
    (kind, q_len, cached_len) triples (q_start is then filled in order)."""
    arr = np.asarray(seq_meta, dtype=np.int64)
    if arr.ndim != 2 or arr.shape[1] not in (3, 4):
        raise ValueError("seq_meta must be [R, 4] (kind, q_start, q_len, cached_len) or [R, 3] (kind, q_len, cached)")
    if arr.shape[1] == 3:
        starts = np.concatenate([[0], np.cumsum(arr[:, 1])[:-1]]) if len(arr) else np.zeros(0, np.int64)
        arr = np.stack([arr[:, 0], starts, arr[:, 1], arr[:, 2]], axis=1)
    return np.ascontiguousarray(arr.astype(np.int32))


class _BatchC:
    """Keeps the ctypes array alive alongside the struct that points into it."""

    def __init__(self, seq_meta):
        rows = _meta_rows(seq_meta)
        self.rows = rows
        self.arr = (N.SeqMeta * max(1, len(rows)))()
        if len(rows):
            ctypes.memmove(self.arr, rows.ctypes.data, rows.nbytes)
        self.c = N.Batch(self.arr, len(rows))


class Model:
    """The host-side roofline latency model (owns a duet_model unless borrowed from a Context)."""

    def __init__(self, handle=None, owner=None):
        if handle is None:
            h = ctypes.c_void_p()
            N.check(N.lib().duet_model_create(ctypes.byref(h)), "duet_model_create")
            handle, self._owned = h, True
        else:
            handle, self._owned = ctypes.c_void_p(handle), False
        self.handle = handle
        self._owner = owner

    def __del__(self):
        if getattr(self, "_owned", False) and self.handle:
            N.lib().duet_model_destroy(self.handle)
            self.handle = None

    def set_tables(self, flops_per_s, bytes_per_s):
        n = N.TOTAL_CUS // N.CU_STEP
        cus = (ctypes.c_int32 * n)(*range(N.CU_STEP, N.TOTAL_CUS + 1, N.CU_STEP))
        fl = (ctypes.c_double * n)(*[float(x) for x in flops_per_s])
        by = (ctypes.c_double * n)(*[float(x) for x in bytes_per_s])
        N.check(N.lib().duet_model_set_tables(self.handle, n, cus, fl, by), "duet_model_set_tables")

    def tables(self):
        n = N.TOTAL_CUS // N.CU_STEP
        cus, fl, by = (ctypes.c_int32 * n)(), (ctypes.c_double * n)(), (ctypes.c_double * n)()
        N.check(N.lib().duet_model_get_tables(self.handle, n, cus, fl, by), "duet_model_get_tables")
        return list(cus), list(fl), list(by)

    def set_sharing_tables(self, flops_per_s, bytes_per_s):
        n = N.TOTAL_CUS // N.CU_STEP
        cus = (ctypes.c_int32 * n)(*range(N.CU_STEP, N.TOTAL_CUS + 1, N.CU_STEP))
        fl = (ctypes.c_double * n)(*[float(x) for x in flops_per_s])
        by = (ctypes.c_double * n)(*[float(x) for x in bytes_per_s])
        N.check(N.lib().duet_model_set_sharing_tables(self.handle, n, cus, fl, by), "duet_model_set_sharing_tables")

    def sharing_tables(self):
        """(cus, flops, bytes, is_set): the standalone tables when no sharing tables are set."""
        n = N.TOTAL_CUS // N.CU_STEP
        cus, fl, by = (ctypes.c_int32 * n)(), (ctypes.c_double * n)(), (ctypes.c_double * n)()
        flag = ctypes.c_int32()
        N.check(N.lib().duet_model_get_sharing_tables(self.handle, n, cus, fl, by, ctypes.byref(flag)),
                "duet_model_get_sharing_tables")
        return list(cus), list(fl), list(by), bool(flag.value)

    def set_launch_tables(self, prefill_s, decode_s):
        """Fixed seconds per layer of each partition kind on every share (zero: the paper's model)."""
        n = N.TOTAL_CUS // N.CU_STEP
        cus = (ctypes.c_int32 * n)(*range(N.CU_STEP, N.TOTAL_CUS + 1, N.CU_STEP))
        lp = (ctypes.c_double * n)(*[float(x) for x in prefill_s])
        ld = (ctypes.c_double * n)(*[float(x) for x in decode_s])
        N.check(N.lib().duet_model_set_launch_tables(self.handle, n, cus, lp, ld), "duet_model_set_launch_tables")

    def launch_tables(self):
        n = N.TOTAL_CUS // N.CU_STEP
        cus, lp, ld = (ctypes.c_int32 * n)(), (ctypes.c_double * n)(), (ctypes.c_double * n)()
        N.check(N.lib().duet_model_get_launch_tables(self.handle, n, cus, lp, ld), "duet_model_get_launch_tables")
        return list(cus), list(lp), list(ld)

    def set_efficiency(self, prefill_eff: float, decode_eff: float):
        N.check(N.lib().duet_model_set_efficiency(self.handle, prefill_eff, decode_eff), "duet_model_set_efficiency")

    def save(self, path: str):
        N.check(N.lib().duet_model_save(self.handle, path.encode()), "duet_model_save")

    def load(self, path: str):
        N.check(N.lib().duet_model_load(self.handle, path.encode()), "duet_model_load")


def predict_iter_latency(batch, cu_split: CuSplit, shape: AttnShape, model: Model | None = None) -> float:
    """Predicted latency (us) of one iteration of shape.num_layers layers."""
    b = _BatchC(batch)
    us = ctypes.c_double()
    N.check(N.lib().duet_predict_iter_latency(model.handle if model else None, ctypes.byref(_shape_c(shape)),
                                              ctypes.byref(b.c), cu_split.to_c(), ctypes.byref(us)),
            "duet_predict_iter_latency")
    return us.value


def predict_partition_latency(batch, kind: int, cus: int, shape: AttnShape, model: Model | None = None,
                              shared: bool = True) -> float:
    """Predicted time (us) of one partition: the requests of `kind` on `cus` CUs (t_d or t_p)."""
    b = _BatchC(batch)
    us = ctypes.c_double()
    N.check(N.lib().duet_predict_partition_latency(model.handle if model else None, ctypes.byref(_shape_c(shape)),
                                                   ctypes.byref(b.c), int(kind), int(cus), int(bool(shared)),
                                                   ctypes.byref(us)), "duet_predict_partition_latency")
    return us.value


def choose_cu_split(batch, tbt_slo_us: float, shape: AttnShape, model: Model | None = None,
                    max_decode_steps: int = 0):
    """Algorithm 1: returns (CuSplit, predicted_us, rho, status_flags).  max_decode_steps > 0
    caps k, the decode steps run per prefill step."""
    b = _BatchC(batch)
    out, us, rho, flags = N.CuSplit(), ctypes.c_double(), ctypes.c_double(), ctypes.c_int32()
    N.check(N.lib().duet_choose_cu_split(model.handle if model else None, ctypes.byref(_shape_c(shape)),
                                         ctypes.byref(b.c), float(tbt_slo_us), int(max_decode_steps),
                                         ctypes.byref(out), ctypes.byref(us),
                                         ctypes.byref(rho), ctypes.byref(flags)), "duet_choose_cu_split")
    return CuSplit(out.mode, out.cus_prefill, out.cus_decode, out.k_decode_steps), us.value, rho.value, flags.value


BLOCK_GQA_QKV = 1
BLOCK_FUSED_GATE_UP = 2


@dataclass(frozen=True)
class BlockShape:
    """Dense dimensions of the block around the attention layers (duet_block_shape)."""
    ffn_dim: int
    vocab_size: int = 0
    flags: int = 0

    def to_c(self) -> N.BlockShape:
        return N.BlockShape(int(self.ffn_dim), int(self.vocab_size), int(self.flags))


def predict_model_latency(batch, cu_split: CuSplit, shape: AttnShape, block: BlockShape,
                          model: Model | None = None) -> float:
    """Full-model latency (us): token-level operators, attention and classifier (duet_predict_model_latency)."""
    b = _BatchC(batch)
    us = ctypes.c_double()
    N.check(N.lib().duet_predict_model_latency(model.handle if model else None, ctypes.byref(_shape_c(shape)),
                                               ctypes.byref(block.to_c()), ctypes.byref(b.c), cu_split.to_c(),
                                               ctypes.byref(us)), "duet_predict_model_latency")
    return us.value


def choose_cu_split_model(batch, tbt_slo_us: float, shape: AttnShape, block: BlockShape, model: Model | None = None,
                          max_decode_steps: int = 0):
    """Algorithm 1 on the full-model estimate: (CuSplit, predicted_us, rho, status_flags)."""
    b = _BatchC(batch)
    out, us, rho, flags = N.CuSplit(), ctypes.c_double(), ctypes.c_double(), ctypes.c_int32()
    N.check(N.lib().duet_choose_cu_split_model(model.handle if model else None, ctypes.byref(_shape_c(shape)),
                                               ctypes.byref(block.to_c()), ctypes.byref(b.c), float(tbt_slo_us),
                                               int(max_decode_steps), ctypes.byref(out), ctypes.byref(us),
                                               ctypes.byref(rho), ctypes.byref(flags)), "duet_choose_cu_split_model")
    return CuSplit(out.mode, out.cus_prefill, out.cus_decode, out.k_decode_steps), us.value, rho.value, flags.value


def batch_work(batch, shape: AttnShape, kind: int = -1) -> tuple[float, float]:
    """The model's (FLOPs, bytes) for the requests of `kind` (-1 = all), shape.num_layers layers."""
    b = _BatchC(batch)
    f, by = ctypes.c_double(), ctypes.c_double()
    N.check(N.lib().duet_batch_work(ctypes.byref(_shape_c(shape)), ctypes.byref(b.c), int(kind), ctypes.byref(f),
                                    ctypes.byref(by)), "duet_batch_work")
    return f.value, by.value


def workspace_bytes(shape: AttnShape, seq_meta) -> int:
    b = _BatchC(seq_meta)
    n = ctypes.c_size_t()
    N.check(N.lib().duet_workspace_bytes(ctypes.byref(_shape_c(shape)), ctypes.byref(b.c), ctypes.byref(n)),
            "duet_workspace_bytes")
    return n.value


def block_workspace_bytes(shape: AttnShape, block: BlockShape, seq_meta, k_decode_steps: int = 1) -> int:
    """Device workspace of duet_block_forward for this batch."""
    b = _BatchC(seq_meta)
    n = ctypes.c_size_t()
    N.check(N.lib().duet_block_workspace_bytes(ctypes.byref(_shape_c(shape)), ctypes.byref(block.to_c()),
                                               ctypes.byref(b.c), int(k_decode_steps), ctypes.byref(n)),
            "duet_block_workspace_bytes")
    return n.value


BLOCK_BUFFER_NAMES = ("norm", "qkv", "q", "attn", "gate_up", "act")


def block_buffers(shape: AttnShape, block: BlockShape, seq_meta, k_decode_steps: int = 1) -> dict:
    """Byte offsets of the block forward's activation buffers in its workspace (duet_block_buffers)."""
    b = _BatchC(seq_meta)
    offs = (ctypes.c_size_t * 6)()
    N.check(N.lib().duet_block_buffers(ctypes.byref(_shape_c(shape)), ctypes.byref(block.to_c()), ctypes.byref(b.c),
                                       int(k_decode_steps), offs), "duet_block_buffers")
    return dict(zip(BLOCK_BUFFER_NAMES, (int(x) for x in offs)))


class Engine:
    """The serving engine's batch former and page allocator (duet_engine_*), host only."""

    def __init__(self, token_budget: int, num_pages: int, max_pages_per_req: int, *, page_size: int = 16,
                 shuffle_seed: int = 0):
        h = ctypes.c_void_p()
        N.check(N.lib().duet_engine_create(int(token_budget), int(page_size), int(num_pages), int(max_pages_per_req),
                                           int(shuffle_seed), ctypes.byref(h)), "duet_engine_create")
        self.handle, self.max_pages, self.budget = h, int(max_pages_per_req), int(token_budget)

    def add_request(self, prompt_len: int, output_len: int) -> int:
        rid = ctypes.c_int64()
        N.check(N.lib().duet_engine_add_request(self.handle, int(prompt_len), int(output_len), ctypes.byref(rid)),
                "duet_engine_add_request")
        return rid.value

    def stats(self) -> tuple[int, int, int]:
        """(waiting, running, free pages)."""
        w, r, f = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
        N.check(N.lib().duet_engine_stats(self.handle, ctypes.byref(w), ctypes.byref(r), ctypes.byref(f)),
                "duet_engine_stats")
        return w.value, r.value, f.value

    def step(self, decode_steps: int = 1):
        """The next step: (seq_meta int32 [R, 4], page_table int32 [R, max_pages], request ids int64 [R]).
        decode_steps > 1: a look-ahead step (duet_engine_step_lookahead)."""
        w, r, _ = self.stats()
        cap = int(w + r) + 1
        meta = np.zeros((cap, 4), dtype=np.int32)
        table = np.zeros((cap, self.max_pages), dtype=np.int32)
        ids = np.zeros(cap, dtype=np.int64)
        n = ctypes.c_int32()
        if decode_steps == 1:
            N.check(N.lib().duet_engine_step(self.handle, meta.ctypes.data, table.ctypes.data, ids.ctypes.data, cap,
                                             ctypes.byref(n)), "duet_engine_step")
        else:
            N.check(N.lib().duet_engine_step_lookahead(self.handle, int(decode_steps), meta.ctypes.data,
                                                       table.ctypes.data, ids.ctypes.data, cap, ctypes.byref(n)),
                    "duet_engine_step_lookahead")
        return meta[:n.value].copy(), table[:n.value].copy(), ids[:n.value].copy()

    def complete(self, decode_steps_run: int | None = None) -> None:
        """Completes the step; decode_steps_run: of a look-ahead step, the steps that ran."""
        if decode_steps_run is None:
            N.check(N.lib().duet_engine_complete(self.handle), "duet_engine_complete")
        else:
            N.check(N.lib().duet_engine_complete_lookahead(self.handle, int(decode_steps_run)),
                    "duet_engine_complete_lookahead")

    def close(self) -> None:
        if self.handle:
            N.lib().duet_engine_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


BLOCK_WEIGHT_NAMES = ("attn_norm", "w_qkv", "w_o", "ffn_norm", "w_gate_up", "w_down")


def lookahead_workspace_bytes(shape: AttnShape, seq_meta, k_decode_steps: int) -> int:
    b = _BatchC(seq_meta)
    n = ctypes.c_size_t()
    N.check(N.lib().duet_lookahead_workspace_bytes(ctypes.byref(_shape_c(shape)), ctypes.byref(b.c),
                                                   int(k_decode_steps), ctypes.byref(n)),
            "duet_lookahead_workspace_bytes")
    return n.value


def shape_of(q, k_cache, num_layers: int = 1) -> AttnShape:
    import torch
    if q.dtype == torch.bfloat16:
        dt = "bf16"
    elif q.dtype == torch.float32:
        dt = "f32"
    else:
        raise TypeError(f"q dtype {q.dtype}: bf16 or float32 expected")
    return AttnShape(int(q.shape[1]), int(k_cache.shape[1]), int(q.shape[2]), dt, int(k_cache.shape[2]), num_layers)


class Context:
    """A duet_ctx on one GPU: CU-masked stream pool, kernels, probes and its latency model.

    Calls run on the current torch stream (or `stream=`).  Spatially shared calls should run on a
    created stream, not the legacy default one: HIP ties every launch on the CU-masked streams to
    work pending on the default stream, which slows back-to-back iterations by about 10%."""

    def __init__(self, device: int = 0, model_path: str | None = None):
        import torch
        if not torch.cuda.is_available():
            raise RuntimeError("no GPU visible: the HIP library needs an MI355X")
        self.device = device
        h = ctypes.c_void_p()
        if model_path is None:
            N.check(N.lib().duet_init(device, ctypes.byref(h)), "duet_init")
        else:
            N.check(N.lib().duet_init_with_model(device, model_path.encode(), ctypes.byref(h)), "duet_init_with_model")
        self.handle = h
        self.model = Model(N.lib().duet_ctx_model(h), owner=self)
        self._ws = None

    def close(self):
        if self.handle:
            N.lib().duet_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def workspace(self, nbytes: int):
        import torch
        if self._ws is None or self._ws.numel() < nbytes:
            self._ws = torch.empty(max(nbytes, 1 << 20), dtype=torch.uint8, device=f"cuda:{self.device}")
        return self._ws

    @staticmethod
    def _check_layer(q, k_cache, v_cache, page_table, b):
        import torch
        for t, name in ((q, "q"), (k_cache, "k_cache"), (v_cache, "v_cache"), (page_table, "page_table")):
            if not t.is_cuda or not t.is_contiguous():
                raise ValueError(f"{name} must be a contiguous device tensor")
        if page_table.dtype != torch.int32:
            raise TypeError("page_table must be int32")
        if v_cache.shape != (k_cache.shape[0], k_cache.shape[1], k_cache.shape[3], k_cache.shape[2]):
            raise ValueError("v_cache must be [P, h_kv, d, page_size] for k_cache [P, h_kv, page_size, d]")
        n_tok = int(b.rows[:, 2].sum()) if len(b.rows) else 0
        if q.shape[0] != n_tok:
            raise ValueError(f"q has {q.shape[0]} rows, the batch schedules {n_tok} tokens")
        if page_table.dim() != 2 or page_table.shape[0] < len(b.rows):
            raise ValueError("page_table must be [R, max_pages] with a row per request")

    def attn_mixed_batch(self, q, k_cache, v_cache, page_table, seq_meta, cu_split: CuSplit = CuSplit.agg(), *,
                         out=None, workspace=None, stream=None, num_layers: int = 1, check_errors: bool = False):
        """One layer (duet_attn_mixed_batch).  num_layers only sizes the workspace and the model."""
        import torch
        shape = shape_of(q, k_cache, num_layers)
        b = _BatchC(seq_meta)
        self._check_layer(q, k_cache, v_cache, page_table, b)
        need = workspace_bytes(shape, b.rows)
        ws = self.workspace(need) if workspace is None else workspace
        if out is None:
            out = torch.empty_like(q)
        st = torch.cuda.current_stream(q.device).cuda_stream if stream is None else stream
        N.check(N.lib().duet_attn_mixed_batch(self.handle, ctypes.byref(_shape_c(shape)), q.data_ptr(),
                                              k_cache.data_ptr(), v_cache.data_ptr(), int(k_cache.shape[0]),
                                              page_table.data_ptr(), int(page_table.shape[1]), ctypes.byref(b.c),
                                              cu_split.to_c(), ws.data_ptr(), ws.numel(), out.data_ptr(),
                                              ctypes.c_void_p(st)), "duet_attn_mixed_batch")
        if check_errors:
            N.check(N.lib().duet_check_device_error(self.handle, ws.data_ptr(), ctypes.c_void_p(st)),
                    "duet_check_device_error")
        return out

    def attn_mixed_batch_noalloc(self, q, k_cache, v_cache, page_table, seq_meta, cu_split: CuSplit = CuSplit.agg(), *,
                                 out=None, stream=None):
        """One layer without a workspace (duet_attn_mixed_batch_noalloc): the library's fixed device
        scratch is used and nothing is allocated (`out` is allocated here when not given)."""
        import torch
        shape = shape_of(q, k_cache, 1)
        b = _BatchC(seq_meta)
        self._check_layer(q, k_cache, v_cache, page_table, b)
        if out is None:
            out = torch.empty_like(q)
        st = torch.cuda.current_stream(q.device).cuda_stream if stream is None else stream
        N.check(N.lib().duet_attn_mixed_batch_noalloc(self.handle, ctypes.byref(_shape_c(shape)), q.data_ptr(),
                                                      k_cache.data_ptr(), v_cache.data_ptr(), int(k_cache.shape[0]),
                                                      page_table.data_ptr(), int(page_table.shape[1]),
                                                      ctypes.byref(b.c), cu_split.to_c(), out.data_ptr(),
                                                      ctypes.c_void_p(st)), "duet_attn_mixed_batch_noalloc")
        return out

    def block_forward(self, x, weights, k_caches, v_caches, page_table, seq_meta, ffn_dim: int,
                      cu_split: CuSplit = CuSplit.agg(), *, x_ahead=None, norm_eps: float = 1e-5, workspace=None,
                      stream=None, check_errors: bool = False):
        """len(weights) transformer blocks in place on the residual stream x [T, h_q d] (duet_block_forward).
        weights: per-layer dicts of contiguous bf16 device tensors named as BLOCK_WEIGHT_NAMES; the caches
        receive every scheduled token's keys and values.  With cu_split.k_decode_steps = k > 1, x_ahead
        holds k - 1 tensors [R_d, h_q d]: the decode requests' residual rows of look-ahead steps 1 .. k - 1
        (updated in place).  Returns x."""
        import torch
        L = len(weights)
        if L < 1 or len(k_caches) != L or len(v_caches) != L:
            raise ValueError("weights, k_caches and v_caches must be non-empty lists of equal length")
        b = _BatchC(seq_meta)
        n_tok = int(b.rows[:, 2].sum()) if len(b.rows) else 0
        kc0 = k_caches[0]
        shape = AttnShape(int(x.shape[1]) // int(kc0.shape[3]), int(kc0.shape[1]), int(kc0.shape[3]), "bf16",
                          int(kc0.shape[2]), L)
        if x.dtype != torch.bfloat16 or not x.is_cuda or not x.is_contiguous() or x.dim() != 2 or x.shape[0] != n_tok:
            raise ValueError(f"x must be a contiguous bf16 device tensor [{n_tok}, d]")
        if page_table.dtype != torch.int32 or not page_table.is_cuda or not page_table.is_contiguous():
            raise ValueError("page_table must be a contiguous int32 device tensor")
        d, dh = int(x.shape[1]), shape.head_dim
        d_qkv = (shape.num_q_heads + 2 * shape.num_kv_heads) * dh
        want = {"attn_norm": (d,), "w_qkv": (d, d_qkv), "w_o": (d, d), "ffn_norm": (d,), "w_gate_up": (d, 2 * ffn_dim),
                "w_down": (ffn_dim, d)}
        for l, w in enumerate(weights):
            for name in BLOCK_WEIGHT_NAMES:
                t = w[name]
                if tuple(t.shape) != want[name] or t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous():
                    raise ValueError(f"layer {l}: {name} must be a contiguous bf16 device tensor {want[name]}")
            self._check_layer(x.view(n_tok, shape.num_q_heads, dh), k_caches[l], v_caches[l], page_table, b)
        block = BlockShape(int(ffn_dim), 0, BLOCK_GQA_QKV | BLOCK_FUSED_GATE_UP)
        k = int(cu_split.k_decode_steps)
        n_dec = int((b.rows[:, 0] == KIND_DECODE).sum()) if len(b.rows) else 0
        xa = list(x_ahead or [])
        if k > 1 and n_dec > 0:
            if len(xa) != k - 1:
                raise ValueError(f"x_ahead must hold k - 1 = {k - 1} tensors")
            for t in xa:
                if t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous() or tuple(t.shape) != (n_dec, d):
                    raise ValueError(f"x_ahead tensors must be contiguous bf16 device tensors [{n_dec}, {d}]")
        need = block_workspace_bytes(shape, block, b.rows, k)
        ws = self.workspace(need) if workspace is None else workspace
        wts = (N.BlockWeights * L)(*[N.BlockWeights(*[w[n].data_ptr() for n in BLOCK_WEIGHT_NAMES]) for w in weights])
        arr = lambda ts: (ctypes.c_void_p * L)(*[t.data_ptr() for t in ts])
        st = torch.cuda.current_stream(x.device).cuda_stream if stream is None else stream
        N.check(N.lib().duet_block_forward(self.handle, ctypes.byref(_shape_c(shape)), ctypes.byref(block.to_c()), wts,
                                           float(norm_eps), x.data_ptr(),
                                           (ctypes.c_void_p * max(1, len(xa)))(*[t.data_ptr() for t in xa]) if xa else None,
                                           arr(k_caches), arr(v_caches),
                                           int(kc0.shape[0]), page_table.data_ptr(), int(page_table.shape[1]),
                                           ctypes.byref(b.c), cu_split.to_c(), ws.data_ptr(), ws.numel(),
                                           ctypes.c_void_p(st)), "duet_block_forward")
        if check_errors:
            N.check(N.lib().duet_check_device_error(self.handle, ws.data_ptr(), ctypes.c_void_p(st)),
                    "duet_check_device_error")
        return x

    def rmsnorm(self, x, weight, eps: float = 1e-5, *, out=None, stream=None):
        """duet_rmsnorm over the rows of a contiguous bf16 device tensor x [rows, d]."""
        import torch
        if out is None:
            out = torch.empty_like(x)
        st = torch.cuda.current_stream(x.device).cuda_stream if stream is None else stream
        N.check(N.lib().duet_rmsnorm(self.handle, x.data_ptr(), weight.data_ptr(), out.data_ptr(), int(x.shape[0]),
                                     int(x.shape[1]), float(eps), ctypes.c_void_p(st)), "duet_rmsnorm")
        return out

    def swiglu(self, gate_up, *, out=None, stream=None):
        """duet_swiglu: gate_up [rows, 2 m] -> [rows, m]."""
        import torch
        rows, m2 = int(gate_up.shape[0]), int(gate_up.shape[1])
        if out is None:
            out = torch.empty(rows, m2 // 2, dtype=gate_up.dtype, device=gate_up.device)
        st = torch.cuda.current_stream(gate_up.device).cuda_stream if stream is None else stream
        N.check(N.lib().duet_swiglu(self.handle, gate_up.data_ptr(), out.data_ptr(), rows, m2 // 2, ctypes.c_void_p(st)),
                "duet_swiglu")
        return out

    def qkv_split(self, qkv, k_cache, v_cache, page_table, seq_meta, shape: AttnShape, *, q=None, workspace=None,
                  stream=None, check_errors: bool = False):
        """duet_qkv_split: the query rows out of qkv [T, (h_q + 2 h_kv) d], keys and values into the cache."""
        import torch
        b = _BatchC(seq_meta)
        T = int(qkv.shape[0])
        if q is None:
            q = torch.empty(T, shape.num_q_heads, shape.head_dim, dtype=qkv.dtype, device=qkv.device)
        ws = self.workspace(workspace_bytes(shape, b.rows)) if workspace is None else workspace
        st = torch.cuda.current_stream(qkv.device).cuda_stream if stream is None else stream
        N.check(N.lib().duet_qkv_split(self.handle, ctypes.byref(_shape_c(shape)), qkv.data_ptr(), q.data_ptr(),
                                       k_cache.data_ptr(), v_cache.data_ptr(), int(k_cache.shape[0]),
                                       page_table.data_ptr(), int(page_table.shape[1]), ctypes.byref(b.c),
                                       ws.data_ptr(), ws.numel(), ctypes.c_void_p(st)), "duet_qkv_split")
        if check_errors:
            N.check(N.lib().duet_check_device_error(self.handle, ws.data_ptr(), ctypes.c_void_p(st)),
                    "duet_check_device_error")
        return q

    def attn_iteration(self, qs, k_caches, v_caches, page_table, seq_meta, cu_split: CuSplit = CuSplit.agg(), *,
                       outs=None, workspace=None, stream=None, check_errors: bool = False):
        """All layers of one iteration (duet_attn_iteration): lists of per-layer tensors sharing the
        batch and the page table.  Returns the list of per-layer outputs."""
        import torch
        L = len(qs)
        if L < 1 or len(k_caches) != L or len(v_caches) != L or (outs is not None and len(outs) != L):
            raise ValueError("qs, k_caches, v_caches (and outs) must be non-empty lists of equal length")
        shape = shape_of(qs[0], k_caches[0], L)
        b = _BatchC(seq_meta)
        for l in range(L):
            if qs[l].shape != qs[0].shape or qs[l].dtype != qs[0].dtype or k_caches[l].shape != k_caches[0].shape:
                raise ValueError(f"layer {l}: shapes differ from layer 0")
            self._check_layer(qs[l], k_caches[l], v_caches[l], page_table, b)
        need = workspace_bytes(shape, b.rows)
        ws = self.workspace(need) if workspace is None else workspace
        if outs is None:
            outs = [torch.empty_like(x) for x in qs]
        arr = lambda ts: (ctypes.c_void_p * L)(*[t.data_ptr() for t in ts])
        st = torch.cuda.current_stream(qs[0].device).cuda_stream if stream is None else stream
        N.check(N.lib().duet_attn_iteration(self.handle, ctypes.byref(_shape_c(shape)), arr(qs), arr(k_caches),
                                            arr(v_caches), int(k_caches[0].shape[0]), page_table.data_ptr(),
                                            int(page_table.shape[1]), ctypes.byref(b.c), cu_split.to_c(),
                                            ws.data_ptr(), ws.numel(), arr(outs), ctypes.c_void_p(st)),
                "duet_attn_iteration")
        if check_errors:
            N.check(N.lib().duet_check_device_error(self.handle, ws.data_ptr(), ctypes.c_void_p(st)),
                    "duet_check_device_error")
        return outs

    def attn_lookahead(self, qs, q_ahead, k_ahead, v_ahead, k_caches, v_caches, page_table, seq_meta,
                       cu_split: CuSplit, *, outs=None, outs_ahead=None, workspace=None, stream=None,
                       check_errors: bool = False):
        """One prefill step and k = cu_split.k_decode_steps decode steps (duet_attn_lookahead).

        qs, k_caches, v_caches, outs: per-layer lists as in attn_iteration (step 0).  q_ahead,
        k_ahead, v_ahead, outs_ahead: lists of (k - 1) * L tensors, index (s - 1) * L + l, of shape
        [R_d, h_q or h_kv, d] with the decode requests in seq_meta order.  The caches are written
        (steps >= 1 append their tokens).  Returns (outs, outs_ahead)."""
        import torch
        L = len(qs)
        k = int(cu_split.k_decode_steps)
        n_ahead = (k - 1) * L
        if L < 1 or len(k_caches) != L or len(v_caches) != L or (outs is not None and len(outs) != L):
            raise ValueError("qs, k_caches, v_caches (and outs) must be non-empty lists of equal length")
        if len(q_ahead) != n_ahead or len(k_ahead) != n_ahead or len(v_ahead) != n_ahead:
            raise ValueError(f"q_ahead, k_ahead and v_ahead need (k - 1) * L = {n_ahead} tensors")
        shape = shape_of(qs[0], k_caches[0], L)
        b = _BatchC(seq_meta)
        n_dec = int((b.rows[:, 0] == 1).sum()) if len(b.rows) else 0
        for l in range(L):
            if qs[l].shape != qs[0].shape or qs[l].dtype != qs[0].dtype or k_caches[l].shape != k_caches[0].shape:
                raise ValueError(f"layer {l}: shapes differ from layer 0")
            self._check_layer(qs[l], k_caches[l], v_caches[l], page_table, b)
        for x in range(n_ahead):
            for t, name, h in ((q_ahead[x], "q_ahead", shape.num_q_heads), (k_ahead[x], "k_ahead", shape.num_kv_heads),
                               (v_ahead[x], "v_ahead", shape.num_kv_heads)):
                if not t.is_cuda or not t.is_contiguous() or t.dtype != qs[0].dtype or \
                        tuple(t.shape) != (n_dec, h, shape.head_dim):
                    raise ValueError(f"{name}[{x}] must be a contiguous {qs[0].dtype} device tensor "
                                     f"[{n_dec}, {h}, {shape.head_dim}]")
        need = lookahead_workspace_bytes(shape, b.rows, k)
        ws = self.workspace(need) if workspace is None else workspace
        if outs is None:
            outs = [torch.empty_like(x) for x in qs]
        if outs_ahead is None:
            outs_ahead = [torch.empty_like(x) for x in q_ahead]
        if len(outs_ahead) != n_ahead:
            raise ValueError(f"outs_ahead needs {n_ahead} tensors")
        arr = lambda ts, n: (ctypes.c_void_p * max(n, 1))(*[t.data_ptr() for t in ts])
        st = torch.cuda.current_stream(qs[0].device).cuda_stream if stream is None else stream
        N.check(N.lib().duet_attn_lookahead(self.handle, ctypes.byref(_shape_c(shape)), arr(qs, L),
                                            arr(q_ahead, n_ahead), arr(k_ahead, n_ahead), arr(v_ahead, n_ahead),
                                            arr(k_caches, L), arr(v_caches, L), int(k_caches[0].shape[0]),
                                            page_table.data_ptr(), int(page_table.shape[1]), ctypes.byref(b.c),
                                            cu_split.to_c(), ws.data_ptr(), ws.numel(), arr(outs, L),
                                            arr(outs_ahead, n_ahead), ctypes.c_void_p(st)), "duet_attn_lookahead")
        if check_errors:
            N.check(N.lib().duet_check_device_error(self.handle, ws.data_ptr(), ctypes.c_void_p(st)),
                    "duet_check_device_error")
        return outs, outs_ahead

    def set_decode_graphs(self, enable: bool):
        N.check(N.lib().duet_set_decode_graphs(self.handle, 1 if enable else 0), "duet_set_decode_graphs")

    def decode_graph_stats(self) -> dict:
        c, cap, rep = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
        N.check(N.lib().duet_decode_graph_stats(self.handle, ctypes.byref(c), ctypes.byref(cap), ctypes.byref(rep)),
                "duet_decode_graph_stats")
        return {"cached": c.value, "captured": cap.value, "replayed": rep.value}

    def gather_kv(self, cache, which: int, page_table, req: int, kv_len: int, shape: AttnShape):
        import torch
        if not 0 <= req < page_table.shape[0]:
            raise ValueError(f"request {req} outside the page table's {page_table.shape[0]} rows")
        out = torch.empty(kv_len, shape.num_kv_heads, shape.head_dim, dtype=cache.dtype, device=cache.device)
        st = torch.cuda.current_stream(cache.device).cuda_stream
        N.check(N.lib().duet_gather_kv(self.handle, ctypes.byref(_shape_c(shape)), which, cache.data_ptr(),
                                       int(cache.shape[0]), page_table.data_ptr(), int(page_table.shape[1]), req,
                                       kv_len, out.data_ptr(), ctypes.c_void_p(st)), "duet_gather_kv")
        return out

    def set_profiling(self, level):
        """0 off, 1 iteration events, 2 per-kernel events (True means 2)."""
        level = 2 if level is True else int(level)
        N.check(N.lib().duet_set_profiling(self.handle, level), "duet_set_profiling")

    def last_kernel_times(self) -> dict:
        t = N.KernelTimes()
        N.check(N.lib().duet_last_kernel_times(self.handle, ctypes.byref(t)), "duet_last_kernel_times")
        return {f: getattr(t, f) for f, _ in N.KernelTimes._fields_}

    def probe_read_bw(self, cus: int, buf, iters: int = 3) -> float:
        v = ctypes.c_double()
        N.check(N.lib().duet_probe_read_bw(self.handle, cus, buf.data_ptr(), buf.numel() * buf.element_size(), iters,
                                           ctypes.byref(v)), "duet_probe_read_bw")
        return v.value

    def probe_mfma(self, cus: int, iters: int = 8192) -> float:
        v = ctypes.c_double()
        N.check(N.lib().duet_probe_mfma(self.handle, cus, iters, ctypes.byref(v)), "duet_probe_mfma")
        return v.value

    def probe_placement(self, cus: int, high_end: bool, blocks: int):
        import torch
        out = torch.zeros(2 * blocks, dtype=torch.int32, device=f"cuda:{self.device}")
        N.check(N.lib().duet_probe_placement(self.handle, cus, 1 if high_end else 0, blocks, out.data_ptr()),
                "duet_probe_placement")
        return out.cpu().numpy().astype(np.uint32).reshape(blocks, 2)

    def calibrate(self, scratch=None) -> Model:
        import torch
        if scratch is None:
            scratch = torch.empty(1 << 30, dtype=torch.uint8, device=f"cuda:{self.device}")
        N.check(N.lib().duet_calibrate(self.handle, self.model.handle, scratch.data_ptr(), scratch.numel()),
                "duet_calibrate")
        return self.model


_default = None


def default_context() -> Context:
    global _default
    if _default is None:
        _default = Context(0)
    return _default


def attn_mixed_batch(q, k_cache, v_cache, page_table, seq_meta, cu_split: CuSplit = CuSplit.agg(), **kw):
    """One iteration's attention on the default context; see Context.attn_mixed_batch."""
    return default_context().attn_mixed_batch(q, k_cache, v_cache, page_table, seq_meta, cu_split, **kw)
