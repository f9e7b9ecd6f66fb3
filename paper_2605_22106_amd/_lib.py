"""ctypes binding of libarbor.so (the C ABI in include/arbor.h).

Argument marshalling only: torch tensors on the GPU are handed over as raw
device pointers together with torch's current HIP stream.  Every function has
the name of the C entry point it calls and returns the C return code (the host
validation / launch result); device-determined outcomes land in the int32
`status` tensor.  There is no fallback: without the built library, or without
a GPU tensor where the C ABI expects device memory, these functions raise.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libarbor.so")

OK, OVER_BUDGET = 0, 1
EINVAL, ENOPAGES, EHIP, EUNSUPPORTED, ENONFINITE, EWORKSPACE, ECORRUPT = -1, -2, -3, -4, -5, -6, -7
BF16, F32 = 0, 1
# kernels a call can time on their own (arbor_timing_t)
KERNEL_SCORE_ATTN, KERNEL_SELECT, KERNEL_COMPACT_MOVE, KERNEL_DECODE_ATTN = 0, 1, 2, 3
KERNEL_DECODE_CREDIT, KERNEL_COUNT = 4, 5
SELECT_TAIL_HEAVY, SELECT_TAIL_ONLY, SELECT_SINKS_TAIL = 0, 1, 2
MAX_DEPTH = 63


class Timing(ctypes.Structure):
    _fields_ = [("kernel", ctypes.c_int32), ("start", ctypes.c_void_p), ("stop", ctypes.c_void_p)]


class Geom(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("q_per_kv", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("num_pages", ctypes.c_int64), ("timing", ctypes.POINTER(Timing))]


class TreeS(ctypes.Structure):
    _fields_ = [("num_nodes", ctypes.c_int32), ("num_tokens", ctypes.c_int64),
                ("parent", ctypes.c_void_p), ("n_full", ctypes.c_void_p),
                ("tok_off", ctypes.c_void_p), ("page_off", ctypes.c_void_p),
                ("n_kept", ctypes.c_void_p), ("page_table", ctypes.c_void_p)]


class PoolS(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("slot_pos", ctypes.c_void_p),
                ("free_stack", ctypes.c_void_p), ("free_top", ctypes.c_void_p)]


class Params(ctypes.Structure):
    _fields_ = [("alpha_max", ctypes.c_double), ("gamma", ctypes.c_double),
                ("lambda_d", ctypes.c_double), ("lambda_delta", ctypes.c_double),
                ("eta", ctypes.c_double), ("r_min", ctypes.c_double),
                ("k_min", ctypes.c_int32), ("l_tail", ctypes.c_int32),
                ("theta", ctypes.c_float * 3), ("softmax_scale", ctypes.c_float),
                ("select_mode", ctypes.c_int32), ("score_self_window", ctypes.c_int32),
                ("lazy_rehydration", ctypes.c_int32), ("n_sinks", ctypes.c_int32),
                ("k_protect", ctypes.c_int32)]


class DecodeCredit(ctypes.Structure):
    _fields_ = [("slice_layers", ctypes.POINTER(ctypes.c_int32)), ("n_slice", ctypes.c_int32),
                ("self_window", ctypes.c_int32), ("A", ctypes.c_void_p),
                ("rows_seen", ctypes.c_void_p)]


class Walk(ctypes.Structure):
    _fields_ = [("targets", ctypes.c_void_p), ("n_steps", ctypes.c_int32),
                ("budget_tokens", ctypes.c_int64), ("pressure_margin", ctypes.c_int64),
                ("q_win", ctypes.c_void_p), ("window", ctypes.c_int32),
                ("slice_layers", ctypes.POINTER(ctypes.c_int32)), ("n_slice", ctypes.c_int32),
                ("v_in", ctypes.c_void_p), ("u_in", ctypes.c_void_p), ("A", ctypes.c_void_p),
                ("rows_seen", ctypes.c_void_p), ("a_out", ctypes.c_void_p), ("s", ctypes.c_void_p),
                ("host_k", ctypes.c_void_p), ("host_v", ctypes.c_void_p), ("k", ctypes.c_void_p),
                ("delta", ctypes.c_void_p), ("on_path", ctypes.c_void_p),
                ("sel_pos", ctypes.c_void_p), ("stats", ctypes.c_void_p)]


class Sizes(ctypes.Structure):
    _fields_ = [("num_nodes", ctypes.c_int32), ("num_tokens", ctypes.c_int64),
                ("max_context", ctypes.c_int64), ("max_observers", ctypes.c_int32),
                ("window", ctypes.c_int32), ("n_slice", ctypes.c_int32),
                ("max_leaves", ctypes.c_int32), ("max_layers", ctypes.c_int32)]


_lib = None


def load() -> ctypes.CDLL:
    """The HIP library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2605_22106_amd.build`")
        lib = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        G, T, Pl, Pa = (ctypes.POINTER(Geom), ctypes.POINTER(TreeS), ctypes.POINTER(PoolS),
                        ctypes.POINTER(Params))
        sig = {
            "arbor_workspace_size": (sz, [G, ctypes.POINTER(Sizes)]),
            "arbor_strerror": (ctypes.c_char_p, [ctypes.c_int]),
            "arbor_score": (ctypes.c_int, [G, T, Pl, vp, i32, vp, i32, ctypes.POINTER(i32), i32,
                                           vp, vp, vp, vp, vp, vp, Pa, vp, vp, sz, vp]),
            "arbor_allocate": (ctypes.c_int, [T, vp, i32, i64, vp, Pa, vp, vp, vp, vp, vp, sz, vp]),
            "arbor_select": (ctypes.c_int, [G, T, Pl, vp, vp, Pa, vp, vp, vp]),
            "arbor_compact": (ctypes.c_int, [G, T, Pl, vp, vp, vp, vp, sz, vp]),
            "arbor_compact_noalloc": (ctypes.c_int, [G, T, Pl, vp, vp, vp, vp]),
            "arbor_select_compact": (ctypes.c_int, [G, T, Pl, vp, vp, Pa, vp, vp, vp, sz, vp]),
            "arbor_rehydrate": (ctypes.c_int, [G, T, Pl, vp, vp, vp, vp, vp, sz, vp]),
            "arbor_tree_decode_attn": (ctypes.c_int, [G, T, Pl, vp, i32, i32, i32, vp, vp, i32,
                                                      vp, ctypes.c_float, vp, vp, sz, vp]),
            "arbor_tree_decode_attn_scored": (ctypes.c_int,
                                              [G, T, Pl, vp, i32, i32, i32, vp, vp, i32, vp,
                                               ctypes.c_float, ctypes.POINTER(DecodeCredit), vp,
                                               vp, sz, vp]),
            "arbor_uncertainty": (ctypes.c_int, [vp, i32, i32, i64, i32, vp, vp, i32, vp, vp, sz,
                                                 vp]),
            "arbor_uncertainty_workspace_size": (sz, [i32, i64, i32]),
            "arbor_walk": (ctypes.c_int, [G, T, Pl, ctypes.POINTER(Walk), Pa, vp, vp, sz, vp]),
        }
        for name, (res, args) in sig.items():
            f = getattr(lib, name)
            f.restype = res
            f.argtypes = args
        _lib = lib
    return _lib


def exported_symbols():
    return ["arbor_workspace_size", "arbor_strerror", "arbor_score", "arbor_allocate",
            "arbor_select", "arbor_compact", "arbor_compact_noalloc", "arbor_select_compact",
            "arbor_rehydrate", "arbor_tree_decode_attn",
            "arbor_tree_decode_attn_scored", "arbor_uncertainty",
            "arbor_uncertainty_workspace_size", "arbor_walk"]


def _dev(t: torch.Tensor | None, name: str):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def params_struct(p: dict, softmax_scale: float = 0.0) -> Params:
    th = p.get("theta", (1.0, 1.0, 1.0))
    return Params(float(p.get("alpha_max", math.inf)), float(p["gamma"]), float(p["lambda_d"]),
                  float(p["lambda_delta"]), float(p["eta"]), float(p["r_min"]), int(p["k_min"]),
                  int(p["l_tail"]), (ctypes.c_float * 3)(*[float(x) for x in th]),
                  float(p.get("softmax_scale", softmax_scale)), int(p.get("select_mode", 0)),
                  int(p.get("score_self_window", 0)), int(p.get("lazy_rehydration", 1)),
                  int(p.get("n_sinks", 0)), int(p.get("k_protect", 0)))


@dataclass
class KVState:
    """Device tensors of one tree and its paged KV pool."""
    parent: torch.Tensor
    n_full: torch.Tensor
    tok_off: torch.Tensor
    page_off: torch.Tensor
    n_kept: torch.Tensor
    page_table: torch.Tensor
    k: torch.Tensor
    v: torch.Tensor
    slot_pos: torch.Tensor
    free_stack: torch.Tensor
    free_top: torch.Tensor
    layers: int
    kv_heads: int
    q_per_kv: int
    head_dim: int
    page_size: int
    dtype: int
    num_tokens: int

    @property
    def num_nodes(self) -> int:
        return int(self.parent.numel())

    @property
    def num_pages(self) -> int:
        return int(self.k.shape[1])

    def geom(self, timing: "Timing | None" = None) -> Geom:
        g = Geom(self.layers, self.kv_heads, self.q_per_kv, self.head_dim, self.page_size,
                 self.dtype, self.num_pages)
        if timing is not None:
            g.timing = ctypes.pointer(timing)
        return g

    def tree(self) -> TreeS:
        return TreeS(self.num_nodes, self.num_tokens, _dev(self.parent, "parent"),
                     _dev(self.n_full, "n_full"), _dev(self.tok_off, "tok_off"),
                     _dev(self.page_off, "page_off"), _dev(self.n_kept, "n_kept"),
                     _dev(self.page_table, "page_table"))

    def pool(self) -> PoolS:
        return PoolS(_dev(self.k, "k"), _dev(self.v, "v"), _dev(self.slot_pos, "slot_pos"),
                     _dev(self.free_stack, "free_stack"), _dev(self.free_top, "free_top"))

    def clone(self) -> "KVState":
        f = {k: (getattr(self, k).clone() if isinstance(getattr(self, k), torch.Tensor)
                 else getattr(self, k)) for k in self.__dataclass_fields__}
        return KVState(**f)

    def copy_from(self, other: "KVState") -> None:
        for k in self.__dataclass_fields__:
            a = getattr(self, k)
            if isinstance(a, torch.Tensor):
                a.copy_(getattr(other, k))


def kv_state_from(st: dict, device="cuda") -> KVState:
    """Move a generator state (see synth.build_state) to the GPU."""
    d = torch.device(device)
    dt = BF16 if st["dtype"] == "bf16" else F32
    return KVState(st["parent"].to(d), st["n_full"].to(d), st["tok_off"].to(d),
                   st["page_off"].to(d), st["n_kept"].to(d).clone(), st["page_table"].to(d).clone(),
                   st["k"].to(d).contiguous(), st["v"].to(d).contiguous(),
                   st["slot_pos"].to(d).clone(), st["free_stack"].to(d).clone(),
                   st["free_top"].to(d).clone(), st["layers"], st["kv_heads"], st["q_per_kv"],
                   st["head_dim"], st["page_size"], dt, st["num_tokens"])


def arbor_workspace_size(kv: KVState, *, max_context=None, max_observers=0, window=0, n_slice=0,
                         max_leaves=0, max_layers=0) -> int:
    g = kv.geom()
    sz = Sizes(kv.num_nodes, kv.num_tokens,
               int(max_context if max_context is not None else kv.num_tokens),
               int(max_observers), int(window), int(n_slice), int(max_leaves), int(max_layers))
    return int(load().arbor_workspace_size(ctypes.byref(g), ctypes.byref(sz)))


def arbor_strerror(code: int) -> str:
    return load().arbor_strerror(int(code)).decode()


def timing(kernel: int, start, stop) -> Timing:
    """A per-call timing request: `start` / `stop` (torch.cuda.Event with timing
    enabled) are recorded around the call's launches of `kernel`."""
    return Timing(int(kernel), ctypes.c_void_p(start.cuda_event), ctypes.c_void_p(stop.cuda_event))


def arbor_score(kv: KVState, observers, q_win, window, slice_layers, v_in, u_in, A, rows_seen,
                a_out, s_out, params: dict, status, workspace, stream=None, timing=None) -> int:
    g, t, p = kv.geom(timing), kv.tree(), kv.pool()
    pa = params_struct(params)
    sl = (ctypes.c_int32 * len(slice_layers))(*[int(x) for x in slice_layers])
    return load().arbor_score(ctypes.byref(g), ctypes.byref(t), ctypes.byref(p),
                              _dev(observers, "observers"), int(observers.numel()),
                              _dev(q_win, "q_win"), int(window), sl, len(slice_layers),
                              _dev(v_in, "v_in"), _dev(u_in, "u_in"), _dev(A, "A"),
                              _dev(rows_seen, "rows_seen"), _dev(a_out, "a_out"),
                              _dev(s_out, "s_out"), ctypes.byref(pa), _dev(status, "status"),
                              _dev(workspace, "workspace"), int(workspace.numel()),
                              _stream(stream))


def arbor_allocate(kv: KVState, active, budget, s, params: dict, k_out, delta_out, on_path_out,
                   status, workspace, stream=None) -> int:
    t = kv.tree()
    pa = params_struct(params)
    return load().arbor_allocate(ctypes.byref(t), _dev(active, "active"), int(active.numel()),
                                 int(budget), _dev(s, "s"), ctypes.byref(pa),
                                 _dev(k_out, "k_out"), _dev(delta_out, "delta_out"),
                                 _dev(on_path_out, "on_path_out"), _dev(status, "status"),
                                 _dev(workspace, "workspace"), int(workspace.numel()),
                                 _stream(stream))


def arbor_select(kv: KVState, A, k, params: dict, sel_pos, status, stream=None,
                 timing=None) -> int:
    g, t, p = kv.geom(timing), kv.tree(), kv.pool()
    pa = params_struct(params)
    return load().arbor_select(ctypes.byref(g), ctypes.byref(t), ctypes.byref(p), _dev(A, "A"),
                               _dev(k, "k"), ctypes.byref(pa), _dev(sel_pos, "sel_pos"),
                               _dev(status, "status"), _stream(stream))


def arbor_compact(kv: KVState, k, sel_pos, status, workspace, stream=None, timing=None) -> int:
    g, t, p = kv.geom(timing), kv.tree(), kv.pool()
    return load().arbor_compact(ctypes.byref(g), ctypes.byref(t), ctypes.byref(p), _dev(k, "k"),
                                _dev(sel_pos, "sel_pos"), _dev(status, "status"),
                                _dev(workspace, "workspace"), int(workspace.numel()),
                                _stream(stream))


def arbor_select_compact(kv: KVState, A, k, params: dict, sel_pos, status, workspace,
                         stream=None, timing=None) -> int:
    """arbor_select then arbor_compact on the same k, as one entry point."""
    g, t, p = kv.geom(timing), kv.tree(), kv.pool()
    pa = params_struct(params)
    return load().arbor_select_compact(ctypes.byref(g), ctypes.byref(t), ctypes.byref(p),
                                       _dev(A, "A"), _dev(k, "k"), ctypes.byref(pa),
                                       _dev(sel_pos, "sel_pos"), _dev(status, "status"),
                                       _dev(workspace, "workspace"), int(workspace.numel()),
                                       _stream(stream))


def arbor_compact_noalloc(kv: KVState, k, sel_pos, status, stream=None) -> int:
    """arbor_compact with the library's own scratch (no workspace argument)."""
    g, t, p = kv.geom(), kv.tree(), kv.pool()
    return load().arbor_compact_noalloc(ctypes.byref(g), ctypes.byref(t), ctypes.byref(p),
                                        _dev(k, "k"), _dev(sel_pos, "sel_pos"),
                                        _dev(status, "status"), _stream(stream))


def _host_or_dev(t: torch.Tensor, name: str):
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if not t.is_cuda and not t.is_pinned():
        raise ValueError(f"{name} must be pinned host memory or a GPU tensor")
    return ctypes.c_void_p(t.data_ptr())


def arbor_rehydrate(kv: KVState, on_path, host_k, host_v, status, workspace, stream=None) -> int:
    g, t, p = kv.geom(), kv.tree(), kv.pool()
    return load().arbor_rehydrate(ctypes.byref(g), ctypes.byref(t), ctypes.byref(p),
                                  _dev(on_path, "on_path"), _host_or_dev(host_k, "host_k"),
                                  _host_or_dev(host_v, "host_v"), _dev(status, "status"),
                                  _dev(workspace, "workspace"), int(workspace.numel()),
                                  _stream(stream))


def arbor_tree_decode_attn(kv: KVState, leaves, layer_begin, layer_end, q, out, lse_out,
                           softmax_scale, status, workspace, stream=None, timing=None) -> int:
    g, t, p = kv.geom(timing), kv.tree(), kv.pool()
    out_dtype = BF16 if out.dtype == torch.bfloat16 else F32
    return load().arbor_tree_decode_attn(ctypes.byref(g), ctypes.byref(t), ctypes.byref(p),
                                         _dev(leaves, "leaves"), int(leaves.numel()),
                                         int(layer_begin), int(layer_end), _dev(q, "q"),
                                         _dev(out, "out"), out_dtype, _dev(lse_out, "lse_out"),
                                         float(softmax_scale), _dev(status, "status"),
                                         _dev(workspace, "workspace"), int(workspace.numel()),
                                         _stream(stream))


def arbor_tree_decode_attn_scored(kv: KVState, leaves, layer_begin, layer_end, q, out, lse_out,
                                  softmax_scale, slice_layers, self_window, A, rows_seen, status,
                                  workspace, stream=None, timing=None) -> int:
    """arbor_tree_decode_attn plus the decode-time credit of this step's
    attention weights on the slice layers into A (fp32 [N]) and rows_seen
    (int64 [V])."""
    g, t, p = kv.geom(timing), kv.tree(), kv.pool()
    out_dtype = BF16 if out.dtype == torch.bfloat16 else F32
    sl = (ctypes.c_int32 * max(1, len(slice_layers)))(*[int(x) for x in slice_layers])
    cr = DecodeCredit(sl, len(slice_layers), int(self_window), _dev(A, "A"),
                      _dev(rows_seen, "rows_seen"))
    return load().arbor_tree_decode_attn_scored(ctypes.byref(g), ctypes.byref(t),
                                                ctypes.byref(p), _dev(leaves, "leaves"),
                                                int(leaves.numel()), int(layer_begin),
                                                int(layer_end), _dev(q, "q"), _dev(out, "out"),
                                                out_dtype, _dev(lse_out, "lse_out"),
                                                float(softmax_scale), ctypes.byref(cr),
                                                _dev(status, "status"),
                                                _dev(workspace, "workspace"),
                                                int(workspace.numel()), _stream(stream))


def arbor_walk(kv: KVState, targets, budget, params: dict, A, s, k, delta, on_path, sel_pos,
               status, workspace, host_k=None, host_v=None, pressure_margin=0, q_win=None,
               window=0, slice_layers=(), v_in=None, u_in=None, rows_seen=None, a_out=None,
               stats=None, stream=None) -> int:
    """Alg. 2's controller over the Transition events to targets[0..n) on the
    device (see include/arbor.h)."""
    g, t, p = kv.geom(), kv.tree(), kv.pool()
    pa = params_struct(params)
    sl = (ctypes.c_int32 * max(1, len(slice_layers)))(*[int(x) for x in slice_layers])
    hk = None if host_k is None else _host_or_dev(host_k, "host_k")
    hv = None if host_v is None else _host_or_dev(host_v, "host_v")
    w = Walk(_dev(targets, "targets"), int(targets.numel()), int(budget), int(pressure_margin),
             _dev(q_win, "q_win"), int(window), sl, len(slice_layers), _dev(v_in, "v_in"),
             _dev(u_in, "u_in"), _dev(A, "A"), _dev(rows_seen, "rows_seen"),
             _dev(a_out, "a_out"), _dev(s, "s"), hk, hv, _dev(k, "k"), _dev(delta, "delta"),
             _dev(on_path, "on_path"), _dev(sel_pos, "sel_pos"), _dev(stats, "stats"))
    return load().arbor_walk(ctypes.byref(g), ctypes.byref(t), ctypes.byref(p), ctypes.byref(w),
                             ctypes.byref(pa), _dev(status, "status"), _dev(workspace, "workspace"),
                             int(workspace.numel()), _stream(stream))


def arbor_uncertainty_workspace_size(n_rows: int, vocab: int, dtype: int) -> int:
    return int(load().arbor_uncertainty_workspace_size(int(n_rows), int(vocab), int(dtype)))


def arbor_uncertainty(logits, top_k, u_out, status, workspace, dst=None, stream=None) -> int:
    """u_out[dst[r]] (or u_out[r]) = 1 - H / ln(vocab) of row r of `logits`
    ([n_rows, vocab], bf16 or fp32), H over the whole row or its top_k plus one
    "other" outcome."""
    if logits.dim() != 2:
        raise ValueError("logits must be [n_rows, vocab]")
    if logits.dtype not in (torch.bfloat16, torch.float32):
        raise ValueError("logits must be bfloat16 or float32")
    dtype = BF16 if logits.dtype == torch.bfloat16 else F32
    return load().arbor_uncertainty(_dev(logits, "logits"), dtype, int(logits.shape[0]),
                                    int(logits.shape[1]), int(top_k), _dev(dst, "dst"),
                                    _dev(u_out, "u_out"), int(u_out.numel()),
                                    _dev(status, "status"), _dev(workspace, "workspace"),
                                    int(workspace.numel()), _stream(stream))
