"""ctypes binding of libbranchattn.so (argument marshalling only).

Every function here has the name of the C entry point it wraps
(include/branch_attn.h) and does nothing but convert arguments: torch
tensors become device pointers, the current torch stream becomes the
hipStream_t, host arrays become ctypes arrays.  All computation happens in
the library's HIP kernels; if the library is missing, loading fails loudly.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "_lib", "libbranchattn.so")

BA_OK = 0
BA_E_INVAL = -1
BA_E_UNSUPPORTED = -2
BA_E_HIP = -3
BA_E_WORKSPACE = -4

BA_KIND_EAGLE_CHAIN = 0
BA_KIND_DFLASH_BLOCK = 1
BA_DTYPE_BF16 = 0
BA_DTYPE_F32 = 1
BA_MODE_PER_STEP = 0
BA_MODE_FUSED = 1
BA_MODE_AUTO = 2

EXPORTED = ("zigzag_partition", "branch_attn_plan_create", "branch_attn_plan_destroy",
            "branch_attn_workspace_size", "branch_attn_plan_info", "branch_attn_useful_flops",
            "branch_attn_pair_counts", "branch_attn_last_error", "branch_attn_fwd", "branch_attn_fwd_noalloc",
            "branch_attn_bwd",
            "lse_merge", "branch_attn_plan_set_rope", "branch_attn_plan_positions", "branch_attn_qkv_fwd",
            "branch_attn_qkv_bwd", "branch_attn_qkv_workspace_size", "branch_attn_plan_mode")

c_i32 = ctypes.c_int32
c_vp = ctypes.c_void_p


class BaGroup(ctypes.Structure):
    _fields_ = [("seq", c_i32), ("anchor", c_i32), ("kind", c_i32), ("len", c_i32),
                ("row0", c_i32), ("row_stride", c_i32)]


class BaProblem(ctypes.Structure):
    _fields_ = [("num_seqs", c_i32), ("cu_seqlens", ctypes.POINTER(c_i32)),
                ("has_main", ctypes.POINTER(ctypes.c_uint8)), ("cp_size", c_i32), ("cp_rank", c_i32),
                ("hq", c_i32), ("hkv", c_i32), ("head_dim", c_i32), ("softmax_scale", ctypes.c_float),
                ("num_groups", c_i32), ("groups", ctypes.POINTER(BaGroup)), ("num_branch_rows", c_i32)]


class BaFwdIO(ctypes.Structure):
    _fields_ = [("q_main", c_vp), ("q_br", c_vp), ("k_br", c_vp), ("v_br", c_vp),
                ("k_step", ctypes.POINTER(c_vp)), ("v_step", ctypes.POINTER(c_vp)),
                ("o_main", c_vp), ("o_br", c_vp), ("lse_main", c_vp), ("lse_br", c_vp),
                ("ring_begin", c_vp), ("ring_end", c_vp)]


class BaBwdIO(ctypes.Structure):
    _fields_ = [("q_main", c_vp), ("q_br", c_vp), ("k_br", c_vp), ("v_br", c_vp),
                ("k_step", ctypes.POINTER(c_vp)), ("v_step", ctypes.POINTER(c_vp)),
                ("o_main", c_vp), ("o_br", c_vp), ("lse_main", c_vp), ("lse_br", c_vp),
                ("do_main", c_vp), ("do_br", c_vp), ("dq_main", c_vp), ("dq_br", c_vp),
                ("dk_step", ctypes.POINTER(c_vp)), ("dv_step", ctypes.POINTER(c_vp)),
                ("dk_br", c_vp), ("dv_br", c_vp), ("grad_dtype", c_i32), ("ring_begin", c_vp),
                ("ring_end", c_vp), ("kv_end", c_vp)]


class BranchAttnError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"[{code}] {msg}")
        self.code = code


_lib = None


def lib() -> ctypes.CDLL:
    """Load the library (once).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_07108_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        L.zigzag_partition.argtypes = [ctypes.POINTER(c_i32), c_i32, c_i32, c_i32, ctypes.POINTER(c_i32),
                                       ctypes.POINTER(c_i32), ctypes.POINTER(c_i32)]
        L.branch_attn_plan_create.argtypes = [ctypes.POINTER(BaProblem), ctypes.POINTER(c_vp)]
        L.branch_attn_plan_destroy.argtypes = [c_vp]
        L.branch_attn_plan_destroy.restype = None
        L.branch_attn_plan_set_rope.argtypes = [c_vp, ctypes.c_float]
        L.branch_attn_workspace_size.argtypes = [c_vp, c_i32, ctypes.POINTER(ctypes.c_size_t),
                                                 ctypes.POINTER(ctypes.c_size_t)]
        L.branch_attn_plan_mode.argtypes = [c_vp, c_i32, ctypes.POINTER(c_i32)]
        L.branch_attn_plan_info.argtypes = [c_vp, ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int64)]
        L.branch_attn_useful_flops.argtypes = [c_vp, ctypes.POINTER(ctypes.c_double),
                                               ctypes.POINTER(ctypes.c_double)]
        L.branch_attn_pair_counts.argtypes = [c_vp, ctypes.POINTER(ctypes.c_double),
                                              ctypes.POINTER(ctypes.c_double)]
        L.branch_attn_last_error.restype = ctypes.c_char_p
        L.branch_attn_fwd.argtypes = [c_vp, c_vp, c_i32, ctypes.POINTER(BaFwdIO), c_vp, ctypes.c_size_t]
        L.branch_attn_fwd_noalloc.argtypes = [c_vp, c_vp, c_i32, ctypes.POINTER(BaFwdIO)]
        L.branch_attn_bwd.argtypes = [c_vp, c_vp, c_i32, ctypes.POINTER(BaBwdIO), c_vp, ctypes.c_size_t]
        L.lse_merge.argtypes = [c_vp, ctypes.c_int64, c_i32, c_i32, c_vp, c_vp, c_vp, c_i32, c_vp]
        L.branch_attn_plan_positions.argtypes = [c_vp, ctypes.POINTER(c_i32), ctypes.POINTER(c_i32)]
        L.branch_attn_qkv_fwd.argtypes = [c_vp, ctypes.c_int64, c_i32, c_i32, c_i32, c_vp, c_vp, c_vp,
                                          ctypes.c_float, c_vp, c_vp, c_vp]
        L.branch_attn_qkv_bwd.argtypes = [c_vp, ctypes.c_int64, c_i32, c_i32, c_i32, c_vp, c_vp, c_vp,
                                          ctypes.c_float, c_vp, c_vp, c_vp, c_i32, c_vp, c_i32, c_vp, c_i32,
                                          c_vp, ctypes.c_size_t]
        L.branch_attn_qkv_workspace_size.argtypes = [ctypes.c_int64, c_i32, c_i32, ctypes.POINTER(ctypes.c_size_t)]
        _lib = L
    return _lib


def _check(rc: int):
    if rc != BA_OK:
        raise BranchAttnError(rc, lib().branch_attn_last_error().decode())


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream=None):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return c_vp(s.cuda_stream)


def _ptr_array(ts: Sequence) -> ctypes.Array:
    return (c_vp * len(ts))(*[_ptr(t) for t in ts])


# ----------------------------------------------------------------- host calls

def zigzag_partition(cu_seqlens, cp_size: int, cp_rank: int):
    """Returns (local_cu_seqlens, local_to_global, local_pos) as int32 arrays."""
    cu = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
    S = len(cu) - 1
    n_local = int(cu[-1]) // max(int(cp_size), 1) if S >= 1 else 0
    lcu = np.zeros(max(S + 1, 1), np.int32)
    l2g = np.zeros(max(n_local, 1), np.int32)
    lpos = np.zeros(max(n_local, 1), np.int32)
    P = ctypes.POINTER(c_i32)
    _check(lib().zigzag_partition(cu.ctypes.data_as(P), S, int(cp_size), int(cp_rank),
                                  lcu.ctypes.data_as(P), l2g.ctypes.data_as(P), lpos.ctypes.data_as(P)))
    return lcu, l2g[:n_local], lpos[:n_local]


class Plan:
    """Owns a ba_plan built by branch_attn_plan_create."""

    def __init__(self, cu_seqlens, has_main, cp_size, cp_rank, hq, hkv, head_dim, softmax_scale,
                 groups: np.ndarray, num_branch_rows: int):
        cu = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
        hm = np.ascontiguousarray(np.asarray(has_main, dtype=np.uint8))
        g = np.ascontiguousarray(np.asarray(groups, dtype=np.int32).reshape(-1, 6))
        garr = (BaGroup * max(len(g), 1))()
        for i, row in enumerate(g):
            garr[i] = BaGroup(*[int(x) for x in row])
        prob = BaProblem(len(cu) - 1, cu.ctypes.data_as(ctypes.POINTER(c_i32)),
                         hm.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)), int(cp_size), int(cp_rank),
                         int(hq), int(hkv), int(head_dim), float(softmax_scale), len(g), garr,
                         int(num_branch_rows))
        h = c_vp()
        _check(lib().branch_attn_plan_create(ctypes.byref(prob), ctypes.byref(h)))
        self._h = h
        self.cp_size = int(cp_size)

    @property
    def handle(self):
        return self._h

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value and _lib is not None:
            _lib.branch_attn_plan_destroy(h)
            self._h = None

    def set_rope(self, theta: float):
        """Rotary position embedding in front of the attention (theta 0: off)."""
        _check(lib().branch_attn_plan_set_rope(self._h, float(theta)))

    def positions(self, n_local: int, num_branch_rows: int):
        """(main_pos [n_local], br_pos [num_branch_rows]) int32 host arrays."""
        mp = np.zeros(max(n_local, 1), np.int32)
        bp = np.zeros(max(num_branch_rows, 1), np.int32)
        P = ctypes.POINTER(c_i32)
        _check(lib().branch_attn_plan_positions(self._h, mp.ctypes.data_as(P), bp.ctypes.data_as(P)))
        return mp[:n_local], bp[:num_branch_rows]

    def mode(self, mode: int = BA_MODE_AUTO) -> int:
        """The schedule `mode` stands for with this plan (BA_MODE_AUTO resolved)."""
        r = c_i32()
        _check(lib().branch_attn_plan_mode(self._h, int(mode), ctypes.byref(r)))
        return r.value

    def workspace_size(self, mode: int):
        f, b = ctypes.c_size_t(), ctypes.c_size_t()
        _check(lib().branch_attn_workspace_size(self._h, int(mode), ctypes.byref(f), ctypes.byref(b)))
        return f.value, b.value

    def info(self):
        n, t = ctypes.c_int64(), ctypes.c_int64()
        _check(lib().branch_attn_plan_info(self._h, ctypes.byref(n), ctypes.byref(t)))
        return n.value, t.value

    def pair_counts(self):
        m, l = ctypes.c_double(), ctypes.c_double()
        _check(lib().branch_attn_pair_counts(self._h, ctypes.byref(m), ctypes.byref(l)))
        return m.value, l.value

    def useful_flops(self):
        f, b = ctypes.c_double(), ctypes.c_double()
        _check(lib().branch_attn_useful_flops(self._h, ctypes.byref(f), ctypes.byref(b)))
        return f.value, b.value


# --------------------------------------------------------------- device calls

def branch_attn_fwd(plan: Plan, mode: int, q_main, q_br, k_br, v_br, k_step, v_step, o_main, o_br,
                    lse_main, lse_br, workspace, stream=None, ring_events=(None, None)):
    ks, vs = _ptr_array(k_step), _ptr_array(v_step)
    io = BaFwdIO(_ptr(q_main), _ptr(q_br), _ptr(k_br), _ptr(v_br), ks, vs, _ptr(o_main), _ptr(o_br),
                 _ptr(lse_main), _ptr(lse_br), ring_events[0], ring_events[1])
    _check(lib().branch_attn_fwd(_stream(stream), plan.handle, int(mode), ctypes.byref(io),
                                 _ptr(workspace), workspace.numel() * workspace.element_size()))


def branch_attn_fwd_noalloc(plan: Plan, mode: int, q_main, q_br, k_br, v_br, k_step, v_step, o_main, o_br,
                            lse_main, lse_br, stream=None):
    """branch_attn_fwd with the library's static per-GPU scratch instead of a workspace."""
    ks, vs = _ptr_array(k_step), _ptr_array(v_step)
    io = BaFwdIO(_ptr(q_main), _ptr(q_br), _ptr(k_br), _ptr(v_br), ks, vs, _ptr(o_main), _ptr(o_br),
                 _ptr(lse_main), _ptr(lse_br), None, None)
    _check(lib().branch_attn_fwd_noalloc(_stream(stream), plan.handle, int(mode), ctypes.byref(io)))


def branch_attn_bwd(plan: Plan, mode: int, q_main, q_br, k_br, v_br, k_step, v_step, o_main, o_br,
                    lse_main, lse_br, do_main, do_br, dq_main, dq_br, dk_step, dv_step, dk_br, dv_br,
                    grad_dtype: int, workspace, stream=None, ring_events=(None, None)):
    ks, vs = _ptr_array(k_step), _ptr_array(v_step)
    dks, dvs = _ptr_array(dk_step), _ptr_array(dv_step)
    io = BaBwdIO(_ptr(q_main), _ptr(q_br), _ptr(k_br), _ptr(v_br), ks, vs, _ptr(o_main), _ptr(o_br),
                 _ptr(lse_main), _ptr(lse_br), _ptr(do_main), _ptr(do_br), _ptr(dq_main), _ptr(dq_br),
                 dks, dvs, _ptr(dk_br), _ptr(dv_br), int(grad_dtype), ring_events[0], ring_events[1],
                 ring_events[2] if len(ring_events) > 2 else None)
    _check(lib().branch_attn_bwd(_stream(stream), plan.handle, int(mode), ctypes.byref(io),
                                 _ptr(workspace), workspace.numel() * workspace.element_size()))


def lse_merge(o_acc, lse_acc, o_part, lse_part, stream=None):
    """In place: (o_acc [rows, H, d] f32, lse_acc [H, rows] f32) <- merge with the partial."""
    import torch
    rows, heads, d = o_acc.shape
    dt = BA_DTYPE_BF16 if o_part.dtype == torch.bfloat16 else BA_DTYPE_F32
    _check(lib().lse_merge(_stream(stream), rows, heads, d, _ptr(o_acc), _ptr(lse_acc), _ptr(o_part), dt,
                           _ptr(lse_part)))


# ------------------------------------------------------- QKV projection

def branch_attn_qkv_workspace_size(rows: int, hq: int, hkv: int) -> int:
    n = ctypes.c_size_t()
    _check(lib().branch_attn_qkv_workspace_size(int(rows), int(hq), int(hkv), ctypes.byref(n)))
    return n.value


def branch_attn_qkv_fwd(x, w, hq: int, hkv: int, pos, theta: float, q, k, v, stream=None):
    """x [rows, hidden] bf16, w [(hq + 2 hkv) * 128, hidden] bf16, pos [rows] int32 (or None when
    theta == 0); writes q [rows, hq, 128], k and v [rows, hkv, 128] (bf16)."""
    rows, hidden = x.shape
    _check(lib().branch_attn_qkv_fwd(_stream(stream), int(rows), int(hidden), int(hq), int(hkv), _ptr(x), _ptr(w),
                                     _ptr(pos), float(theta), _ptr(q), _ptr(k), _ptr(v)))


def branch_attn_qkv_bwd(x, w, hq: int, hkv: int, pos, theta: float, dq, dk, dv, dx, dw,
                        accumulate_dw: bool, workspace, stream=None):
    """Gradients dx (dtype of the dx tensor) and dw (fp32, overwritten or accumulated) of the
    projection for dq / dk / dv of one dtype (bf16 or fp32)."""
    import torch
    rows, hidden = x.shape
    gd = BA_DTYPE_F32 if dq.dtype == torch.float32 else BA_DTYPE_BF16
    xd = BA_DTYPE_F32 if dx.dtype == torch.float32 else BA_DTYPE_BF16
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().branch_attn_qkv_bwd(_stream(stream), int(rows), int(hidden), int(hq), int(hkv), _ptr(x), _ptr(w),
                                     _ptr(pos), float(theta), _ptr(dq), _ptr(dk), _ptr(dv), gd, _ptr(dx), xd,
                                     _ptr(dw), 1 if accumulate_dw else 0, _ptr(workspace), ws_bytes))
