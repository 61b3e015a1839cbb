"""ctypes binding of libmla_online.so (argument marshalling only).

Every step runs in the HIP library; PyTorch supplies device memory and the
stream.  Importing this module loads the library and raises if it is missing
or cannot be loaded: there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch  # loads the HIP runtime the library binds to

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmla_online.so")

MLA_OK = 0
MLA_BF16, MLA_F32 = 0, 1
STATUS = {0: "MLA_OK", 1: "MLA_ERR_NULL", 2: "MLA_ERR_SHAPE", 3: "MLA_ERR_UNSUPPORTED",
          4: "MLA_ERR_SEGMENTS", 5: "MLA_ERR_ROWS", 6: "MLA_ERR_WORKSPACE", 7: "MLA_ERR_HIP"}
EXPORTS = ("mla_online_attend_query", "mla_online_attend", "mla_segment_merge", "mla_sliced_oproj_add",
           "mla_online_plan_query", "mla_online_plan", "mla_online_attend_planned",
           "mla_online_attend_planned_noalloc", "mla_sliced_oproj_add_planned",
           "mla_offline_produce_query", "mla_offline_produce", "mla_protected_rows_query", "mla_protected_rows",
           "mla_protected_rows_planned_query", "mla_protected_rows_planned",
           "mla_moe_fanout", "mla_shared_wb", "mla_probe_mfma_bf16", "mla_status_str", "mla_last_error_detail",
           "mla_version")


class MlaError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(f"{STATUS.get(status, status)}: {detail}")
        self.status = status
        self.detail = detail


class Geom(ctypes.Structure):
    _fields_ = [("n_heads", ctypes.c_int32), ("n_groups", ctypes.c_int32), ("d_latent", ctypes.c_int32),
                ("d_rope", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_proj_groups", ctypes.c_int32),
                ("softmax_scale", ctypes.c_float), ("rope_base", ctypes.c_double), ("value_rope", ctypes.c_int32)]


class Segment(ctypes.Structure):
    _fields_ = [("kv_start", ctypes.c_int64), ("length", ctypes.c_int64), ("req_offset", ctypes.c_int64)]


class PlanInfo(ctypes.Structure):
    """mla_plan_info: host description of a plan built by mla_online_plan."""
    _fields_ = [("geom", Geom), ("n_rows", ctypes.c_int64), ("split_keys", ctypes.c_int64),
                ("max_slots", ctypes.c_int64), ("max_parts", ctypes.c_int64), ("n_segs", ctypes.c_int32),
                ("prot_cap", ctypes.c_int32), ("max_items", ctypes.c_int32), ("one_chunk", ctypes.c_int32),
                ("plan_bytes", ctypes.c_size_t), ("ws_bytes", ctypes.c_size_t), ("layout", ctypes.c_int64 * 24),
                ("check", ctypes.c_uint64)]


class ProtectCfg(ctypes.Structure):
    _fields_ = [("query_seg", ctypes.c_int32), ("edge_rows", ctypes.c_int32), ("tail_rows", ctypes.c_int64),
                ("budget", ctypes.c_double)]


def _load(path: str = LIB_PATH):
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built; run `python -m paper_2609_07008_amd.build`")
    lib = ctypes.CDLL(path)
    P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    GP, SP = ctypes.POINTER(Geom), ctypes.POINTER(Segment)
    lib.mla_online_attend_query.argtypes = [GP, SP, I32, P, I32, I64, ctypes.POINTER(I64), ctypes.POINTER(I64),
                                            ctypes.POINTER(SZ)]
    lib.mla_online_attend.argtypes = [GP, SP, I32, P, I32, I64, P, P, P, P, P, P, P, P, P, SZ, P]
    lib.mla_segment_merge.argtypes = [I64, I32, P, P, P, I32, P, P, P]
    lib.mla_sliced_oproj_add.argtypes = [GP, I64, P, P, P, P, I32, P, P, P, P]
    IP = ctypes.POINTER(PlanInfo)
    lib.mla_online_plan_query.argtypes = [GP, SP, I32, I64, I32, IP]
    lib.mla_online_plan.argtypes = [GP, SP, I32, I64, I32, IP, P, SZ, P]
    lib.mla_online_attend_planned.argtypes = [GP, IP, P, P, P, P, P, P, I32, P, P, P, P, P, P, P, SZ, P]
    lib.mla_online_attend_planned_noalloc.argtypes = [GP, IP, P, P, P, P, P, P, I32, P, P, P, P, P, P, P]
    lib.mla_sliced_oproj_add_planned.argtypes = [GP, IP, P, P, P, P, P, P, P, I32, P, P]
    lib.mla_offline_produce_query.argtypes = [GP, SP, I32, ctypes.POINTER(SZ)]
    lib.mla_offline_produce.argtypes = [GP, SP, I32, P, P, P, P, I32, P, P, SZ, P]
    lib.mla_protected_rows_query.argtypes = [SP, I32, ctypes.POINTER(SZ)]
    lib.mla_protected_rows.argtypes = [SP, I32, ctypes.POINTER(ProtectCfg), P, P, P, P, P, SZ, P]
    lib.mla_protected_rows_planned_query.argtypes = [IP, ctypes.POINTER(SZ)]
    lib.mla_protected_rows_planned.argtypes = [IP, P, ctypes.POINTER(ProtectCfg), P, P, P, P, P, SZ, P]
    lib.mla_moe_fanout.argtypes = [I64, I32, P, I32, I32, ctypes.c_float, P, P, P, P, P]
    lib.mla_shared_wb.argtypes = [I64, I32, I32, P, P, I32, P, P]
    lib.mla_probe_mfma_bf16.argtypes = [I32, ctypes.POINTER(ctypes.c_double), P, P]
    for f in ("mla_online_attend_query", "mla_online_attend", "mla_segment_merge", "mla_sliced_oproj_add",
              "mla_online_plan_query", "mla_online_plan", "mla_online_attend_planned",
              "mla_online_attend_planned_noalloc", "mla_sliced_oproj_add_planned", "mla_offline_produce_query",
              "mla_offline_produce", "mla_protected_rows_query", "mla_protected_rows",
              "mla_protected_rows_planned_query", "mla_protected_rows_planned", "mla_moe_fanout", "mla_shared_wb",
              "mla_probe_mfma_bf16"):
        getattr(lib, f).restype = ctypes.c_int
    lib.mla_status_str.argtypes = [ctypes.c_int]
    lib.mla_status_str.restype = ctypes.c_char_p
    lib.mla_last_error_detail.argtypes = []
    lib.mla_last_error_detail.restype = ctypes.c_char_p
    lib.mla_version.restype = ctypes.c_char_p
    return lib


LIB = _load()


def _check(status: int):
    if status != MLA_OK:
        raise MlaError(status, LIB.mla_last_error_detail().decode())


def make_geom(g) -> Geom:
    """Geometry from any object with the fields of mla_geom."""
    return Geom(int(g.n_heads), int(g.n_groups), int(g.d_latent), int(g.d_rope), int(g.d_model),
                int(g.n_proj_groups), float(g.softmax_scale), float(g.rope_base),
                int(bool(getattr(g, "value_rope", False))))


def head_width(g) -> int:
    """d_v: width of one head output (d_c, or d_c + d_r with a rotary value)."""
    return int(g.d_latent) + (int(g.d_rope) if getattr(g, "value_rope", False) else 0)


def make_segments(segs) -> ctypes.Array:
    segs = np.asarray(segs, dtype=np.int64).reshape(-1, 3)
    arr = (Segment * max(1, segs.shape[0]))()
    for i, (ks, ln, ro) in enumerate(segs):
        arr[i] = Segment(int(ks), int(ln), int(ro))
    return arr, int(segs.shape[0])


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, torch.Tensor):
        return ctypes.c_void_p(t.data_ptr())
    if isinstance(t, np.ndarray):
        return t.ctypes.data_as(ctypes.c_void_p)
    return ctypes.c_void_p(int(t))


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def attend_query(geom, segs, prot_rows, split_keys: int):
    """Host-only size query: (n_slots, n_parts, workspace bytes)."""
    g = make_geom(geom)
    sarr, ns = make_segments(segs)
    prot = np.ascontiguousarray(prot_rows, dtype=np.int32)
    n_slots, n_parts, ws = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_size_t()
    _check(LIB.mla_online_attend_query(ctypes.byref(g), sarr, ns, _ptr(prot), int(prot.shape[0]),
                                       int(split_keys), ctypes.byref(n_slots), ctypes.byref(n_parts),
                                       ctypes.byref(ws)))
    return n_slots.value, n_parts.value, ws.value


def online_attend(geom, segs, prot_rows, split_keys, kv, q_glob, q_loc, part_o, part_lse, part_ptr,
                  part_seg, row_src, workspace, stream=None):
    """Relocation + segment-wise attention (mla_online_attend).  Device tensors in,
    device tensors out; prot_rows is a host int32 array."""
    g = make_geom(geom)
    sarr, ns = make_segments(segs)
    prot = np.ascontiguousarray(prot_rows, dtype=np.int32)
    _check(LIB.mla_online_attend(ctypes.byref(g), sarr, ns, _ptr(prot), int(prot.shape[0]), int(split_keys),
                                 _ptr(kv), _ptr(q_glob), _ptr(q_loc), _ptr(part_o), _ptr(part_lse),
                                 _ptr(part_ptr), _ptr(part_seg), _ptr(row_src), _ptr(workspace),
                                 workspace.numel() * workspace.element_size(), _stream(stream)))


def segment_merge(n_slots, d_latent, part_o, part_lse, part_ptr, out_dtype, out_o, out_lse, stream=None):
    _check(LIB.mla_segment_merge(int(n_slots), int(d_latent), _ptr(part_o), _ptr(part_lse), _ptr(part_ptr),
                                 int(out_dtype), _ptr(out_o), _ptr(out_lse), _stream(stream)))


def sliced_oproj_add(geom, n_rows, o_glob, o_loc, glob_head, prot_rows_d, n_prot, w_o, z_off, z, stream=None):
    g = make_geom(geom)
    gh = np.ascontiguousarray(glob_head, dtype=np.int32)
    _check(LIB.mla_sliced_oproj_add(ctypes.byref(g), int(n_rows), _ptr(o_glob), _ptr(o_loc), _ptr(gh),
                                    _ptr(prot_rows_d), int(n_prot), _ptr(w_o), _ptr(z_off), _ptr(z),
                                    _stream(stream)))


def plan_query(geom, segs, split_keys: int, prot_cap: int) -> PlanInfo:
    """Host-only: the PlanInfo (sizes and bounds) of a plan."""
    g = make_geom(geom)
    sarr, ns = make_segments(segs)
    info = PlanInfo()
    _check(LIB.mla_online_plan_query(ctypes.byref(g), sarr, ns, int(split_keys), int(prot_cap), ctypes.byref(info)))
    return info


def online_plan(geom, segs, split_keys: int, prot_cap: int, plan, stream=None) -> PlanInfo:
    """mla_online_plan: writes the plan image into the device tensor `plan` and
    returns its PlanInfo."""
    g = make_geom(geom)
    sarr, ns = make_segments(segs)
    info = PlanInfo()
    _check(LIB.mla_online_plan(ctypes.byref(g), sarr, ns, int(split_keys), int(prot_cap), ctypes.byref(info),
                               _ptr(plan), plan.numel() * plan.element_size(), _stream(stream)))
    return info


def online_attend_planned(geom, info, plan, prot_rows, n_prot, kv, q_glob, q_loc, out_o, out_lse=None,
                          part_ptr=None, part_seg=None, row_src=None, status=None, workspace=None, stream=None):
    """mla_online_attend_planned: every argument a device tensor (prot_rows int32,
    n_prot int32 [1]); out_o bfloat16 or float32 [info.max_slots, d_v]."""
    g = make_geom(geom)
    out = MLA_BF16 if out_o.dtype == torch.bfloat16 else MLA_F32
    _check(LIB.mla_online_attend_planned(ctypes.byref(g), ctypes.byref(info), _ptr(plan), _ptr(prot_rows),
                                         _ptr(n_prot), _ptr(kv), _ptr(q_glob), _ptr(q_loc), out, _ptr(out_o),
                                         _ptr(out_lse), _ptr(part_ptr), _ptr(part_seg), _ptr(row_src), _ptr(status),
                                         _ptr(workspace), workspace.numel() * workspace.element_size(),
                                         _stream(stream)))


NOALLOC_SCRATCH_BYTES = 16 << 20   # MLA_NOALLOC_SCRATCH_BYTES


def online_attend_planned_noalloc(geom, info, plan, prot_rows, n_prot, kv, q_glob, q_loc, out_o, out_lse=None,
                                  part_ptr=None, part_seg=None, row_src=None, status=None, stream=None):
    """mla_online_attend_planned_noalloc: as online_attend_planned, with the
    library's per-GPU scratch array in place of a workspace (nothing allocated)."""
    g = make_geom(geom)
    out = MLA_BF16 if out_o.dtype == torch.bfloat16 else MLA_F32
    _check(LIB.mla_online_attend_planned_noalloc(ctypes.byref(g), ctypes.byref(info), _ptr(plan), _ptr(prot_rows),
                                                 _ptr(n_prot), _ptr(kv), _ptr(q_glob), _ptr(q_loc), out, _ptr(out_o),
                                                 _ptr(out_lse), _ptr(part_ptr), _ptr(part_seg), _ptr(row_src),
                                                 _ptr(status), _stream(stream)))


def sliced_oproj_add_planned(geom, info, o_glob, o_loc, glob_head, prot_rows, n_prot, w_o, z_off, z, stream=None):
    """mla_sliced_oproj_add_planned: |A| from the device tensor n_prot; z float32
    or bfloat16."""
    g = make_geom(geom)
    gh = np.ascontiguousarray(glob_head, dtype=np.int32)
    zt = MLA_BF16 if z.dtype == torch.bfloat16 else MLA_F32
    _check(LIB.mla_sliced_oproj_add_planned(ctypes.byref(g), ctypes.byref(info), _ptr(o_glob), _ptr(o_loc), _ptr(gh),
                                            _ptr(prot_rows), _ptr(n_prot), _ptr(w_o), _ptr(z_off), zt, _ptr(z),
                                            _stream(stream)))


def offline_produce_query(geom, segs) -> int:
    """Host-only: workspace bytes of mla_offline_produce."""
    g = make_geom(geom)
    sarr, ns = make_segments(segs)
    ws = ctypes.c_size_t()
    _check(LIB.mla_offline_produce_query(ctypes.byref(g), sarr, ns, ctypes.byref(ws)))
    return ws.value


def offline_produce(geom, segs, kv, q_loc, glob_head, w_o, out_dtype, z_off, workspace, stream=None):
    """MLA-Off producer (mla_offline_produce): the Local-head artifact z_off of
    every row.  Device tensors in and out; segs and glob_head are host arrays."""
    g = make_geom(geom)
    sarr, ns = make_segments(segs)
    gh = np.ascontiguousarray(glob_head, dtype=np.int32)
    _check(LIB.mla_offline_produce(ctypes.byref(g), sarr, ns, _ptr(kv), _ptr(q_loc), _ptr(gh), _ptr(w_o),
                                   int(out_dtype), _ptr(z_off), _ptr(workspace),
                                   workspace.numel() * workspace.element_size(), _stream(stream)))


def protected_rows_query(segs) -> int:
    """Host-only: workspace bytes of mla_protected_rows."""
    sarr, ns = make_segments(segs)
    ws = ctypes.c_size_t()
    _check(LIB.mla_protected_rows_query(sarr, ns, ctypes.byref(ws)))
    return ws.value


def protected_rows(segs, query_seg, edge_rows, tail_rows, budget, row_flags, scores, prot_rows, n_prot,
                   workspace, stream=None):
    """The protected token-row set (mla_protected_rows) into the device tensors
    prot_rows [N] int32 and n_prot [1] int32; row_flags and scores are device
    tensors or None."""
    sarr, ns = make_segments(segs)
    cfg = ProtectCfg(int(query_seg), int(edge_rows), int(tail_rows), float(budget))
    _check(LIB.mla_protected_rows(sarr, ns, ctypes.byref(cfg), _ptr(row_flags), _ptr(scores), _ptr(prot_rows),
                                  _ptr(n_prot), _ptr(workspace), workspace.numel() * workspace.element_size(),
                                  _stream(stream)))


def protected_rows_planned_query(info) -> int:
    """Host-only: workspace bytes of mla_protected_rows_planned."""
    ws = ctypes.c_size_t()
    _check(LIB.mla_protected_rows_planned_query(ctypes.byref(info), ctypes.byref(ws)))
    return ws.value


def protected_rows_planned(info, plan, query_seg, edge_rows, tail_rows, budget, row_flags, scores, prot_rows, n_prot,
                           workspace, stream=None):
    """mla_protected_rows_planned: the protected set with the segment table taken
    from the plan image; kernels only."""
    cfg = ProtectCfg(int(query_seg), int(edge_rows), int(tail_rows), float(budget))
    _check(LIB.mla_protected_rows_planned(ctypes.byref(info), _ptr(plan), ctypes.byref(cfg), _ptr(row_flags),
                                          _ptr(scores), _ptr(prot_rows), _ptr(n_prot), _ptr(workspace),
                                          workspace.numel() * workspace.element_size(), _stream(stream)))


def moe_fanout(router, tau, expert_idx, expert_w, fanout, expert_count=None, top_k: int = 6, min_k: int = 3,
               stream=None):
    """Adaptive MoE fanout (mla_moe_fanout) of the device tensor router [N, E]
    float32 into expert_idx [N, top_k] int32, expert_w [N, top_k] float32,
    fanout [N] int32 and, if given, expert_count [E] int32."""
    n, e = (int(router.shape[0]), int(router.shape[1])) if router is not None else (0, 0)
    _check(LIB.mla_moe_fanout(n, e, _ptr(router), int(top_k), int(min_k), float(tau), _ptr(expert_idx),
                              _ptr(expert_w), _ptr(fanout), _ptr(expert_count), _stream(stream)))


def shared_wb(z, w_b, y, stream=None):
    """y = W_b z (mla_shared_wb): z [N, d_in] bf16 and w_b [d_out, d_in] bf16 device
    tensors, y [N, d_out] float32 or bfloat16."""
    n, d_in = int(z.shape[0]), int(z.shape[1])
    d_out = int(w_b.shape[0])
    out = MLA_BF16 if y.dtype == torch.bfloat16 else MLA_F32
    _check(LIB.mla_shared_wb(n, d_in, d_out, _ptr(z), _ptr(w_b), out, _ptr(y), _stream(stream)))


def probe_mfma_bf16(iters, sink, stream=None) -> float:
    """Enqueue the matrix-core rate probe (mla_probe_mfma_bf16, a diagnostic of
    mla_probe.h) with `iters` products per chain; sink is a device tensor of at
    least 4 bytes.  Returns the launch's flop; time it with events on `stream`."""
    flop = ctypes.c_double(0.0)
    _check(LIB.mla_probe_mfma_bf16(int(iters), ctypes.byref(flop), _ptr(sink), _stream(stream)))
    return flop.value


def version() -> str:
    return LIB.mla_version().decode()
