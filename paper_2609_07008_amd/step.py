"""One MLA-Online step on device tensors: attend -> merge -> sliced o-proj + artifact.

Holds the output and scratch buffers for a fixed geometry, segment table and
protected set, sized by the library's own size query.  Argument marshalling
and allocation only; every computation is a call into libmla_online.so.
"""
from __future__ import annotations

import numpy as np
import torch

from . import mla


class OnlineStep:
    def __init__(self, geom, segs, prot_rows, glob_head, split_keys: int, device="cuda",
                 with_part_seg: bool = True, out_dtype: int = mla.MLA_BF16):
        self.geom = geom
        self.segs = np.asarray(segs, dtype=np.int64).reshape(-1, 3)
        self.prot = np.ascontiguousarray(prot_rows, dtype=np.int32)
        self.glob_head = np.ascontiguousarray(glob_head, dtype=np.int32)
        self.split_keys = int(split_keys)
        self.n_rows = int(self.segs[:, 1].sum())
        self.n_slots, self.n_parts, ws = mla.attend_query(geom, self.segs, self.prot, self.split_keys)
        d_c = mla.head_width(geom)
        dev = torch.device(device)
        self.part_o = torch.empty((self.n_parts, d_c), dtype=torch.float32, device=dev)
        self.part_lse = torch.empty((self.n_parts,), dtype=torch.float32, device=dev)
        self.part_ptr = torch.empty((self.n_slots + 1,), dtype=torch.int64, device=dev)
        self.part_seg = (torch.empty((self.n_parts, 2), dtype=torch.int32, device=dev)
                         if with_part_seg else None)
        self.row_src = torch.empty((self.n_rows,), dtype=torch.uint8, device=dev)
        self.ws = torch.empty((max(ws, 256),), dtype=torch.uint8, device=dev)
        self.out_dtype = out_dtype
        self.out_o = torch.empty((self.n_slots, d_c),
                                 dtype=torch.bfloat16 if out_dtype == mla.MLA_BF16 else torch.float32,
                                 device=dev)
        self.out_lse = torch.empty((self.n_slots,), dtype=torch.float32, device=dev)
        self.z = torch.empty((self.n_rows, int(geom.d_model)), dtype=torch.float32, device=dev)
        self.prot_d = torch.from_numpy(self.prot.copy()).to(dev)
        G = int(geom.n_groups)
        self.n_glob_slots = self.n_rows * G

    def attend(self, kv, q_glob, q_loc, stream=None):
        mla.online_attend(self.geom, self.segs, self.prot, self.split_keys, kv, q_glob, q_loc, self.part_o,
                          self.part_lse, self.part_ptr, self.part_seg, self.row_src, self.ws, stream)

    def merge(self, stream=None):
        mla.segment_merge(self.n_slots, mla.head_width(self.geom), self.part_o, self.part_lse, self.part_ptr,
                          self.out_dtype, self.out_o, self.out_lse, stream)

    def oproj(self, w_o, z_off, stream=None):
        if self.out_dtype != mla.MLA_BF16:
            raise ValueError("the sliced o-proj consumes bf16 head outputs")
        o_glob = self.out_o[: self.n_glob_slots]
        o_loc = self.out_o[self.n_glob_slots:] if self.n_slots > self.n_glob_slots else None
        mla.sliced_oproj_add(self.geom, self.n_rows, o_glob, o_loc, self.glob_head, self.prot_d,
                             int(self.prot.shape[0]), w_o, z_off, self.z, stream)

    def run(self, kv, q_glob, q_loc, w_o, z_off, stream=None):
        self.attend(kv, q_glob, q_loc, stream)
        self.merge(stream)
        self.oproj(w_o, z_off, stream)
        return self.z


class PlannedStep:
    """The step with the protected set in device memory: the plan is built once
    for a segment table, split mode and capacity (mla_online_plan); each call then
    takes prot_rows / |A| from device tensors and only enqueues kernels
    (mla_online_attend_planned, mla_sliced_oproj_add_planned).  Buffers are sized
    for the capacity; argument marshalling and allocation only."""

    def __init__(self, geom, segs, glob_head, split_keys: int, prot_cap: int, device="cuda",
                 out_dtype: int = mla.MLA_BF16, z_dtype=torch.float32, bookkeeping: bool = True,
                 with_lse: bool = True):
        self.geom = geom
        self.segs = np.asarray(segs, dtype=np.int64).reshape(-1, 3)
        self.glob_head = np.ascontiguousarray(glob_head, dtype=np.int32)
        dev = torch.device(device)
        info = mla.plan_query(geom, self.segs, split_keys, prot_cap)
        self.plan = torch.empty((max(int(info.plan_bytes), 256),), dtype=torch.uint8, device=dev)
        self.info = mla.online_plan(geom, self.segs, split_keys, prot_cap, self.plan)
        self.ws = torch.empty((max(int(self.info.ws_bytes), 256),), dtype=torch.uint8, device=dev)
        self.n_rows = int(self.info.n_rows)
        self.n_glob_slots = self.n_rows * int(geom.n_groups)
        d_v = mla.head_width(geom)
        self.out_o = torch.empty((int(self.info.max_slots), d_v),
                                 dtype=torch.bfloat16 if out_dtype == mla.MLA_BF16 else torch.float32, device=dev)
        self.out_lse = torch.empty((int(self.info.max_slots),), dtype=torch.float32, device=dev) if with_lse else None
        self.part_ptr = (torch.empty((int(self.info.max_slots) + 1,), dtype=torch.int64, device=dev)
                         if bookkeeping else None)
        self.part_seg = (torch.empty((max(int(self.info.max_parts), 1), 2), dtype=torch.int32, device=dev)
                         if bookkeeping else None)
        self.row_src = torch.empty((self.n_rows,), dtype=torch.uint8, device=dev) if bookkeeping else None
        self.status = torch.empty((1,), dtype=torch.int32, device=dev)
        self.z = torch.empty((self.n_rows, int(geom.d_model)), dtype=z_dtype, device=dev)

    def attend(self, prot_rows, n_prot, kv, q_glob, q_loc, stream=None):
        mla.online_attend_planned(self.geom, self.info, self.plan, prot_rows, n_prot, kv, q_glob, q_loc, self.out_o,
                                  self.out_lse, self.part_ptr, self.part_seg, self.row_src, self.status, self.ws,
                                  stream)

    def oproj(self, prot_rows, n_prot, w_o, z_off, stream=None):
        if self.out_o.dtype != torch.bfloat16:
            raise ValueError("the sliced o-proj consumes bf16 head outputs")
        o_glob = self.out_o[: self.n_glob_slots]
        o_loc = self.out_o[self.n_glob_slots:] if self.out_o.shape[0] > self.n_glob_slots else None
        mla.sliced_oproj_add_planned(self.geom, self.info, o_glob, o_loc, self.glob_head, prot_rows, n_prot, w_o,
                                     z_off, self.z, stream)

    def run(self, prot_rows, n_prot, kv, q_glob, q_loc, w_o, z_off, stream=None):
        self.attend(prot_rows, n_prot, kv, q_glob, q_loc, stream)
        self.oproj(prot_rows, n_prot, w_o, z_off, stream)
        return self.z
