"""Drive a synthetic workload through the C ABI on one GPU.

Setup (untimed): replay the workload's scenario on the library's block
manager (new / append / fork), write every appended token's K and V into the
device pools through ``spork_kv_write`` (running ``spork_kv_copy`` first when
an append reports a copy-on-write), build each step's plan and upload its
image. ``Step.run()`` then issues exactly one hot-path call. Marshalling only:
every number is computed by the library's kernels.
"""

import numpy as np
import torch

from . import spork
from .synth import BF16

_TORCH_DTYPE = {BF16: torch.bfloat16, "f32": torch.float32}
_SPORK_DTYPE = {BF16: spork.SPORK_DTYPE_BF16, "f32": spork.SPORK_DTYPE_F32}


def to_device(arr, dtype, device):
    """Host storage array (uint16 bf16 bits or float32) -> device tensor of ``dtype``."""
    if dtype == BF16:
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).to(device)


class Step:
    """One planned call of the hot path with its device buffers."""

    def __init__(self, dw, index):
        wl = dw.wl
        st = wl.steps[index]
        dev = dw.device
        self.index = index
        self.spec = st
        self.plan = spork.spork_plan_create(dw.cache, dw.shape, st.seqs, st.n_rows, st.groups, dw.n_cu)
        self.info = spork.spork_plan_get_info(self.plan)
        image = spork.spork_plan_image(self.plan)
        self.image = torch.from_numpy(image).to(dev)
        rows = sum(st.n_rows)
        td = _TORCH_DTYPE[wl.dtype]
        self.q = to_device(st.q, wl.dtype, dev)
        self.out = torch.empty((rows, wl.hq, wl.d), dtype=td, device=dev)
        self.lse = torch.empty((rows, wl.hq), dtype=torch.float32, device=dev)
        att_ws = (self.info["workspace_bytes"] + 255) // 256 * 256
        self.verify = st.verify_k > 0
        acc_ws = 0
        if self.verify:
            self.n_verify = st.drafts.shape[0]
            self.vocab = st.logits.shape[1]
            acc_ws = spork.spork_verify_workspace_bytes(self.n_verify, st.verify_k, self.vocab)
            self.logits = to_device(st.logits, wl.logits_dtype, dev)
            self.drafts = torch.from_numpy(st.drafts).to(dev)
            self.accept_len = torch.full((self.n_verify,), -1, dtype=torch.int32, device=dev)
            self.next_token = torch.full((self.n_verify,), -1, dtype=torch.int32, device=dev)
            self.argmax = torch.full((self.n_verify * (st.verify_k + 1),), -1, dtype=torch.int32, device=dev)
        self.workspace = torch.empty(max(att_ws + acc_ws, 256), dtype=torch.uint8, device=dev)
        spork.spork_workspace_clear(self.plan, self.workspace)
        self.dw = dw

    def poison(self):
        """Fill outputs and workspace with NaN / -1 so unwritten values show
        (the workspace's control words are then zeroed again, as a call
        requires)."""
        self.out.fill_(float("nan"))
        self.lse.fill_(float("nan"))
        self.workspace.fill_(0xFF)
        spork.spork_workspace_clear(self.plan, self.workspace)
        if self.verify:
            self.accept_len.fill_(-1)
            self.next_token.fill_(-1)
            self.argmax.fill_(-1)

    def run(self, stream=None, attention=True):
        dw = self.dw
        if self.verify:
            spork.spork_verify_accept(self.plan if attention else None, self.image, self.q, dw.k_pool,
                                      dw.v_pool, self.out, self.lse, self.logits,
                                      _SPORK_DTYPE[dw.wl.logits_dtype], self.vocab, self.drafts,
                                      self.n_verify, self.spec.verify_k, self.accept_len,
                                      self.next_token, self.argmax, self.workspace, stream)
        else:
            spork.spork_attn_decode(self.plan, self.image, self.q, dw.k_pool, dw.v_pool, self.out,
                                    self.lse, self.workspace, stream)

    def close(self):
        if self.plan is not None:
            spork.spork_plan_destroy(self.plan)
            self.plan = None


class DeviceWorkload:
    """A workload's pools and block manager on one GPU."""

    def __init__(self, wl, device="cuda:0", n_cu=0, poison_pool=True):
        self.wl = wl
        self.device = torch.device(device)
        self.n_cu = n_cu
        self.shape = spork.make_shape(wl.hq, wl.hkv, wl.d, wl.block_size, _SPORK_DTYPE[wl.dtype],
                                      wl.sm_scale)
        self.cache = spork.spork_cache_create(wl.num_blocks, wl.block_size, wl.free_order)
        td = _TORCH_DTYPE[wl.dtype]
        nb, h, bs, d = wl.num_blocks, wl.hkv, wl.block_size, wl.d
        self.k_pool = torch.empty((nb, h, bs, d), dtype=td, device=self.device)
        self.v_pool = torch.empty((nb, h, d, bs), dtype=td, device=self.device)
        if poison_pool:  # unwritten slots hold NaN: reading one would show in the results
            self.k_pool.fill_(float("nan"))
            self.v_pool.fill_(float("nan"))
        self.bad_slots = torch.zeros(1, dtype=torch.int32, device=self.device)
        self.written = {}
        self.steps = []

    def apply(self, ops):
        wl = self.wl
        for op in ops:
            if op[0] == "new":
                sid = spork.spork_seq_new(self.cache)
                assert sid == op[1], (sid, op)
                self.written[sid] = 0
            elif op[0] == "fork":
                sid = spork.spork_fork(self.cache, op[1])
                assert sid == op[2], (sid, op)
                self.written[sid] = self.written[op[1]]
            elif op[0] == "append":
                seq, n = op[1], op[2]
                slots, cow = spork.spork_seq_append(self.cache, seq, n)
                for src, dst, nv in cow:
                    spork.spork_kv_copy(self.shape, self.k_pool, self.v_pool, wl.num_blocks, src, dst, nv)
                k, v = wl.context(seq)
                lo = self.written[seq]
                kd = to_device(k[lo:lo + n], wl.dtype, self.device)
                vd = to_device(v[lo:lo + n], wl.dtype, self.device)
                sd = torch.from_numpy(slots).to(self.device)
                spork.spork_kv_write(self.shape, self.k_pool, self.v_pool, wl.num_blocks, sd, kd, vd,
                                     self.bad_slots)
                self.written[seq] = lo + n
            elif op[0] == "free":
                spork.spork_seq_free(self.cache, op[1])
            else:
                raise ValueError(op)

    def prepare(self, index):
        """Apply the scenario up to step ``index`` and plan that step."""
        self.apply(self.wl.steps[index].ops_before)
        step = Step(self, index)
        self.steps.append(step)
        return step

    def advance(self, step, index):
        """Apply the scenario up to step ``index`` and reuse ``step``'s plan
        for it (spork_plan_advance patches the device image); the step's
        query rows take step ``index``'s Q. Returns the same Step object."""
        st = self.wl.steps[index]
        self.apply(st.ops_before)
        spork.spork_plan_advance(step.plan, self.cache, step.image)
        step.q.copy_(to_device(st.q, self.wl.dtype, self.device))
        step.index = index
        step.spec = st
        step.info = spork.spork_plan_get_info(step.plan)
        return step

    def prepare_all(self):
        return [self.prepare(i) for i in range(len(self.wl.steps))]

    def close(self):
        for s in self.steps:
            s.close()
        if self.cache is not None:
            spork.spork_cache_destroy(self.cache)
            self.cache = None

