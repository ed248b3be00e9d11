"""Device-side setup for one planned step: pool, inputs, plan, outputs.

Product side: it uses only the binding (and torch for memory), never the
oracle.  Tests, the smoke check and the benchmark build on it.
"""

from __future__ import annotations

import numpy as np
import torch

from . import binding as B
from .workloads import POISON_BF16, Batch, HostValues


def to_device_bits(bits: np.ndarray, device="cuda") -> torch.Tensor:
    """uint16 bf16 patterns -> a bf16 tensor holding exactly those bits."""
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.to(device).view(torch.bfloat16)


def to_host_bits(t: torch.Tensor) -> np.ndarray:
    return t.detach().view(torch.int16).cpu().numpy().view(np.uint16)


class DeviceStep:
    """One batch resident on the GPU.

    The pool is poisoned with a NaN pattern, then the pages a step owns are
    written; slots that the step's append fills stay poisoned until
    ``append`` runs.  Pages of agents listed in ``host_resident`` are kept
    out of the pool and placed in a pinned host page store instead, to be
    brought in by ``gather_evicted``.
    """

    def __init__(self, batch: Batch, hv: HostValues, device="cuda", mode=B.PFX_MODE_MIXED,
                 host_resident=(), decode_workers=0, piece_steps=0, poison=True, decode_engine=B.PFX_DECODE_MFMA):
        self.batch = batch
        self.device = device
        n, hkv, d = batch.num_pages, batch.num_kv_heads, batch.head_dim
        shape = (n, hkv, 16, d)
        self.k_pool = torch.empty(shape, dtype=torch.bfloat16, device=device)
        self.v_pool = torch.empty(shape, dtype=torch.bfloat16, device=device)
        if poison:
            self.k_pool.view(torch.int16).fill_(POISON_BF16)
            self.v_pool.view(torch.int16).fill_(POISON_BF16)
        # Split the generated pages into pool-resident and host-resident ones.
        host_pages = set()
        for a in host_resident:
            host_pages.update(int(p) for p in batch.prefix_pages[a])
        keep = np.array([int(p) not in host_pages for p in hv.pages], bool)
        self._write_pages(hv.pages[keep], hv.k_pages[keep], hv.v_pages[keep])
        self.host_store = None
        if host_pages:
            idx = np.nonzero(~keep)[0]
            self.host_dst = hv.pages[idx].astype(np.int32)           # pool page each store page belongs to
            self.host_src = np.arange(len(idx), dtype=np.int32)
            hk = torch.empty((len(idx), hkv, 16, d), dtype=torch.bfloat16, pin_memory=True)
            hvv = torch.empty_like(hk, pin_memory=True)
            hk.view(torch.int16).copy_(torch.from_numpy(hv.k_pages[idx].view(np.int16)))
            hvv.view(torch.int16).copy_(torch.from_numpy(hv.v_pages[idx].view(np.int16)))
            self.host_store = (hk, hvv)
            self.host_pool = B.make_pool(len(idx), hkv, d, hk, hvv)
            self.copy_ws = torch.empty(B.pfx_page_copy_workspace_bytes(len(idx)) + 256, dtype=torch.uint8,
                                       device=device)
        self.q = to_device_bits(hv.q, device)
        self.k_new = to_device_bits(hv.k_new, device)
        self.v_new = to_device_bits(hv.v_new, device)
        t = batch.num_tokens
        self.o = torch.empty((t, batch.num_q_heads, d), dtype=torch.bfloat16, device=device)
        self.lse = torch.empty((t, batch.num_q_heads), dtype=torch.float32, device=device)
        self.pool = B.make_pool(n, hkv, d, self.k_pool, self.v_pool)
        self.plan = B.plan_from_batch(self.pool, batch, mode, decode_workers=decode_workers,
                                      piece_steps=piece_steps, decode_engine=decode_engine).upload(device=device)

    def _write_pages(self, pages, kp, vp, chunk=4096):
        for s in range(0, len(pages), chunk):
            idx = torch.from_numpy(np.asarray(pages[s:s + chunk], np.int64)).to(self.device)
            self.k_pool.view(torch.int16).index_copy_(0, idx, torch.from_numpy(kp[s:s + chunk].view(np.int16)).to(self.device))
            self.v_pool.view(torch.int16).index_copy_(0, idx, torch.from_numpy(vp[s:s + chunk].view(np.int16)).to(self.device))

    def gather_evicted(self):
        """Bring host-resident prefix pages into their pool pages (prefix movement)."""
        if self.host_store is None:
            return
        B.pfx_page_copy(self.pool, self.host_pool, self.host_dst, self.host_src, self.copy_ws)

    def append(self):
        B.pfx_append_kv(self.pool, self.plan, self.k_new, self.v_new)

    def attention(self, sm_scale=0.0):
        B.pfx_attention(self.pool, self.plan, self.q, self.o, self.lse, sm_scale)

    def step(self):
        self.append()
        self.attention()

    def read_pages(self, pages):
        idx = torch.from_numpy(np.asarray(pages, np.int64)).to(self.device)
        k = self.k_pool.view(torch.int16).index_select(0, idx).cpu().numpy().view(np.uint16)
        v = self.v_pool.view(torch.int16).index_select(0, idx).cpu().numpy().view(np.uint16)
        return k, v

    def outputs(self):
        return to_host_bits(self.o), self.lse.detach().cpu().numpy()
