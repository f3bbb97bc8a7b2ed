"""Moves a synthetic call (``workloads.Call``) to the GPU: device tensors for
the packed metadata and queries, and pools filled through ``vd_kv_write``.

Pure data movement; the attention itself runs in the library's kernels."""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import torch

from . import workloads as W
from .vdattn import Batch, VdAttn


def bf16_tensor(bits: np.ndarray, device) -> torch.Tensor:
    """uint16 bf16 bit patterns (numpy) -> torch.bfloat16 on ``device``."""
    a = np.ascontiguousarray(bits, dtype=np.uint16).view(np.int16)
    return torch.from_numpy(a).to(device).view(torch.bfloat16)


def bits_of(t: torch.Tensor) -> np.ndarray:
    """torch.bfloat16 -> uint16 bit patterns (numpy, host)."""
    return t.detach().view(torch.int16).cpu().numpy().view(np.uint16)


@dataclass
class DeviceCall:
    call: W.Call
    batch: Batch

    @property
    def kv_bytes(self) -> int:
        return self.call.kv_bytes()


def clone_device_call(dc: DeviceCall) -> DeviceCall:
    """A device copy of a staged call: every tensor of its batch cloned on the
    device (pools, page table, queries, lengths, optional outputs)."""
    from dataclasses import fields, replace

    b = dc.batch
    kw = {f.name: getattr(b, f.name).clone() for f in fields(b)
          if isinstance(getattr(b, f.name), torch.Tensor)}
    return DeviceCall(dc.call, replace(b, **kw))


def handle_for(shape: W.Shape) -> VdAttn:
    return VdAttn(shape.num_q_heads, shape.num_kv_heads, shape.head_dim, shape.page_size,
                  window=shape.window)


def fill_pool(attn: VdAttn, call: W.Call, k_pool: torch.Tensor, v_pool: torch.Tensor,
              chunk_tokens: int = 1 << 16, exclude_new: bool = False):
    """Writes every valid slot of ``call`` into the pools with vd_kv_write
    (without this call's own tokens when ``exclude_new``)."""
    k, v, slots = call.write_list(exclude_new=exclude_new)
    dev = k_pool.device
    for lo in range(0, slots.shape[0], chunk_tokens):
        hi = min(lo + chunk_tokens, slots.shape[0])
        attn.kv_write(bf16_tensor(k[lo:hi], dev), bf16_tensor(v[lo:hi], dev),
                      torch.from_numpy(slots[lo:hi]).to(dev), k_pool, v_pool, call.num_pages)


def to_device(attn: VdAttn, call: W.Call, device="cuda", poison: bool = True,
              hint_extra_q: int = 0, hint_extra_ctx: int = 0, append: bool = False,
              shared_pages=None, lse: bool = False) -> DeviceCall:
    """Device copy of ``call``.  Pools start as bf16 NaN (``poison``) or zero,
    then receive every valid slot; host hints are the call's true maxima plus
    the given extras.  With ``append``, this call's own tokens are not written
    to the pool but handed to the batch (k_new, v_new: the K/V of the query
    rows), for the library to write before attention.  ``shared_pages`` is
    set when some page is read by several requests (or as given).  With
    ``lse`` the batch carries a NaN-filled [T, Hq] float32 log-sum-exp output."""
    fill = int(np.int16(np.uint16(W.BF16_QNAN).view(np.int16))) if poison else 0
    k_pool = attn.new_pool(call.num_pages, device)
    v_pool = attn.new_pool(call.num_pages, device)
    k_pool.view(torch.int16).fill_(fill)
    v_pool.view(torch.int16).fill_(fill)
    fill_pool(attn, call, k_pool, v_pool, exclude_new=append)
    extra = {}
    if append:
        kn, vn = call.query_kv()
        extra = dict(k_new=bf16_tensor(kn, device), v_new=bf16_tensor(vn, device))
    if lse:
        extra["lse"] = torch.full((call.total_q_tokens, call.shape.num_q_heads), float("nan"),
                                  dtype=torch.float32, device=device)
    batch = Batch(
        q=bf16_tensor(call.q_bits(), device),
        cu_q_lens=torch.from_numpy(call.cu_q_lens).to(device),
        context_lens=torch.from_numpy(call.context_lens).to(device),
        page_table=torch.from_numpy(np.ascontiguousarray(call.page_table)).to(device),
        k_pool=k_pool, v_pool=v_pool, num_pages=call.num_pages,
        max_q_len=max(call.max_q_len, 1) + hint_extra_q,
        max_context_len=max(call.max_context_len, 1) + hint_extra_ctx,
        shared_pages=call.shares_pages() if shared_pages is None else bool(shared_pages),
        **extra)
    return DeviceCall(call, batch)
