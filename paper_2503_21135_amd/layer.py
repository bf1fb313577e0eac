"""A packed mixed-precision MoE layer resident in device memory, and the
route -> expert FFN -> combine pipeline over it.

Layout in HBM (all torch-allocated, 256-byte aligned by the caching
allocator), per weight kind (gate, up, down):
  codes      int32 words, expert after expert (routed 0..E-1, then shared),
             each expert's rows row-major in the packed layout of moe_quant.h,
             expert starts rounded up to 16 bytes
  sz         {fp16 scale, fp16 zero} words, group-major per expert
  copy_*     resident copies of the channel cache in the 8-bit code format,
             one row per slot (8-bit codes of the original rows at load time,
             b-bit codes after a requantization)
  cache16    the retained original channels as binary16, one row per slot
             (uploaded on first requantization)
  row_slot   int32 [E][R] switch table
Plus order_gu [E][d_ff] and order_dn [E][d_model] (visiting orders rebuilt by
the switch) and a staging buffer for the host slot list.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, Optional

import numpy as np
import torch

from . import api
from ._lib import KIND_DOWN, KindDesc, LayerDesc, MoEError


def _u32_to_i32(a: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(a).view(np.int32)


@dataclass
class Buffers:
    """Per-batch-size device buffers of the pipeline (allocated once)."""

    T: int
    topk_ids: torch.Tensor
    topk_w: torch.Tensor
    offsets: torch.Tensor
    perm: torch.Tensor
    inv: torch.Tensor
    route_ws: torch.Tensor
    o: torch.Tensor
    ffn_ws: torch.Tensor
    y: torch.Tensor
    n_split: int


class MoELayer:
    """Packs a layer's fp32 expert weights on the GPU with moe_quant_pack and
    runs the hot path through the C ABI."""

    def __init__(self, inputs, device: str = "cuda", keep_status: bool = True):
        cfg = inputs.cfg
        self.cfg = cfg
        self.inputs = inputs
        self.device = torch.device(device)
        dev = self.device
        E, S, g = cfg.n_experts, cfg.n_shared, cfg.group
        self.E, self.S, self.k = E, S, cfg.top_k
        self.bits_host = np.ascontiguousarray(inputs.bits, np.int32)
        self.bits = torch.tensor(self.bits_host, dtype=torch.int32, device=dev)
        self.router = torch.tensor(inputs.router, dtype=torch.float32, device=dev)
        self.status = torch.zeros(1, dtype=torch.int32, device=dev)
        self.ffn_status = torch.zeros(1, dtype=torch.int32, device=dev)
        self._keep = []            # host arrays the descriptor points into
        self.kinds = []
        desc = LayerDesc()
        desc.n_experts, desc.n_shared = E, S
        desc.d_model, desc.d_ff = cfg.d_model, cfg.d_ff
        desc.d_ff_shared = cfg.d_ff_shared if S > 0 else 0
        desc.group = g
        desc.bits_host = self.bits_host.ctypes.data
        desc.bits = self.bits.data_ptr()
        max_slots = 0
        for kind in range(3):
            kd = self._pack_kind(kind)
            self.kinds.append(kd)
            max_slots = max(max_slots, kd["n_slots"])
            K = desc.kind[kind]
            K.codes = kd["codes"].data_ptr()
            K.sz = kd["sz"].data_ptr()
            K.code_off = kd["code_off"].data_ptr()
            K.sz_off = kd["sz_off"].data_ptr()
            K.code_off_host = kd["code_off_host"].ctypes.data
            K.n_slots = kd["n_slots"]
            K.copy_codes = kd["copy_codes"].data_ptr()
            K.copy_sz = kd["copy_sz"].data_ptr()
            K.copy_hdr = kd["copy_hdr"].data_ptr()
            K.copy_hdr_host = kd["copy_hdr_host"].ctypes.data
            K.row_slot = kd["row_slot"].data_ptr()
        self.order_gu = torch.empty(E * cfg.d_ff, dtype=torch.int32, device=dev)
        self.order_dn = torch.empty(E * cfg.d_model, dtype=torch.int32, device=dev)
        self.class_cnt = torch.empty(8 * E, dtype=torch.int32, device=dev)
        self.staging = torch.empty(max_slots + 1, dtype=torch.int32, device=dev)
        desc.order_gu = self.order_gu.data_ptr()
        desc.order_dn = self.order_dn.data_ptr()
        desc.class_cnt = self.class_cnt.data_ptr()
        desc.staging = self.staging.data_ptr()
        self.desc = desc
        api.moe_set_channel_switch(desc, -1, None)
        torch.cuda.synchronize(dev)
        if keep_status and int(self.status.item()) != 0:
            raise MoEError("moe_quant_pack reported status %d" % int(self.status.item()))
        self._bufs: Dict[int, Buffers] = {}
        self.cache16: Dict[int, torch.Tensor] = {}
        # precision of each routed expert's copies per kind: 0 = the 8-bit
        # copies made at load time, b > 0 = requantized at b bits
        self.copy_bits = {kind: np.zeros(E, np.int32) for kind in range(3)}

    # ------------------------------------------------------------------ packing
    def _pack_kind(self, kind: int) -> dict:
        cfg, inp, dev = self.cfg, self.inputs, self.device
        E, S, g = cfg.n_experts, cfg.n_shared, cfg.group
        code_off, sz_off = [], []
        cw = sw = 0
        for e in range(E + S):
            R, K, b = cfg.rows(kind, e), cfg.cols(kind, e), int(self.bits_host[e])
            code_off.append(cw)
            sz_off.append(sw)
            cw += (R * api.moe_code_row_words(K, b) + 3) // 4 * 4
            sw += R * (K // g)
        codes = torch.empty(max(cw, 4), dtype=torch.int32, device=dev)
        sz = torch.empty(max(sw, 1), dtype=torch.int32, device=dev)
        hdr = np.ascontiguousarray(inp.copy_headers(kind), np.int32).reshape(-1, 2)
        n_slots = hdr.shape[0]
        Kr = cfg.cols(kind, 0)
        crw = api.moe_code_row_words(Kr, 8)
        copy_codes = torch.empty(max(n_slots * crw, 4), dtype=torch.int32, device=dev)
        copy_sz = torch.empty(max(n_slots * (Kr // g), 1), dtype=torch.int32, device=dev)
        for e in range(E + S):
            R, K, b = cfg.rows(kind, e), cfg.cols(kind, e), int(self.bits_host[e])
            w = torch.from_numpy(inp.weight(e, kind)).to(dev)
            api.moe_quant_pack(w, b, g, codes[code_off[e]:], sz[sz_off[e]:], n=R,
                               ld_codes=api.moe_code_row_words(K, b), sz_row_stride=1,
                               sz_group_stride=R,
                               status=self.status)
            if e < E and n_slots:
                sl = np.nonzero(hdr[:, 0] == e)[0]
                if len(sl):
                    s0, s1 = int(sl[0]), int(sl[-1]) + 1
                    if s1 - s0 != len(sl):
                        raise MoEError("copy headers must be grouped by expert")
                    rows = torch.tensor(hdr[s0:s1, 1], dtype=torch.int32, device=dev)
                    api.moe_quant_pack(w, 8, g, copy_codes[s0 * crw:],
                                       copy_sz[s0 * (K // g):], rows=rows, ld_codes=crw,
                                       sz_row_stride=K // g, sz_group_stride=1,
                                       status=self.status)
            del w
        R0 = cfg.rows(kind, 0)
        code_off_host = np.asarray(code_off, np.int64)
        return dict(
            codes=codes, sz=sz,
            code_off=torch.tensor(code_off_host, dtype=torch.int64, device=dev),
            sz_off=torch.tensor(np.asarray(sz_off, np.int64), dtype=torch.int64, device=dev),
            code_off_host=code_off_host, sz_off_host=np.asarray(sz_off, np.int64),
            n_slots=n_slots, copy_codes=copy_codes, copy_sz=copy_sz,
            copy_hdr=torch.tensor(hdr.ravel(), dtype=torch.int32, device=dev),
            copy_hdr_host=np.ascontiguousarray(hdr.ravel()),
            row_slot=torch.empty(E * R0, dtype=torch.int32, device=dev))

    # ------------------------------------------------------------------ switch
    def set_switch(self, kind: int, slots_on: Optional[np.ndarray]) -> None:
        api.moe_set_channel_switch(self.desc, kind, slots_on)

    def set_epoch(self, epoch: int = 0) -> None:
        """Install the copy-pool mask of a mask epoch for all three kinds."""
        for kind in range(3):
            self.set_switch(kind, self.inputs.slots_on(kind, epoch))

    def reset_switch(self) -> None:
        api.moe_set_channel_switch(self.desc, -1, None)

    # ------------------------------------------------------------ requantization
    def channel_cache(self, kind: int) -> torch.Tensor:
        """Device float16 [n_slots][K]: the retained original channels of one
        kind in slot order (kept in device memory, Sec. V-A)."""
        if kind not in self.cache16:
            c16 = np.ascontiguousarray(self.inputs.channel_cache(kind))
            n, K = self.kinds[kind]["n_slots"], self.cfg.cols(kind, 0)
            if c16.shape != (n, K):
                raise MoEError("channel cache of kind %d has shape %s" % (kind, c16.shape))
            self.cache16[kind] = torch.from_numpy(c16.view(np.float16)).to(self.device)
        return self.cache16[kind]

    def requant(self, kind: int, expert_bits, stream=None) -> None:
        """Requantize the cached channels of one kind at each expert's new
        precision (0 = leave the expert's copies), Sec. IV-B."""
        eb = np.ascontiguousarray(expert_bits, np.int32)
        api.moe_requant_channels(self.desc, kind, self.channel_cache(kind), eb,
                                 status=self.status, stream=stream)
        self.copy_bits[kind] = np.where(eb > 0, eb, self.copy_bits[kind]).astype(np.int32)

    def switch_dataset(self, expert_bits, epoch: int = 0, stream=None) -> None:
        """Dynamic switch for a new dataset: requantize every kind's cached
        channels at the new per-expert precisions and install the copy-pool
        mask of `epoch`."""
        for kind in range(3):
            self.requant(kind, expert_bits, stream)
        for kind in range(3):
            api.moe_set_channel_switch(self.desc, kind, self.inputs.slots_on(kind, epoch),
                                       stream)

    # ------------------------------------------------------------------ forward
    def buffers(self, T: int) -> Buffers:
        if T in self._bufs:
            return self._bufs[T]
        dev, E, S, k, d = self.device, self.E, self.S, self.k, self.cfg.d_model
        n_split, ffn_bytes = api.moe_ffn_plan(self.desc, T, k)
        rb = api.moe_route_workspace_bytes(T, E, k, S)
        rows = T * (k + S)
        b = Buffers(
            T=T,
            topk_ids=torch.empty(T, k, dtype=torch.int32, device=dev),
            topk_w=torch.empty(T, k, dtype=torch.float32, device=dev),
            offsets=torch.empty(E + S + 1, dtype=torch.int32, device=dev),
            perm=torch.empty(max(rows, 1), dtype=torch.int32, device=dev),
            inv=torch.empty(T, k + S, dtype=torch.int32, device=dev),
            route_ws=torch.empty(max(rb, 256), dtype=torch.uint8, device=dev),
            o=torch.empty(n_split, max(rows, 1), d, dtype=torch.float32, device=dev),
            ffn_ws=torch.empty(max(ffn_bytes, 256), dtype=torch.uint8, device=dev),
            y=torch.empty(T, d, dtype=torch.float32, device=dev),
            n_split=n_split)
        self._bufs[T] = b
        return b

    def route(self, x: torch.Tensor, bias: Optional[torch.Tensor] = None, stream=None) -> Buffers:
        b = self.buffers(x.shape[0])
        api.moe_route_permute(x, self.router, bias, self.k, self.S, b.topk_ids, b.topk_w,
                              b.offsets, b.perm, b.inv, b.route_ws, stream=stream)
        return b

    def ffn(self, x: torch.Tensor, b: Buffers, stream=None) -> None:
        api.moe_expert_ffn_mixed(self.desc, x, self.k, b.offsets, b.perm, b.o, b.ffn_ws,
                                 status=self.ffn_status, stream=stream)

    def ffn_status_value(self) -> int:
        """The FFN's device status word (0, or MOE_ERR_RANGE once the fp16
        operand path has met a value beyond fp16's range); reads it back."""
        return int(self.ffn_status.item())

    def clear_ffn_status(self) -> None:
        self.ffn_status.zero_()

    def combine(self, b: Buffers, stream=None) -> torch.Tensor:
        api.moe_unpermute_combine(b.o, b.n_split, b.inv, b.topk_w, self.k, self.S, b.y,
                                  stream=stream)
        return b.y

    def forward(self, x: torch.Tensor, bias: Optional[torch.Tensor] = None,
                stream=None) -> torch.Tensor:
        """x bf16 [T][d_model] on the device -> y fp32 [T][d_model]."""
        if x.dtype != torch.bfloat16 or not x.is_cuda or not x.is_contiguous():
            raise MoEError("x must be a contiguous bfloat16 device tensor")
        b = self.route(x, bias, stream)
        self.ffn(x, b, stream)
        return self.combine(b, stream)

    # ------------------------------------------------------------------ readback
    def packed_expert(self, kind: int, e: int):
        """(codes uint32 [R][K*b/32], sz uint32 [K/g][R]) of one expert, on the host."""
        cfg, kd = self.cfg, self.kinds[kind]
        R, K, b, g = cfg.rows(kind, e), cfg.cols(kind, e), int(self.bits_host[e]), cfg.group
        o = int(kd["code_off_host"][e])
        so = int(kd["sz_off_host"][e])
        rw = api.moe_code_row_words(K, b)
        codes = kd["codes"][o:o + R * rw].cpu().numpy().view(np.uint32).reshape(R, rw)[:, :K * b // 32]
        sz = kd["sz"][so:so + R * (K // g)].cpu().numpy().view(np.uint32).reshape(K // g, R)
        return codes, sz

    def packed_copies(self, kind: int):
        kd, cfg = self.kinds[kind], self.cfg
        K, g, n = cfg.cols(kind, 0), cfg.group, kd["n_slots"]
        rw = api.moe_code_row_words(K, 8)
        codes = kd["copy_codes"][:n * rw].cpu().numpy().view(np.uint32).reshape(n, rw)[:, :K // 4]
        sz = kd["copy_sz"][:n * (K // g)].cpu().numpy().view(np.uint32).reshape(n, K // g)
        return codes, sz

    def row_slot(self, kind: int) -> np.ndarray:
        R = self.cfg.rows(kind, 0)
        return self.kinds[kind]["row_slot"].cpu().numpy().reshape(self.E, R)

    def packed_bytes(self) -> int:
        """Bytes of base codes and {scale, zero} words of every expert."""
        tot = 0
        for kind in range(3):
            for e in range(self.E + self.S):
                R, K = self.cfg.rows(kind, e), self.cfg.cols(kind, e)
                tot += R * K * int(self.bits_host[e]) // 8 + R * (K // self.cfg.group) * 4
        return tot
