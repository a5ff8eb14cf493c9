"""One transfer of a batch through the C ABI, with its device buffers.

``TransferPath`` owns (as torch tensors) everything the four calls of the
path need -- the character spans on the device, the alignment table, the
packed maps, the receiver cache and the workspaces -- and ``step()`` runs the
path once: ``hf_build_alignment`` -> ``hf_build_layer_map`` ->
``hf_transfer_kv`` (with ``layer_map="neighbor3"``: ``hf_build_layer_taps`` ->
``hf_transfer_kv_taps``).  It does no arithmetic of the method itself.
"""

from __future__ import annotations

from typing import Optional

import numpy as np

from . import heterofold as hf


class TransferPath:
    def __init__(self, seg, S, A, bias, rope: Optional[dict], L_r: int, H_r: int,
                 mode: str = "overlap", R=None, pack_stream=None, layer_map: str = "interp2",
                 opts: Optional[dict] = None, staged: Optional[bool] = None):
        import torch

        if layer_map not in ("interp2", "neighbor3"):
            raise ValueError(f"layer map {layer_map!r} unknown")
        self.torch = torch
        self.layer_mode = layer_map
        self.opts = opts
        dev = S.device
        self.seg = seg
        self.mode = mode
        self.S = S
        self.L_s = int(S.shape[1])
        self.L_r = int(L_r)
        self.H_r = int(H_r)
        self.d_h = int(S.shape[5])
        self.bias = bias
        self.rope = None if rope is None else dict(rope)
        if self.rope is not None:
            B = seg.batch
            if self.rope.get("pos0_s") is None:
                self.rope["pos0_s"] = np.zeros(B, np.int32)
            if self.rope.get("pos0_r") is None:
                self.rope["pos0_r"] = np.zeros(B, np.int32)
        as_dev = lambda a: torch.as_tensor(np.ascontiguousarray(a, np.int32), device=dev)  # noqa: E731
        self.s_beg, self.s_end = as_dev(seg.s_beg), as_dev(seg.s_end)
        self.r_beg, self.r_end = as_dev(seg.r_beg), as_dev(seg.r_end)
        self.s_len, self.r_len = seg.s_len, seg.r_len
        cap = hf.hf_alignment_nnz_capacity(seg.s_len, seg.r_len, mode)
        nR = int(seg.r_cu[-1])
        self.alignment = hf.Alignment(
            torch.zeros(nR + 1, dtype=torch.int32, device=dev),
            torch.zeros(max(cap, 1), dtype=torch.int32, device=dev),
            torch.zeros(max(cap, 1), dtype=torch.int32, device=dev),
            torch.zeros(max(nR, 1), dtype=torch.int32, device=dev), seg.s_cu, seg.r_cu)
        self.align_ws = torch.empty(max(hf.hf_alignment_workspace_bytes(seg.r_cu), 16),
                                    dtype=torch.uint8, device=dev)
        self.A_packed = hf.hf_pack_maps(A, stream=pack_stream)
        if R is None:
            T_cap_r = max(1, int(self.r_len.max()) if self.r_len.size else 1)
            R = torch.zeros((seg.batch, self.L_r, 2, self.H_r, T_cap_r, self.d_h), dtype=S.dtype,
                            device=dev)
        self.R = R
        # The library takes its staged path when the workspace holds its slabs.
        # staged=None picks the faster path as measured at 32K on one MI355X:
        # staged for concatenated taps, fused for the interpolating map.
        wsb = hf.hf_transfer_workspace_bytes(self.s_len, self.r_len, S, R, self.rope)
        if staged is None:
            staged = layer_map == "neighbor3" and hf.hf_transfer_staged_workspace_bytes(
                self.s_len, self.r_len, S, R, self.rope, 3) > 0
        self.staged = bool(staged)  # the path the library takes for this batch
        if staged:
            n_taps = 3 if layer_map == "neighbor3" else 0
            st = hf.hf_transfer_staged_workspace_bytes(self.s_len, self.r_len, S, R, self.rope,
                                                       n_taps)
            if st == 0:
                raise ValueError("the staged path does not serve this shape")
            wsb = max(wsb, st)
        self.transfer_ws = torch.empty(max(wsb, 256), dtype=torch.uint8, device=dev)
        self.layer_map = None

    def build_alignment(self, stream=None):
        return hf.hf_build_alignment(self.seg.s_cu, self.seg.r_cu, self.s_beg, self.s_end,
                                     self.r_beg, self.r_end, self.mode, out=self.alignment,
                                     workspace=self.align_ws, stream=stream)

    def build_layer_map(self):
        if self.layer_mode == "neighbor3":
            self.layer_map = hf.hf_build_layer_taps(self.L_s, self.L_r)
        else:
            self.layer_map = hf.hf_build_layer_map(self.L_s, self.L_r)
        return self.layer_map

    def transfer(self, stream=None):
        if self.layer_mode == "neighbor3":
            return hf.hf_transfer_kv_taps(self.s_len, self.r_len, self.alignment, self.layer_map,
                                          self.S, self.R, self.A_packed, self.bias, self.rope,
                                          workspace=self.transfer_ws, stream=stream,
                                          opts=self.opts)
        return hf.hf_transfer_kv(self.s_len, self.r_len, self.alignment, self.layer_map, self.S,
                                 self.R, self.A_packed, self.bias, self.rope,
                                 workspace=self.transfer_ws, stream=stream, opts=self.opts)

    def step(self, stream=None):
        """One pass of the whole path (asynchronous on the stream)."""
        self.build_alignment(stream)
        self.build_layer_map()
        self.transfer(stream)
        return self.R
