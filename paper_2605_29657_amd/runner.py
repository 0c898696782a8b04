"""Device staging for one stage of a batch: tensors in HBM, outputs, workspace, calls.

Plumbing only (no arithmetic of the method): it copies a
:class:`~paper_2605_29657_amd.synth.StageBatch` to the GPU once, builds the
``occam_problem`` and the row-tensor descriptors, allocates worst-case output
buffers and the workspace, and calls :func:`occam.prune` (or the unfused
entry points) on them.
"""
from __future__ import annotations

import numpy as np
import torch

from . import occam
from .synth import StageBatch


def to_device(a: np.ndarray, dtype: str, device="cuda") -> torch.Tensor:
    """Host array -> device tensor with the same bytes (bf16 bits become torch.bfloat16)."""
    if dtype == "bf16" and a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def _i32(x, device):
    return torch.as_tensor(np.asarray(x, dtype=np.int32), device=device)


class DeviceStage:
    """One stage of a batch resident in HBM, ready for the library's calls.

    ``ragged``: pass device offsets (True) or the uniform shape (False); defaults to
    whether the batch actually is ragged.  ``row_offsets`` (ragged only): False passes the
    key offsets alone, with the uniform row count, for batches whose samples all have the
    same number of anchor rows; None or True passes both.
    """

    def __init__(self, sb: StageBatch, device="cuda", ragged=None, payload=True,
                 softmax_scale: float = 0.0, max_cands=None, row_offsets=None):
        self.sb = sb
        self.device = device
        self.ragged = sb.ragged if ragged is None else bool(ragged)
        if sb.ragged and not self.ragged:
            raise ValueError("a ragged batch needs device offsets (ragged=True)")
        self.q = to_device(sb.q, sb.dtype, device)
        self.k = to_device(sb.k, sb.dtype, device)
        self.total_keys = int(sb.k_off[-1])
        self.total_cands = int(sb.N.sum())
        # The mutual-scoring stage reduces every key by the mean over its anchor rows.
        rr = occam.ROWS_MEAN if sb.stage == "mut" else occam.ROWS_MAX
        if self.ragged:
            if row_offsets is False and np.any(sb.T != sb.T[0]):
                raise ValueError("row_offsets=False needs the same row count in every sample")
            self.q_off = None if row_offsets is False else _i32(sb.q_off, device)
            self.k_off = _i32(sb.k_off, device)
            self.problem = occam.Problem(sb.B, sb.H, sb.Hkv, sb.d, sb.R, rows=int(sb.T[0]),
                                         q_offsets=self.q_off,
                                         key_offsets=self.k_off, max_rows=int(sb.T.max()),
                                         max_cands=int(sb.N.max()) if max_cands is None
                                         else int(max_cands), dtype=sb.dtype,
                                         softmax_scale=softmax_scale, visual_row_reduce=rr)
        else:
            self.q_off = self.k_off = None
            self.problem = occam.Problem(sb.B, sb.H, sb.Hkv, sb.d, sb.R, rows=int(sb.T[0]),
                                         cands=int(sb.N[0]), dtype=sb.dtype,
                                         softmax_scale=softmax_scale, visual_row_reduce=rr)
        self.ws = occam.workspace(self.problem, device)
        self.out = occam.prune_outputs(sb.B, self.total_cands, self.total_keys, device)
        self.rows = []
        self.row_src, self.row_dst = [], []
        if payload:
            for pl in sb.payload:
                if pl.name == "k_rows":
                    src = self.k.view(self.k.shape[0], -1)
                else:
                    src = to_device(pl.rows, sb.dtype, device)
                dst = torch.zeros((max(self.total_cands, 1), src.shape[1]), dtype=src.dtype,
                                  device=device)
                self.row_src.append(src)
                self.row_dst.append(dst)
                self.rows.append(occam.Rows(src, dst, src_pad_rows=pl.pad_rows, src_row0=pl.row0))

    def prune(self, lam: float, reduce: int = occam.REG_MEAN, with_rows: bool = True,
              with_scores: bool = True, row_lse=None, index_map=None, stream=None):
        o = self.out
        occam.prune(self.problem, self.q, self.k, lam, o["kept_idx"], o["kept_count"],
                    o["kept_offsets"], self.ws, reduce=reduce,
                    rows=self.rows if with_rows else None,
                    scores=o["scores"] if with_scores else None, tau=o["tau"],
                    row_lse=row_lse, index_map=index_map, stream=stream)

    def host(self, with_rows: bool = True) -> dict:
        """Copy the outputs back (synchronises the device)."""
        torch.cuda.synchronize()
        o = {k: v.cpu().numpy() for k, v in self.out.items()}
        total = int(o["kept_offsets"][-1])
        res = dict(scores=o["scores"][:self.total_keys], tau=o["tau"], kept_count=o["kept_count"],
                   kept_offsets=o["kept_offsets"], kept_idx=o["kept_idx"][:total])
        if with_rows:
            rows = []
            for dst in self.row_dst:
                a = dst[:total].cpu()
                if a.dtype == torch.bfloat16:
                    a = a.view(torch.int16)
                rows.append(a.numpy().view(np.uint16) if a.dtype == torch.int16 else a.numpy())
            res["rows"] = rows
        return res
