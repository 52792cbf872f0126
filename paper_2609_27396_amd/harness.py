"""Device-side setup of one DPara round for tests, the smoke check and the benchmark.

Uploads a drafter's weights and one round's synthetic inputs to HBM, prefills
the context cache through ``dpara_ctx_append`` and exposes the four calls of a
round on preallocated output tensors.  Marshalling only: all computation runs
in libdpara's kernels.
"""
from __future__ import annotations

import numpy as np
import torch

from . import dpara as D
from .synth import RoundInputs


def round_up(x: int, m: int) -> int:
    return (x + m - 1) // m * m


class DeviceRound:
    def __init__(self, shape, weights: dict, ri: RoundInputs, ctx_cap: int | None = None, device="cuda",
                 drafter: D.DeviceDrafter | None = None):
        self.shape = shape
        self.ri = ri
        self.dev = device
        self.d = drafter if drafter is not None else D.DeviceDrafter(shape, weights, device)
        B, g, H, V = len(ri.ctx_lens), shape.gamma, shape.hidden, shape.vocab
        self.B = B
        need = int(max(ri.ctx_lens)) + 2 * (g + 1)
        self.ctx_cap = ctx_cap or max(64, round_up(need, 64))
        self.ctx = D.DeviceContext(shape, B, self.ctx_cap, device)
        self.ws = D.Workspace(self.d.cfg, B, self.ctx_cap, device)
        mdt = self.d.mat_dtype
        i32 = dict(dtype=torch.int32, device=device)
        self.spine = torch.from_numpy(ri.spine.astype(np.int32)).to(device)
        ldt = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
        self.logits = torch.from_numpy(ri.target_logits).to(device=device, dtype=ldt)
        self.new_feats = torch.from_numpy(ri.new_feats).to(device=device, dtype=mdt)
        self.reps = torch.empty((B, g + 1, g, H), dtype=torch.float32, device=device)
        self.accept = torch.empty(B, **i32)
        self.bonus = torch.empty(B, **i32)
        self.targmax = torch.empty((B, g + 1), **i32)
        self.gathered = torch.empty((B, g, H), dtype=torch.float32, device=device)
        self.drafts = torch.empty((B, g), **i32)
        self.next_spine = torch.empty((B, g + 1), **i32)
        self.margins = torch.empty((B, g), dtype=torch.float32, device=device)
        D.dpara_clear_status(self.ws.ptr, D._stream(None))
        self.prefill()

    def prefill(self):
        """Fill the cache with the round's context features (positions 0..n_b-1)."""
        B, H = self.B, self.shape.hidden
        n_max = int(max(self.ri.ctx_lens))
        self.ctx.ctx_len.zero_()
        if n_max == 0:
            return
        feats = torch.zeros((B, n_max, H), dtype=self.d.mat_dtype, device=self.dev)
        for b, f in enumerate(self.ri.ctx_feats):
            if f.shape[0]:
                feats[b, :f.shape[0]] = torch.from_numpy(f).to(device=self.dev, dtype=self.d.mat_dtype)
        n_new = torch.from_numpy(self.ri.ctx_lens.astype(np.int32)).to(self.dev)
        D.ctx_append(self.d, self.ctx, feats, n_new, self.ws)
        torch.cuda.synchronize()
        del feats

    def append(self, n_new, feats=None, stream=None):
        feats = self.new_feats if feats is None else feats
        D.ctx_append(self.d, self.ctx, feats, n_new, self.ws, stream)

    def backbone(self, stream=None):
        D.backbone_all_boundaries(self.d, self.ctx, self.spine, self.reps, self.ws, stream)

    def verify(self, stream=None):
        D.verify_greedy(self.d, self.logits, self.spine, self.accept, self.bonus, self.targmax, self.ws, stream)

    def head(self, stream=None):
        D.select_and_head(self.d, self.reps, self.accept, self.bonus, self.gathered, self.drafts,
                          self.next_spine, self.margins, self.ws, stream)

    def head_sampled(self, temperature: float, seed: int, scores=None, stream=None):
        D.select_and_head_sampled(self.d, self.reps, self.accept, self.bonus, self.gathered, self.drafts,
                                  self.next_spine, self.margins, temperature, seed, scores, self.ws, stream)

    def verify_sampled(self, scores, temperature: float, seed: int, stream=None):
        D.verify_sampled(self.d, self.logits, scores, self.spine, temperature, seed, self.accept, self.bonus,
                         self.ws, stream)

    def candidates(self, stream=None):
        """Every branch row's head candidates (the off-serial-path head variant)."""
        if getattr(self, "cand", None) is None:
            self.cand = D.branch_candidates_buffer(self.d, self.B)
        D.branch_candidates(self.d, self.reps, self.cand, self.ws, stream)

    def head_cand(self, stream=None):
        D.select_and_head_cand(self.d, self.reps, self.cand, self.accept, self.bonus, self.gathered, self.drafts,
                               self.next_spine, self.margins, self.ws, stream)

    def status(self) -> int:
        torch.cuda.synchronize()
        return self.ws.status()

    def head_fallback(self) -> int:
        """Nonzero if the last head call needed the full head (a step the pruned head could not prove)."""
        torch.cuda.synchronize()
        return self.ws.head_fallback()


def upload_cache(ctx, k, v, ctx_lens, dtype):
    """Write host K/V (k[l][b], v[l][b]: [n_b, n_kv, hd]) into a DeviceContext and set ctx_len."""
    for l in range(len(k)):
        for b, n in enumerate(ctx_lens):
            n = int(n)
            if n == 0:
                continue
            ctx.k[l, b, :, :n, :] = torch.from_numpy(k[l][b]).to(dtype=dtype).permute(1, 0, 2).cuda()
            ctx.v[l, b, :, :, :n] = torch.from_numpy(v[l][b]).to(dtype=dtype).permute(1, 2, 0).cuda()
    ctx.ctx_len[:len(ctx_lens)] = torch.tensor(np.asarray(ctx_lens, np.int32)).cuda()
