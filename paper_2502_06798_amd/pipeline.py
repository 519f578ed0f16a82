"""One matching step over a batch: match, assign, gather.

Holds the output and workspace buffers of a batch size so repeated steps
allocate nothing; every call goes straight to the C ABI on one stream.
"""
from __future__ import annotations

from typing import Optional, Sequence

import numpy as np
import torch

from . import binding as B


class MatchStep:
    def __init__(self, cache: B.Cache, b: int, k: int, theta: Sequence[float], K: Sequence[int],
                 inst_level: Sequence[int], inst_cap: Sequence[int],
                 inst_queue: Optional[Sequence[int]] = None, slots_per_inst: Optional[int] = None,
                 latent_bytes: int = 0, device="cuda", route: str = "rounds", resident_fallback: bool = False):
        if route not in ("rounds", "planned"):
            raise ValueError("route is 'rounds' (preference-order rounds) or 'planned' (Route-Plan quotas)")
        self.cache, self.b, self.k, self.route = cache, b, k, route
        # with resident_fallback, the level and the latent follow the best
        # neighbour whose latent is resident (apc_resident_best), not the top-1
        self.resident_fallback = resident_fallback
        self.theta = np.ascontiguousarray(theta, dtype=np.float32)
        self.K = np.ascontiguousarray(K, dtype=np.int32)
        self.inst_level = np.ascontiguousarray(inst_level, dtype=np.int32)
        self.inst_cap = np.ascontiguousarray(inst_cap, dtype=np.int32)
        self.inst_queue = None if inst_queue is None else np.ascontiguousarray(inst_queue, dtype=np.int32)
        self.n_inst = int(self.inst_level.size)
        self.spi = int(self.inst_cap.max()) if slots_per_inst is None and self.n_inst else (slots_per_inst or 0)
        i32 = dict(dtype=torch.int32, device=device)
        self.top_score = torch.empty((b, k), dtype=torch.float32, device=device)
        self.top_idx = torch.empty((b, k), **i32)
        self.ws = B.workspace_tensor(cache, b, k, device)
        self.opt_level = torch.empty(b, **i32)
        self.out_level = torch.empty(b, **i32)
        self.out_inst = torch.empty(b, **i32)
        self.out_slot = torch.empty(b, **i32)
        self.inst_fill = torch.empty(max(self.n_inst, 1), **i32)
        self.hit = torch.empty(b, **i32)
        self.res_score = torch.empty(b, dtype=torch.float32, device=device) if resident_fallback else None
        self.res_idx = torch.empty(b, **i32) if resident_fallback else None
        n_lv = self.K.size + 1
        self.plan = torch.empty(n_lv * n_lv, **i32) if route == "planned" else None
        self.latent_bytes = latent_bytes
        self.batch = (torch.empty((self.n_inst * self.spi, latent_bytes), dtype=torch.uint8, device=device)
                      if latent_bytes else None)

    def match(self, q: torch.Tensor, q_scale: Optional[torch.Tensor] = None, stream=None):
        B.apc_match_batch(self.cache, q, q_scale, self.k, self.top_score, self.top_idx, self.ws, stream)
        if self.resident_fallback:
            B.apc_resident_best(self.cache, self.top_score, self.top_idx, self.k, self.k, self.b,
                                self.res_score, self.res_idx, stream)

    def _best(self):
        """(scores, entries, row stride) that the level and the gather follow."""
        if self.resident_fallback:
            return self.res_score, self.res_idx, 1
        return self.top_score, self.top_idx, self.k

    def assign(self, stream=None):
        sc, _, ld = self._best()
        if self.route == "planned":
            B.apc_assign_planned(sc, ld, self.b, self.theta, self.K, self.inst_level,
                                 self.inst_cap, self.inst_queue, self.plan, self.opt_level, self.out_level,
                                 self.out_inst, self.out_slot, self.inst_fill, stream)
            return
        B.apc_assign(sc, ld, self.b, self.theta, self.K, self.inst_level, self.inst_cap,
                     self.inst_queue, self.opt_level, self.out_level, self.out_inst, self.out_slot,
                     self.inst_fill, stream)

    def gather(self, stream=None):
        if self.batch is None:
            return
        _, ix, ld = self._best()
        B.apc_gather_latents(self.cache, ix, ld, self.b, self.out_level, self.out_inst,
                             self.out_slot, self.n_inst, self.spi, self.batch, self.hit, stream)

    def run(self, q: torch.Tensor, q_scale: Optional[torch.Tensor] = None, stream=None):
        self.match(q, q_scale, stream)
        self.assign(stream)
        self.gather(stream)
