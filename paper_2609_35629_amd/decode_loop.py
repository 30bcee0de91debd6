"""A multi-layer decode loop over the library: per layer a team table of the
prompt and a growing exact suffix (the paragraph "Cache state and budget"
and Alg. "SANTA++ attention for one query head": the generated rows
E = {N+1, .., N+t} are attended exactly, and E is empty at the first sparse
prediction).

Each step decodes every layer with the suffix rows generated so far, then
appends the step's new key/value row of each (b, kv) to that layer's suffix
cache.  The caches, tables and workspaces are allocated once, for the loop's
capacity; a step allocates nothing on the device beyond what the caller's
row copies need.
"""
from __future__ import annotations

from typing import List, Optional, Sequence

import torch

from . import Teams, build_teams, decode, decode_workspace, dense_decode, dense_workspace


class LayerCache:
    """One layer: its team table (or, for the dense baseline, its prompt
    K/V) and its suffix cache [B, Hkv, capacity, d] of which the first T rows
    are filled."""

    def __init__(self, K: torch.Tensor, V: torch.Tensor, capacity: int, Hq: int, budget: int,
                 P: int, R: int, dense: bool = False):
        B, Hkv, N, d = K.shape
        self.B, self.Hkv, self.N, self.d, self.Hq = B, Hkv, N, d, Hq
        self.capacity = capacity
        self.budget = budget
        self.dense = dense
        self.T = 0
        self.sK = torch.zeros((B, Hkv, capacity, d), dtype=K.dtype, device=K.device)
        self.sV = torch.zeros_like(self.sK)
        self.out = torch.empty((B, Hq, d), dtype=torch.float32, device=K.device)
        if dense:
            self.K, self.V = K, V
            self.teams = None
            self.ws = dense_workspace(B, Hq, Hkv, N, capacity, d)
        else:
            self.teams: Optional[Teams] = build_teams(K, V, P, R)
            self.ws = decode_workspace(self.teams, Hq, capacity, budget)

    def attend(self, q: torch.Tensor, seed: int, step: int, scale: float = 0.0, debug=None) -> torch.Tensor:
        """The layer's attention output for queries q [B, Hq, d] over the
        prompt (sampled, or dense) and the T suffix rows generated so far."""
        if self.dense:
            return dense_decode(q, self.K, self.V, self.sK, self.sV, scale=scale, out=self.out, workspace=self.ws,
                                T=self.T)
        return decode(self.teams, q, self.sK, self.sV, self.budget, seed=seed, step=step, scale=scale,
                      out=self.out, workspace=self.ws, debug=debug, T=self.T)

    def append(self, k: torch.Tensor, v: torch.Tensor) -> None:
        """Append one generated row per (b, kv): k, v [B, Hkv, d]."""
        if self.T >= self.capacity:
            raise ValueError(f"suffix cache full ({self.capacity} rows)")
        self.sK[:, :, self.T].copy_(k)
        self.sV[:, :, self.T].copy_(v)
        self.T += 1

    def close(self) -> None:
        if self.teams is not None:
            self.teams.close()
            self.teams = None


class DecodeLoop:
    """Layers decoded in order at every step; layer l draws its sampling
    noise with seed `seed + l` (each layer's noise stream is its own)."""

    def __init__(self, prompts: Sequence[tuple], capacity: int, Hq: int, budget: int, P: int, R: int,
                 seed: int = 0, dense: bool = False):
        self.layers: List[LayerCache] = [LayerCache(K, V, capacity, Hq, budget, P, R, dense) for K, V in prompts]
        self.seed = seed
        self.step_id = 0

    def step(self, qs: Sequence[torch.Tensor], ks: Sequence[torch.Tensor], vs: Sequence[torch.Tensor],
             scale: float = 0.0, debugs=None) -> List[torch.Tensor]:
        """One decode step: layer l attends with qs[l], then appends ks[l],
        vs[l].  Returns each layer's output (views of the layer's buffer,
        valid until the next step)."""
        outs = []
        for li, layer in enumerate(self.layers):
            dbg = debugs[li] if debugs is not None else None
            outs.append(layer.attend(qs[li], self.seed + li, self.step_id, scale, dbg))
            layer.append(ks[li], vs[li])
        self.step_id += 1
        return outs

    def close(self) -> None:
        for layer in self.layers:
            layer.close()
