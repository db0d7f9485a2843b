"""The whole eviction pass (score -> select -> compact) on torch device tensors.

`EvictionPass` allocates every output and the workspace once for a given
shape, so that `run()` only enqueues the three library calls -- the form the
benchmark times.  All arithmetic happens inside libecokv.
"""
from __future__ import annotations

from typing import Optional

import torch

from . import ecokv as E


class EvictionPass:
    def __init__(self, shape: E.Shape, budget, mode: int = E.PER_HEAD,
                 params: Optional[E.Params] = None, dtype: torch.dtype = torch.bfloat16,
                 device: str = "cuda"):
        self.shape, self.budget, self.mode = shape, E._flat_ints(budget), mode
        self.params = params or E.Params()
        c = shape.c
        L, Hkv, D, w, B = c.num_layers, c.num_kv_heads, c.head_dim, c.window, c.num_seqs
        cu = shape.cu_seqlens
        self.Ptot = cu[-1] - B * w
        U = L * Hkv * B
        self.scores = torch.empty(L * Hkv * self.Ptot, dtype=torch.float32, device=device)
        self.lambda_ = torch.empty(U, dtype=torch.float32, device=device)
        self.stats = torch.empty(U * E.NSTATS, dtype=torch.float32, device=device)
        ws = E.ecokv_workspace_size(shape, self.params)
        self.workspace = torch.empty(max(ws, 256), dtype=torch.uint8, device=device)
        self.n_idx = E.ecokv_index_count_mode(shape, mode, self.budget)
        self.idx = torch.empty(max(self.n_idx, 1), dtype=torch.int32, device=device)
        self.counts = torch.empty(max(U, 1), dtype=torch.int32, device=device)
        self.offsets = torch.empty(max(U, 1), dtype=torch.int32, device=device)
        self.Kc = torch.empty((max(self.n_idx, 1), D), dtype=dtype, device=device)
        self.Vc = torch.empty((max(self.n_idx, 1), D), dtype=dtype, device=device)

    def score(self, K: torch.Tensor, Q_win: torch.Tensor, stream=None, V: Optional[torch.Tensor] = None,
              pre: Optional[torch.Tensor] = None):
        if pre is not None:
            E.ecokv_score_pre(K, V, Q_win, self.shape, self.params, pre, self.scores, self.lambda_, self.stats,
                              self.workspace, stream)
        elif self.params.imp_mode == E.IMP_ATTN_VNORM:
            E.ecokv_score_v(K, V, Q_win, self.shape, self.params, self.scores, self.lambda_, self.stats,
                            self.workspace, stream)
        else:
            E.ecokv_score(K, Q_win, self.shape, self.params, self.scores, self.lambda_, self.stats,
                          self.workspace, stream)

    def select(self, stream=None):
        E.ecokv_select(self.scores, self.shape, self.mode, self.budget, self.idx, self.counts,
                       self.offsets, stream)

    def compact(self, K: torch.Tensor, V: torch.Tensor, stream=None):
        E.ecokv_compact(K, V, self.shape, self.mode, self.budget, self.idx, self.counts, self.offsets,
                        self.Kc, self.Vc, stream)

    def run(self, K: torch.Tensor, V: torch.Tensor, Q_win: torch.Tensor, stream=None,
            pre: Optional[torch.Tensor] = None):
        self.score(K, Q_win, stream, V, pre)
        self.select(stream)
        self.compact(K, V, stream)
        return self
