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
                 device: str = "cuda", workspace: Optional[torch.Tensor] = None):
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
        if workspace is not None and workspace.numel() >= ws:
            self.workspace = workspace  # (shared with passes that never run at the same time)
        else:
            # zero-filled: its first word is the status that ecokv_workspace_status reads
            self.workspace = torch.zeros(max(ws, 256), dtype=torch.uint8, device=device)
        # zero-filled, as ecokv_select leaves it
        self.sel_workspace = torch.zeros(max(E.ecokv_select_workspace_size(shape, mode), 256), dtype=torch.uint8,
                                         device=device)
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
                       self.offsets, self.sel_workspace, stream)

    def compact(self, K: torch.Tensor, V: torch.Tensor, stream=None):
        E.ecokv_compact(K, V, self.shape, self.mode, self.budget, self.idx, self.counts, self.offsets,
                        self.Kc, self.Vc, stream)

    def run(self, K: torch.Tensor, V: torch.Tensor, Q_win: torch.Tensor, stream=None,
            pre: Optional[torch.Tensor] = None):
        self.score(K, Q_win, stream, V, pre)
        self.select(stream)
        self.compact(K, V, stream)
        return self

    def check(self, stream=None):
        """Synchronise `stream` and raise if a score call since the last check
        had a wait between blocks give up (see ecokv_workspace_status)."""
        E.ecokv_workspace_status(self.workspace, stream)


class LayerwiseEviction:
    """The pass layer by layer as a prefill finishes the layers, one call per
    layer or per group of consecutive layers.

    `shape` is the shape of one call: num_layers = 1 for a call per layer, or
    k > 1 for a call per group of k consecutive layers (whose K, V and Q_win
    the caller passes as [k][...] tensors, e.g. views of a cache laid out layer
    by layer).  Call c runs on the c % 2-th of two side streams (default
    priority), with its own outputs (`passes[c]`: scores, idx, counts, offsets,
    Kc, Vc) and the workspace of its stream.  One call's select and epilogue
    occupy only a few compute units; on two streams they overlap the next
    call's sweeps (28 layers of 28q/4kv at 32768 tokens: 77 -> 48 us per layer
    with a call per layer); a group of layers per call fills more of the chip
    per launch.  `run_layer` / `run_group` order the call after the work
    already queued on the caller's stream; `wait` makes the caller's stream
    wait for every call queued so far.  The caller keeps a call's K, V and
    Q_win alive until `wait` (they are read on a side stream, which torch's
    allocator does not track).  The host work per call is one event record
    and wait plus the three library calls.
    """

    def __init__(self, shape: E.Shape, budget, num_layers: int, mode: int = E.PER_HEAD,
                 params: Optional[E.Params] = None, dtype: torch.dtype = torch.bfloat16, device: str = "cuda"):
        k = shape.c.num_layers
        if k < 1 or num_layers % k != 0:
            raise ValueError(f"the call shape's {k} layers must divide the {num_layers} layers")
        self.layers_per_call = k
        params = params or E.Params()
        ws = max(E.ecokv_workspace_size(shape, params), 256)
        self.streams = [torch.cuda.Stream(device=device), torch.cuda.Stream(device=device)]
        self.workspaces = [torch.zeros(ws, dtype=torch.uint8, device=device) for _ in range(2)]
        self.passes = [EvictionPass(shape, budget, mode, params, dtype, device, self.workspaces[c % 2])
                       for c in range(num_layers // k)]
        self._ready = [torch.cuda.Event(), torch.cuda.Event()]
        self._done = [torch.cuda.Event(), torch.cuda.Event()]

    def run_group(self, call: int, K: torch.Tensor, V: torch.Tensor, Q_win: torch.Tensor) -> EvictionPass:
        """Call `call`: layers call * k .. call * k + k - 1 (K, V, Q_win over them)."""
        i = call % 2
        s, ready = self.streams[i], self._ready[i]
        ready.record(torch.cuda.current_stream(K.device))
        s.wait_event(ready)
        return self.passes[call].run(K, V, Q_win, stream=s)

    def run_layer(self, layer: int, K: torch.Tensor, V: torch.Tensor, Q_win: torch.Tensor) -> EvictionPass:
        """One layer per call (the call shape's num_layers = 1)."""
        if self.layers_per_call != 1:
            raise ValueError("this instance takes groups of layers: use run_group")
        return self.run_group(layer, K, V, Q_win)

    def run_layers(self, calls, K, V, Q_win):
        """Several calls whose inputs are all ready: one ordering event for
        all of them (per-call events cost 48 -> 54 us per layer on the
        28-layer stack with a call per layer).  K, V, Q_win: sequences indexed
        like `calls`."""
        cur = torch.cuda.current_stream(self.workspaces[0].device)
        for s, ready in zip(self.streams, self._ready):
            ready.record(cur)
            s.wait_event(ready)
        for j, c in enumerate(calls):
            self.passes[c].run(K[j], V[j], Q_win[j], stream=self.streams[c % 2])

    def wait(self):
        cur = torch.cuda.current_stream(self.workspaces[0].device)
        for s, done in zip(self.streams, self._done):
            done.record(s)
            cur.wait_event(done)

    def check(self):
        """Synchronise both side streams and raise if a layer's score call had a
        wait between blocks give up (see ecokv_workspace_status)."""
        for s, ws in zip(self.streams, self.workspaces):
            E.ecokv_workspace_status(ws, s)
