"""One router + controller step on device buffers, built on the C ABI binding.

A :class:`RouterStep` owns the per-step outputs (expert indices, gate weights,
counts, load statistics), the router workspace and the controller state of one
MoE layer, all as device tensors, and issues the ABI calls of one iteration of
Alg. 1: route the batch with the current bias, update the bias from the
counts, and compute MaxVio/MinVio.
"""
from __future__ import annotations

import torch

from . import binding as B


class RouterStep:
    def __init__(self, T: int, d: int, E: int, K: int, dtype: torch.dtype = torch.bfloat16,
                 cfg: B.ControllerCfg | None = None, variant: int = 0, device: str = "cuda"):
        self.T, self.d, self.E, self.K, self.dtype, self.variant = T, d, E, K, dtype, variant
        code = B.IDB_DTYPE_BF16 if dtype == torch.bfloat16 else B.IDB_DTYPE_F32
        self.dtype_code = code
        self.cfg = cfg or B.ControllerCfg(E)
        self.state = B.ControllerState(E, device)
        self.idx = torch.empty((T, K), dtype=torch.int32, device=device)
        self.w = torch.empty((T, K), dtype=torch.float32, device=device)
        self.counts = torch.zeros(E, dtype=torch.int32, device=device)
        self.stats = torch.zeros(2, dtype=torch.float64, device=device)
        nbytes = B.idb_router_workspace_bytes(T, d, E, K, code, variant)
        self.workspace = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=device)
        self.info = B.idb_router_variant_info(T, d, E, K, code, variant)
        self.W_packed = None

    def pack(self, W, stream=None):
        """Pack the router matrix (once per weight update); later calls with ``W=None`` read the packed copy.

        The packed buffer is allocated on the first call and reused after, so
        the call can be captured in a graph."""
        if self.W_packed is None or self.W_packed.shape != W.shape or self.W_packed.dtype != W.dtype:
            self.W_packed = torch.empty_like(W)
        B.idb_router_pack_weight(W, self.W_packed, stream)
        return self.W_packed

    def _weights(self, W):
        if W is None:
            return self.W_packed, B.IDB_WEIGHT_PACKED
        return W, B.IDB_WEIGHT_ROW_MAJOR

    def route(self, x, W=None, accumulate: bool = False, scores_dump=None, stream=None):
        """Route with row-major ``W``, or with the packed copy from :meth:`pack` when ``W`` is None."""
        Wt, layout = self._weights(W)
        B.idb_router_forward(x, Wt, self.state.bias, self.K, self.idx, self.w, self.counts, accumulate, scores_dump,
                             self.workspace, self.variant, stream, layout)

    def score_select(self, x, W=None, accumulate: bool = False, scores_dump=None, stream=None, events=None):
        """The router's first launch; ``events`` = (start, stop) ``torch.cuda.Event`` pair that then takes the
        fused kernel's own start and end timestamps."""
        Wt, layout = self._weights(W)
        if events is None:
            B.idb_router_score_select(x, Wt, self.state.bias, self.K, self.idx, self.w, self.counts, accumulate,
                                      scores_dump, self.workspace, self.variant, stream, layout)
        else:
            B.idb_router_score_select_timed(x, Wt, self.state.bias, self.K, self.idx, self.w, self.counts,
                                            events[0], events[1], accumulate, scores_dump, self.workspace,
                                            self.variant, stream, layout)

    def merge(self, stream=None):
        B.idb_router_merge(self.T, self.d, self.E, self.K, self.dtype_code, self.idx, self.w, self.counts,
                           self.workspace, self.variant, stream)

    def update(self, stream=None):
        B.idb_controller_update(self.counts, self.cfg, self.state, stream)

    def load_stats(self, stream=None):
        B.idb_load_stats(self.counts, self.stats, stream)

    def update_and_stats(self, stream=None):
        """MaxVio/MinVio of this step's counts and the bias update, one launch."""
        B.idb_controller_step(self.counts, self.cfg, self.state, self.stats, stream)

    def step(self, x, W=None, accumulate: bool = False, stream=None):
        """Route, then compute MaxVio/MinVio and update the bias (all asynchronous; the update runs in
        the slice merge's last workgroup when the tiling has several slices)."""
        Wt, layout = self._weights(W)
        B.idb_router_step(x, Wt, self.K, self.cfg, self.state, self.idx, self.w, self.counts, accumulate,
                          self.stats, self.workspace, self.variant, stream, layout)

    def merge_step(self, stream=None):
        """The second launch of :meth:`step` after :meth:`score_select` (same bias, same outputs): slice merge,
        MaxVio/MinVio and the bias update."""
        B.idb_router_merge_step(self.T, self.d, self.K, self.dtype_code, self.cfg, self.state, self.idx, self.w,
                                self.counts, self.stats, self.workspace, self.variant, stream)

    # ------------------------------------------------------------ Quantile Balancing

    def qb_buffers(self):
        """Allocate (once) the Quantile Balancing inputs and its larger workspace."""
        if getattr(self, "scores_t", None) is None:
            dev = self.idx.device
            self.scores_t = torch.empty((self.E, self.T), dtype=torch.float32, device=dev)
            self.alpha = torch.empty(self.T, dtype=torch.float32, device=dev)
            n = B.idb_qb_router_workspace_bytes(self.T, self.d, self.E, self.K, self.dtype_code, self.variant)
            self.qb_workspace = torch.empty(max(n, 16), dtype=torch.uint8, device=dev)

    def qb_route(self, x, W=None, accumulate: bool = False, stream=None):
        """Route with the current bias and write Quantile Balancing's cutoffs and expert-major scores."""
        self.qb_buffers()
        Wt, layout = self._weights(W)
        B.idb_qb_router_forward(x, Wt, self.state.bias, self.K, self.idx, self.w, self.counts, self.scores_t,
                                self.alpha, accumulate, self.qb_workspace, self.variant, stream, layout)

    def qb_step(self, x, W=None, rho: float = 0.0, stream=None):
        """One Quantile Balancing iteration (Eq. pid-quantile): route, then the bias target and MaxVio/MinVio of
        the counts (one launch)."""
        self.qb_route(x, W, stream=stream)
        B.idb_qb_update(self.scores_t, self.alpha, self.K, rho, self.state.bias, stream, counts=self.counts,
                        stats=self.stats)

    # ------------------------------------------------------------ auxiliary-loss statistics

    def aux_buffers(self, variant: int = 0):
        """Allocate (once) the auxiliary-loss outputs f, P, loss and their workspace (one-slice tiling)."""
        if getattr(self, "aux_P", None) is None:
            dev = self.idx.device
            self.aux_variant = variant
            self.aux_f = torch.empty(self.E, dtype=torch.float64, device=dev)
            self.aux_P = torch.empty(self.E, dtype=torch.float64, device=dev)
            self.aux_loss = torch.empty(1, dtype=torch.float64, device=dev)
            n = B.idb_aux_router_workspace_bytes(self.T, self.d, self.E, self.K, self.dtype_code, variant)
            if n == 0:
                raise B.IdbError("idb_aux_router_workspace_bytes", B.IDB_ERR_UNSUPPORTED,
                                 f"no one-slice router tiling for E={self.E} (variant {variant})")
            self.aux_workspace = torch.empty(n, dtype=torch.uint8, device=dev)
            self.aux_info = B.idb_router_variant_info(self.T, self.d, self.E, self.K, self.dtype_code, variant) \
                if variant else None

    def aux_step(self, x, W=None, alpha: float = 0.05, stream=None):
        """Softmax routing without bias, the auxiliary-loss statistics f, P and alpha sum f P
        (Eq. pid-auxloss) and MaxVio/MinVio of the counts (two launches)."""
        self.aux_buffers()
        Wt, layout = self._weights(W)
        B.idb_aux_router_forward(x, Wt, self.K, alpha, self.idx, self.w, self.counts, self.aux_f, self.aux_P,
                                 self.aux_loss, self.aux_workspace, None, self.aux_variant, stream, layout,
                                 stats=self.stats)
