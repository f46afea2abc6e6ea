"""RSC training of a GCN on top of the library (sections 3.1-3.3 and 5.1).

Each aggregation `P_l = SpMM(A_hat, J_l)` runs exactly in the forward pass
(rsc_spmm). Its backward `grad J_l = SpMM(A_hat^T, grad P_l)` runs in one of
three modes, chosen per step by `RscController`:

* "sampled": on the layer's cached top-k slice (rsc_spmm_sampled) — the
  approximation of section 3.1, reused across steps (section 3.3.1);
* "resample": without caching, each approximated step scores, selects and
  slices against its own gradient (rsc_cache_refresh with the current k_l)
  before the sampled product;
* "score": exactly, and the pairs (column i of A_hat^T, row i of grad P_l)
  are scored into the layer's cache (rsc_cache_score) — a refresh step;
  after the backward the controller allocates k_l across layers with the
  greedy of section 3.2.1 (each layer's ranking profiled on the device by
  rsc_greedy_profile, the greedy loop on the host by
  rsc_greedy_allocate_profiles) and selects/slices each layer's columns
  (rsc_cache_select);
* "exact": plain exact backward (no approximation, or the final phase of
  training after switching back, section 3.3.2).

With track_staleness, every refresh after the first also records, per
layer, the AUC of the selection it replaced under the new ranking and the
overlap of the two selections (section 3.3.1, Fig. 4), computed on the
device by rsc_cache_staleness from rsc_greedy_profile's ranking.

The dense update phase (MatMul, ReLU, loss, optimizer) uses torch; it is not
part of the aggregation path.
"""
from __future__ import annotations

import math
import time
from dataclasses import dataclass, field

import torch

from . import Cache, DeviceCsr, SpmmPlan, _check, _stream, greedy_allocate_profiles, lib


class _Aggregate(torch.autograd.Function):
    @staticmethod
    def forward(ctx, J: torch.Tensor, layer: "AggregationLayer") -> torch.Tensor:
        ctx.layer = layer
        t = layer._tick()
        P = layer.plan.run(J.contiguous())
        layer._tock(t, "forward")
        return P

    @staticmethod
    def backward(ctx, grad_P: torch.Tensor):
        layer = ctx.layer
        g = grad_P.contiguous()
        t = layer._tick()
        if layer.mode == "resample":
            # no caching: this step's own top-k and slice, then the sampled product
            layer.cache.refresh(g, layer.k, step=layer.step)
            grad_J = layer.cache.spmm_sampled(g)
        elif layer.mode == "sampled":
            grad_J = layer.cache.spmm_sampled(g)
        else:
            grad_J = layer.plan_t.run(g)
        layer._tock(t, "backward")
        if layer.mode == "score":
            layer.cache.score(g)
        return grad_J, None


class AggregationLayer:
    """One SpMM site: the operand A_hat (CSR), the CSR of its transpose for
    the backward, and the sampled-matrix cache of the backward operand."""

    def __init__(self, A: DeviceCsr, AT: DeviceCsr | None, width: int, refresh_interval: int):
        self.A = A
        self.AT = A if AT is None else AT
        self.width = width
        # the backward multiplies by A_hat^T: its columns are scored and sliced;
        # the CSR of its transpose (A_hat) gives the column norms
        self.cache = Cache(self.AT, self.A, refresh_interval=refresh_interval)
        # exact products with the static operands go through plans (prepared once)
        self.plan = SpmmPlan(A)
        self.plan_t = self.plan if self.AT is A else SpmmPlan(self.AT)
        self.mode = "exact"
        self.k = A.n_cols       # columns kept by the approximation (set by the allocation)
        self.step = 0
        self.timings = None  # set to a list to record (kind, start, end) events of each SpMM

    def _tick(self):
        if self.timings is None:
            return None
        e = torch.cuda.Event(enable_timing=True)
        e.record()
        return e

    def _tock(self, start, kind: str) -> None:
        if start is not None:
            e = torch.cuda.Event(enable_timing=True)
            e.record()
            self.timings.append((kind, start, e))

    def __call__(self, J: torch.Tensor) -> torch.Tensor:
        return _Aggregate.apply(J, self)


@dataclass
class RscConfig:
    budget: tuple = (1, 10)          # C of Eq. 4b as num/den
    alpha: tuple = (2, 100)          # greedy step alpha |V| (section 5.1)
    refresh_interval: int = 10       # allocation and cache refresh period (section 5.1)
    switch_fraction: tuple = (8, 10)  # approximate for this share of the steps (section 5.1)
    total_steps: int | None = None
    enabled: bool = True
    cache: bool = True               # reuse each slice until the next refresh (section 3.3.1); if
                                     # False every approximated step selects and slices anew
    track_staleness: bool = False    # record AUC / overlap of successive selections


@dataclass
class StepRecord:
    step: int
    mode: str
    k: list = field(default_factory=list)
    greedy_s: float = 0.0
    auc: list = field(default_factory=list)      # previous selection under the new ranking
    overlap: list = field(default_factory=list)  # |S_prev & S_new| / |S_prev|


class RscController:
    """Decides each step's backward mode and, at refresh steps, allocates
    k_l with the greedy and refreshes every layer's slice."""

    def __init__(self, layers: list, cfg: RscConfig):
        self.layers = layers
        self.cfg = cfg
        A = layers[0].AT
        self.n = A.n_cols
        self.nnz = A.nnz
        self.colnnz_ptr = layers[0].cache.buffers()[1]
        # ||A_hat^T||_F^2 (Eq. 4a's normaliser), summed on the device in a fixed order
        self.fro_a2 = layers[0].cache.norms(scored=False)[0]
        dev = A.rowptr.device
        nb = lib().rsc_greedy_blocks(self.n, cfg.alpha[0], cfg.alpha[1])
        self.mass = torch.empty((len(layers), max(nb, 1)), dtype=torch.float64, device=dev)
        self.count = torch.empty((len(layers), max(nb, 1)), dtype=torch.int64, device=dev)
        self.nb = nb
        self.ws = torch.empty(max(lib().rsc_greedy_profile_workspace_bytes(self.n), 1), dtype=torch.uint8,
                              device=dev)
        # each layer's pair ranking at the latest refresh (for the staleness record)
        self.order = torch.empty((len(layers), max(self.n, 1)), dtype=torch.int32, device=dev) \
            if cfg.track_staleness else None
        self.last_refresh = None
        self.k = [self.n] * len(layers)
        self.history: list[StepRecord] = []

    def begin(self, step: int) -> str:
        cfg = self.cfg
        if not cfg.enabled:
            mode = "exact"
        elif cfg.total_steps is not None and \
                step * cfg.switch_fraction[1] >= cfg.total_steps * cfg.switch_fraction[0]:
            mode = "exact"
        elif self.last_refresh is None or step - self.last_refresh >= cfg.refresh_interval:
            mode = "score"
        else:
            mode = "sampled" if cfg.cache else "resample"
        for layer in self.layers:
            layer.mode = mode
            layer.step = step
        self.history.append(StepRecord(step, mode))
        return mode

    def end(self, step: int) -> None:
        rec = self.history[-1]
        if rec.mode != "score":
            rec.k = list(self.k) if rec.mode in ("sampled", "resample") else [self.n] * len(self.layers)
            return
        torch.cuda.synchronize()  # time the allocation alone, not the backward before it
        t0 = time.perf_counter()
        # device: rank each layer's pairs and profile the ranking (sum of
        # sqrt(q) and of column entry counts per block of `step` ranks)
        fro_b2 = []
        for l, layer in enumerate(self.layers):
            ptrs = layer.cache.buffers()
            _check(lib().rsc_greedy_profile(ptrs[2], self.colnnz_ptr, self.n, self.cfg.alpha[0],
                                            self.cfg.alpha[1], self.mass[l].data_ptr(),
                                            self.count[l].data_ptr(),
                                            None if self.order is None else self.order[l].data_ptr(),
                                            self.ws.data_ptr(), self.ws.numel(), _stream()))
            fro_b2.append(layer.cache.norms()[1])   # ||grad H||_F^2 of the scored gradient (device sum)
        masses = self.mass[:, :self.nb].cpu().numpy()
        counts = self.count[:, :self.nb].cpu().numpy()
        widths = [layer.width for layer in self.layers]
        # host: the greedy loop over the profiles
        self.k, _ = greedy_allocate_profiles(list(masses), list(counts), self.n, self.nnz, widths,
                                             self.fro_a2, fro_b2, self.cfg.budget, self.cfg.alpha)
        for layer, k in zip(self.layers, self.k):
            layer.cache.select(k, step)
            layer.k = k
        rec.greedy_s = time.perf_counter() - t0
        if self.order is not None and self.last_refresh is not None:
            # the selection each cache just replaced, under the new ranking
            # (section 3.3.1, Fig. 4), on the device
            for l, layer in enumerate(self.layers):
                auc, both, k_prev = layer.cache.staleness(self.order[l])
                rec.auc.append(auc)
                if k_prev:
                    rec.overlap.append(both / k_prev)
        rec.k = list(self.k)
        self.last_refresh = step

    def close(self):
        for layer in self.layers:
            layer.cache.close()
            layer.plan.close()
            layer.plan_t.close()


class GCN(torch.nn.Module):
    """Two-layer GCN (Eq. 1): logits = A_hat ReLU(A_hat X W1) W2, each
    aggregation an AggregationLayer."""

    def __init__(self, A: DeviceCsr, in_features: int, hidden: int, classes: int, cfg: RscConfig,
                 seed: int = 2, AT: DeviceCsr | None = None):
        super().__init__()
        g = torch.Generator().manual_seed(seed)

        def glorot(fan_in, fan_out):
            a = math.sqrt(6.0 / (fan_in + fan_out))
            return torch.nn.Parameter(((torch.rand(fan_in, fan_out, generator=g) * 2 - 1) * a).cuda())

        self.W1 = glorot(in_features, hidden)
        self.W2 = glorot(hidden, classes)
        self.agg1 = AggregationLayer(A, AT, hidden, cfg.refresh_interval)
        self.agg2 = AggregationLayer(A, AT, classes, cfg.refresh_interval)
        self.controller = RscController([self.agg1, self.agg2], cfg)

    def forward(self, X: torch.Tensor) -> torch.Tensor:
        H1 = torch.relu(self.agg1(X @ self.W1))
        return self.agg2(H1 @ self.W2)

    def train_step(self, X, targets, optimizer, step: int):
        """One RSC training step: forward, multi-label BCE loss, backward
        (mode set by the controller), optional optimizer update."""
        self.controller.begin(step)
        if optimizer is not None:
            optimizer.zero_grad(set_to_none=True)
        logits = self(X)
        loss = torch.nn.functional.binary_cross_entropy_with_logits(logits, targets)
        loss.backward()
        self.controller.end(step)
        if optimizer is not None:
            optimizer.step()
        return loss

    def close(self):
        self.controller.close()
