"""Reference RSC training step of a two-layer GCN, in fp64 (oracle).

TEST INFRASTRUCTURE ONLY. It follows the paper's procedure directly:
forward H1 = ReLU(A J1), J1 = X W1; logits P2 = A J2, J2 = H1 W2 (Eq. 1 and
its SpMM/MatMul form, section 2.1); mean binary cross-entropy with logits;
backward through each aggregation as grad J = A^T grad P exactly, or on the
top-k column slice of A^T (section 2.2.1, section 3.1: only the backward is
approximated); at a refresh step the backward is exact, both layers' pairs are
scored (O4 keys of the fp32-rounded gradients), k_l comes from the greedy of
section 3.2.1 (O8) and each layer's columns are selected (O5) and sliced (O6).
Products are scipy sparse / numpy dense in fp64.

With track_staleness, each refresh after the first also records, per layer,
the staleness of the cached selection (section 3.3.1, Fig. 4): the AUC of
the previous selection under the new ranking and the overlap of the two
selections, counted by orc_selection_auc; with the k_l of every refresh this
is the trace of Fig. 7.

Pins (tests/test_oracle_pins.py): the exact-mode gradients against central
differences of the reported loss, the loss at zero logits (ln 2), and a
full-budget step between refreshes against the exact gradients; the
aggregation steps it uses (O3-O8) are pinned there too; the staleness
record against brute force over all (selected, unselected) pairs.
"""
from __future__ import annotations

import numpy as np
import scipy.sparse as sp

from . import col_sqnorms, greedy, pair_keys, rank_order, selection_staleness, slice_csr, sum_sequential, topk


class RscReference:
    """cache=False: every approximated step selects (O4, O5) and slices (O6)
    against that step's own gradient with the current k_l before the
    product, instead of reusing the slice of the last refresh (the
    no-caching arm of section 3.3.1's comparison)."""

    def __init__(self, rowptr, col, val, n, widths, budget, alpha, refresh_interval, cache=True,
                 track_staleness=False):
        self.n = n
        self.A = sp.csr_matrix((val.astype(np.float64), col, rowptr), shape=(n, n))
        self.AT = self.A.T.tocsr()
        self.csr_t = (rowptr, col, val)  # A^T of a symmetric A is A itself
        self.cn2, self.colnnz = col_sqnorms(rowptr, val)
        self.fro_a2 = sum_sequential(self.cn2)      # ||A||_F^2 (Eq. 4a)
        self.nnz = int(rowptr[-1])
        self.widths = list(widths)
        self.budget, self.alpha, self.R = budget, alpha, refresh_interval
        self.last = None
        self.k = [n] * len(widths)
        self.idx = [None] * len(widths)
        self.masks = [None] * len(widths)
        self.refresh_masks = [None] * len(widths)   # the selections of the last refresh
        self.slices = [None] * len(widths)
        self.cache = cache
        self.track = track_staleness
        self.history = []   # one record per refresh: step, k, auc, overlap

    def _select(self, l, key):
        rowptr, col, val = self.csr_t
        self.idx[l], mask = topk(key, self.k[l])
        self.masks[l] = mask
        ro, co, vo = slice_csr(rowptr, col, val, mask)
        self.slices[l] = sp.csr_matrix((vo.astype(np.float64), co, ro), shape=(self.n, self.n))

    def _backward_spmm(self, l, g, mode):
        if mode == "sampled":
            if not self.cache:
                self._select(l, pair_keys(self.cn2, g.astype(np.float32))["key"])
            return self.slices[l] @ g
        return self.AT @ g

    def step(self, X, W1, W2, Y, step):
        """One training step with weights W1, W2. At a refresh step the keys
        and ||grad H||_F^2 it scored are also returned (keys, fro_b2)."""
        mode = "score" if (self.last is None or step - self.last >= self.R) else "sampled"
        J1 = X @ W1
        P1 = self.A @ J1
        H1 = np.maximum(P1, 0.0)
        J2 = H1 @ W2
        P2 = self.A @ J2
        loss = float(np.mean(np.maximum(P2, 0) - P2 * Y + np.log1p(np.exp(-np.abs(P2)))))
        gP2 = (1.0 / (1.0 + np.exp(-P2)) - Y) / P2.size
        gJ2 = self._backward_spmm(1, gP2, mode)
        gW2 = H1.T @ gJ2
        gP1 = (gJ2 @ W2.T) * (P1 > 0)
        gJ1 = self._backward_spmm(0, gP1, mode)
        gW1 = X.T @ gJ1
        out = {"mode": mode, "loss": loss, "gW1": gW1, "gW2": gW2}
        if mode == "score":
            keys, fro_b2 = [], []
            for g in (gP1, gP2):
                o = pair_keys(self.cn2, g.astype(np.float32))
                keys.append(o["key"])
                fro_b2.append(sum_sequential(o["rn2"]))     # ||grad H||_F^2 (Eq. 4a)
            out["keys"], out["fro_b2"] = keys, fro_b2
            self.k, _ = greedy(keys, self.colnnz, self.nnz, self.widths, self.fro_a2, fro_b2,
                               self.budget, self.alpha)
            rec = {"step": step, "k": list(self.k), "auc": [], "overlap": []}
            for l in range(2):
                prev = self.refresh_masks[l]
                self._select(l, keys[l])
                self.refresh_masks[l] = self.masks[l]
                if self.track and prev is not None:
                    auc, overlap = selection_staleness(rank_order(keys[l]), prev, self.masks[l])
                    rec["auc"].append(auc)
                    rec["overlap"].append(overlap)
            self.history.append(rec)
            self.last = step
        out["k"] = list(self.k)
        out["idx"] = [None if i is None else i.copy() for i in self.idx]
        return out
