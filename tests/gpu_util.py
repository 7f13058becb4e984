"""Helpers for the GPU tests: run a layer through the C ABI, run the oracle on
the same inputs, and compare under the rules in tests/parity.py."""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np
import torch

import oracle
import paper_2508_02401_amd as ckv
from tests import parity

POOL = {"avg": ckv.CKV_POOL_AVG, "max": ckv.CKV_POOL_MAX}
ORACLE_POOL = {"avg": oracle.POOL_AVG, "max": oracle.POOL_MAX}


@dataclass
class Case:
    H: int
    n_kv: int
    d: int
    w: int
    pool: str
    kp: int
    dtype: torch.dtype
    shared: bool = False  # layer-shared selection (CKV_SHARE_LAYER)
    explicit_scale: float = 0.0  # desc.scale; 0 selects the default 1/sqrt(d)
    keep_window: bool = True     # CKV_KEEP_WINDOW: the window is kept by rule, not ranked

    @property
    def tail(self) -> int:
        """Tokens at the end kept by rule (the window), 0 when all compete."""
        return self.w if self.keep_window else 0

    def desc(self):
        flags = (ckv.CKV_KEEP_WINDOW if self.keep_window else 0) | \
            (ckv.CKV_SHARE_LAYER if self.shared else 0)
        return ckv.layer_desc(self.H, self.n_kv, self.d, self.w, self.dtype, self.explicit_scale,
                              POOL[self.pool], self.kp, flags)

    @property
    def scale(self) -> float:
        return self.explicit_scale if self.explicit_scale > 0 else 1.0 / math.sqrt(self.d)


def run_gpu(case: Case, mask, q_list, k_list, v_list, budgets: Sequence[int],
            scores_out: bool = True):
    """ckv_compress_layer on a batch; returns per prompt dict of numpy arrays."""
    desc = case.desc()
    seqs = []
    for q, k, v, b in zip(q_list, k_list, v_list, budgets):
        s = ckv.Seq(q, k, v, int(b))
        ckv.alloc_outputs(desc, s, with_scores=scores_out)
        seqs.append(s)
    ws = ckv.alloc_workspace(desc, seqs, k_list[0].device)
    ckv.ckv_compress_layer(desc, mask, seqs, ws)
    torch.cuda.synchronize()
    out = []
    for s in seqs:
        out.append(dict(scores=s.scores.cpu().numpy() if s.scores is not None else None,
                        idx=s.idx.cpu().numpy(), k_out=s.k_out.cpu(), v_out=s.v_out.cpu()))
    return out


def chosen_heads(mask, H: int, n_kv: int, g: int) -> List[int]:
    G = H // n_kv
    return [g * G + t for t in range(G) if mask[g * G + t]]


def oracle_group(case: Case, mask, q: torch.Tensor, k: torch.Tensor, g: int, budget: int):
    heads = chosen_heads(mask, case.H, case.n_kv, g)
    q_sel = q[heads].double().cpu().numpy()
    kg = k[g].double().cpu().numpy()
    if not case.keep_window:
        return oracle.select_group_all(q_sel, kg, case.w, case.scale, ORACLE_POOL[case.pool],
                                       case.kp, int(budget))
    scores, idx, _ = oracle.select_group(q_sel, kg, case.w, case.scale, ORACLE_POOL[case.pool],
                                         case.kp, int(budget))
    return scores, idx


def oracle_shared(case: Case, mask, q: torch.Tensor, k: torch.Tensor, budget: int):
    """The layer-shared selection of the oracle: (scores [L-w] or [L], idx [min(B, L)])."""
    if not case.keep_window:
        return oracle.select_layer_shared_all(q.double().cpu().numpy(), mask,
                                              k.double().cpu().numpy(), case.w, case.scale,
                                              ORACLE_POOL[case.pool], case.kp, int(budget))
    return oracle.select_layer_shared(q.double().cpu().numpy(), mask, k.double().cpu().numpy(),
                                      case.w, case.scale, ORACLE_POOL[case.pool], case.kp,
                                      int(budget))


def check_shared(case: Case, gpu: dict, ref_scores, ref_idx, k: torch.Tensor, v: torch.Tensor,
                 label: str = ""):
    """Assert parity of a layer-shared selection: the one score and index row,
    and every KV head's compact rows at those indices."""
    rel, swaps = check_group(case, gpu, 0, ref_scores, ref_idx, k, v, label, heads=range(k.shape[0]))
    return rel, swaps


def check_group(case: Case, gpu: dict, g: int, ref_scores, ref_idx, k: torch.Tensor,
                v: torch.Tensor, label: str = "", heads=None):
    """Assert parity of selection row g of one prompt (KV head g, or the shared
    row 0) and of the compact rows of `heads` (default: head g) at its indices.
    Returns (max rel err, swaps)."""
    L = k.shape[1]
    gs = gpu["scores"][g] if gpu["scores"] is not None else None
    if gs is not None:
        ok, rel, bad = parity.score_errors(gs, ref_scores)
        assert ok, "%s group %d: %d scores off, max rel %.3g" % (label, g, bad, rel)
    else:
        rel = float("nan")
    gi = gpu["idx"][g]
    ok, swaps, msg = parity.index_swaps(gi, ref_idx, ref_scores, L, case.tail)
    assert ok, "%s group %d: %s" % (label, g, msg)
    # the GPU's selection is exactly the top-N of the GPU's own scores
    n_keep = len(gi) - case.tail
    if gs is not None and len(gi) < L:
        own = parity.topn_reference(np.asarray(gs, dtype=np.float64), n_keep)
        np.testing.assert_array_equal(gi[:n_keep], own, err_msg="%s group %d own top-N" % (label, g))
    # compact cache: bit-exact rows of the input at the GPU's indices
    ii = torch.from_numpy(gi.astype(np.int64))
    for h in (heads if heads is not None else [g]):
        assert torch.equal(gpu["k_out"][h], k[h].cpu()[ii]), "%s head %d k_out" % (label, h)
        assert torch.equal(gpu["v_out"][h], v[h].cpu()[ii]), "%s head %d v_out" % (label, h)
    return rel, swaps


def random_inputs(case: Case, L: int, seed: int, device, n_sel: Optional[int] = None,
                  mask=None):
    gen = torch.Generator(device="cpu").manual_seed(seed)
    q = torch.randn((case.H, case.w, case.d), generator=gen).to(case.dtype).to(device)
    k = torch.randn((case.n_kv, L, case.d), generator=gen).to(case.dtype).to(device)
    v = torch.randn((case.n_kv, L, case.d), generator=gen).to(case.dtype).to(device)
    if mask is None:
        rng = np.random.default_rng(seed)
        G = case.H // case.n_kv
        mask = np.zeros(case.H, np.uint8)
        for g in range(case.n_kv):
            n = n_sel if n_sel is not None else int(rng.integers(1, G + 1))
            for t in rng.choice(G, size=min(n, G), replace=False):
                mask[g * G + int(t)] = 1
    return q, k, v, mask
