"""A seeded sweep of random layer shapes through the C ABI against the fp64
oracle: head counts and grouping, head_dim, dtype, window, pool kind and
kernel, explicit scale, window kept or ranked, per-group or layer-shared
selection, ragged batches of prompts, budgets from the window up to past the
prompt, through ckv_compress_layer or ckv_compress_stack (two layers, one
batch). Each draw is printed before it runs, so a failure names its seed."""
import numpy as np
import pytest
import torch

import paper_2508_02401_amd as ckv
from tests.gpu_util import (Case, check_group, check_shared, oracle_group, oracle_shared,
                            random_inputs, run_gpu)

pytestmark = pytest.mark.gpu

N_DRAWS = 64
DTYPES = (torch.bfloat16, torch.float16, torch.float32)


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ckv.load()
    return torch.device("cuda:0")


def draw(i: int):
    rng = np.random.default_rng(9000 + i)
    G = int(rng.choice([1, 2, 4, 7, 8]))
    n_kv = int(rng.choice([1, 2, 4]))
    case = Case(G * n_kv, n_kv, int(rng.choice([64, 128])), int(rng.integers(1, 97)),
                str(rng.choice(["avg", "max"])), int(rng.choice([1, 3, 5, 7, 9, 15, 31])),
                DTYPES[int(rng.integers(0, 3))], shared=bool(rng.integers(0, 4) == 0),
                explicit_scale=float(rng.choice([0.0, 0.0, 0.07, 0.2])),
                keep_window=bool(rng.integers(0, 3) > 0))
    top = int(rng.choice([600, 2600, 9000]))
    lens = [int(rng.integers(case.w + 1, top)) for _ in range(int(rng.integers(1, 4)))]
    lo = case.w if case.keep_window else 1
    budgets = [int(rng.integers(lo, L + 40)) for L in lens]
    return case, lens, budgets, bool(rng.integers(0, 2)), int(rng.integers(0, 1 << 30))


def _check_prompt(case, out, mask, q, k, v, budget, label):
    if case.shared:
        rs, ri = oracle_shared(case, mask, q, k, budget)
        check_shared(case, out, rs, ri, k, v, label)
        return
    groups = range(case.n_kv) if case.n_kv <= 2 else (0, case.n_kv - 1)
    for g in groups:
        rs, ri = oracle_group(case, mask, q, k, g, budget)
        check_group(case, out, g, rs, ri, k, v, label)


@pytest.mark.parametrize("i", range(N_DRAWS))
def test_random_layer_shapes(dev, i):
    case, lens, budgets, stack, seed = draw(i)
    label = "draw %d: %s L=%s B=%s %s" % (i, case, lens, budgets, "stack" if stack else "layer")
    print(label, flush=True)
    n_layers = 2 if stack else 1
    layers = []
    mask = None
    for l in range(n_layers):
        qs, ks, vs = [], [], []
        for p, L in enumerate(lens):
            q, k, v, m = random_inputs(case, L, seed=seed + 31 * l + p, device="cpu", mask=mask)
            mask = m  # one head mask per layer, shared by its prompts
            qs.append(q)
            ks.append(k)
            vs.append(v)
        layers.append((mask, qs, ks, vs))
        mask = None
    desc = case.desc()
    if stack:
        seqs, masks = [], []
        for mask, qs, ks, vs in layers:
            row = []
            for q, k, v, b in zip(qs, ks, vs, budgets):
                s = ckv.Seq(q.to(dev), k.to(dev), v.to(dev), int(b))
                ckv.alloc_outputs(desc, s, with_scores=True)
                row.append(s)
            seqs.append(row)
            masks.append(mask)
        ws = torch.empty(2 * ckv.ckv_workspace_bytes(desc, seqs[0]) + 64, dtype=torch.uint8,
                         device=dev)
        ckv.ckv_compress_stack(desc, np.stack(masks), seqs, ws, torch.cuda.current_stream(), None)
        torch.cuda.synchronize()
        outs = [[dict(scores=s.scores.cpu().numpy(), idx=s.idx.cpu().numpy(), k_out=s.k_out.cpu(),
                      v_out=s.v_out.cpu()) for s in row] for row in seqs]
    else:
        mask, qs, ks, vs = layers[0]
        outs = [run_gpu(case, mask, [q.to(dev) for q in qs], [k.to(dev) for k in ks],
                        [v.to(dev) for v in vs], budgets)]
    for l, (mask, qs, ks, vs) in enumerate(layers):
        for p in range(len(lens)):
            _check_prompt(case, outs[l][p], mask, qs[p], ks[p], vs[p], budgets[p],
                          "%s layer %d prompt %d" % (label, l, p))
