"""The largest shapes the build accepts, through the C ABI against the oracle:
128 query heads over 64 KV heads with the widest window (128) and pool kernel
(31), and a batch of CKV_MAX_SEQS ragged prompts, each through
ckv_compress_layer and ckv_compress_stack."""
import numpy as np
import pytest
import torch

import paper_2508_02401_amd as ckv
from tests.gpu_util import Case, check_group, oracle_group, random_inputs, run_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ckv.load()
    return torch.device("cuda:0")


def _stack(desc, layers, dev):
    """ckv_compress_stack over layers [(mask, qs, ks, vs, budgets)], one batch."""
    seqs, masks = [], []
    for mask, qs, ks, vs, budgets in layers:
        row = []
        for q, k, v, b in zip(qs, ks, vs, budgets):
            s = ckv.Seq(q.to(dev), k.to(dev), v.to(dev), int(b))
            ckv.alloc_outputs(desc, s, with_scores=True)
            row.append(s)
        seqs.append(row)
        masks.append(mask)
    ws = torch.empty(len(layers) * ckv.ckv_workspace_bytes(desc, seqs[0]) + 64, dtype=torch.uint8,
                     device=dev)
    ckv.ckv_compress_stack(desc, np.stack(masks), seqs, ws, torch.cuda.current_stream(), None)
    torch.cuda.synchronize()
    return [[dict(scores=s.scores.cpu().numpy(), idx=s.idx.cpu().numpy(), k_out=s.k_out.cpu(),
                  v_out=s.v_out.cpu()) for s in row] for row in seqs]


def test_most_heads_widest_window_and_pool(dev):
    # CKV_MAX_Q_HEADS, CKV_MAX_KV_HEADS, CKV_MAX_WINDOW and CKV_MAX_POOL_KERNEL
    case = Case(128, 64, 128, 128, "max", 31, torch.bfloat16)
    L, budget = 1500, 300
    layers = []
    for l in range(2):
        q, k, v, mask = random_inputs(case, L, seed=77 + l, device="cpu", n_sel=2)
        layers.append((mask, [q], [k], [v], [budget]))
    print("limits: 128 q / 64 kv heads, w=128, k=31", flush=True)
    mask, qs, ks, vs, bs = layers[0]
    out_layer = run_gpu(case, mask, [qs[0].to(dev)], [ks[0].to(dev)], [vs[0].to(dev)], bs)[0]
    out_stack = _stack(case.desc(), layers, dev)
    for f in ("scores", "idx"):
        assert np.array_equal(out_layer[f], out_stack[0][0][f]), f
    for l, (mask, qs, ks, vs, bs) in enumerate(layers):
        for g in (0, 17, 40, 63):
            rs, ri = oracle_group(case, mask, qs[0], ks[0], g, bs[0])
            check_group(case, out_stack[l][0], g, rs, ri, ks[0], vs[0], "layer %d" % l)


def test_largest_batch_of_ragged_prompts(dev):
    n = ckv.CKV_MAX_SEQS
    case = Case(8, 2, 64, 16, "avg", 5, torch.float16)
    rng = np.random.default_rng(5)
    lens = [int(x) for x in rng.integers(17, 1200, size=n)]
    budgets = [int(rng.integers(16, L + 20)) for L in lens]
    layers = []
    for l in range(2):
        qs, ks, vs, mask = [], [], [], None
        for p, L in enumerate(lens):
            q, k, v, mask = random_inputs(case, L, seed=500 + 37 * l + p, device="cpu", mask=mask)
            qs.append(q)
            ks.append(k)
            vs.append(v)
        layers.append((mask, qs, ks, vs, budgets))
    print("limits: %d prompts, L=%s" % (n, lens), flush=True)
    mask, qs, ks, vs, bs = layers[0]
    outs_layer = run_gpu(case, mask, [q.to(dev) for q in qs], [k.to(dev) for k in ks],
                         [v.to(dev) for v in vs], bs)
    outs_stack = _stack(case.desc(), layers, dev)
    for p in range(n):
        for f in ("scores", "idx"):
            assert np.array_equal(outs_layer[p][f], outs_stack[0][p][f]), (p, f)
    for l, (mask, qs, ks, vs, bs) in enumerate(layers):
        for p in range(n):
            for g in range(case.n_kv):
                rs, ri = oracle_group(case, mask, qs[p], ks[p], g, bs[p])
                check_group(case, outs_stack[l][p], g, rs, ri, ks[p], vs[p],
                            "layer %d prompt %d" % (l, p))
