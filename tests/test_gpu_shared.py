"""GPU parity of the layer-shared selection (CKV_SHARE_LAYER) against the
oracle, through the C ABI: the chosen heads of the whole layer rank the tokens
together and one index set is kept for every KV head (paper Sec. 3.3)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2508_02401_amd as ckv
from paper_2508_02401_amd import synth
from tests.gpu_util import (Case, check_group, check_shared, oracle_group, oracle_shared,
                            random_inputs, run_gpu)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ckv.load()
    return torch.device("cuda:0")


def _mask(H, heads):
    m = np.zeros(H, np.uint8)
    m[list(heads)] = 1
    return m


SHARED_CASES = [
    # (label, Case, L, chosen heads, budget)
    ("llama-4srh-spread", Case(32, 8, 128, 32, "max", 7, torch.bfloat16, True), 4095,
     (1, 9, 18, 30), 512),
    ("llama-4srh-one-group", Case(32, 8, 128, 32, "max", 7, torch.bfloat16, True), 3001,
     (4, 5, 6, 7), 300),
    ("paper-defaults-w8-avg5", Case(32, 8, 128, 8, "avg", 5, torch.bfloat16, True), 2600,
     (0, 13, 14, 27), 128),
    ("f16-d64-3heads", Case(16, 4, 64, 16, "max", 3, torch.float16, True), 2049,
     (2, 3, 12), 100),
    ("f32-d128-w64", Case(8, 2, 128, 64, "avg", 7, torch.float32, True), 1500,
     (0, 1, 6), 200),
    ("bf16-w48-two-per-group", Case(16, 4, 128, 48, "max", 9, torch.bfloat16, True), 3333,
     (0, 1, 8, 9), 250),
    ("single-head", Case(8, 2, 128, 16, "max", 5, torch.bfloat16, True), 1100, (5,), 64),
    # the paper's top-4 heads of a layer all in one group at w = 64: 256 rows,
    # read as two row groups of 128
    ("llama-4srh-one-group-w64", Case(32, 8, 128, 64, "max", 7, torch.bfloat16, True), 3001,
     (8, 9, 10, 11), 300),
]


@pytest.mark.parametrize("label,case,L,heads,budget", SHARED_CASES, ids=[c[0] for c in SHARED_CASES])
def test_shared_parity(dev, label, case, L, heads, budget):
    mask = _mask(case.H, heads)
    q, k, v, _ = random_inputs(case, L, seed=hash(label) % 1000, device="cpu", mask=mask)
    out = run_gpu(case, mask, [q.to(dev)], [k.to(dev)], [v.to(dev)], [budget])[0]
    assert out["scores"].shape == (1, L - case.w) and out["idx"].shape == (1, min(budget, L))
    rs, ri = oracle_shared(case, mask, q, k, budget)
    check_shared(case, out, rs, ri, k, v, label)


@pytest.mark.parametrize("budget", [32, 33, 1023, 1024, 5000])
def test_shared_edge_budgets(dev, budget):
    case = Case(32, 8, 128, 32, "max", 7, torch.bfloat16, True)
    mask = _mask(32, (3, 10, 17, 31))
    q, k, v, _ = random_inputs(case, 1024, seed=budget, device="cpu", mask=mask)
    out = run_gpu(case, mask, [q.to(dev)], [k.to(dev)], [v.to(dev)], [budget])[0]
    rs, ri = oracle_shared(case, mask, q, k, budget)
    check_shared(case, out, rs, ri, k, v, "budget %d" % budget)


def test_shared_one_group_equals_group_selection(dev):
    # all chosen heads in one group: the shared set is that group's own set
    case = Case(32, 8, 128, 32, "max", 7, torch.bfloat16, True)
    per_group = Case(32, 8, 128, 32, "max", 7, torch.bfloat16, False)
    heads = (20, 21, 23)
    mask_sh = _mask(32, heads)
    q, k, v, _ = random_inputs(case, 6000, seed=21, device=dev, mask=mask_sh)
    sh = run_gpu(case, mask_sh, [q], [k], [v], [400])[0]
    mask_pg = np.ones(32, np.uint8)  # every other group needs heads in per-group scope
    mask_pg[20:24] = 0  # group 5 keeps exactly the shared heads
    mask_pg[list(heads)] = 1
    pg = run_gpu(per_group, mask_pg, [q], [k], [v], [400])[0]
    np.testing.assert_array_equal(sh["scores"][0], pg["scores"][5])
    np.testing.assert_array_equal(sh["idx"][0], pg["idx"][5])


def test_shared_split_calls_match_fused(dev):
    # ckv_score, ckv_select and ckv_gather in turn give the fused result
    case = Case(32, 8, 128, 32, "avg", 5, torch.bfloat16, True)
    mask = _mask(32, (0, 7, 8, 25))
    q, k, v, _ = random_inputs(case, 7000, seed=22, device=dev, mask=mask)
    fused = run_gpu(case, mask, [q], [k], [v], [700])[0]
    desc = case.desc()
    s = ckv.alloc_outputs(desc, ckv.Seq(q, k, v, 700))
    ws = ckv.alloc_workspace(desc, [s], dev)
    ckv.ckv_score(desc, mask, [s], ws)
    ckv.ckv_select(desc, [s], ws)
    ckv.ckv_gather(desc, [s])
    torch.cuda.synchronize()
    np.testing.assert_array_equal(s.scores.cpu().numpy(), fused["scores"])
    np.testing.assert_array_equal(s.idx.cpu().numpy(), fused["idx"])
    assert torch.equal(s.k_out.cpu(), fused["k_out"]) and torch.equal(s.v_out.cpu(), fused["v_out"])


def test_shared_ragged_batch(dev):
    case = Case(28, 4, 128, 32, "max", 7, torch.bfloat16, True)
    mask = _mask(28, (2, 9, 15, 26))
    lens, budgets = (1500, 4097, 9000), (100, 300, 1000)
    ins = [random_inputs(case, L, seed=30 + i, device=dev, mask=mask) for i, L in enumerate(lens)]
    out = run_gpu(case, mask, [x[0] for x in ins], [x[1] for x in ins], [x[2] for x in ins], budgets)
    for i, (q, k, v, _) in enumerate(ins):
        rs, ri = oracle_shared(case, mask, q, k, budgets[i])
        check_shared(case, out[i], rs, ri, k.cpu(), v.cpu(), "ragged %d" % i)
        single = run_gpu(case, mask, [q], [k], [v], [budgets[i]])[0]
        np.testing.assert_array_equal(single["scores"], out[i]["scores"])


def test_shared_full_size_128k(dev):
    # the 128K Llama shape with the paper's four retrieval heads per layer
    wl = synth.WORKLOADS["llama8b-128k-stack"]
    case = Case(wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.window, "max", wl.pool_kernel,
                wl.dtype, True)
    inp = synth.layer_inputs(wl, 0, dev)
    mask = _mask(32, (1, 6, 22, 29))
    out = run_gpu(case, mask, inp.q_win, inp.k, inp.v, [128])[0]
    rs, ri = oracle_shared(case, mask, inp.q_win[0], inp.k[0], 128)
    check_shared(case, out, rs, ri, inp.k[0].cpu(), inp.v[0].cpu(), "128k shared")
