"""GPU parity with CKV_KEEP_WINDOW off: the window tokens are not kept by rule,
every one of the L tokens is scored (a window column only by the window rows
that see it), pooled over [0, L), and the best B of all L tokens are kept.
Against the oracle's whole-prompt selection (select_group_all /
select_layer_shared_all) under the rules in tests/parity.py, through every
entry point that scores or selects: ckv_compress_layer, the split calls with
caller scores, caller row statistics, the layer-shared scope and
ckv_compress_stack."""
import zlib

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


def _off(H, n_kv, d, w, pool, kp, dtype, shared=False):
    return Case(H, n_kv, d, w, pool, kp, dtype, shared, keep_window=False)


CASES = [
    # (label, Case, L, n_sel, budget)
    ("bf16-d128-G4-ragged", _off(32, 8, 128, 32, "max", 7, torch.bfloat16), 4095, 2, 512),
    ("bf16-d64-w8-budget-below-window", _off(8, 2, 64, 8, "avg", 5, torch.bfloat16), 257, 1, 5),
    ("f16-w13-3heads", _off(8, 1, 128, 13, "max", 3, torch.float16), 2000, 3, 100),
    ("f32-d64-avg7", _off(8, 2, 64, 16, "avg", 7, torch.float32), 1024, 1, 128),
    # w8 = 64, two heads: each wave's query blocks are whole heads (direct stores)
    ("bf16-w64-2heads-direct", _off(8, 2, 128, 64, "max", 7, torch.bfloat16), 3000, 2, 300),
    # w8 = 32, four heads: a query block per head, pair mapping
    ("bf16-w32-4heads", _off(16, 4, 128, 32, "max", 7, torch.bfloat16), 2999, 4, 300),
    # the largest window, and windows straddling the 32-row query blocks
    ("bf16-w128", _off(8, 2, 128, 128, "max", 7, torch.bfloat16), 3000, 1, 400),
    ("bf16-w48-straddle", _off(8, 2, 128, 48, "max", 9, torch.bfloat16), 3333, 2, 200),
    ("bf16-w1-k31", _off(16, 4, 128, 1, "avg", 31, torch.bfloat16), 5000, 4, 1000),
    # more than 128 chosen rows: two row groups per KV head
    ("bf16-w64-4heads-256rows", _off(8, 2, 128, 64, "max", 7, torch.bfloat16), 3000, 4, 300),
    # the window starting exactly on a stage boundary, and one past it
    ("bf16-window-on-stage-edge", _off(8, 2, 128, 32, "avg", 5, torch.bfloat16), 64 * 40 + 32, 2, 128),
    ("bf16-window-past-stage-edge", _off(8, 2, 128, 32, "max", 5, torch.bfloat16), 64 * 40 + 33, 2, 128),
    ("bf16-budget-1", _off(8, 2, 128, 32, "max", 7, torch.bfloat16), 1500, 2, 1),
    ("bf16-budget-L-minus-1", _off(8, 2, 128, 32, "max", 7, torch.bfloat16), 2000, 2, 1999),
    ("bf16-budget-L", _off(8, 2, 128, 32, "max", 7, torch.bfloat16), 700, 2, 700),
]


@pytest.mark.parametrize("label,case,L,n_sel,budget", CASES, ids=[c[0] for c in CASES])
def test_keep_window_off_parity(dev, label, case, L, n_sel, budget):
    q, k, v, mask = random_inputs(case, L, seed=zlib.crc32(label.encode()) % 10000, device="cpu",
                                  n_sel=n_sel)
    print("case", label, flush=True)
    out = run_gpu(case, mask, [q.to(dev)], [k.to(dev)], [v.to(dev)], [budget])[0]
    assert out["scores"].shape == (case.n_kv, L) and out["idx"].shape == (case.n_kv, min(budget, L))
    for g in range(case.n_kv):
        rs, ri = oracle_group(case, mask, q, k, g, budget)
        check_group(case, out, g, rs, ri, k, v, label)


def test_keep_window_off_window_tokens_can_be_evicted(dev):
    # planted high-scoring keys far from the window and a small budget: the
    # kept set leaves out most of the window (which the default mode keeps)
    case = _off(8, 2, 128, 32, "max", 3, torch.bfloat16)
    L, budget = 4000, 48
    q, k, v, mask = random_inputs(case, L, seed=77, device="cpu", n_sel=2)
    for g in range(2):
        heads = [g * 4 + t for t in range(4) if mask[g * 4 + t]]
        qbar = q[heads].float().reshape(-1, 128).mean(0)
        k[g, 100:140] = (k[g, 100:140].float() + 4.0 * qbar / (qbar @ qbar).sqrt()).to(k.dtype)
    out = run_gpu(case, mask, [q.to(dev)], [k.to(dev)], [v.to(dev)], [budget])[0]
    for g in range(2):
        rs, ri = oracle_group(case, mask, q, k, g, budget)
        check_group(case, out, g, rs, ri, k, v, "evict-window")
        kept = set(out["idx"][g].tolist())
        assert len(kept & set(range(L - 32, L))) < 32
        assert len(kept & set(range(100, 140))) >= 20


def test_keep_window_off_split_calls_and_caller_lse(dev):
    # ckv_score + ckv_select + ckv_gather, then the same with the window rows'
    # log-sum-exp supplied by the caller: both equal ckv_compress_layer
    case = _off(32, 8, 128, 32, "max", 7, torch.bfloat16)
    L, budget = 3001, 250
    q, k, v, mask = random_inputs(case, L, seed=5, device="cpu", n_sel=2)
    desc = case.desc()
    ref = run_gpu(case, mask, [q.to(dev)], [k.to(dev)], [v.to(dev)], [budget])[0]
    lse = torch.full((case.H, case.w), float("nan"), dtype=torch.float32)
    for g in range(case.n_kv):
        heads = [g * 4 + t for t in range(4) if mask[g * 4 + t]]
        vals = oracle.window_lse(q[heads].double().numpy(), k[g].double().numpy(), case.scale)
        for t, h in enumerate(heads):
            lse[h] = torch.from_numpy(vals[t]).float()
    for with_lse in (False, True):
        s = ckv.Seq(q.to(dev), k.to(dev), v.to(dev), budget, lse=lse.to(dev) if with_lse else None)
        ckv.alloc_outputs(desc, s)
        ws = ckv.alloc_workspace(desc, [s], dev)
        ckv.ckv_score(desc, mask, [s], ws)
        ckv.ckv_select(desc, [s], ws)
        ckv.ckv_gather(desc, [s])
        torch.cuda.synchronize()
        out = dict(scores=s.scores.cpu().numpy(), idx=s.idx.cpu().numpy(), k_out=s.k_out.cpu(),
                   v_out=s.v_out.cpu())
        if not with_lse:
            np.testing.assert_array_equal(out["scores"], ref["scores"])
            np.testing.assert_array_equal(out["idx"], ref["idx"])
        for g in range(case.n_kv):
            rs, ri = oracle_group(case, mask, q, k, g, budget)
            check_group(case, out, g, rs, ri, k, v, "split lse=%s" % with_lse)


def test_keep_window_off_select_on_oracle_scores_is_exact(dev):
    # ckv_select alone on caller scores over all L tokens (rounded, many
    # ties): exactly the oracle's whole-prompt top-B of the same values
    case = _off(8, 2, 64, 8, "max", 7, torch.bfloat16)
    rng = np.random.default_rng(9)
    L = 20000
    desc = case.desc()
    for budget in (1, 7, 100, 4096, 19999, 20000):
        scores = np.round(rng.random((2, L)), 3).astype(np.float32)
        sc = torch.from_numpy(scores).to(dev)
        idx = torch.empty((2, min(budget, L)), dtype=torch.int32, device=dev)
        s = ckv.Seq(None, None, None, budget, scores=sc, idx=idx, seq_len=L)
        ckv.ckv_select(desc, [s], ckv.alloc_workspace(desc, [s], dev))
        torch.cuda.synchronize()
        for g in range(2):
            ref = oracle.select_tokens_all(scores[g].astype(np.float64), L, budget)
            np.testing.assert_array_equal(idx[g].cpu().numpy(), ref)


SHARED = [
    ("llama-4srh-spread", _off(32, 8, 128, 32, "max", 7, torch.bfloat16, True), 4095,
     (1, 9, 18, 30), 512),
    ("w64-one-group-256rows", _off(32, 8, 128, 64, "max", 7, torch.bfloat16, True), 3001,
     (8, 9, 10, 11), 300),
    ("f16-d64-avg", _off(16, 4, 64, 16, "avg", 5, torch.float16, True), 2049, (2, 3, 12), 60),
]


@pytest.mark.parametrize("label,case,L,heads,budget", SHARED, ids=[c[0] for c in SHARED])
def test_keep_window_off_shared(dev, label, case, L, heads, budget):
    mask = np.zeros(case.H, np.uint8)
    mask[list(heads)] = 1
    q, k, v, _ = random_inputs(case, L, seed=zlib.crc32(label.encode()) % 1000, device="cpu",
                               mask=mask)
    out = run_gpu(case, mask, [q.to(dev)], [k.to(dev)], [v.to(dev)], [budget])[0]
    assert out["scores"].shape == (1, L)
    rs, ri = oracle_shared(case, mask, q, k, budget)
    check_shared(case, out, rs, ri, k, v, label)


def test_keep_window_off_ragged_batch_and_stack(dev):
    # three layers of a ragged two-prompt batch through ckv_compress_stack
    # (side stream, one slot): bit-exact against per-layer calls, and every
    # (layer, prompt, KV head) against the oracle
    case = _off(16, 4, 128, 32, "max", 7, torch.bfloat16)
    desc = case.desc()
    lens, budgets = (3100, 1777), (300, 40)
    layers = []
    for l in range(3):
        ins = [random_inputs(case, L, seed=500 + 10 * l + i, device="cpu", n_sel=1 + (l + i) % 2)
               for i, L in enumerate(lens)]
        mask = ins[0][3]
        layers.append((mask, [x[:3] for x in ins]))
    seqs = []
    for mask, ins in layers:
        row = []
        for (q, k, v), b in zip(ins, budgets):
            row.append(ckv.alloc_outputs(desc, ckv.Seq(q.to(dev), k.to(dev), v.to(dev), b)))
        seqs.append(row)
    ws = torch.empty(ckv.ckv_workspace_bytes(desc, seqs[0]), dtype=torch.uint8, device=dev)
    ckv.ckv_compress_stack(desc, np.stack([m for m, _ in layers]), seqs, ws,
                           torch.cuda.current_stream(), torch.cuda.Stream())
    torch.cuda.synchronize()
    for l, (mask, ins) in enumerate(layers):
        per = run_gpu(case, mask, [x[0].to(dev) for x in ins], [x[1].to(dev) for x in ins],
                      [x[2].to(dev) for x in ins], budgets)
        for s, (q, k, v) in enumerate(ins):
            got = dict(scores=seqs[l][s].scores.cpu().numpy(), idx=seqs[l][s].idx.cpu().numpy(),
                       k_out=seqs[l][s].k_out.cpu(), v_out=seqs[l][s].v_out.cpu())
            np.testing.assert_array_equal(got["scores"], per[s]["scores"])
            np.testing.assert_array_equal(got["idx"], per[s]["idx"])
            for g in range(case.n_kv):
                rs, ri = oracle_group(case, mask, q, k, g, budgets[s])
                check_group(case, got, g, rs, ri, k, v, "stack layer %d prompt %d" % (l, s))


def test_keep_window_off_full_size_128k_sampled_heads(dev):
    # a layer of the 128K Llama workload with the window ranked like any other
    # token, budget 128 per KV head; three KV heads against the oracle
    wl = synth.WORKLOADS["llama8b-128k-stack"]
    inp = synth.layer_inputs(wl, 2, dev)
    case = _off(wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.window, "max", wl.pool_kernel,
                wl.dtype)
    print("case 128k keep-window off", flush=True)
    out = run_gpu(case, inp.mask, inp.q_win, inp.k, inp.v, [128])[0]
    k_cpu, v_cpu = inp.k[0].cpu(), inp.v[0].cpu()
    for g in (0, 3, 7):
        rs, ri = oracle_group(case, inp.mask, inp.q_win[0], k_cpu, g, 128)
        check_group(case, out, g, rs, ri, k_cpu, v_cpu, "128k off g%d" % g)
