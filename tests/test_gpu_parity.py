"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Small cases run the oracle on every KV head; the full-size workloads run it on
sampled KV heads (each head's selection is independent). Tolerances and the
tie rule are in tests/parity.py.
"""
import zlib

import numpy as np
import pytest
import torch

import oracle
import paper_2508_02401_amd as ckv
from paper_2508_02401_amd import synth
from tests import parity
from tests.gpu_util import (Case, check_group, chosen_heads, oracle_group, random_inputs,
                            run_gpu, ORACLE_POOL)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ckv.load()
    return torch.device("cuda:0")


def _full_check(case, mask, q, k, v, budget, label, dev):
    out = run_gpu(case, mask, [q.to(dev)], [k.to(dev)], [v.to(dev)], [budget])[0]
    for g in range(case.n_kv):
        rs, ri = oracle_group(case, mask, q, k, g, budget)
        check_group(case, out, g, rs, ri, k, v, label)
    return out


CASES = [
    # (label, Case, L, n_sel, budget)
    ("bf16-d128-G4-ragged", Case(32, 8, 128, 32, "max", 7, torch.bfloat16), 4095, 2, 512),
    ("bf16-d64-paper-defaults", Case(8, 2, 64, 8, "avg", 5, torch.bfloat16), 257, 1, 64),
    ("f16-w13-3heads", Case(8, 1, 128, 13, "max", 3, torch.float16), 2000, 3, 100),
    ("bf16-w64-128rows", Case(8, 2, 128, 64, "max", 7, torch.bfloat16), 3000, 2, 300),
    ("f32-d128-64rows", Case(8, 2, 128, 16, "avg", 1, torch.float32), 1500, 4, 200),
    ("f32-d64", Case(8, 2, 64, 16, "avg", 7, torch.float32), 1024, 1, 128),
    ("bf16-w1-allheads-k31", Case(16, 4, 128, 1, "avg", 31, torch.bfloat16), 5000, 4, 1000),
    ("bf16-maxpool-k1", Case(8, 2, 64, 24, "max", 1, torch.bfloat16), 1100, 2, 90),
    ("f16-d64-G7", Case(28, 4, 64, 32, "max", 7, torch.float16), 2500, 2, 75),
    ("bf16-tile-boundary", Case(8, 2, 128, 32, "max", 7, torch.bfloat16), 992 * 3 + 32, 1, 500),
    ("bf16-chunk-boundary", Case(8, 2, 128, 32, "avg", 7, torch.bfloat16), 1024 * 2 + 1, 2, 100),
    # one KV head: 257 workgroups share its 64-token stages round-robin
    ("bf16-one-kv-head-many-splits", Case(4, 1, 128, 32, "max", 7, torch.bfloat16), 65536 + 17, 1,
     256),
    # prefix of 40 whole 64-token stages plus one token
    ("bf16-stage-edge", Case(8, 2, 128, 32, "avg", 5, torch.bfloat16), 64 * 40 + 32 + 1, 2, 128),
    # w8 = 48: query blocks straddle heads (8-row group sums)
    ("bf16-w48-straddle", Case(8, 2, 128, 48, "max", 9, torch.bfloat16), 3333, 2, 200),
    # 3-4 query blocks: each wave takes two of them; whole heads inside one
    # wave store their window sums directly (w8 = 32 and w8 = 64)
    ("bf16-w32-4heads-per-group", Case(16, 4, 128, 32, "max", 7, torch.bfloat16), 2999, 4, 300),
    ("f16-d64-w32-3heads", Case(28, 4, 64, 32, "avg", 5, torch.float16), 2100, 3, 150),
    ("bf16-w57-2heads-padded", Case(8, 2, 128, 57, "max", 7, torch.bfloat16), 2345, 2, 222),
    # the largest window: one head fills all 128 rows of its group (its four
    # query blocks span two waves, so the window sums go through the fold)
    ("bf16-w128-max-window", Case(8, 2, 128, 128, "max", 7, torch.bfloat16), 3000, 1, 400),
    ("f16-d64-w128-max-window", Case(8, 2, 64, 128, "avg", 9, torch.float16), 1500, 1, 300),
    # everything but one prefix token kept
    ("bf16-budget-L-minus-1", Case(8, 2, 128, 32, "max", 7, torch.bfloat16), 2000, 2, 1999),
    # more than 128 chosen rows in a group: the K passes read it in row groups
    # of at most 128 rows (2 x 128 at w = 64, 3 x 128 at w = 128, 120 + 40 at w = 40)
    ("bf16-w64-4heads-256rows", Case(8, 2, 128, 64, "max", 7, torch.bfloat16), 3000, 4, 300),
    ("f16-d64-w128-3heads-384rows", Case(8, 2, 64, 128, "avg", 5, torch.float16), 2000, 3, 200),
    ("bf16-w40-4heads-uneven-row-groups", Case(16, 4, 128, 40, "max", 7, torch.bfloat16), 2500, 4, 256),
]


@pytest.mark.parametrize("label,case,L,n_sel,budget", CASES, ids=[c[0] for c in CASES])
def test_layer_parity(dev, label, case, L, n_sel, budget):
    q, k, v, mask = random_inputs(case, L, seed=zlib.crc32(label.encode()) % 10000, device="cpu", n_sel=n_sel)
    print("case", label, "L", L, flush=True)
    _full_check(case, mask, q, k, v, budget, label, dev)


@pytest.mark.parametrize("scale", [0.03, 0.2])
def test_explicit_scale(dev, scale):
    # desc.scale given explicitly (not the default 1/sqrt(d) = 0.088): a
    # flatter (0.03) and a sharper (0.2) softmax, against the oracle at the
    # same scale
    case = Case(32, 8, 128, 32, "max", 7, torch.bfloat16, explicit_scale=scale)
    q, k, v, mask = random_inputs(case, 3001, seed=int(scale * 1000), device="cpu", n_sel=2)
    print("case explicit scale %g" % scale, flush=True)
    out = _full_check(case, mask, q, k, v, 400, "scale %g" % scale, dev)
    # the default scale gives different scores: the explicit one is really used
    d_case = Case(32, 8, 128, 32, "max", 7, torch.bfloat16)
    rs, _ = oracle_group(d_case, mask, q, k, 0, 400)
    assert not np.allclose(out["scores"][0], rs, rtol=1e-2)


@pytest.mark.parametrize("budget", [32, 33, 40, 1000])
def test_window_edge_budgets(dev, budget):
    # L = w + 1: a one-token prefix; B = w keeps only the window, B >= L keeps all
    case = Case(8, 2, 128, 32, "max", 7, torch.bfloat16)
    q, k, v, mask = random_inputs(case, 33, seed=5, device="cpu", n_sel=2)
    _full_check(case, mask, q, k, v, budget, "edge-%d" % budget, dev)


@pytest.mark.parametrize("pool", ["avg", "max"])
def test_constant_keys_tie_break(dev, pool):
    # identical keys: every prefix score is equal away from the edges, so the
    # selection is decided by the lower-index rule alone and must match exactly
    case = Case(8, 2, 128, 16, pool, 5, torch.bfloat16)
    q, k, v, mask = random_inputs(case, 3000, seed=9, device="cpu", n_sel=2)
    k[:] = k[:, :1, :]
    out = _full_check(case, mask, q, k, v, 400, "const-" + pool, dev)
    for g in range(case.n_kv):
        _, ri = oracle_group(case, mask, q, k, g, 400)
        np.testing.assert_array_equal(out["idx"][g], ri)


def test_tiny_workload(dev):
    wl = synth.WORKLOADS["tiny-fp32"]
    inp = synth.layer_inputs(wl, 0, dev)
    case = Case(wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.window, "avg", wl.pool_kernel,
                wl.dtype)
    out = run_gpu(case, inp.mask, inp.q_win, inp.k, inp.v, [wl.budget])[0]
    for g in range(wl.num_kv_heads):
        rs, ri = oracle_group(case, inp.mask, inp.q_win[0], inp.k[0], g, wl.budget)
        check_group(case, out, g, rs, ri, inp.k[0], inp.v[0], "tiny")
        # planted sinks and span survive
        assert set(inp.planted[0].tolist()) <= set(out["idx"][g].tolist())


def _workload_case(wl):
    return Case(wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.window,
                "max" if wl.pool == 1 else "avg", wl.pool_kernel, wl.dtype)


def test_llama_32k_layer_all_heads(dev):
    wl = synth.WORKLOADS["llama8b-32k-layer"]
    inp = synth.layer_inputs(wl, 0, dev)
    case = _workload_case(wl)
    out = run_gpu(case, inp.mask, inp.q_win, inp.k, inp.v, [wl.budget])[0]
    q64 = inp.q_win[0].double().cpu().numpy()
    k64 = inp.k[0].double().cpu().numpy()
    rs, ri = oracle.select_layer(q64, inp.mask, k64, case.w, case.scale, ORACLE_POOL[case.pool],
                                 case.kp, wl.budget)
    k_cpu, v_cpu = inp.k[0].cpu(), inp.v[0].cpu()
    for g in range(case.n_kv):
        check_group(case, out, g, rs[g], ri[g], k_cpu, v_cpu, "llama32k")
        assert set(inp.planted[0].tolist()) <= set(out["idx"][g].tolist())


@pytest.mark.parametrize("name,layer,groups", [
    ("llama8b-128k-stack", 0, (0, 5)),
    ("llama8b-32k-stack", 7, (3,)),
])
def test_full_size_sampled_heads(dev, name, layer, groups):
    wl = synth.WORKLOADS[name]
    inp = synth.layer_inputs(wl, layer, dev)
    case = _workload_case(wl)
    e = synth.layer_errors(wl)
    total, m, M = synth.budget_params(wl, wl.seq_lens[0])
    budgets, st = ckv.ckv_allocate_budgets(e, total, m, M)
    ref_b, _ = oracle.allocate_budgets(e, total, m, M)
    assert st == ckv.CKV_OK and budgets.tolist() == ref_b.tolist()
    b = int(budgets[layer])
    out = run_gpu(case, inp.mask, inp.q_win, inp.k, inp.v, [b])[0]
    k_cpu, v_cpu = inp.k[0].cpu(), inp.v[0].cpu()
    for g in groups:
        rs, ri = oracle_group(case, inp.mask, inp.q_win[0], inp.k[0], g, b)
        check_group(case, out, g, rs, ri, k_cpu, v_cpu, "%s L%d" % (name, layer))
    # on every head, the selection is the top-N of the GPU's own scores
    for g in range(case.n_kv):
        own = parity.topn_reference(out["scores"][g].astype(np.float64), b - case.w)
        np.testing.assert_array_equal(out["idx"][g][: b - case.w], own)


def test_sixteen_prompts_in_one_call(dev):
    # the most prompts one call takes (CKV_MAX_SEQS): lengths and budgets all
    # differ, including a one-token prefix and a budget past the prompt
    case = Case(8, 2, 128, 16, "max", 5, torch.bfloat16)
    rng = np.random.default_rng(16)
    lens = [17, 40, 3000] + [int(x) for x in rng.integers(50, 2500, size=13)]
    budgets = [16, 64, 100] + [int(x) for x in rng.integers(16, 600, size=13)]
    budgets[5] = lens[5] + 10
    assert len(lens) == ckv.CKV_MAX_SEQS
    ins = [random_inputs(case, L, seed=200 + i, device="cpu", n_sel=1 + i % 2) for i, L in enumerate(lens)]
    mask = ins[0][3]
    ins = [(q, k, v) for q, k, v, _ in ins]
    print("case sixteen prompts", flush=True)
    out = run_gpu(case, mask, [q.to(dev) for q, _, _ in ins], [k.to(dev) for _, k, _ in ins],
                  [v.to(dev) for _, _, v in ins], budgets)
    for s, ((q, k, v), B) in enumerate(zip(ins, budgets)):
        g = s % case.n_kv
        rs, ri = oracle_group(case, mask, q, k, g, B)
        check_group(case, out[s], g, rs, ri, k, v, "prompt%d" % s)


def test_ragged_batch_sampled_heads(dev):
    wl = synth.WORKLOADS["qwen7b-ragged-batch"]
    inp = synth.layer_inputs(wl, 3, dev)
    case = _workload_case(wl)
    e = synth.layer_errors(wl)
    budgets = []
    for L in wl.seq_lens:
        total, m, M = synth.budget_params(wl, L)
        b, st = ckv.ckv_allocate_budgets(e, total, m, M)
        assert st == ckv.CKV_OK
        budgets.append(int(b[3]))
    out = run_gpu(case, inp.mask, inp.q_win, inp.k, inp.v, budgets)
    for s, L in enumerate(wl.seq_lens):
        g = s % case.n_kv
        rs, ri = oracle_group(case, inp.mask, inp.q_win[s], inp.k[s], g, budgets[s])
        check_group(case, out[s], g, rs, ri, inp.k[s].cpu(), inp.v[s].cpu(), "qwen seq%d" % s)
    # the batched call equals one call per prompt
    for s in range(len(wl.seq_lens)):
        single = run_gpu(case, inp.mask, [inp.q_win[s]], [inp.k[s]], [inp.v[s]], [budgets[s]])[0]
        np.testing.assert_array_equal(single["scores"], out[s]["scores"])
        np.testing.assert_array_equal(single["idx"], out[s]["idx"])


def test_select_on_oracle_scores_is_exact(dev):
    # ckv_select alone, fed the oracle's scores rounded to fp32: the indices
    # must equal the oracle's selection on the same fp32 values exactly
    case = Case(8, 2, 64, 8, "max", 7, torch.bfloat16)
    rng = np.random.default_rng(3)
    L = 20000
    desc = case.desc()
    for budget in (8, 9, 100, 4096, 19991, 19999, 20000):
        scores = np.round(rng.random((2, L - 8)), 3).astype(np.float32)  # many ties
        sc = torch.from_numpy(scores).to(dev)
        idx = torch.empty((2, min(budget, L)), dtype=torch.int32, device=dev)
        s = ckv.Seq(None, None, None, budget, scores=sc, idx=idx, seq_len=L)
        ckv.ckv_select(desc, [s], ckv.alloc_workspace(desc, [s], dev))
        torch.cuda.synchronize()
        for g in range(2):
            ref = oracle.select_tokens(scores[g].astype(np.float64), L, 8, budget)
            np.testing.assert_array_equal(idx[g].cpu().numpy(), ref)


def test_gather_is_bitwise(dev):
    case = Case(8, 2, 128, 8, "max", 7, torch.bfloat16)
    L = 5000
    desc = case.desc()
    k = torch.randn((2, L, 128), device=dev).to(torch.bfloat16)
    v = torch.randn((2, L, 128), device=dev).to(torch.bfloat16)
    rng = np.random.default_rng(4)
    idx_np = np.stack([np.sort(rng.choice(L, 300, replace=False)) for _ in range(2)]).astype(np.int32)
    s = ckv.Seq(None, k, v, 300, idx=torch.from_numpy(idx_np).to(dev),
                k_out=torch.empty((2, 300, 128), dtype=torch.bfloat16, device=dev),
                v_out=torch.empty((2, 300, 128), dtype=torch.bfloat16, device=dev))
    ckv.ckv_gather(desc, [s])
    torch.cuda.synchronize()
    kc = k.cpu().view(torch.int16).numpy()
    for g in range(2):
        np.testing.assert_array_equal(s.k_out[g].cpu().view(torch.int16).numpy(),
                                      oracle.gather_rows(kc[g], idx_np[g]))


def test_strided_inputs(dev):
    # K/V stored token-major [L, n_kv, d] and Q a slice of a wider buffer
    case = Case(8, 2, 128, 16, "max", 7, torch.bfloat16)
    q, k, v, mask = random_inputs(case, 3000, seed=12, device="cpu", n_sel=2)
    big_q = torch.zeros((case.H, case.w + 3, case.d), dtype=case.dtype)
    big_q[:, 2:2 + case.w] = q
    q_view = big_q.to(dev)[:, 2:2 + case.w]
    k_t = k.permute(1, 0, 2).contiguous().to(dev).permute(1, 0, 2)
    v_t = v.permute(1, 0, 2).contiguous().to(dev).permute(1, 0, 2)
    assert k_t.stride() == (case.d, case.n_kv * case.d, 1)
    out = run_gpu(case, mask, [q_view], [k_t], [v_t], [300])[0]
    for g in range(case.n_kv):
        rs, ri = oracle_group(case, mask, q, k, g, 300)
        check_group(case, out, g, rs, ri, k, v, "strided")


def test_deterministic(dev):
    case = Case(32, 8, 128, 32, "max", 7, torch.bfloat16)
    q, k, v, mask = random_inputs(case, 20000, seed=13, device=dev, n_sel=2)
    a = run_gpu(case, mask, [q], [k], [v], [700])[0]
    b = run_gpu(case, mask, [q], [k], [v], [700])[0]
    np.testing.assert_array_equal(a["scores"], b["scores"])
    np.testing.assert_array_equal(a["idx"], b["idx"])


def test_graph_replay_matches_eager(dev):
    case = Case(32, 8, 128, 32, "max", 7, torch.bfloat16)
    q, k, v, mask = random_inputs(case, 10000, seed=14, device=dev, n_sel=2)
    eager = run_gpu(case, mask, [q], [k], [v], [500])[0]
    desc = case.desc()
    s = ckv.alloc_outputs(desc, ckv.Seq(q, k, v, 500))
    ws = ckv.alloc_workspace(desc, [s], dev)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        ckv.ckv_compress_layer(desc, mask, [s], ws)  # warm-up outside capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        ckv.ckv_compress_layer(desc, mask, [s], ws)
    for rep in range(3):
        s.scores.fill_(-1.0)
        s.idx.fill_(-1)
        s.k_out.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(s.scores.cpu().numpy(), eager["scores"], err_msg="rep %d" % rep)
        np.testing.assert_array_equal(s.idx.cpu().numpy(), eager["idx"], err_msg="rep %d" % rep)
        assert torch.equal(s.k_out.cpu(), eager["k_out"])
