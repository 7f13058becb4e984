"""GPU parity of ckv_compress_stack (the whole path over a stack of layers:
the K passes layer by layer, the selection stages in launches that cover a
batch of layers, on a side stream beside the next batch's K passes or on the
same stream): every layer's scores, indices and compact K/V equal those of
ckv_compress_layer on the same inputs bit for bit, for several batch sizes
with and without the side stream, and match the fp64 oracle under the rules
in tests/parity.py."""
import numpy as np
import pytest
import torch

import paper_2508_02401_amd as ckv
from paper_2508_02401_amd import synth
from tests.gpu_util import Case, check_group, oracle_group, random_inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ckv.load()
    return torch.device("cuda:0")


def _outputs(desc, layer_inputs):
    """Fresh output buffers for every layer: [layer][prompt] Seq."""
    out = []
    for mask, qs, ks, vs, budgets in layer_inputs:
        seqs = []
        for q, k, v, b in zip(qs, ks, vs, budgets):
            s = ckv.alloc_outputs(desc, ckv.Seq(q, k, v, int(b)), with_scores=True)
            s.scores.fill_(-1.0)
            s.idx.fill_(-7)
            seqs.append(s)
        out.append(seqs)
    return out


def _run_stack(desc, layer_inputs, dev, side, slots=None):
    """ckv_compress_stack with `slots` layer slots of workspace (default: the
    fewest the schedule accepts; more slots mean larger selection batches)."""
    seqs = _outputs(desc, layer_inputs)
    one = ckv.ckv_workspace_bytes(desc, seqs[0])
    slots = slots if slots is not None else (2 if side else 1)
    ws = torch.empty(slots * one + 100, dtype=torch.uint8, device=dev)
    masks = np.stack([li[0] for li in layer_inputs])
    side_stream = torch.cuda.Stream() if side else None
    ckv.ckv_compress_stack(desc, masks, seqs, ws, torch.cuda.current_stream(), side_stream)
    torch.cuda.synchronize()
    return seqs


def _run_layers(desc, layer_inputs, dev):
    seqs = _outputs(desc, layer_inputs)
    ws = ckv.alloc_workspace(desc, seqs[0], dev)
    for (mask, *_), layer in zip(layer_inputs, seqs):
        ckv.ckv_compress_layer(desc, mask, layer, ws)
    torch.cuda.synchronize()
    return seqs


def _assert_same(a, b, label):
    for l, (la, lb) in enumerate(zip(a, b)):
        for p, (sa, sb) in enumerate(zip(la, lb)):
            for f in ("scores", "idx", "k_out", "v_out"):
                assert torch.equal(getattr(sa, f), getattr(sb, f)), "%s layer %d prompt %d %s" % (
                    label, l, p, f)


def _as_dict(s):
    return dict(scores=s.scores.cpu().numpy(), idx=s.idx.cpu().numpy(), k_out=s.k_out.cpu(),
                v_out=s.v_out.cpu())


@pytest.mark.parametrize("side,slots", [(True, 2), (False, 1), (False, 2), (False, 5),
                                        (True, 4), (True, 10)],
                         ids=["side-batch1", "one-batch1", "one-batch2-ragged", "one-batch5",
                              "side-batch2-ragged", "side-batch5"])
def test_small_stack_matches_layer_calls_and_oracle(dev, side, slots):
    case = Case(16, 4, 128, 32, "max", 7, torch.bfloat16)
    lens = (3000, 1100)
    # per-layer budgets per prompt: ordinary, the window alone, keep-all,
    # one past the window, and large
    budgets = [(200, 64), (32, 32), (5000, 1100), (33, 1099), (2999, 500)]
    layer_inputs = []
    for l, bl in enumerate(budgets):
        qs, ks, vs = [], [], []
        mask = None
        for p, L in enumerate(lens):
            q, k, v, m = random_inputs(case, L, seed=100 * l + p, device="cpu", mask=mask)
            mask = m  # one mask per layer, shared by its prompts
            qs.append(q.to(dev))
            ks.append(k.to(dev))
            vs.append(v.to(dev))
        layer_inputs.append((mask, qs, ks, vs, bl))
    desc = case.desc()
    got = _run_stack(desc, layer_inputs, dev, side, slots)
    ref = _run_layers(desc, layer_inputs, dev)
    _assert_same(got, ref, "stack vs layer calls")
    for l, (mask, qs, ks, vs, bl) in enumerate(layer_inputs):
        for p in range(len(lens)):
            out = _as_dict(got[l][p])
            for g in range(case.n_kv):
                rs, ri = oracle_group(case, mask, qs[p].cpu(), ks[p].cpu(), g, bl[p])
                check_group(case, out, g, rs, ri, ks[p].cpu(), vs[p].cpu(),
                            "stack layer %d prompt %d" % (l, p))


def test_full_size_stack_128k(dev):
    # four layers of the 32-layer Llama-3.1-8B-shaped L = 131072 workload, with
    # their Algorithm 1 budgets; bit-exact against per-layer calls, and one
    # sampled KV head of every layer against the oracle
    wl = synth.WORKLOADS["llama8b-128k-stack"]
    total, m, M = synth.budget_params(wl, wl.seq_lens[0])
    budgets, st = ckv.ckv_allocate_budgets(synth.layer_errors(wl), total, m, M)
    assert st == ckv.CKV_OK
    case = Case(wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.window, "max", wl.pool_kernel,
                wl.dtype)
    layer_inputs = []
    for l in range(4):
        inp = synth.layer_inputs(wl, l, dev)
        layer_inputs.append((inp.mask, inp.q_win, inp.k, inp.v, [int(budgets[l])]))
    desc = case.desc()
    print("stack of 4 layers at L=131072", flush=True)
    got = _run_stack(desc, layer_inputs, dev, False, slots=4)
    ref = _run_layers(desc, layer_inputs, dev)
    _assert_same(got, ref, "128k stack (one batch) vs layer calls")
    got = _run_stack(desc, layer_inputs, dev, True)
    ref = _run_layers(desc, layer_inputs, dev)
    _assert_same(got, ref, "128k stack vs layer calls")
    for l, (mask, qs, ks, vs, bl) in enumerate(layer_inputs):
        g = (3 * l + 1) % case.n_kv
        k_cpu = ks[0].cpu()
        rs, ri = oracle_group(case, mask, qs[0].cpu(), k_cpu, g, bl[0])
        check_group(case, _as_dict(got[l][0]), g, rs, ri, k_cpu, vs[0].cpu(), "128k layer %d" % l)


def test_stack_rejects_a_bad_layer_before_launching(dev):
    case = Case(8, 2, 64, 16, "avg", 5, torch.bfloat16)
    layer_inputs = []
    for l in range(3):
        q, k, v, mask = random_inputs(case, 700, seed=l, device="cpu", n_sel=1)
        layer_inputs.append((mask, [q.to(dev)], [k.to(dev)], [v.to(dev)], [100]))
    bad = layer_inputs[2][0].copy()
    bad[4:] = 0  # group 1 has no chosen head
    layer_inputs[2] = (bad,) + layer_inputs[2][1:]
    desc = case.desc()
    seqs = _outputs(desc, layer_inputs)
    ws = torch.empty(2 * ckv.ckv_workspace_bytes(desc, seqs[0]), dtype=torch.uint8, device=dev)
    with pytest.raises(ckv.CkvError) as err:
        ckv.ckv_compress_stack(desc, np.stack([li[0] for li in layer_inputs]), seqs, ws,
                               torch.cuda.current_stream(), torch.cuda.Stream())
    assert err.value.status == ckv.CKV_ERR_MASK
    torch.cuda.synchronize()
    for layer in seqs:  # nothing was launched: the sentinels are intact
        assert bool((layer[0].idx == -7).all()) and bool((layer[0].scores == -1.0).all())


def test_stack_ties_long_prompts_and_big_budgets(dev):
    # The stack's selection (one workgroup per layer and KV head) against the
    # per-layer kernels and the oracle where its rarer paths run:
    #   layer 0: constant keys, so every prefix score ties; the threshold bin
    #            holds all 139968 keys and is ranked by histogram passes down
    #            to the exact key, and the lowest indices win;
    #   layer 1: random keys with a budget of 20000 (kept rows copied in many
    #            rounds), the output in two 131072-token segments;
    #   layer 2: constant keys plus a planted high-scoring span, so the span
    #            is kept and the remaining slots go to the lowest indices.
    case = Case(8, 2, 128, 32, "max", 7, torch.bfloat16)
    L = 140000
    layer_inputs = []
    for l, budget in enumerate((10032, 20000, 6000)):
        q, k, v, mask = random_inputs(case, L, seed=900 + l, device="cpu", n_sel=2)
        if l != 1:
            k = k[:, :1, :].expand(-1, L, -1).contiguous()
        if l == 2:
            G = case.H // case.n_kv
            for g in range(case.n_kv):
                qbar = q[g * G:(g + 1) * G].float().mean(dim=(0, 1))
                k[g, 50000:50400] = (k[g, 50000:50400].float()
                                     + 4.0 * qbar / qbar.norm() ** 2 * case.d ** 0.5).to(k.dtype)
        layer_inputs.append((mask, [q.to(dev)], [k.to(dev)], [v.to(dev)], [budget]))
    desc = case.desc()
    print("stack of 3 layers at L=140000", flush=True)
    got = _run_stack(desc, layer_inputs, dev, False, slots=3)
    ref = _run_layers(desc, layer_inputs, dev)
    _assert_same(got, ref, "ties/long stack vs layer calls")
    for l, (mask, qs, ks, vs, bl) in enumerate(layer_inputs):
        g = l % case.n_kv
        k_cpu = ks[0].cpu()
        rs, ri = oracle_group(case, mask, qs[0].cpu(), k_cpu, g, bl[0])
        check_group(case, _as_dict(got[l][0]), g, rs, ri, k_cpu, vs[0].cpu(), "ties layer %d" % l)
    # the tie rule itself: with constant keys the kept prefix is 0..n_keep-1
    assert np.array_equal(got[0][0].idx.cpu().numpy()[0, :10000], np.arange(10000))


def test_stack_with_row_groups_beyond_128_rows(dev):
    # layers whose groups hold 3-4 chosen heads at w = 64 (192-256 rows, read
    # as two row groups): the stack equals the per-layer calls bit for bit and
    # matches the oracle
    case = Case(16, 4, 128, 64, "max", 7, torch.bfloat16)
    layer_inputs, cpu = [], []
    for l in range(3):
        q, k, v, mask = random_inputs(case, 1700, seed=60 + l, device="cpu", n_sel=3 + l % 2)
        layer_inputs.append((mask, [q.to(dev)], [k.to(dev)], [v.to(dev)], [200 + 50 * l]))
        cpu.append((mask, q, k, v, 200 + 50 * l))
    desc = case.desc()
    print("case stack row groups", flush=True)
    stacked = _run_stack(desc, layer_inputs, dev, side=False, slots=2)
    _assert_same(stacked, _run_layers(desc, layer_inputs, dev), "row groups")
    for l, (mask, q, k, v, b) in enumerate(cpu):
        out = _as_dict(stacked[l][0])
        for g in range(case.n_kv):
            rs, ri = oracle_group(case, mask, q, k, g, b)
            check_group(case, out, g, rs, ri, k, v, "layer %d" % l)


@pytest.mark.parametrize("pool,kp", [("max", 1), ("avg", 3), ("max", 9), ("avg", 15), ("max", 31)],
                         ids=["max-k1", "avg-k3", "max-k9", "avg-k15", "max-k31"])
def test_stack_pooling_radii_and_gather_split(dev, pool, kp):
    # The stack's pooling kernel at halo widths 0-4 chunks (radius 0 to 15) over
    # a ragged 8192-score span and tail, and both ways of copying the kept rows:
    # budgets of 512 rows per unit copy in the selection launch, 513 in a gather
    # launch of their own. One layer per batch (each way alone) and both layers in
    # one batch (the split then covers both); bit-exact against per-layer calls,
    # and every KV head of both layers against the oracle.
    case = Case(8, 2, 64, 16, pool, kp, torch.bfloat16)
    L = 8192 + 2 * 1024 + 16 + 5  # ragged: the scored span is not a multiple of 4
    layer_inputs, cpu = [], []
    for l, budget in enumerate((512, 513)):
        q, k, v, mask = random_inputs(case, L, seed=700 + 10 * kp + l, device="cpu", n_sel=1 + l)
        layer_inputs.append((mask, [q.to(dev)], [k.to(dev)], [v.to(dev)], [budget]))
        cpu.append((mask, q, k, v, budget))
    desc = case.desc()
    print("stack pool %s k=%d" % (pool, kp), flush=True)
    ref = _run_layers(desc, layer_inputs, dev)
    for slots in (1, 2):
        got = _run_stack(desc, layer_inputs, dev, False, slots=slots)
        _assert_same(got, ref, "pool %s k=%d slots %d" % (pool, kp, slots))
    for l, (mask, q, k, v, b) in enumerate(cpu):
        out = _as_dict(got[l][0])
        for g in range(case.n_kv):
            rs, ri = oracle_group(case, mask, q, k, g, b)
            check_group(case, out, g, rs, ri, k, v, "pool %s k=%d layer %d" % (pool, kp, l))
