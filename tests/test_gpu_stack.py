"""GPU parity of ckv_compress_stack (the whole path over a stack of layers,
with the selection of layer l on a side stream beside the K passes of layer
l+1): every layer's scores, indices and compact K/V equal those of
ckv_compress_layer on the same inputs bit for bit, with and without the side
stream, and match the fp64 oracle under the rules in tests/parity.py."""
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


def _run_stack(desc, layer_inputs, dev, side):
    seqs = _outputs(desc, layer_inputs)
    one = ckv.ckv_workspace_bytes(desc, seqs[0])
    ws = torch.empty((2 if side else 1) * one, dtype=torch.uint8, device=dev)
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


@pytest.mark.parametrize("side", [True, False], ids=["side-stream", "one-stream"])
def test_small_stack_matches_layer_calls_and_oracle(dev, side):
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
    got = _run_stack(desc, layer_inputs, dev, side)
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
