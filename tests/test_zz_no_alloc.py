"""ckv_compress_layer_noalloc (library-held workspace) against
ckv_compress_layer (caller workspace) on the same inputs: two calls in a row,
the second smaller, on the same GPU, so the second runs on what the first left
in the library's array. Same kernels and arguments apart from the workspace
address, so every output must match bit for bit; one KV head of the small call
is also checked against the oracle.
"""
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


def _seqs(desc, qs, ks, vs, budgets):
    seqs = []
    for q, k, v, b in zip(qs, ks, vs, budgets):
        s = ckv.Seq(q, k, v, int(b))
        ckv.alloc_outputs(desc, s, with_scores=True)
        seqs.append(s)
    return seqs


def _both(desc, mask, qs, ks, vs, budgets, stream=None):
    """Run the no-allocation entry point, then ckv_compress_layer with a
    caller workspace filled with a nonzero pattern; return both outputs."""
    a = _seqs(desc, qs, ks, vs, budgets)
    b = _seqs(desc, qs, ks, vs, budgets)
    need = ckv.ckv_workspace_bytes(desc, a)
    assert 0 < need <= ckv.CKV_NOALLOC_MAX_WORKSPACE_BYTES
    ckv.ckv_compress_layer_noalloc(desc, mask, a, stream=stream)
    ws = torch.full((need,), 0xA5, dtype=torch.uint8, device=ks[0].device)
    ckv.ckv_compress_layer(desc, mask, b, ws, stream=stream)
    torch.cuda.synchronize()
    return a, b


def _assert_same(a, b, label):
    for i, (x, y) in enumerate(zip(a, b)):
        for name in ("scores", "idx", "k_out", "v_out"):
            tx, ty = getattr(x, name), getattr(y, name)
            assert torch.equal(tx.view(torch.uint8) if tx.dtype != torch.int32 else tx,
                               ty.view(torch.uint8) if ty.dtype != torch.int32 else ty), \
                "%s prompt %d: %s differs" % (label, i, name)


def test_noalloc_matches_caller_workspace_twice(dev):
    # call 1: one 131072-token prompt of the llama8b-128k-stack layer shape
    # (32 query / 8 KV heads, dim 128, w = 64), about 36 MiB of workspace
    wl = synth.WORKLOADS["llama8b-128k-stack"]
    inp = synth.layer_inputs(wl, 5, dev)
    case = Case(wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.window,
                "max" if wl.pool == 1 else "avg", wl.pool_kernel, wl.dtype)
    desc = case.desc()
    budgets = [1500 + 37 * i for i in range(len(wl.seq_lens))]
    print("case noalloc call 1: llama8b 131072 tokens", flush=True)
    a, b = _both(desc, inp.mask, inp.q_win, inp.k, inp.v, budgets)
    _assert_same(a, b, "call 1")
    del inp, a, b

    # call 2: smaller, other shape and parameters (28 query / 4 KV heads,
    # w = 32, avg pooling, fp16, two ragged prompts), on a side stream
    case2 = Case(28, 4, 128, 32, "avg", 5, torch.float16)
    desc2 = case2.desc()
    ins = [random_inputs(case2, L, seed=91 + i, device=dev, n_sel=2) for i, L in enumerate((3001, 1234))]
    mask2 = ins[0][3]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    print("case noalloc call 2: 28/4 heads, 3001 + 1234 tokens, side stream", flush=True)
    with torch.cuda.stream(side):
        a2, b2 = _both(desc2, mask2, [x[0] for x in ins], [x[1] for x in ins], [x[2] for x in ins],
                       [300, 200], stream=side)
    _assert_same(a2, b2, "call 2")
    # and the oracle on one KV head of the first prompt
    q, k, v, _ = ins[0]
    rs, ri = oracle_group(case2, mask2, q.cpu(), k.cpu(), 1, 300)
    out = dict(scores=a2[0].scores.cpu().numpy(), idx=a2[0].idx.cpu().numpy(),
               k_out=a2[0].k_out.cpu(), v_out=a2[0].v_out.cpu())
    check_group(case2, out, 1, rs, ri, k.cpu(), v.cpu(), "noalloc call 2")


def test_noalloc_rejects_oversize_and_bad_args(dev):
    # a prompt whose workspace exceeds the library's array is refused before
    # anything runs; invalid arguments give ckv_compress_layer's status
    case = Case(32, 8, 128, 64, "max", 7, torch.bfloat16)
    desc = case.desc()
    L = 600000
    k = torch.empty((8, L, 128), dtype=torch.bfloat16, device=dev)
    q = torch.empty((32, 64, 128), dtype=torch.bfloat16, device=dev)
    s = _seqs(desc, [q], [k], [k], [1000])
    assert ckv.ckv_workspace_bytes(desc, s) > ckv.CKV_NOALLOC_MAX_WORKSPACE_BYTES
    mask = np.ones(32, np.uint8)
    with pytest.raises(ckv.CkvError) as e:
        ckv.ckv_compress_layer_noalloc(desc, mask, s)
    assert e.value.status == ckv.CKV_ERR_WORKSPACE
    bad = case.desc()
    bad.pool_kernel = 4
    with pytest.raises(ckv.CkvError) as e:
        ckv.ckv_compress_layer_noalloc(bad, mask, s)
    assert e.value.status == ckv.CKV_ERR_INVALID_ARG
