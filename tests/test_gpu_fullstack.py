"""Whole-stack GPU parity: ckv_compress_stack over every layer of the three
multi-layer workloads (the configurations the throughput is quoted on),
with their Algorithm 1 budgets, and every (layer, prompt, KV head) compared
with the fp64 oracle under the rules in tests/parity.py:

  * llama8b-128k-stack: 32 layers, L = 131072, w = 64, 1-2 heads per group;
  * llama8b-32k-stack:  32 layers, L = 32768,  w = 32, 1-2 heads per group;
  * qwen7b-ragged-batch: 28 layers, 4 ragged prompts per layer
    (L = 8192, 24576, 65536, 98304), 28 query / 4 KV heads, w = 32.

The stack runs as the benchmark runs it (one workspace slot per layer, the
selection of all layers in one batch). The oracle's group selection is
single-threaded C, so independent (layer, prompt, KV head) checks run
concurrently on a thread pool sized to the host's CPU share.
"""
import concurrent.futures as cf
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2508_02401_amd as ckv
from paper_2508_02401_amd import synth
from tests.gpu_util import Case, check_group, oracle_group

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ckv.load()
    return torch.device("cuda:0")


def _threads() -> int:
    n = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    return max(1, min(n or 1, 16))


def _budgets(wl):
    """[prompt][layer] Algorithm 1 budgets from the library, checked against
    the oracle's allocation."""
    out = []
    errs = synth.layer_errors(wl)
    for L in wl.seq_lens:
        total, m, M = synth.budget_params(wl, L)
        b, st = ckv.ckv_allocate_budgets(errs, total, m, M)
        assert st == ckv.CKV_OK
        ref, rst = oracle.allocate_budgets(errs, total, m, M)
        assert rst == oracle.OK and [int(x) for x in b] == [int(x) for x in ref]
        out.append([int(x) for x in b])
    return out


def _check_whole_stack(name, dev):
    wl = synth.WORKLOADS[name]
    case = Case(wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.window,
                "max" if wl.pool == 1 else "avg", wl.pool_kernel, wl.dtype)
    desc = case.desc()
    budgets = _budgets(wl)
    print("case %s: drawing %d layers" % (name, wl.n_layers), flush=True)
    inputs, seqs = [], []
    for l in range(wl.n_layers):
        inp = synth.layer_inputs(wl, l, dev)
        inputs.append(inp)
        layer = []
        for s in range(len(wl.seq_lens)):
            x = ckv.alloc_outputs(desc, ckv.Seq(inp.q_win[s], inp.k[s], inp.v[s], budgets[s][l]))
            x.scores.fill_(-1.0)
            x.idx.fill_(-7)
            layer.append(x)
        seqs.append(layer)
    one = max(ckv.ckv_workspace_bytes(desc, layer) for layer in seqs)
    ws = torch.empty(wl.n_layers * one, dtype=torch.uint8, device=dev)
    masks = np.stack([inp.mask for inp in inputs])
    print("case %s: ckv_compress_stack" % name, flush=True)
    ckv.ckv_compress_stack(desc, masks, seqs, ws, torch.cuda.current_stream(), None)
    torch.cuda.synchronize()
    del ws

    def check(l, s, g, out):
        inp = inputs[l]
        rs, ri = oracle_group(case, inp.mask, inp.q_win[s], inp.k[s], g, budgets[s][l])
        return check_group(case, out, g, rs, ri, inp.k[s], inp.v[s],
                           "%s layer %d prompt %d" % (name, l, s))

    jobs = []
    with cf.ThreadPoolExecutor(max_workers=_threads()) as ex:
        for l in range(wl.n_layers):
            for s, x in enumerate(seqs[l]):
                out = dict(scores=x.scores.cpu().numpy(), idx=x.idx.cpu().numpy(),
                           k_out=x.k_out.cpu(), v_out=x.v_out.cpu())
                for g in range(wl.num_kv_heads):
                    jobs.append(ex.submit(check, l, s, g, out))
        worst, swaps = 0.0, 0
        for j in jobs:
            rel, sw = j.result()
            worst, swaps = max(worst, rel), swaps + sw
    n = wl.n_layers * len(wl.seq_lens) * wl.num_kv_heads
    assert len(jobs) == n
    print("case %s: %d (layer, prompt, KV head) selections match the oracle; max score rel err "
          "%.2e, %d tie swaps" % (name, n, worst, swaps), flush=True)


def test_whole_stack_llama8b_128k(dev):
    _check_whole_stack("llama8b-128k-stack", dev)


def test_whole_stack_llama8b_32k(dev):
    _check_whole_stack("llama8b-32k-stack", dev)


def test_whole_stack_qwen7b_ragged_batch(dev):
    _check_whole_stack("qwen7b-ragged-batch", dev)
