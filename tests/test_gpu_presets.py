"""GPU parity of the comparison presets the paper discusses in Sec. 2:
StreamingLLM-style retention (first and last tokens; ckv_streaming_select)
and SnapKV-style selection (every head of a group scores its tokens;
ckv_compress_layer with snapkv_mask). Index rows and compact caches are
integer / byte results: bit-exact against the oracle."""
import zlib

import numpy as np
import pytest
import torch

import oracle
import paper_2508_02401_amd as ckv
from tests.gpu_util import Case, check_group, oracle_group, random_inputs, run_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ckv.load()
    return torch.device("cuda:0")


def _bits(t: torch.Tensor) -> np.ndarray:
    """The raw bit patterns of a bf16 / f16 / f32 tensor."""
    return t.contiguous().view(torch.int32 if t.dtype == torch.float32 else torch.int16).numpy()


STREAM_CASES = [
    # (label, Case, [(L, budget), ...] prompts, n_sink)
    ("bf16-d128-llama", Case(32, 8, 128, 32, "max", 7, torch.bfloat16), [(5000, 256)], 4),
    ("bf16-ragged-batch", Case(8, 2, 128, 16, "max", 7, torch.bfloat16),
     [(300, 64), (1000, 1000), (77, 500), (4097, 129)], 4),
    ("f16-d64-no-sinks", Case(28, 4, 64, 32, "avg", 5, torch.float16), [(2500, 100)], 0),
    ("f32-sinks-exceed-budget", Case(8, 2, 64, 16, "avg", 3, torch.float32), [(900, 40)], 64),
    ("bf16-shared", Case(32, 8, 128, 32, "max", 7, torch.bfloat16, shared=True), [(3000, 200)], 4),
]


@pytest.mark.parametrize("label,case,prompts,n_sink", STREAM_CASES, ids=[c[0] for c in STREAM_CASES])
def test_streaming_select_parity(dev, label, case, prompts, n_sink):
    desc = case.desc()
    seqs, inputs = [], []
    for i, (L, B) in enumerate(prompts):
        _, k, v, _ = random_inputs(case, L, seed=zlib.crc32(label.encode()) % 1000 + i, device="cpu")
        s = ckv.Seq(None, k.to(dev), v.to(dev), B)
        ckv.alloc_outputs(desc, s, with_scores=False)
        seqs.append(s)
        inputs.append((k, v))
    print("case", label, flush=True)
    ckv.ckv_streaming_select(desc, seqs, n_sink)
    torch.cuda.synchronize()
    for (L, B), s, (k, v) in zip(prompts, seqs, inputs):
        ref = oracle.streaming_indices(L, B, n_sink)
        idx = s.idx.cpu().numpy()
        rows = [idx[0]] if case.shared else list(idx)
        for r in rows:
            np.testing.assert_array_equal(r, ref, err_msg=label)
        kout, vout = s.k_out.cpu(), s.v_out.cpu()
        for g in range(case.n_kv):
            np.testing.assert_array_equal(_bits(kout[g]), oracle.gather_rows(_bits(k[g]), ref))
            np.testing.assert_array_equal(_bits(vout[g]), oracle.gather_rows(_bits(v[g]), ref))


SNAP_CASES = [
    # (label, Case, L, budget): every query head of every group chosen
    ("bf16-llama-G4", Case(32, 8, 128, 32, "max", 7, torch.bfloat16), 4000, 300),
    ("f16-d64-G7", Case(28, 4, 64, 16, "avg", 5, torch.float16), 2100, 200),
]


@pytest.mark.parametrize("label,case,L,budget", SNAP_CASES, ids=[c[0] for c in SNAP_CASES])
def test_snapkv_preset_parity(dev, label, case, L, budget):
    mask = ckv.snapkv_mask(case.H)
    q, k, v, _ = random_inputs(case, L, seed=zlib.crc32(label.encode()) % 10000, device="cpu",
                               mask=mask)
    print("case", label, flush=True)
    out = run_gpu(case, mask, [q.to(dev)], [k.to(dev)], [v.to(dev)], [budget])[0]
    for g in range(case.n_kv):
        rs, ri = oracle_group(case, mask, q, k, g, budget)
        check_group(case, out, g, rs, ri, k, v, label)
