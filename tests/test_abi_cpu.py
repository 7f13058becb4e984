"""Host-side checks of libckv.so that need no GPU: it loads, exports every
symbol include/ckv.h declares, rejects bad arguments before launching
anything, and its Algorithm 1 agrees with the oracle's."""
import ctypes
import os
import re

import numpy as np
import pytest
import torch

import oracle
import paper_2508_02401_amd as ckv
from paper_2508_02401_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    text = open(os.path.join(ROOT, "include", "ckv.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ckv_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(ckv.LIB_PATH)
    names = _declared_functions()
    assert set(names) == set(ckv.EXPORTED)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings():
    for code in (0, -1, -2, -3, -4, -5, -6):
        assert ckv.ckv_status_string(code) != "unknown status"
    assert ckv.ckv_status_string(-99) == "unknown status"


# Fake device buffers: validation only looks at null/alignment, and every
# case below must fail before any HIP call.
_BUF = np.zeros(1 << 16, dtype=np.uint8)
_BASE = (_BUF.ctypes.data + 255) & ~255


def _desc(**kw):
    base = dict(num_q_heads=8, num_kv_heads=2, head_dim=64, window=4, dtype=ckv.CKV_BF16,
                scale=0.0, pool=ckv.CKV_POOL_MAX, pool_kernel=7, flags=ckv.CKV_KEEP_WINDOW)
    base.update(kw)
    d = ckv._binding.ckv_layer_desc()
    for k, v in base.items():
        setattr(d, k, v)
    return d


def _seq(**kw):
    s = ckv._binding.ckv_seq()
    vals = dict(q_win=_BASE, q_stride_head=4 * 64, q_stride_row=64, k=_BASE + 4096,
                v=_BASE + 8192, kv_stride_head=100 * 64, kv_stride_tok=64, seq_len=100, budget=16,
                scores=_BASE + 12288, idx=_BASE + 16384, k_out=_BASE + 20480,
                v_out=_BASE + 24576)
    vals.update(kw)
    for k, v in vals.items():
        setattr(s, k, v)
    return s


def _call(fn, desc, seq, mask=None, ws=True, n=1):
    lib = ckv.load()
    arr = (ckv._binding.ckv_seq * n)(*([seq] * n))
    ws_ptr = _BASE + 32768 if ws else None
    ws_n = 1 << 40 if ws else 0
    if fn == "score" or fn == "compress":
        m = np.ones(desc.num_q_heads, np.uint8) if mask is None else np.asarray(mask, np.uint8)
        mm = (ctypes.c_uint8 * m.size)(*m.tolist())
        f = lib.ckv_score if fn == "score" else lib.ckv_compress_layer
        return f(ctypes.byref(desc), mm, arr, n, ws_ptr, ws_n, None)
    if fn == "select":
        return lib.ckv_select(ctypes.byref(desc), arr, n, ws_ptr, ws_n, None)
    return lib.ckv_gather(ctypes.byref(desc), arr, n, None)


@pytest.mark.parametrize("fn", ["score", "compress", "select", "gather"])
@pytest.mark.parametrize("bad,expect", [
    (dict(pool_kernel=4), ckv.CKV_ERR_INVALID_ARG),
    (dict(pool_kernel=0), ckv.CKV_ERR_INVALID_ARG),
    (dict(pool_kernel=33), ckv.CKV_ERR_UNSUPPORTED),
    (dict(pool=5), ckv.CKV_ERR_INVALID_ARG),
    (dict(head_dim=96), ckv.CKV_ERR_UNSUPPORTED),
    (dict(dtype=7), ckv.CKV_ERR_UNSUPPORTED),
    (dict(num_q_heads=7), ckv.CKV_ERR_INVALID_ARG),
    (dict(window=0), ckv.CKV_ERR_INVALID_ARG),
    (dict(window=129), ckv.CKV_ERR_UNSUPPORTED),
    (dict(flags=4), ckv.CKV_ERR_UNSUPPORTED),
    (dict(flags=ckv.CKV_KEEP_WINDOW | ckv.CKV_SHARE_LAYER | 8), ckv.CKV_ERR_UNSUPPORTED),
    (dict(scale=float("nan")), ckv.CKV_ERR_INVALID_ARG),
])
def test_bad_descriptor(fn, bad, expect):
    assert _call(fn, _desc(**bad), _seq()) == expect


def test_keep_window_off_budget_rules_and_workspace():
    # without CKV_KEEP_WINDOW every token competes: a budget below the window
    # is fine, a budget of 0 is not; all L columns are scored, so the
    # workspace grows by the window's columns
    lib = ckv.load()
    on, off = _desc(), _desc(flags=0)
    arr = (ckv._binding.ckv_seq * 1)(_seq())
    w_on = lib.ckv_workspace_bytes(ctypes.byref(on), arr, 1)
    w_off = lib.ckv_workspace_bytes(ctypes.byref(off), arr, 1)
    assert w_off > w_on > 0
    assert _call("compress", on, _seq(budget=on.window - 1)) == ckv.CKV_ERR_BUDGET
    assert _call("compress", off, _seq(budget=0)) == ckv.CKV_ERR_BUDGET
    # validation passes (the launch then fails here, where there is no GPU)
    assert _call("compress", off, _seq(budget=1)) not in (ckv.CKV_ERR_BUDGET,
                                                           ckv.CKV_ERR_INVALID_ARG,
                                                           ckv.CKV_ERR_UNSUPPORTED)


@pytest.mark.parametrize("fn", ["score", "compress", "select", "gather"])
@pytest.mark.parametrize("bad,expect", [
    (dict(budget=3), ckv.CKV_ERR_BUDGET),          # below the window of 4
    (dict(seq_len=4), ckv.CKV_ERR_INVALID_ARG),    # L must exceed w
    (dict(seq_len=1 << 31), ckv.CKV_ERR_INVALID_ARG),
])
def test_bad_sequence(fn, bad, expect):
    assert _call(fn, _desc(), _seq(**bad)) == expect


@pytest.mark.parametrize("fn,field", [
    ("score", "q_win"), ("score", "k"), ("score", "scores"), ("compress", "v"),
    ("compress", "idx"), ("compress", "k_out"), ("select", "scores"), ("select", "idx"),
    ("gather", "k"), ("gather", "v_out"), ("gather", "idx"),
])
def test_null_pointer(fn, field):
    assert _call(fn, _desc(), _seq(**{field: None})) == ckv.CKV_ERR_INVALID_ARG


@pytest.mark.parametrize("field", ["q_win", "k", "scores"])
def test_misaligned_pointer(field):
    s = _seq()
    assert _call("score", _desc(), _seq(**{field: getattr(s, field) + 2})) == ckv.CKV_ERR_INVALID_ARG


def test_misaligned_stride():
    assert _call("score", _desc(), _seq(kv_stride_tok=65)) == ckv.CKV_ERR_INVALID_ARG
    assert _call("score", _desc(), _seq(q_stride_row=63)) == ckv.CKV_ERR_INVALID_ARG


def test_group_without_chosen_head():
    mask = [1, 0, 0, 0, 0, 0, 0, 0]  # group 1 (heads 4..7) has none
    assert _call("score", _desc(), _seq(), mask=mask) == ckv.CKV_ERR_MASK
    assert _call("compress", _desc(), _seq(), mask=mask) == ckv.CKV_ERR_MASK


def test_row_groups_size_the_workspace():
    # a group's chosen rows are read in row groups of at most 128, each with
    # its own K-pass partials: the workspace grows with the row groups a
    # group can need (1 at w = 32 with 4 heads, 2 at w = 64, 4 at w = 128)
    sizes = [ckv.ckv_workspace_bytes(_desc(window=w), [ckv.Seq(None, None, None, 200, seq_len=4000)])
             for w in (32, 64, 128)]
    assert 0 < sizes[0] < sizes[1] < sizes[2]


def test_missing_or_small_workspace():
    assert _call("score", _desc(), _seq(), ws=False) == ckv.CKV_ERR_WORKSPACE
    lib = ckv.load()
    d, s = _desc(), _seq()
    arr = (ckv._binding.ckv_seq * 1)(s)
    need = lib.ckv_workspace_bytes(ctypes.byref(d), arr, 1)
    assert need > 0
    m = (ctypes.c_uint8 * 8)(*([1] * 8))
    rc = lib.ckv_score(ctypes.byref(d), m, arr, 1, _BASE + 32768, need - 1, None)
    assert rc == ckv.CKV_ERR_WORKSPACE


def test_too_many_sequences():
    assert _call("select", _desc(), _seq(), n=17) == ckv.CKV_ERR_UNSUPPORTED


def test_workspace_bytes_grows_with_length():
    lib = ckv.load()
    d = _desc()
    a = (ckv._binding.ckv_seq * 1)(_seq(seq_len=1000))
    b = (ckv._binding.ckv_seq * 1)(_seq(seq_len=100000))
    assert 0 < lib.ckv_workspace_bytes(ctypes.byref(d), a, 1) < lib.ckv_workspace_bytes(
        ctypes.byref(d), b, 1)
    bad = (ckv._binding.ckv_seq * 1)(_seq(seq_len=2))
    assert lib.ckv_workspace_bytes(ctypes.byref(d), bad, 1) == 0


# ---------------------------------------------------------------------------
# Algorithm 1: the library's host implementation against the oracle's.
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("seed", range(200))
def test_allocate_budgets_matches_oracle(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 64))
    e = rng.dirichlet(np.ones(n) * float(rng.choice([0.05, 0.5, 1.0, 20.0])))
    if seed % 7 == 0:
        e = np.round(e, 2)  # exact ties and half-way shares
    per = int(rng.integers(8, 3000))
    m = int(rng.integers(0, per + 1))
    M = int(rng.integers(per, 4 * per))
    total = int(n * per + rng.integers(-3 * per, 3 * per))
    got, st = ckv.ckv_allocate_budgets(e, total, m, M)
    ref, rst = oracle.allocate_budgets(e, total, m, M)
    assert got.tolist() == ref.tolist()
    assert (st == ckv.CKV_OK) == (rst == oracle.OK)


def test_allocate_budgets_workload_parameters():
    for name in ("llama8b-32k-stack", "llama8b-128k-stack", "qwen7b-ragged-batch"):
        wl = synth.WORKLOADS[name]
        e = synth.layer_errors(wl)
        for L in wl.seq_lens:
            total, m, M = synth.budget_params(wl, L)
            got, st = ckv.ckv_allocate_budgets(e, total, m, M)
            assert st == ckv.CKV_OK
            assert got.sum() == total and got.min() >= max(m, wl.window) and got.max() <= M


def test_allocate_budgets_rejects_bad_input():
    with pytest.raises(ckv.CkvError):
        ckv.ckv_allocate_budgets([0.5, float("nan")], 100, 10, 60)
    with pytest.raises(ckv.CkvError):
        ckv.ckv_allocate_budgets([0.5, 0.5], 100, 60, 10)


# ---------------------------------------------------------------------------
# Synthetic workloads: deterministic, shaped as documented.
# ---------------------------------------------------------------------------
def test_synth_mask_and_planting():
    wl = synth.WORKLOADS["llama8b-32k-stack"]
    G = wl.num_q_heads // wl.num_kv_heads
    for layer in range(4):
        m = synth.head_mask(wl, layer)
        per = m.reshape(wl.num_kv_heads, G).sum(axis=1)
        assert set(per.tolist()) <= set(wl.n_sel_choices)
        np.testing.assert_array_equal(m, synth.head_mask(wl, layer))
        pos = synth.planted_positions(wl, layer, 0, 32768)
        assert len(pos) == wl.sinks + wl.n_spans * wl.span_len
        assert len(np.unique(pos)) == len(pos)
        assert pos.max() < 32768 - wl.window


def test_synth_tiny_inputs_on_cpu():
    wl = synth.WORKLOADS["tiny-fp32"]
    a = synth.layer_inputs(wl, 0, "cpu")
    b = synth.layer_inputs(wl, 0, "cpu")
    assert a.q_win[0].shape == (8, 16, 64) and a.k[0].shape == (2, 1024, 64)
    assert torch.equal(a.k[0], b.k[0]) and torch.equal(a.q_win[0], b.q_win[0])
    # planted keys raise the mean scaled logit of a group's chosen rows by 3
    G = 4
    q = a.q_win[0].double()
    planted = a.planted[0]
    others = np.setdiff1d(np.arange(1024 - 16), planted)
    for g in range(2):
        chosen = [g * G + t for t in range(G) if a.mask[g * G + t]]
        qbar = q[chosen].reshape(-1, 64).mean(0)
        logit = (a.k[0][g].double() @ qbar) / 8.0
        assert 2.5 < float(logit[planted].mean()) < 3.5
        assert abs(float(logit[others].mean())) < 0.5


def test_shared_scope_mask_rules():
    # layer-shared scope: a layer with no chosen head at all is rejected before
    # any launch; an unknown flag bit is unsupported
    shared = _desc(flags=ckv.CKV_KEEP_WINDOW | ckv.CKV_SHARE_LAYER)
    for fn in ("score", "compress"):
        assert _call(fn, shared, _seq(), mask=[0] * 8) == ckv.CKV_ERR_MASK
        assert _call(fn, _desc(flags=ckv.CKV_KEEP_WINDOW | 4), _seq()) == ckv.CKV_ERR_UNSUPPORTED


def test_shared_scope_workspace_is_smaller():
    # one selection per prompt instead of one per KV group
    per_group = ckv.layer_desc(32, 8, 128, 32, torch.bfloat16, 0.0, ckv.CKV_POOL_MAX, 7)
    shared = ckv.layer_desc(32, 8, 128, 32, torch.bfloat16, 0.0, ckv.CKV_POOL_MAX, 7,
                            ckv.CKV_KEEP_WINDOW | ckv.CKV_SHARE_LAYER)
    s = ckv.Seq(None, None, None, 512, seq_len=65536)
    assert 0 < ckv.ckv_workspace_bytes(shared, [s]) < ckv.ckv_workspace_bytes(per_group, [s])


_RESOURCE_USAGE = {}


def _resource_usage():
    """Per-kernel resource use of every HIP source as the compiler reports it
    ({kernel: {"scratch": bytes/lane, "lds": bytes/block}}), compiled once per
    session, the sources side by side."""
    import re
    import subprocess
    from paper_2508_02401_amd import build as B

    if _RESOURCE_USAGE:
        return _RESOURCE_USAGE
    procs = {}
    for src in B.SOURCES:
        if not src.endswith(".hip"):
            continue
        cmd = [B.HIPCC, "-x", "hip"] + B.COMMON + [
            "--cuda-device-only", "-c", os.path.join(B.CSRC, src), "-o", os.devnull,
            "-Rpass-analysis=kernel-resource-usage"]
        procs[src] = subprocess.Popen(cmd, stdout=subprocess.DEVNULL, stderr=subprocess.PIPE,
                                      text=True)
    for src, proc in procs.items():
        out = proc.communicate(timeout=900)[1]
        names = re.findall(r"Function Name: (\S+)", out)
        scratch = [int(x) for x in re.findall(r"ScratchSize \[bytes/lane\]: (\d+)", out)]
        lds = [int(x) for x in re.findall(r"LDS Size \[bytes/block\]: (\d+)", out)]
        with open(os.path.join(B.CSRC, src)) as f:
            has_kernels = "__global__" in f.read()
        assert len(names) == len(scratch) == len(lds) and bool(names) == has_kernels, src
        for n, sc, l in zip(names, scratch, lds):
            _RESOURCE_USAGE[n] = {"scratch": sc, "lds": l, "src": src}
    return _RESOURCE_USAGE


def test_kernels_use_no_scratch_memory():
    # every kernel keeps its arrays in registers and LDS; per-lane scratch (a
    # register array the compiler could not promote, or the argument block
    # copied to private memory) is a large silent slowdown
    usage = _resource_usage()
    assert any("score_kernel" in k for k in usage) and any("decode_kernel" in k for k in usage)
    bad = [k for k, u in usage.items() if u["scratch"]]
    assert not bad, "kernels with scratch memory: %s" % bad


# ---------------------------------------------------------------------------
# ckv_compress_stack: every layer is validated before anything is enqueued.
# ---------------------------------------------------------------------------
def _stack_call(desc, layers, masks, ws_bytes=1 << 40, side=None):
    """layers: list of per-layer ckv_seq lists; masks: [n_layers][H]."""
    lib = ckv.load()
    flat = [s for layer in layers for s in layer]
    arr = (ckv._binding.ckv_seq * max(1, len(flat)))(*flat)
    m = np.asarray(masks, np.uint8).reshape(-1)
    mm = (ctypes.c_uint8 * max(1, m.size))(*m.tolist())
    return lib.ckv_compress_stack(ctypes.byref(desc), len(layers), mm, arr,
                                  len(layers[0]) if layers else 1, _BASE + 32768, ws_bytes, None,
                                  side)


def test_stack_rejects_bad_layers():
    d, ok_mask = _desc(), [1] * 8
    three = [[_seq()], [_seq()], [_seq()]]
    assert _stack_call(d, [], [ok_mask]) == ckv.CKV_ERR_INVALID_ARG
    # a later layer with another prompt length, budget below the window, a
    # null output, or a group without a chosen head
    assert _stack_call(d, [[_seq()], [_seq(seq_len=99)]], [ok_mask] * 2) == ckv.CKV_ERR_INVALID_ARG
    assert _stack_call(d, [[_seq()], [_seq(budget=3)]], [ok_mask] * 2) == ckv.CKV_ERR_BUDGET
    assert _stack_call(d, [[_seq()], [_seq(k_out=None)]], [ok_mask] * 2) == ckv.CKV_ERR_INVALID_ARG
    assert _stack_call(d, three, [ok_mask, ok_mask, [1, 0, 0, 0, 0, 0, 0, 0]]) == ckv.CKV_ERR_MASK
    assert _stack_call(_desc(pool_kernel=4), three, [ok_mask] * 3) == ckv.CKV_ERR_INVALID_ARG


def test_stack_workspace_needs_one_slot():
    lib = ckv.load()
    d = _desc()
    arr = (ckv._binding.ckv_seq * 1)(_seq())
    one = lib.ckv_workspace_bytes(ctypes.byref(d), arr, 1)
    # one layer slot is the least the stack takes, with or without a side
    # stream; the (fake) stream handle is never touched because the size check
    # fails first
    assert _stack_call(d, [[_seq()], [_seq()]], [[1] * 8] * 2, ws_bytes=one - 1,
                       side=0x1000) == ckv.CKV_ERR_WORKSPACE
    assert _stack_call(d, [[_seq()], [_seq()]], [[1] * 8] * 2, ws_bytes=0,
                       side=None) == ckv.CKV_ERR_WORKSPACE


def test_selection_kernels_fit_beside_two_k_pass_workgroups():
    # A caller that runs layers on several streams can overlap one layer's
    # selection kernels with another layer's K passes: each of those kernels
    # must fit in the LDS that two K-pass
    # workgroups leave free on a CU (160 KB). The stack's one-workgroup-per-
    # group selection kernel is not among them (it holds a 131072-token
    # segment's bitmaps in LDS and waits for CUs to drain).
    usage = _resource_usage()
    lds = {k: u["lds"] for k, u in usage.items()}
    # the K-pass kernels of 16-bit d = 128 layers (the Llama / Qwen shapes)
    kpass = max(v for k, v in lds.items()
                if ("rowstats_kernel" in k or "score_kernel" in k) and ("ILi0ELi128" in k or "ILi1ELi128" in k))
    free = 160 * 1024 - 2 * kpass
    for k in ("pool_units_kernel", "pool_kernel", "hist_kernel", "filter_kernel", "resolve_kernel",
              "compact_kernel"):
        size = max(v for n, v in lds.items() if k in n)
        assert size <= free, "%s uses %d B of LDS, %d B are free beside two K-pass workgroups" % (
            k, size, free)


# ---- caller row statistics (the lse field) --------------------------------
@pytest.mark.parametrize("fn", ["score", "compress"])
@pytest.mark.parametrize("bad", [
    dict(lse=_BASE + 40962),                        # not 4-byte aligned
    dict(lse=_BASE + 40960, lse_stride_head=3),     # head stride below the window of 4
    dict(lse=_BASE + 40960, lse_stride_head=-4),
])
def test_bad_lse(fn, bad):
    assert _call(fn, _desc(), _seq(**bad)) == ckv.CKV_ERR_INVALID_ARG


@pytest.mark.parametrize("fn", ["score", "compress"])
def test_lse_for_some_prompts_only_is_rejected(fn):
    lib = ckv.load()
    arr = (ckv._binding.ckv_seq * 2)(_seq(lse=_BASE + 40960, lse_stride_head=4), _seq())
    m = (ctypes.c_uint8 * 8)(*([1] * 8))
    f = lib.ckv_score if fn == "score" else lib.ckv_compress_layer
    assert f(ctypes.byref(_desc()), m, arr, 2, _BASE + 32768, 1 << 40, None) == \
        ckv.CKV_ERR_INVALID_ARG


def test_lse_binding_rejects_wrong_layout():
    s = ckv.Seq(None, None, None, 16, lse=torch.zeros(4, 8, dtype=torch.float64))
    with pytest.raises(ValueError):
        ckv._binding._seq_array([s])
    s = ckv.Seq(None, None, None, 16, lse=torch.zeros(8, 4).t())
    with pytest.raises(ValueError):
        ckv._binding._seq_array([s])


# ---- compression-error profile: host normalisation and validation ----------
@pytest.mark.parametrize("seed", range(8))
def test_normalize_errors_matches_oracle(seed):
    rng = np.random.default_rng(seed)
    e = rng.random((int(rng.integers(1, 5)), int(rng.integers(1, 40)))) + 1e-3
    np.testing.assert_allclose(ckv.ckv_normalize_errors(e), oracle.normalize_errors(e),
                               rtol=1e-13, atol=0)


@pytest.mark.parametrize("bad", [np.zeros((2, 3)), np.array([[1.0, -1.0, 0.5]]),
                                 np.array([[1.0, np.nan]])])
def test_normalize_errors_rejects(bad):
    with pytest.raises(ckv.CkvError) as err:
        ckv.ckv_normalize_errors(bad)
    assert err.value.status == ckv.CKV_ERR_INVALID_ARG


def _adesc(**kw):
    base = dict(num_q_heads=8, num_kv_heads=2, head_dim=64, dtype=ckv.CKV_BF16, scale=0.0)
    base.update(kw)
    d = ckv._binding.ckv_attn_desc()
    for k, v in base.items():
        setattr(d, k, v)
    return d


def _cache(**kw):
    c = ckv._binding.ckv_kv_cache()
    vals = dict(k=_BASE + 4096, v=_BASE + 8192, stride_head=100 * 64, stride_tok=64, n=100)
    vals.update(kw)
    for k, v in vals.items():
        setattr(c, k, v)
    return c


def _decode(desc, cache, T=4, q=_BASE, qst=8 * 64, qsh=64, out=_BASE + 12288, ws=True):
    lib = ckv.load()
    return lib.ckv_decode_attention(ctypes.byref(desc), q, qst, qsh, T, ctypes.byref(cache), out,
                                    _BASE + 32768 if ws else None, 1 << 40 if ws else 0, None)


@pytest.mark.parametrize("bad,expect", [
    (dict(head_dim=96), ckv.CKV_ERR_UNSUPPORTED),
    (dict(dtype=9), ckv.CKV_ERR_UNSUPPORTED),
    (dict(num_q_heads=7), ckv.CKV_ERR_INVALID_ARG),
    (dict(scale=float("inf")), ckv.CKV_ERR_INVALID_ARG),
])
def test_decode_bad_descriptor(bad, expect):
    assert _decode(_adesc(**bad), _cache()) == expect


@pytest.mark.parametrize("kw,expect", [
    (dict(T=0), ckv.CKV_ERR_INVALID_ARG),
    (dict(T=33), ckv.CKV_ERR_UNSUPPORTED),       # 4 heads per group x 33 tokens > 128 rows
    (dict(q=None), ckv.CKV_ERR_INVALID_ARG),
    (dict(q=_BASE + 8), ckv.CKV_ERR_INVALID_ARG),
    (dict(qsh=32), ckv.CKV_ERR_INVALID_ARG),
    (dict(out=None), ckv.CKV_ERR_INVALID_ARG),
    (dict(ws=False), ckv.CKV_ERR_WORKSPACE),
])
def test_decode_bad_arguments(kw, expect):
    assert _decode(_adesc(), _cache(), **kw) == expect


@pytest.mark.parametrize("kw", [dict(n=0), dict(k=None), dict(v=_BASE + 8200), dict(stride_tok=32),
                                dict(stride_tok=65), dict(n=1 << 31)])
def test_decode_bad_cache(kw):
    assert _decode(_adesc(), _cache(**kw)) == ckv.CKV_ERR_INVALID_ARG


def test_layer_error_validation():
    lib = ckv.load()
    d = _adesc()
    full, comp = _cache(), _cache(n=20, stride_head=20 * 64)

    def call(w_o=_BASE + 16384, w_stride=8 * 64, D=256, eps=1e-6, ratio=_BASE + 20480,
             e=_BASE + 24576, ws=True):
        return lib.ckv_layer_error(ctypes.byref(d), _BASE, 8 * 64, 64, 4, ctypes.byref(full),
                                   ctypes.byref(comp), w_o, w_stride, D, eps, ratio, e,
                                   _BASE + 32768 if ws else None, 1 << 40 if ws else 0, None)
    assert call(w_o=None) == ckv.CKV_ERR_INVALID_ARG
    assert call(w_stride=8 * 64 - 8) == ckv.CKV_ERR_INVALID_ARG
    assert call(D=0) == ckv.CKV_ERR_INVALID_ARG
    assert call(eps=-1.0) == ckv.CKV_ERR_INVALID_ARG
    assert call(ratio=None) == ckv.CKV_ERR_INVALID_ARG
    assert call(e=_BASE + 24578) == ckv.CKV_ERR_INVALID_ARG
    assert call(ws=False) == ckv.CKV_ERR_WORKSPACE
    assert ckv.ckv_layer_error_workspace_bytes(d, 4, 100, 20, 256) > 0
    assert ckv.ckv_layer_error_workspace_bytes(d, 0, 100, 20, 256) == 0


def _dseq(T=4, q=_BASE, qst=8 * 64, qsh=64, out=_BASE + 12288, **cache_kw):
    return ckv.ckv_decode_seq(q, qst, qsh, T, 0, _cache(**cache_kw), out)


def _decode_batch(desc, seqs, ws=True):
    lib = ckv.load()
    arr = (ckv.ckv_decode_seq * max(len(seqs), 1))(*seqs)
    return lib.ckv_decode_attention_batch(ctypes.byref(desc), arr, len(seqs),
                                          _BASE + 65536 if ws else None, 1 << 40 if ws else 0,
                                          None)


@pytest.mark.parametrize("bad", [dict(T=0), dict(q=None), dict(qsh=32), dict(out=_BASE + 2),
                                 dict(n=0), dict(stride_tok=65), dict(k=None)])
def test_decode_batch_rejects_any_bad_prompt(bad):
    # the bad prompt is the second of three; nothing may be launched
    seqs = [_dseq(), _dseq(**bad), _dseq(T=1, n=7)]
    assert _decode_batch(_adesc(), seqs) == ckv.CKV_ERR_INVALID_ARG
    assert ckv.ckv_decode_batch_workspace_bytes(_adesc(), seqs) == 0


def test_decode_batch_argument_errors():
    assert _decode_batch(_adesc(), []) == ckv.CKV_ERR_INVALID_ARG
    assert _decode_batch(_adesc(head_dim=96), [_dseq()]) == ckv.CKV_ERR_UNSUPPORTED
    assert _decode_batch(_adesc(), [_dseq(T=33)]) == ckv.CKV_ERR_UNSUPPORTED
    assert _decode_batch(_adesc(), [_dseq(), _dseq(n=3)], ws=False) == ckv.CKV_ERR_WORKSPACE
    lib = ckv.load()
    assert lib.ckv_decode_attention_batch(ctypes.byref(_adesc()), None, 2, _BASE, 1 << 40,
                                          None) == ckv.CKV_ERR_INVALID_ARG


def test_decode_batch_workspace_arithmetic():
    d = _adesc()
    # one prompt needs what the single-cache entry point needs
    for T, n in ((1, 1), (4, 100), (2, 70000)):
        assert ckv.ckv_decode_batch_workspace_bytes(d, [_dseq(T=T, n=n, stride_head=n * 64)]) == \
            ckv.ckv_decode_workspace_bytes(d, T, n)
    # launches hold at most 24 prompts: prompt 25 starts a new launch of its own
    seqs = [_dseq(T=1 + i % 3, n=50 + 37 * i, stride_head=(50 + 37 * i) * 64) for i in range(25)]
    whole = ckv.ckv_decode_batch_workspace_bytes(d, seqs)
    assert whole == (ckv.ckv_decode_batch_workspace_bytes(d, seqs[:24]) +
                     ckv.ckv_decode_batch_workspace_bytes(d, seqs[24:]))
    assert whole > ckv.ckv_decode_batch_workspace_bytes(d, seqs[:24])


def test_streaming_select_validation():
    lib = ckv.load()

    def call(n_sink=4, **kw):
        arr = (ckv._binding.ckv_seq * 1)(_seq(**kw))
        return lib.ckv_streaming_select(ctypes.byref(_desc()), arr, 1, n_sink, None)
    assert call(n_sink=-1) == ckv.CKV_ERR_INVALID_ARG
    assert call(idx=None) == ckv.CKV_ERR_INVALID_ARG
    assert call(k_out=None) == ckv.CKV_ERR_INVALID_ARG
    assert call(k=None) == ckv.CKV_ERR_INVALID_ARG
    assert lib.ckv_streaming_select(ctypes.byref(_desc(pool_kernel=4)),
                                    (ckv._binding.ckv_seq * 1)(_seq()), 1, 4,
                                    None) == ckv.CKV_ERR_INVALID_ARG
