"""C-ABI checks that need no GPU.

* libflexattn.so loads and exports every function include/flexattn.h declares.
* flex_attn_plan (C++) equals the Python re-derivation (oracle/plan.py)
  word for word on the five workloads and on fuzzed batches, and returns the
  same status on malformed inputs.
* Run calls reject bad arguments before touching the GPU.
"""
import ctypes
import os
import random
import re

import pytest
import torch

from oracle import plan as OP
from paper_2606_04415_amd import flexattn as F
from paper_2606_04415_amd.workloads import WORKLOADS, draw_lengths

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "flexattn.h")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(flex_(?:attn|ctl|ts)_\w+)\s*\(", text)))


def test_exports_every_declared_symbol():
    lib = F.lib()
    declared = header_functions()
    assert len(declared) >= 15
    for name in declared:
        assert hasattr(lib, name), f"{name} declared in flexattn.h but not exported"
    assert sorted(F.EXPORTED) == declared


def c_plan(sh_py, opts_py, qsl, ls, maxp):
    sh = F.make_shape(sh_py.num_q_heads, sh_py.num_kv_heads, sh_py.head_dim_qk, sh_py.head_dim_v,
                      sh_py.page_size, sh_py.sm_scale, sh_py.v_aliases_k)
    opts = None
    if opts_py is not None:
        opts = F.make_opts(**{k: getattr(opts_py, k) for k in OP.Opts.__dataclass_fields__})
    st = F.plan_status(sh, opts, qsl, ls, maxp)
    if st != F.FLEX_OK:
        return st, None, None
    p = F.flex_attn_plan(sh, opts, qsl, ls, maxp)
    return st, p.export(), p.info


def compare(sh, opts, qsl, ls, maxp):
    st, words, info = c_plan(sh, opts, qsl, ls, maxp)
    ref = OP.build_plan(sh, opts, qsl, ls, maxp)
    assert st == ref.status
    if st == OP.OK:
        assert words == ref.blob
        for k in ("n_decode_items", "n_prefill_items", "n_split_seqs", "pages_per_split", "cus_decode", "cus_prefill",
                  "workspace_bytes", "device_plan_bytes", "plan_words", "decode_wg_width", "n_fused_wgs"):
            assert info[k] == ref.info[k], k
        assert info["decode_bytes"] == ref.info["decode_bytes"]
        assert info["prefill_flops"] == ref.info["prefill_flops"]


@pytest.mark.parametrize("name", sorted(WORKLOADS))
@pytest.mark.parametrize("cus_decode", [0, 128, -1])
def test_plan_matches_rederivation_on_workloads(name, cus_decode):
    w = WORKLOADS[name]
    ns, ls = draw_lengths(w, torch.Generator().manual_seed(0))
    qsl = [0]
    for n in ns:
        qsl.append(qsl[-1] + n)
    sh = OP.Shape(w.num_q_heads, w.num_kv_heads, w.head_dim_qk, w.head_dim_v, w.page_size,
                  w.sm_scale, int(w.v_aliases_k))
    compare(sh, OP.Opts(cus_decode=cus_decode), qsl, ls, w.max_pages_per_seq)


def test_plan_matches_rederivation_fuzz():
    rng = random.Random(1)
    shapes = [OP.Shape(28, 4, 128, 128, 16, 128 ** -0.5, 0), OP.Shape(4, 1, 64, 64, 16, 0.125, 0),
              OP.Shape(32, 2, 128, 128, 64, 0.1, 0), OP.Shape(128, 1, 576, 512, 64, 192 ** -0.5, 1),
              OP.Shape(64, 1, 576, 512, 64, 0.07, 1), OP.Shape(16, 16, 192, 128, 64, 192 ** -0.5, 0),
              OP.Shape(8, 4, 192, 128, 64, 0.1, 0), OP.Shape(40, 5, 64, 64, 16, 0.125, 0),
              OP.Shape(48, 3, 128, 128, 64, 0.09, 0), OP.Shape(64, 8, 128, 128, 16, 0.088, 0)]
    for trial in range(400):
        sh = rng.choice(shapes)
        P = sh.page_size
        B = rng.randint(0, 50)
        ns, ls = [], []
        for _ in range(B):
            kind = rng.random()
            L = rng.choice([0, 1, 15, 16, 17, 129, 4095, rng.randint(1, 20000)])
            n = 0 if L == 0 else (1 if kind < 0.6 else rng.randint(0, L))
            ns.append(n)
            ls.append(L)
        qsl = [0]
        for n in ns:
            qsl.append(qsl[-1] + n)
        maxp = max([1] + [-(-L // P) for L in ls]) + rng.randint(0, 3)
        opts = OP.Opts(cus_decode=rng.choice([0, 64, 192, -1]),
                       wg_per_cu=rng.choice([0, 2]), min_split_tokens=rng.choice([0, 16, 1000]),
                       bm=(rng.choice([0, 0, 16, 32, 128]) if sh.head_dim_qk in (64, 128)
                           else rng.choice([0, 64]) if sh.head_dim_qk == 576 else rng.choice([0, 128])),
                       cus_total=rng.choice([0, 256, 240, 16]),
                       hbm_gbps=rng.choice([0.0, 5000.0]), decode_gbps_per_cu=rng.choice([0.0, 25.0]))
        compare(sh, opts, qsl, ls, maxp)


@pytest.mark.parametrize("qsl,ls,maxp", [
    ([1, 2], [4], 16),
    ([0, 3, 2], [4, 4], 16),
    ([0, 5], [4], 16),
    ([0, 1], [10 ** 6], 16),
    ([0, 0], [0], 16),
    ([0], [], 16),
    ([0, 1], [-3], 16),
    ([0, 1], [5], -1),
])
def test_plan_status_matches(qsl, ls, maxp):
    compare(OP.Shape(28, 4, 128, 128, 16, 0.088, 0), None, qsl, ls, maxp)


@pytest.mark.parametrize("sh", [
    OP.Shape(28, 4, 96, 96, 16, 0.1, 0), OP.Shape(28, 4, 128, 128, 32, 0.1, 0),
    OP.Shape(28, 3, 128, 128, 16, 0.1, 0), OP.Shape(28, 4, 128, 128, 16, -1.0, 0),
    OP.Shape(28, 4, 128, 128, 16, float("nan"), 0), OP.Shape(128, 1, 576, 512, 64, 0.1, 0),
    OP.Shape(96, 1, 576, 512, 64, 0.1, 1), OP.Shape(34, 2, 128, 128, 16, 0.1, 0),
    OP.Shape(8, 2, 128, 128, 16, 0.1, 1),
])
def test_shape_status_matches(sh):
    compare(sh, None, [0, 1], [5], 4)


@pytest.mark.parametrize("opts", [OP.Opts(cus_decode=-2), OP.Opts(cus_decode=300), OP.Opts(bm=96),
                                  OP.Opts(wg_per_cu=-1), OP.Opts(min_split_tokens=-4)])
def test_opts_status_matches(opts):
    compare(OP.Shape(28, 4, 128, 128, 16, 0.1, 0), opts, [0, 1, 3], [5, 9], 4)


def test_run_calls_reject_bad_args_without_gpu():
    sh = F.make_shape(28, 4, 128, 128, 16, 0.088)
    plan = F.flex_attn_plan(sh, F.make_opts(min_split_tokens=16), [0, 1, 3], [40, 50], 4)
    assert plan.info["n_split_seqs"] == 1 and plan.info["workspace_bytes"] > 0
    a = F.Args()   # all NULL
    for fn in (F.lib().flex_attn_decode, F.lib().flex_attn_prefill):
        st = fn(plan.handle, ctypes.byref(a), None)
        assert st == F.FLEX_ERR_INVALID_ARG
    assert F.lib().flex_attn_mixed(plan.handle, ctypes.byref(a), 7, None, None) == F.FLEX_ERR_INVALID_ARG
    # plausible-looking but misaligned pointers are refused before any launch
    a.q = 0x1001
    a.k_cache = a.v_cache = a.block_table = a.seq_lens = a.query_start_loc = a.out = a.d_plan = 0x1000
    assert F.lib().flex_attn_decode(plan.handle, ctypes.byref(a), None) == F.FLEX_ERR_INVALID_ARG
    assert "aligned" in F.last_error()
    # undersized plan buffer / workspace
    a.q = 0x2000
    a.k_stride = (ctypes.c_int64 * 3)(16 * 4 * 128, 4 * 128, 128)
    a.v_stride = (ctypes.c_int64 * 3)(16 * 4 * 128, 4 * 128, 128)
    a.num_pages = 10
    a.block_table_stride = 4
    # page-local offsets are 32-bit: a page stride or slot span of 2^31 bytes is refused
    a.k_stride = (ctypes.c_int64 * 3)(1 << 30, 4 * 128, 128)
    assert F.lib().flex_attn_decode(plan.handle, ctypes.byref(a), None) == F.FLEX_ERR_INVALID_ARG
    assert "2^31" in F.last_error()
    a.k_stride = (ctypes.c_int64 * 3)(16 * 4 * 128, 1 << 26, 128)
    assert F.lib().flex_attn_decode(plan.handle, ctypes.byref(a), None) == F.FLEX_ERR_INVALID_ARG
    a.k_stride = (ctypes.c_int64 * 3)(16 * 4 * 128, 4 * 128, 128)
    a.d_plan_bytes = 8
    assert F.lib().flex_attn_decode(plan.handle, ctypes.byref(a), None) == F.FLEX_ERR_WORKSPACE
    a.d_plan_bytes = plan.info["device_plan_bytes"]
    a.workspace = 0x3000
    a.workspace_bytes = 16
    assert F.lib().flex_attn_decode(plan.handle, ctypes.byref(a), None) == F.FLEX_ERR_WORKSPACE
    assert F.lib().flex_attn_workspace_init(ctypes.c_void_p(0x3001), 64, None) == F.FLEX_ERR_INVALID_ARG
    assert F.lib().flex_attn_corun_create(100, 50, ctypes.byref(ctypes.c_void_p())) != F.FLEX_OK
    # the one-launch mode: checked like the others, and refused (before any launch)
    # for a plan whose shape has no one-launch form
    assert F.lib().flex_attn_mixed(plan.handle, ctypes.byref(F.Args()), F.FLEX_MODE_FUSED, None, None) == \
        F.FLEX_ERR_INVALID_ARG
    narrow = F.flex_attn_plan(F.make_shape(16, 4, 128, 128, 16, 0.088), None, [0, 1, 3], [40, 50], 4)
    assert narrow.info["n_fused_wgs"] == 0 and plan.info["n_fused_wgs"] > 0
    a.workspace_bytes = 1 << 20
    a.d_plan_bytes = narrow.info["device_plan_bytes"]
    assert F.lib().flex_attn_mixed(narrow.handle, ctypes.byref(a), F.FLEX_MODE_FUSED, None, None) == \
        F.FLEX_ERR_UNSUPPORTED
    assert "one-launch" in F.last_error()


def test_status_strings():
    for st in (0, -1, -2, -3, -4, -5):
        assert F.status_string(st)
    assert F.status_string(-99) == "unknown status"


def test_export_too_small():
    sh = F.make_shape(28, 4, 128, 128, 16, 0.088)
    plan = F.flex_attn_plan(sh, None, [0, 1], [40], 4)
    buf = (ctypes.c_int32 * 4)()
    assert F.lib().flex_attn_plan_export(plan.handle, buf, 4) == F.FLEX_ERR_WORKSPACE


def test_block_table_stride_below_the_plans_rows_is_refused():
    sh = F.make_shape(28, 4, 128, 128, 16, 0.088)
    plan = F.flex_attn_plan(sh, None, [0, 1, 3], [40, 50], 8)     # rows must hold 8 entries
    a = F.Args()
    a.q = a.k_cache = a.v_cache = a.block_table = a.seq_lens = a.query_start_loc = a.out = a.d_plan = 0x1000
    a.k_stride = (ctypes.c_int64 * 3)(16 * 4 * 128, 4 * 128, 128)
    a.v_stride = (ctypes.c_int64 * 3)(16 * 4 * 128, 4 * 128, 128)
    a.num_pages, a.block_table_stride = 10, 4
    a.d_plan_bytes = plan.info["device_plan_bytes"]
    assert F.lib().flex_attn_prefill(plan.handle, ctypes.byref(a), None) == F.FLEX_ERR_INVALID_ARG
    assert "max_pages_per_seq" in F.last_error()


def test_validate_host_catches_bad_metadata():
    """The host-side form of the debug check: a block-table entry outside the
    pool, a negative one, seq_lens or query_start_loc that differ from the
    plan's, and a row stride below the plan's row length are each refused."""
    sh = F.make_shape(28, 4, 128, 128, 16, 0.088)
    qsl, ls = [0, 1, 41, 42], [40, 40, 17]
    plan = F.flex_attn_plan(sh, None, qsl, ls, 4)
    bt = torch.tensor([[0, 1, 2, 99], [3, 4, 5, 99], [6, 7, 99, 99]], dtype=torch.int32)   # 99: unused entries
    F.flex_attn_validate_host(plan, bt, 8, ls, qsl)
    bad = bt.clone()
    bad[1, 2] = 8          # outside [0, 8)
    with pytest.raises(F.FlexAttnError) as e:
        F.flex_attn_validate_host(plan, bad, 8, ls, qsl)
    assert e.value.status == F.FLEX_ERR_INVALID_ARG and "sequence 1, page 2" in str(e.value)
    bad = bt.clone()
    bad[2, 0] = -1
    with pytest.raises(F.FlexAttnError):
        F.flex_attn_validate_host(plan, bad, 8, ls, qsl)
    with pytest.raises(F.FlexAttnError) as e:
        F.flex_attn_validate_host(plan, bt, 8, [40, 41, 17], qsl)
    assert "seq_lens" in str(e.value)
    with pytest.raises(F.FlexAttnError) as e:
        F.flex_attn_validate_host(plan, bt, 8, ls, [0, 1, 40, 42])
    assert "query_start_loc" in str(e.value)
    with pytest.raises(F.FlexAttnError) as e:
        F.flex_attn_validate_host(plan, bt[:, :3], 8, ls, qsl)
    assert "max_pages_per_seq" in str(e.value)


def test_debug_level_switch():
    prev = F.set_debug(1)
    assert F.set_debug(0) == 1
    F.set_debug(prev)
    assert F.lib().flex_attn_set_debug(-1) == F.FLEX_ERR_INVALID_ARG


def test_plan_log_line():
    import subprocess
    import sys
    code = ("import sys; sys.path.insert(0, %r); from paper_2606_04415_amd import flexattn as F; "
            "F.flex_attn_plan(F.make_shape(28, 4, 128, 128, 16, 0.088), None, [0, 1, 3], [40, 50], 4)" % ROOT)
    r = subprocess.run([sys.executable, "-c", code], env=dict(os.environ, FLEX_ATTN_LOG="2"),
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    assert "flexattn plan: 2 seqs (1 decode, 1 prefill)" in r.stderr and "prefill 0: seq 1" in r.stderr


def test_binding_refuses_wrong_dtypes_and_layouts():
    q = torch.zeros(3, 28, 128, dtype=torch.bfloat16)
    k = torch.zeros(4, 16, 4, 128, dtype=torch.bfloat16)
    bt = torch.zeros(2, 4, dtype=torch.int32)
    sl = torch.tensor([40, 50], dtype=torch.int32)
    qsl = torch.tensor([0, 1, 3], dtype=torch.int32)
    out = torch.zeros(3, 28, 128, dtype=torch.bfloat16)
    F.make_args(q, k, k, bt, sl, qsl, out)
    with pytest.raises(ValueError, match="int32"):
        F.make_args(q, k, k, bt.long(), sl, qsl, out)
    with pytest.raises(ValueError, match="bfloat16"):
        F.make_args(q.float(), k, k, bt, sl, qsl, out)
    with pytest.raises(ValueError, match="contiguous"):
        F.make_args(q.transpose(0, 1), k, k, bt, sl, qsl, out)
    with pytest.raises(ValueError, match="innermost"):
        F.make_args(q, k.transpose(2, 3), k, bt, sl, qsl, out)


def test_plan_takes_lists_arrays_and_tensors_alike():
    """The binding passes int32 metadata without a per-element copy; lists,
    numpy arrays and CPU tensors give the same plan words, and values that do
    not fit int32 are refused before the library sees them."""
    import numpy as np
    import torch
    shape = F.make_shape(8, 2, 64, 64, 16, 0.125, False)
    qsl, sl = [0, 1, 40, 41], [300, 40, 900]
    words = F.flex_attn_plan(shape, None, qsl, sl, 64).export()
    assert F.flex_attn_plan(shape, None, np.array(qsl, dtype=np.int64), np.array(sl), 64).export() == words
    assert F.flex_attn_plan(shape, None, torch.tensor(qsl, dtype=torch.int32),
                            torch.tensor(sl, dtype=torch.int32), 64).export() == words
    with pytest.raises(ValueError):
        F.flex_attn_plan(shape, None, qsl, [300, 40, 2 ** 31], 64)
    with pytest.raises(ValueError):
        F.flex_attn_plan(shape, None, [0.0, 1.0, 40.0, 41.0], sl, 64)
