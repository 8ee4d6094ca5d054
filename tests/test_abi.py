"""The C-ABI library loads and exports every function include/*.h declares,
and its host-side validation answers without touching a GPU."""

import glob
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = sorted(glob.glob(os.path.join(ROOT, "include", "*.h")))
LIB = os.path.join(ROOT, "paper_2609_00993_amd", "libmoepd.so")


def declared_functions():
    text = "\n".join(open(h).read() for h in HEADERS)
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(moe_\w+)\s*\(", text, flags=re.M)))


def test_header_declares_the_layer_calls():
    names = declared_functions()
    for n in ("moe_ctx_create", "moe_route", "moe_dispatch", "moe_expert_ffn", "moe_combine", "moe_phase_view",
              "moe_phase_reset", "moe_ctx_destroy", "moe_status_string", "moe_dispatch_layout",
              "moe_dispatch_permute", "moe_turnstile_create", "moe_p_epoch_start", "moe_p_epoch_join"):
        assert n in names


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        pytest.fail("libmoepd.so is not built; run `python -m paper_2609_00993_amd.build`")
    from paper_2609_00993_amd import moepd

    return moepd


def test_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], stdout=subprocess.PIPE, text=True, check=True).stdout
    exported = set(re.findall(r"\sT\s(moe_\w+)$", out, flags=re.M))
    declared = set(declared_functions())
    assert declared <= exported, declared - exported
    assert set(lib.SYMBOLS) == declared


def test_status_strings(lib):
    for code in range(-9, 1):
        s = lib.moe_status_string(code)
        assert s and s != "unknown status"
    assert lib.moe_status_string(-99) == "unknown status"
    assert lib.moe_kernel_name(lib.MOE_KERNEL_GEMM1) == "gemm1_swiglu"
    assert lib.moe_kernel_name(99) == "?"


def _cfg(lib, **kw):
    base = dict(num_experts=8, expert_begin=0, num_local_experts=8, top_k=2, hidden=256, inter=512,
                dtype=lib.MOE_DTYPE_F32, max_tokens_p=64, max_tokens_d=8)
    base.update(kw)
    return lib.make_config(**base)


@pytest.mark.parametrize("bad", [
    dict(num_experts=0), dict(num_experts=2000), dict(num_local_experts=0), dict(num_local_experts=300),
    dict(expert_begin=-1), dict(expert_begin=4), dict(top_k=0), dict(top_k=9), dict(top_k=17, num_experts=32,
                                                                                  num_local_experts=32),
    dict(hidden=100), dict(hidden=32), dict(inter=96), dict(dtype=7), dict(max_tokens_p=-1),
    dict(max_tokens_d=(1 << 20) + 1), dict(flags=1), dict(d_priority_us=-1), dict(d_priority_us=1001),
])
def test_create_rejects_bad_config_without_gpu(lib, bad):
    st, ctx = lib.moe_ctx_create(_cfg(lib, **bad), 0x1000, 0x2000)
    assert st == lib.MOE_ERR_INVALID_ARG and ctx is None


def test_fp8_create_validation_without_gpu(lib):
    # MX FP8 steps through K 128 at a time; its weights carry scale arrays
    st, ctx = lib.moe_ctx_create(_cfg(lib, dtype=lib.MOE_DTYPE_FP8, hidden=192, inter=256), 0x1000, 0x2000, 0x3000,
                                 0x4000)
    assert st == lib.MOE_ERR_INVALID_ARG and ctx is None
    st, ctx = lib.moe_ctx_create(_cfg(lib, dtype=lib.MOE_DTYPE_FP8, hidden=256, inter=192), 0x1000, 0x2000, 0x3000,
                                 0x4000)
    assert st == lib.MOE_ERR_INVALID_ARG and ctx is None
    st, ctx = lib.moe_ctx_create(_cfg(lib, dtype=lib.MOE_DTYPE_FP8, hidden=256, inter=256), 0x1000, 0x2000, None,
                                 0x4000)
    assert st == lib.MOE_ERR_INVALID_ARG and ctx is None


def test_create_rejects_null_weights(lib):
    st, ctx = lib.moe_ctx_create(_cfg(lib), 0, 0x2000)
    assert st == lib.MOE_ERR_INVALID_ARG and ctx is None
    st, ctx = lib.moe_ctx_create(None, 0x1000, 0x2000)
    assert st == lib.MOE_ERR_INVALID_ARG


def test_null_context_calls(lib):
    assert lib.moe_route(None, 0, 0, 0, 1) == lib.MOE_ERR_INVALID_ARG
    assert lib.moe_dispatch(None, 0, 0, 1) == lib.MOE_ERR_INVALID_ARG
    assert lib.moe_expert_ffn(None, 0, 1) == lib.MOE_ERR_INVALID_ARG
    assert lib.moe_combine(None, 0, 0, 1) == lib.MOE_ERR_INVALID_ARG
    assert lib.moe_phase_view(None, 0)[0] == lib.MOE_ERR_INVALID_ARG
    assert lib.moe_phase_reset(None, 0) == lib.MOE_ERR_INVALID_ARG
    assert lib.moe_timing_enable(None, 4) == lib.MOE_ERR_INVALID_ARG
    assert lib.moe_timing_read(None, 0, 0)[0] == lib.MOE_ERR_INVALID_ARG
    assert lib.moe_ctx_destroy(None) == lib.MOE_OK
    assert lib.moe_dispatch_layout(None, 0, 1) == lib.MOE_ERR_INVALID_ARG
    assert lib.moe_dispatch_permute(None, 0, 0, 1) == lib.MOE_ERR_INVALID_ARG


def test_p_epoch_runner_validates_before_touching_the_gpu(lib):
    st, ts = lib.moe_turnstile_create(1, 0)
    lib.check(st)
    try:
        bufs = [0x1000] * 2
        assert lib.moe_p_epoch_start(None, ts, 0, True, 4, bufs, bufs, bufs, 1, 1000)[0] == lib.MOE_ERR_INVALID_ARG
        assert lib.moe_p_epoch_start(0x10, None, 0, True, 4, bufs, bufs, bufs, 1, 1000)[0] == lib.MOE_ERR_INVALID_ARG
        assert lib.moe_p_epoch_start(0x10, ts, 0, True, 4, bufs, bufs, bufs, 0, 1000)[0] == lib.MOE_ERR_INVALID_ARG
        assert lib.moe_p_epoch_start(0x10, ts, 0, True, 4, bufs, bufs, bufs, 1, 0)[0] == lib.MOE_ERR_INVALID_ARG
        assert lib.moe_p_epoch_start(0x10, ts, 0, True, -1, bufs, bufs, bufs, 1, 1000)[0] == lib.MOE_ERR_INVALID_ARG
        assert lib.moe_p_epoch_start(0x10, ts, 0, True, 4, bufs, [0x1000, 0], bufs, 1, 1000)[0] == \
            lib.MOE_ERR_INVALID_ARG
        assert lib.moe_p_epoch_start(0x10, ts, 0, True, 4, [], [], [], 1, 1000)[0] == lib.MOE_ERR_INVALID_ARG
        assert lib.moe_p_epoch_join(None)[0] == lib.MOE_ERR_INVALID_ARG
        st, q = lib.moe_turnstile_query(ts)
        assert q.task == lib.MOE_TS_IDLE and q.epoch == -1  # nothing began
    finally:
        lib.moe_turnstile_destroy(ts)


def test_clock_probe_rejects_bad_arguments(lib):
    """The clock probe validates on the host before any launch (the stream
    and buffer values below are never used)."""
    M = lib
    assert M.moe_clock_probe(None, 100, 16) == M.MOE_ERR_INVALID_ARG  # null stream
    assert M.moe_clock_probe(16, 100, None) == M.MOE_ERR_INVALID_ARG  # null output
    assert M.moe_clock_probe(16, 0, 16) == M.MOE_ERR_INVALID_ARG
    assert M.moe_clock_probe(16, 100001, 16) == M.MOE_ERR_INVALID_ARG


def test_noalloc_layout_validates_on_the_host(lib):
    """The allocation-free layout refuses bad arguments before any HIP call
    (fake pointers, no GPU needed)."""
    fake = 0x1000

    def call(**kw):
        a = dict(topk_idx=fake, T=4, top_k=2, expert_begin=0, num_local_experts=8, counts=fake, offsets=fake,
                 row_of_slot=fake, token_of_row=fake, stream=fake)
        a.update(kw)
        return lib.moe_dispatch_layout_noalloc(**a)

    assert call(T=-1) == lib.MOE_ERR_INVALID_ARG
    assert call(top_k=0) == lib.MOE_ERR_INVALID_ARG
    assert call(top_k=17) == lib.MOE_ERR_INVALID_ARG
    assert call(expert_begin=-1) == lib.MOE_ERR_INVALID_ARG
    assert call(num_local_experts=0) == lib.MOE_ERR_INVALID_ARG
    assert call(num_local_experts=257) == lib.MOE_ERR_INVALID_ARG
    assert call(counts=None) == lib.MOE_ERR_INVALID_ARG
    assert call(offsets=None) == lib.MOE_ERR_INVALID_ARG
    assert call(stream=None) == lib.MOE_ERR_INVALID_ARG
    assert call(topk_idx=None) == lib.MOE_ERR_INVALID_ARG
    assert call(row_of_slot=None) == lib.MOE_ERR_INVALID_ARG
    assert call(T=(1 << 20) + 1) == lib.MOE_ERR_CAPACITY
