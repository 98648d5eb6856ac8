"""C-ABI library checks that need no GPU: the library loads, exports every
symbol the header declares, and its pure host arithmetic (sizes, split plan,
argument validation) matches the oracle's reading of the split."""
import os
import re

import pytest

import oracle
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "moesplit.h")


def _ms():
    from paper_2509_08342_amd import moesplit
    return moesplit


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ms_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    syms = declared_symbols()
    for name in ("ms_create", "ms_configure", "ms_load_top", "ms_evict_top", "ms_predict",
                 "ms_prefetch", "ms_forward", "ms_destroy"):
        assert name in syms


def test_library_exports_every_declared_symbol():
    ms = _ms()
    for name in declared_symbols():
        assert hasattr(ms.lib, name), name


def _desc(shape, max_tokens=1, n_buf=0):
    return _ms().model_desc(shape, max_tokens, n_buf)


@pytest.mark.parametrize("shape", [synth.TINY, synth.MIXTRAL, synth.DEEPSEEK, synth.QWEN3])
def test_sizes(shape):
    ms = _ms()
    s = ms.ms_query_sizes(_desc(shape, 16))
    d, F, el = shape.d_model, shape.d_ff, shape.elem_bytes
    assert s.chunk_bytes == 3 * 64 * d * el
    assert s.n_chunks == -(-F // 64)
    assert s.expert_bytes == s.n_chunks * s.chunk_bytes
    assert s.buffer_bytes == 2 * shape.top_k * s.expert_bytes
    assert s.fixed_pool_bytes >= s.buffer_bytes
    if F % 64 == 0:
        assert s.expert_bytes == shape.expert_bytes


@pytest.mark.parametrize("shape,r", [(synth.MIXTRAL, r) for r in (0.0, 0.25, 0.5, 0.75, 1.0)]
                         + [(synth.DEEPSEEK, 0.5), (synth.QWEN3, 0.5), (synth.TINY, 0.5),
                            (synth.DEEPSEEK, 0.4), (synth.QWEN3, 0.1)])
def test_split_plan_matches_oracle(shape, r):
    ms = _ms()
    desc = _desc(shape)
    units, tb, _ = ms.ms_split_plan(desc, 0, r)
    assert units == oracle.top_units(r, shape.d_ff)
    assert tb == (units // 64) * 3 * 64 * shape.d_model * shape.elem_bytes


def test_split_plan_cache_sizes():
    ms = _ms()
    desc = _desc(synth.MIXTRAL)
    gib = 1 << 30
    # 12 GiB over 32 layers at r = .25/.5/.75 -> 4/2/1 cached tops per layer
    for r, c in ((0.25, 4), (0.5, 2), (0.75, 1)):
        assert ms.ms_split_plan(desc, 12 * gib // 32, r)[2] == c
    # r = 0: no top segment, no cache slots (prefetch only)
    assert ms.ms_split_plan(desc, 12 * gib, 0.0)[2] == 0
    # r = 1: whole experts, capped at E
    assert ms.ms_split_plan(desc, 100 * gib, 1.0)[2] == 8
    assert ms.ms_split_plan(_desc(synth.DEEPSEEK), 4 * gib // 26, 0.5)[2] == 19
    assert ms.ms_split_plan(_desc(synth.QWEN3), 8 * gib // 48, 0.5)[2] == 37


def test_invalid_arguments():
    ms = _ms()
    bad = _desc(synth.TINY)
    bad.d_model = 100
    with pytest.raises(ms.MoeSplitError) as ei:
        ms.ms_query_sizes(bad)
    assert ei.value.status == ms.MS_E_UNSUPPORTED
    bad = _desc(synth.TINY)
    bad.top_k = 9
    with pytest.raises(ms.MoeSplitError) as ei:
        ms.ms_query_sizes(bad)
    assert ei.value.status == ms.MS_E_INVALID
    with pytest.raises(ms.MoeSplitError) as ei:
        ms.ms_split_plan(_desc(synth.TINY), 0, 1.5)
    assert ei.value.status == ms.MS_E_INVALID


@pytest.mark.parametrize("bits", [2, 4])
def test_sizes_of_b_bit_experts(bits):
    """Per chunk: three 64 x d code blocks of b bits plus one 4-byte (scale,
    zero) per group of 64 elements of each matrix (12 d bytes); the expert
    is the whole blob, and a top segment a whole number of chunks."""
    import dataclasses
    ms = _ms()
    shape = dataclasses.replace(synth.MIXTRAL, expert_bits=bits)
    s = ms.ms_query_sizes(_desc(shape))
    d = shape.d_model
    assert s.chunk_bytes == 3 * 64 * d * bits // 8 + 12 * d
    assert s.expert_bytes == s.n_chunks * s.chunk_bytes == shape.expert_bytes
    units, tb, c = ms.ms_split_plan(_desc(shape), 12 * (1 << 30) // 32, 0.5)
    assert units == 7168 and tb == 112 * s.chunk_bytes and c == min(8, (12 * (1 << 30) // 32) // tb)


def test_b_bit_experts_reject_unsupported_shapes():
    import dataclasses
    ms = _ms()
    q = dataclasses.replace(synth.MIXTRAL, expert_bits=2)
    for change, status in ((dict(expert_bits=3), ms.MS_E_INVALID), (dict(dtype="f32"), ms.MS_E_UNSUPPORTED),
                           (dict(d_ff=14300), ms.MS_E_UNSUPPORTED), (dict(d_model=128), ms.MS_E_UNSUPPORTED),
                           (dict(n_shared=1, d_ff_shared=128), ms.MS_E_UNSUPPORTED)):
        with pytest.raises(ms.MoeSplitError) as ei:
            ms.ms_query_sizes(_desc(dataclasses.replace(q, **change)))
        assert ei.value.status == status, change
    desc = _desc(q)
    desc.ffn_splits = 2
    with pytest.raises(ms.MoeSplitError) as ei:
        ms.ms_query_sizes(desc)
    assert ei.value.status == ms.MS_E_UNSUPPORTED


@pytest.mark.parametrize("dtype,d,allowed", [("bf16", 8192, 2), ("f32", 8192, 2), ("bf16", 4096, 4),
                                              ("f32", 4096, 4), ("bf16", 2048, 4)])
def test_ffn_splits_bounded_by_the_kernel_table(dtype, d, allowed):
    """A chunk split over more work-groups needs more column passes per
    thread in the down projection; splits whose one-row accumulators would
    exceed the kernel's register budget (bf16 at d = 8192 beyond 2) are
    refused with MS_E_UNSUPPORTED, and the automatic choice stays within the
    bound."""
    ms = _ms()
    shape = synth.ModelShape("split-limit", 1, d, 256, 8, 2, dtype)
    for splits in (1, 2, 4):
        desc = _desc(shape)
        desc.ffn_splits = splits
        if splits <= allowed:
            ms.ms_query_sizes(desc)
        else:
            with pytest.raises(ms.MoeSplitError) as ei:
                ms.ms_query_sizes(desc)
            assert ei.value.status == ms.MS_E_UNSUPPORTED


@pytest.mark.parametrize("d", [64, 128, 192, 8256])
def test_model_dim_outside_the_kernels_is_refused(d):
    """d_model outside [256, 8192] (the prefill kernels stage 128-wide
    activation slabs) is refused with MS_E_UNSUPPORTED in every dtype."""
    ms = _ms()
    for dtype in ("bf16", "f32"):
        with pytest.raises(ms.MoeSplitError) as ei:
            ms.ms_query_sizes(_desc(synth.ModelShape("narrow", 1, d, 256, 8, 2, dtype)))
        assert ei.value.status == ms.MS_E_UNSUPPORTED
