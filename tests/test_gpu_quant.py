"""GPU parity of the layer over b-bit expert codes (the HQQ format of the
paper's 2-bit Mixtral setting) against the quantized-expert oracle: 2- and
4-bit codes at hidden widths that take every lane layout of the kernel
(d = 256 ... 4096), ragged token counts (many tokens per expert loop over
the kernel's token tile), outputs bitwise independent of residency and split
ratio, and the entry points' error codes."""
import numpy as np
import pytest

import synth
from gpu_helpers import check_layer

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

SHAPES = [
    synth.ModelShape("q2-d256", 1, 256, 512, 8, 2, "bf16", expert_bits=2),
    synth.ModelShape("q4-d512", 1, 512, 256, 8, 2, "bf16", expert_bits=4),
    synth.ModelShape("q2-d1024", 1, 1024, 384, 16, 4, "bf16", expert_bits=2),
    synth.ModelShape("q4-d2048", 2, 2048, 256, 16, 4, "bf16", expert_bits=4),
    synth.ModelShape("q2-d4096", 1, 4096, 256, 8, 2, "bf16", expert_bits=2),
]


def _rig(shape, max_tokens=70):
    from workload import SplitRig, top_bytes
    r = SplitRig(shape, seed=2, max_tokens=max_tokens,
                 budget_bytes=shape.n_layers * shape.n_experts * shape.expert_bytes)
    tb = top_bytes(r, 0.5)
    r.configure([shape.n_experts * tb] * shape.n_layers, [0.5] * shape.n_layers)
    r.load_tops(0, list(range(0, shape.n_experts, 2)))
    return r


@pytest.fixture(scope="module", params=SHAPES, ids=lambda s: s.name)
def rig(request):
    r = _rig(request.param)
    yield r
    r.close()


def _run(rig, h, T, flags=0):
    y, idx, w = rig.outputs(T)
    rig.forward(0, h, T, y, idx, w, flags)
    torch.cuda.synchronize()
    return y, idx, w


@pytest.mark.parametrize("T", [1, 3, 17, 70])
def test_quantized_layer_parity(rig, T):
    h, hf = rig.hidden(T, tag=300 + T)
    y, idx, w = _run(rig, h, T)
    check_layer(rig, 0, hf, y, idx, w)


def test_quantized_outputs_independent_of_residency(rig):
    """Each chunk is computed the same way whether its codes sit in the top
    cache, in a prefetched staging slot or arrive after routing."""
    from paper_2509_08342_amd import moesplit as ms
    from workload import top_bytes
    s = rig.shape
    h, hf = rig.hidden(5, tag=9)
    y0, idx0, w0 = _run(rig, h, 5)
    check_layer(rig, 0, hf, y0, idx0, w0)
    y0 = y0.cpu().numpy()
    for r, tops in ((0.5, []), (0.25, list(range(s.n_experts))), (1.0, [1, 2]), (0.0, [])):
        tb = top_bytes(rig, r)
        rig.configure([s.n_experts * max(tb, 1)] * s.n_layers, [r] * s.n_layers)
        rig.load_tops(0, tops if r > 0 else [])
        ms.ms_drop_buffer(rig.ctx)
        y, idx, w = _run(rig, h, 5, ms.MS_FWD_PREDICT_NEXT if s.n_layers > 1 else 0)
        assert np.array_equal(idx.cpu().numpy(), idx0.cpu().numpy())
        assert np.array_equal(y.cpu().numpy(), y0), "r=%s tops=%s" % (r, tops)


def test_quantized_entry_points_reject_the_other_format():
    from paper_2509_08342_amd import moesplit as ms
    shape = SHAPES[0]
    with _rig(shape, max_tokens=4) as r:
        d, F = shape.d_model, shape.d_ff
        with pytest.raises(ms.MoeSplitError) as ei:
            ms.ms_set_expert(r.ctx, 0, 0, np.zeros((d, F), np.uint16), np.zeros((d, F), np.uint16),
                             np.zeros((F, d), np.uint16))
        assert ei.value.status == ms.MS_E_STATE
    from workload import SplitRig
    plain = synth.ModelShape("bf16-d256", 1, 256, 512, 8, 2, "bf16")
    with SplitRig(plain, seed=1, max_tokens=2, budget_bytes=0) as r2:
        qe = synth.quant_expert(SHAPES[0], 0, 0, 0, 2)
        with pytest.raises(ms.MoeSplitError) as ei:
            ms.ms_set_expert_q(r2.ctx, 0, 0, qe.codes, qe.meta)
        assert ei.value.status == ms.MS_E_STATE


@pytest.mark.parametrize("T", [3, 64, 70])
def test_quantized_matrix_core_and_chunk_paths_match_oracle(rig, T):
    """The matrix-core prefill over b-bit chunks (code pairs as bf16 B
    fragments, scale and zero folded per group) and the chunk kernel both
    match the oracle at partial and full row tiles."""
    from paper_2509_08342_amd import moesplit as ms
    h, hf = rig.hidden(T, tag=600 + T)
    for flag in (ms.MS_FWD_MATRIX_CORES, ms.MS_FWD_NO_MATRIX_CORES):
        y, idx, w = _run(rig, h, T, flag)
        check_layer(rig, 0, hf, y, idx, w)
