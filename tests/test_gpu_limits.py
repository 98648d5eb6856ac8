"""GPU parity at the widest supported model dimension, d_model = 8192, in
bf16 and fp32: two column groups per thread in the FFN's down projection,
tiles limited by the activation rows' LDS size, the few-token logits one
wave per logit where a block of token rows does not fit LDS, the
matrix-core prefill path (bf16, T K >= 8 E) and the many-token
routing at the context's max_tokens.  Selected experts exact, outputs within
the dtype tolerance, and bitwise equal across residency states."""
import numpy as np
import pytest

import synth
from gpu_helpers import check_layer

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

WIDE_D_BF16 = synth.ModelShape("wide-d-bf16", 1, 8192, 256, 8, 2, "bf16")
WIDE_D_F32 = synth.ModelShape("wide-d-f32", 1, 8192, 256, 8, 2, "f32")
MAX_T = 64


@pytest.fixture(scope="module", params=[WIDE_D_BF16, WIDE_D_F32], ids=lambda s: s.name)
def rig(request):
    from workload import SplitRig
    r = SplitRig(request.param, seed=3, max_tokens=MAX_T, budget_bytes=request.param.n_experts * request.param.expert_bytes)
    yield r
    r.close()


def _setup(rig, ratio, tops):
    from workload import top_bytes
    tb = top_bytes(rig, ratio)
    rig.configure([rig.shape.n_experts * tb], [ratio])
    rig.load_tops(0, tops)


def _run(rig, h, T, flags=0):
    y, idx, w = rig.outputs(T)
    rig.forward(0, h, T, y, idx, w, flags)
    torch.cuda.synchronize()
    return y, idx, w


@pytest.mark.parametrize("T", [1, 3, 40, MAX_T])
def test_widest_model_dim_parity(rig, T):
    _setup(rig, 0.5, [0, 2, 4, 6])
    h, hf = rig.hidden(T, tag=900 + T)
    y, idx, w = _run(rig, h, T)
    check_layer(rig, 0, hf, y, idx, w)


@pytest.mark.parametrize("T", [3, 40])
def test_widest_model_dim_independent_of_residency(rig, T):
    h, hf = rig.hidden(T, tag=950 + T)
    outs = []
    for ratio, tops in ((0.5, [0, 2, 4, 6]), (1.0, list(range(8))), (0.0, [])):
        _setup(rig, ratio, tops)
        y, idx, w = _run(rig, h, T)
        outs.append((y.cpu().numpy()[:T], idx.cpu().numpy()[:T]))
    for y, idx in outs[1:]:
        assert np.array_equal(idx, outs[0][1])
        assert np.array_equal(y, outs[0][0])


# the most experts and the largest top-K the kernels take: 512 experts, top-64
# (d_ff 128: two chunks, so r = .5 splits every expert); T = 64 and 100 take
# the many-token routing, and in bf16 the matrix-core path (T K >= 8 E) with
# more experts than one matrix-core launch holds
WIDE_E_F32 = synth.ModelShape("wide-e-f32", 1, 256, 128, 512, 64, "f32")
WIDE_E_BF16 = synth.ModelShape("wide-e-bf16", 1, 256, 128, 512, 64, "bf16")
MAX_T_E = 100


@pytest.fixture(scope="module", params=[WIDE_E_BF16, WIDE_E_F32], ids=lambda s: s.name)
def rig_e(request):
    from workload import SplitRig
    s = request.param
    r = SplitRig(s, seed=4, max_tokens=MAX_T_E, budget_bytes=s.n_experts * s.expert_bytes)
    yield r
    r.close()


@pytest.mark.parametrize("T", [1, 5, 16, 64, MAX_T_E])
def test_most_experts_largest_top_k_parity(rig_e, T):
    _setup(rig_e, 0.5, list(range(0, 512, 2)))
    h, hf = rig_e.hidden(T, tag=980 + T)
    y, idx, w = _run(rig_e, h, T)
    check_layer(rig_e, 0, hf, y, idx, w)


def test_most_experts_independent_of_residency(rig_e):
    T = 5
    h, hf = rig_e.hidden(T, tag=990)
    outs = []
    for ratio, tops in ((0.5, list(range(0, 512, 2))), (1.0, list(range(512))), (0.0, [])):
        _setup(rig_e, ratio, tops)
        y, idx, w = _run(rig_e, h, T)
        outs.append((y.cpu().numpy()[:T], idx.cpu().numpy()[:T]))
    for y, idx in outs[1:]:
        assert np.array_equal(idx, outs[0][1])
        assert np.array_equal(y, outs[0][0])
