"""ms_forward_noalloc (work buffers in the library's static device array)
against ms_forward on the same inputs and residency: selected experts and
gate weights bitwise equal, outputs bitwise equal (the same kernels with the
same work split) and within the oracle's tolerance; two calls in a row, the
second with fewer tokens, on split layers with streamed misses; and the
refusal of a context whose work buffers exceed the array."""
import numpy as np
import pytest

import synth
from gpu_helpers import check_layer

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

TINY_BF16 = synth.ModelShape("tiny-bf16", 2, 256, 512, 8, 2, "bf16")
WIDE_BF16 = synth.ModelShape("wide-bf16", 1, 1024, 512, 40, 6, "bf16", n_shared=1, d_ff_shared=512)


def _pair(r, T, tag, flags):
    """The same tokens through ms_forward and ms_forward_noalloc, the staging
    buffer emptied before each, so both stream the same misses."""
    from paper_2509_08342_amd import moesplit as ms
    h, hf = r.hidden(T, tag=tag)
    out = []
    for fn in (ms.ms_forward, ms.ms_forward_noalloc):
        ms.ms_drop_buffer(r.ctx)
        y, idx, w = r.outputs(T)
        y.fill_(float("nan"))
        fn(r.ctx, 0, h, T, y, idx, w, flags, torch.cuda.current_stream())
        torch.cuda.synchronize()
        out.append((y[:T].clone(), idx[:T].clone(), w[:T].clone()))
    (y0, i0, w0), (y1, i1, w1) = out
    assert torch.equal(i0, i1)
    assert torch.equal(w0.view(torch.int32), w1.view(torch.int32))
    assert torch.equal(y0.view(torch.int32), y1.view(torch.int32))
    check_layer(r, 0, hf, y1, i1, w1)


@pytest.mark.parametrize("shape,T1,T2", [(synth.TINY, 5, 2), (TINY_BF16, 9, 1), (WIDE_BF16, 70, 3)],
                         ids=["tiny-f32", "tiny-bf16", "wide-bf16-many"])
def test_noalloc_forward_equals_forward(shape, T1, T2):
    from paper_2509_08342_amd import moesplit as ms
    from workload import SplitRig, top_bytes
    with SplitRig(shape, seed=21, max_tokens=max(T1, T2), budget_bytes=shape.n_experts * shape.expert_bytes) as r:
        tb = top_bytes(r, 0.5)
        L = shape.n_layers
        r.configure([shape.n_experts // 2 * tb] * L, [0.5] * L)
        r.load_tops(0, range(0, shape.n_experts, 2))
        flags = ms.MS_FWD_PREDICT_NEXT if L > 1 else 0
        _pair(r, T1, 1, flags)
        _pair(r, T2, 2, flags)
        ms.ms_sync(r.ctx)


def test_noalloc_refuses_work_buffers_beyond_the_array():
    from paper_2509_08342_amd import moesplit as ms
    from workload import SplitRig
    shape = synth.ModelShape("big-work", 1, 2048, 1408, 8, 2, "bf16")
    with SplitRig(shape, seed=1, max_tokens=512, budget_bytes=0) as r:
        r.configure([0], [0.0])
        h, _ = r.hidden(4, tag=3)
        y, idx, w = r.outputs(4)
        with pytest.raises(ms.MoeSplitError) as ei:
            ms.ms_forward_noalloc(r.ctx, 0, h, 4, y, idx, w)
        assert ei.value.status == ms.MS_E_UNSUPPORTED
        # the context still works through ms_forward
        ms.ms_forward(r.ctx, 0, h, 4, y, idx, w)
        torch.cuda.synchronize()
