"""stage_backward_noalloc (the backward for callers that cannot allocate:
partial results in the library's static device scratch) against
stage_backward, through the C ABI: two stages with the same parameters, one
differentiated by each entry point after identical forwards, on two calls
in a row, the second with a smaller batch.  The same kernels run on the same
data in the same order, so dx and every gradient must agree bitwise (the
parity bar for this path is the existing entry point's output).  A batch
whose partial results exceed the scratch is rejected with EINVAL and the
saved context is kept."""
import numpy as np
import pytest

import synth
from _parity import IDX, make_stage, to_torch

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_backward_matches_backward(dtype):
    import torch
    if dtype == "bf16":
        cfg = synth.CONFIGS["bert_base_3"].with_(L=2)
        shapes = ((16, 128), (3, 96))
    else:
        cfg = synth.CONFIGS["tiny"].with_(L=2)
        shapes = ((4, 64), (2, 24))
    params = synth.make_params(cfg, perturb=True)
    ref = make_stage(cfg, params)
    na = make_stage(cfg, params)
    try:
        for batch, seq in shapes:
            c = cfg.with_(batch=batch, seq=seq, len_lo=max(1, seq // 2), len_hi=seq)
            _say(f"case no-alloc backward {dtype} B{batch} x S{seq}")
            inp = synth.make_inputs(c, seed=batch * 100 + seq)
            x = to_torch(inp["x"], dtype)
            dy = to_torch(inp["dy"], dtype)
            mask = torch.from_numpy(np.ascontiguousarray(inp["mask"])).cuda()
            ref.forward(x, mask)
            dx_ref = ref.backward(dy)
            na.forward(x, mask)
            dx_na = na.backward_noalloc(dy, torch.empty_like(dy))
            torch.cuda.synchronize()
            assert torch.equal(dx_ref, dx_na)
            for l in range(cfg.L):
                for name in synth.PARAM_NAMES:
                    assert torch.equal(ref.grad(l, IDX[name]), na.grad(l, IDX[name])), (l, name)
    finally:
        ref.close()
        na.close()


def test_noalloc_backward_rejects_a_batch_beyond_the_scratch():
    import torch
    import paper_2202_11836_amd as P
    from paper_2202_11836_amd import Stage
    _say("case no-alloc backward beyond the scratch: h 2048, f 8192, B64 x S512")
    st = Stage(1, 2048, 32, 8192, seed=3, dtype="bf16")
    try:
        x = torch.zeros(64, 512, 2048, dtype=torch.bfloat16, device="cuda")
        st.forward(x)
        with pytest.raises(P.StageError) as e:
            st.backward_noalloc(x, torch.empty_like(x))
        assert e.value.status == P.binding.STAGE_EINVAL and "scratch" in str(e.value)
        st.backward(x)  # the context was kept
        torch.cuda.synchronize()
    finally:
        st.close()
