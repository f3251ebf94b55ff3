"""Contract of the C ABI on the GPU: error codes, state handling, empty
batches, determinism, initialisation and partition invariance (re-splitting
a block of layers into two chained stages must not change the result, the
premise of re-allocating layers between devices, section III / IV-D)."""
import numpy as np
import pytest

import synth
from _parity import IDX, make_stage, to_numpy, to_torch

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


def test_init_rejects_bad_dims():
    from paper_2202_11836_amd import STAGE_BF16, StageError, stage_init
    for args in [(0, 128, 2, 512), (1, 100, 2, 512), (1, 128, 3, 512), (1, 256, 2, 512),
                 (1, 128, 2, 500), (1, 4096, 64, 512)]:
        with pytest.raises(StageError):
            stage_init(*args, 0, STAGE_BF16)


def test_forward_backward_state_errors():
    import torch
    from paper_2202_11836_amd import Stage, StageError
    _say("case abi state errors")
    st = Stage(1, 128, 2, 256, seed=1, dtype="bf16")
    dy = torch.zeros(2, 16, 128, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(StageError) as e:
        st.backward(dy)
    assert e.value.status == 2
    x = torch.randn(2, 16, 128, device="cuda").to(torch.bfloat16)
    st.forward(x)
    st.backward(dy)
    with pytest.raises(StageError) as e:  # context consumed
        st.backward(dy)
    assert e.value.status == 2
    from paper_2202_11836_amd import stage_forward
    with pytest.raises(StageError) as e:  # null y
        stage_forward(st.handle, x, None, 2, 16, None)
    assert e.value.status == 1
    with pytest.raises(StageError) as e:  # x and y alias
        stage_forward(st.handle, x, None, 2, 16, x)
    assert e.value.status == 1
    with pytest.raises(StageError):
        st.param(1, 0)
    with pytest.raises(StageError):
        st.param(0, 12)
    st.close()


def test_empty_batch():
    import torch
    from paper_2202_11836_amd import Stage
    st = Stage(2, 128, 2, 256, seed=1, dtype="f32")
    x = torch.zeros(0, 8, 128, device="cuda")
    y = st.forward(x)
    dx = st.backward(torch.zeros_like(x))
    torch.cuda.synchronize()
    assert y.shape == (0, 8, 128) and dx.shape == (0, 8, 128)
    for l in range(2):
        for w in range(12):
            assert float(st.grad(l, w).abs().max()) == 0.0
    st.close()


def test_init_statistics_and_seed_determinism():
    from paper_2202_11836_amd import Stage
    a = Stage(2, 256, 4, 1024, seed=7, dtype="bf16")
    b = Stage(2, 256, 4, 1024, seed=7, dtype="bf16")
    c = Stage(2, 256, 4, 1024, seed=8, dtype="bf16")
    for l in range(2):
        for w in range(12):
            pa = to_numpy(a.param(l, w))
            pb = to_numpy(b.param(l, w))
            np.testing.assert_array_equal(pa, pb)
            if w in (0, 2, 6, 8):
                assert abs(pa.mean()) < 2e-3 and abs(pa.std() - 0.02) < 1e-3
                assert not np.array_equal(pa, to_numpy(c.param(l, w)))
            elif w in (4, 10):
                assert np.all(pa == 1.0)
            else:
                assert np.all(pa == 0.0)
    # distinct layers / tensors get distinct streams
    assert not np.array_equal(to_numpy(a.param(0, 2)), to_numpy(a.param(1, 2)))
    for s in (a, b, c):
        s.close()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_bitwise_determinism(dtype):
    import torch
    cfg = synth.StageConfig("det", 2, 256, 4, 512, 4, 64, 10, 64, dtype, 5)
    _say(f"case determinism {dtype}")
    inp = synth.make_inputs(cfg)
    params = synth.make_params(cfg, perturb=True)
    st = make_stage(cfg, params)
    x = to_torch(inp["x"], dtype)
    mask = torch.from_numpy(inp["mask"]).cuda()
    dy = to_torch(inp["dy"], dtype)
    outs = []
    for _ in range(2):
        y = st.forward(x, mask)
        dx = st.backward(dy)
        torch.cuda.synchronize()
        outs.append((y.clone(), dx.clone(), [st.grad(l, w) for l in range(2) for w in range(12)]))
    assert torch.equal(outs[0][0], outs[1][0])
    assert torch.equal(outs[0][1], outs[1][1])
    for g0, g1 in zip(outs[0][2], outs[1][2]):
        assert torch.equal(g0, g1)
    st.close()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_partition_invariance(dtype):
    """Layers [0,3) as one stage == stage [0,1) then stage [1,3), chained
    through y -> x forward and dx -> dy backward.  Bitwise on fp32 stages and
    in the bf16 forward pass (the tensor between layers is the bf16 layer
    output either way).  In the bf16 backward pass the gradient crossing
    the boundary is the bf16 dx of the upper stage, while inside one stage
    it stays fp32: there the two agree to the rounding of that one tensor
    (relative L2 <= 1e-2, the bf16 gradient tolerance, on dx and every
    gradient)."""
    import torch
    cfg = synth.StageConfig("part", 3, 128, 2, 256, 2, 32, 8, 32, dtype, 9)
    _say(f"case partition {dtype}")
    inp = synth.make_inputs(cfg)
    params = synth.make_params(cfg, perturb=True)
    whole = make_stage(cfg, params)
    first = make_stage(cfg.with_(L=1), params[:1])
    second = make_stage(cfg.with_(L=2), params[1:])
    x = to_torch(inp["x"], dtype)
    mask = torch.from_numpy(inp["mask"]).cuda()
    dy = to_torch(inp["dy"], dtype)
    y = whole.forward(x, mask)
    dx = whole.backward(dy)
    y1 = first.forward(x, mask)
    y2 = second.forward(y1, mask)
    d1 = second.backward(dy)
    d0 = first.backward(d1)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)
    # (whole stage, chained stages): dx, then layer 0's 12 gradients (in
    # `first`), then layers 1 and 2 (layers 0 and 1 of `second`)
    pairs = [(dx, d0)] + [(whole.grad(l, w), first.grad(0, w) if l == 0 else second.grad(l - 1, w))
                          for l in range(3) for w in range(12)]
    for k, (a, b) in enumerate(pairs):
        if dtype == "f32" or k >= 1 + 12:  # layers above the boundary see the same inputs
            assert torch.equal(a, b), k
        else:
            a, b = a.float(), b.float()
            e = float((a - b).norm() / b.norm().clamp_min(1e-30))
            if k == 1 + 1:  # the key-bias gradient is ~0: its norm against the query's
                e = float((a[128:256] - b[128:256]).norm() / b[:128].norm())
            print(f"  chained vs whole, pair {k}: rel l2 {e:.2e}", flush=True)
            assert e <= 1e-2, (k, e)
    for s in (whole, first, second):
        s.close()


def test_stream_is_respected():
    """Work enqueued on a side stream is ordered on that stream."""
    import torch
    cfg = synth.StageConfig("strm", 1, 128, 2, 256, 2, 32, None, None, "bf16", 4)
    inp = synth.make_inputs(cfg)
    params = synth.make_params(cfg)
    st = make_stage(cfg, params)
    x = to_torch(inp["x"], "bf16")
    ref = st.forward(x)
    st.backward(to_torch(inp["dy"], "bf16"))
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        y = st.forward(x)
        st.backward(to_torch(inp["dy"], "bf16"))
    side.synchronize()
    assert torch.equal(y, ref)
    st.close()


def test_mfma_peak_measurement():
    """The device's achievable dense bf16 MFMA rate and the clock it holds:
    within the physical range of an MI355X (256 compute units, at most
    2.4 GHz, 2516.6 TFLOP/s at that clock) and consistent with each other
    (the rate cannot exceed what the measured clock allows)."""
    import paper_2202_11836_amd as P
    tf, ghz = P.stage_mfma_peak(4000)
    print(f"case mfma peak: {tf:.1f} TFLOP/s at {ghz:.3f} GHz", flush=True)
    assert 0.5 < ghz < 2.6
    assert 200.0 < tf <= 2516.6 * 1.01
    assert tf <= 2516.6 * ghz / 2.4 * 1.05


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_recorded_gradients(dtype):
    """stage_record_grads: after a backward, stage_read kind 3 gives the
    gradient that reached each layer's output: dy at the top layer, and at
    layer 0 what the upper two layers hand down, i.e. the dx of a stage of
    those two layers (bitwise on fp32; on bf16 that dx is the recorded fp32
    value rounded to bf16).  Without recording, or after a new forward,
    kind 3 is a state error."""
    import torch
    import paper_2202_11836_amd as P
    cfg = synth.StageConfig("rec", 3, 128, 2, 256, 2, 32, 8, 32, dtype, 5)
    _say(f"case recorded gradients {dtype}")
    inp = synth.make_inputs(cfg)
    params = synth.make_params(cfg, perturb=True)
    whole = make_stage(cfg, params)
    upper = make_stage(cfg.with_(L=2), params[1:])
    x = to_torch(inp["x"], dtype)
    mask = torch.from_numpy(inp["mask"]).cuda()
    dy = to_torch(inp["dy"], dtype)
    T = cfg.batch * cfg.seq
    whole.forward(x, mask)
    whole.backward(dy)
    with pytest.raises(P.StageError) as e:
        whole.recorded_grad(0, T)
    assert e.value.status == P.binding.STAGE_ESTATE
    whole.record_grads(True)
    y = whole.forward(x, mask)
    dx = whole.backward(dy)
    y0 = whole.saved(1, 0, T).view_as(x)  # layer 0's output = layer 1's input
    upper.forward(y0, mask)
    d1 = upper.backward(dy)
    torch.cuda.synchronize()
    assert torch.equal(whole.recorded_grad(2, T), dy.reshape(T, -1).float())
    r0 = whole.recorded_grad(0, T)
    if dtype == "f32":
        assert torch.equal(r0, d1.reshape(T, -1))
    else:
        assert torch.equal(r0.to(torch.bfloat16), d1.reshape(T, -1))
    assert P.stage_tensor_bytes(whole.handle, 3, 0, 0) == T * cfg.hidden * 4
    whole.forward(x, mask)
    with pytest.raises(P.StageError) as e:
        whole.recorded_grad(0, T)
    assert e.value.status == P.binding.STAGE_ESTATE
    for s in (whole, upper):
        s.close()
