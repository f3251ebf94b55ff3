"""Layer memory model (the lm_j input of the allocator's benchmark stage,
section IV-B): stage_memory_model against a closed form written from the
stage's storage plan, and (GPU) against the bytes the library actually
requests and the device memory it actually takes."""
import pytest

import synth


def closed_form_units(h, H, f, B, S, bf16):
    """(attention unit, feed-forward unit) bytes from the storage plan of a
    half-layer stage: the attention half holds W_qkv, b_qkv, W_o, b_o, g1,
    be1 (with gradients) and saves X, QKV, the fp32 scores (fp32 stages) or
    the log-sum-exp, C, x_hat1, rstd1 and (bf16 stages) C's rounding
    residual; the feed-forward half holds W_1, b_1,
    W_2, b_2, g2, be2 and saves its input H1, GELU'(U), G, x_hat2, rstd2."""
    e = 2 if bf16 else 4
    T = B * S
    a = lambda n: max(n, 256)
    BSS = 0 if bf16 else B * H * S * S
    attn = (a(3 * h * h * e) + a(3 * h * h * 4) + a(h * h * e) + a(h * h * 4)
            + sum(a(n * 4) * 2 for n in (3 * h, h, h, h))
            + a(T * h * e) + a(T * 3 * h * e) + a(BSS * e) + a(B * H * S * 4) + a(T * h * e)
            + a(T * h * e) + a(T * 4) + (a(T * h * e) if bf16 else 0))
    ffn = (a(f * h * e) + a(f * h * 4) + a(h * f * e) + a(h * f * 4)
           + sum(a(n * 4) * 2 for n in (f, h, h, h))
           + a(T * h * e) + a(T * f * e) + a(T * f * e) + a(T * h * e) + a(T * 4))
    return attn, ffn


def closed_form(h, H, f, B, S, bf16):
    """Device bytes of one layer and of the per-stage workspace, from the
    storage plan: parameters in the stage dtype (matrices) or fp32 (vectors)
    with fp32 gradients; the saved activations X, QKV, C, x_hat1, H1,
    GELU'(U), G, x_hat2 (stage dtype), rstd1, rstd2 and the log-sum-exp
    (fp32); the fp32 score matrix is kept only on fp32 stages, the
    context's bf16 rounding residual only on bf16 stages.  Every
    allocation is at least 256 bytes."""
    e = 2 if bf16 else 4
    T = B * S
    a = lambda n: max(n, 256)
    mats = [3 * h * h, h * h, f * h, h * f]
    vecs = [3 * h, h, h, h, f, h, h, h]
    par = sum(a(n * e) + a(n * 4) for n in mats) + sum(a(n * 4) + a(n * 4) for n in vecs)
    BSS = 0 if bf16 else B * H * S * S
    saved = (a(T * h * e) + a(T * 3 * h * e) + a(BSS * e) + a(B * H * S * 4) + a(T * h * e)
             + a(T * h * e) + a(T * 4) + a(T * h * e) + a(T * f * e) + a(T * f * e)
             + a(T * h * e) + a(T * 4) + (a(T * h * e) if bf16 else 0))
    return par + saved


@pytest.mark.parametrize("cfg", ["tiny", "bert_base_3", "bert_large_4"])
def test_memory_model_per_layer_closed_form(cfg):
    import paper_2202_11836_amd as P
    try:
        P.load_library()
    except RuntimeError as e:
        pytest.skip(str(e))
    c = synth.CONFIGS[cfg]
    bf16 = c.dtype == "bf16"
    per_layer, shared = P.stage_memory_model(c.hidden, c.heads, c.ffn, c.batch, c.seq,
                                             P.STAGE_BF16 if bf16 else P.STAGE_F32)
    assert per_layer == closed_form(c.hidden, c.heads, c.ffn, c.batch, c.seq, bf16)
    # the workspace holds at least the fp32 LayerNorm inputs and the data
    # gradients of one layer
    T, h, f = c.batch * c.seq, c.hidden, c.ffn
    assert shared > T * h * 4 + T * f * (2 if bf16 else 4)


@pytest.mark.parametrize("cfg", ["tiny", "bert_base_3", "bert_large_4"])
def test_memory_model_units_closed_form(cfg):
    import paper_2202_11836_amd as P
    try:
        P.load_library()
    except RuntimeError as e:
        pytest.skip(str(e))
    c = synth.CONFIGS[cfg]
    bf16 = c.dtype == "bf16"
    code = P.STAGE_BF16 if bf16 else P.STAGE_F32
    attn, ffn, shared = P.stage_memory_model_units(c.hidden, c.heads, c.ffn, c.batch, c.seq, code)
    assert (attn, ffn) == closed_form_units(c.hidden, c.heads, c.ffn, c.batch, c.seq, bf16)
    per_layer, shared_l = P.stage_memory_model(c.hidden, c.heads, c.ffn, c.batch, c.seq, code)
    assert per_layer == attn + ffn and shared == shared_l


def test_memory_model_rejects_bad_dims():
    import paper_2202_11836_amd as P
    try:
        P.load_library()
    except RuntimeError as e:
        pytest.skip(str(e))
    for args in [(100, 2, 512, 1, 8), (128, 3, 512, 1, 8), (128, 2, 500, 1, 8), (128, 2, 512, -1, 8)]:
        with pytest.raises(P.StageError):
            P.stage_memory_model(*args, P.STAGE_BF16)


@pytest.mark.gpu
@pytest.mark.parametrize("L,cfg,dtype", [(2, "tiny", "f32"), (3, "bert_base_3", "bf16"),
                                         (2, "bert_large_4", "bf16")])
def test_memory_model_matches_allocations(L, cfg, dtype):
    import torch

    import paper_2202_11836_amd as P
    c = synth.CONFIGS[cfg]
    print(f"case memory {cfg} L={L} {dtype}", flush=True)
    code = P.STAGE_BF16 if dtype == "bf16" else P.STAGE_F32
    per_layer, shared = P.stage_memory_model(c.hidden, c.heads, c.ffn, c.batch, c.seq, code)
    # warm the runtime (code objects, streams) before measuring free memory
    warm = P.Stage(1, c.hidden, c.heads, c.ffn, seed=0, dtype=dtype)
    warm.close()
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info()[0]
    st = P.Stage(L, c.hidden, c.heads, c.ffn, seed=1, dtype=dtype)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    x = torch.zeros(c.batch, c.seq, c.hidden, dtype=tdt, device="cuda")
    y = st.forward(x)
    torch.cuda.synchronize()
    held = st.device_bytes()
    assert held == L * per_layer + shared
    free1 = torch.cuda.mem_get_info()[0]
    taken = free0 - free1
    # x and y come from torch's caching allocator (maybe from memory it
    # already held), and the device hands out memory in pages: taken is the
    # prediction up to those two torch tensors and a rounding per allocation
    # (about 100 allocations here)
    slack = 4 * x.numel() * x.element_size() + (128 << 20)
    assert held <= taken + slack and taken <= held + 100 * (2 << 20) + slack
    st.close()
    del y


@pytest.mark.gpu
def test_memory_model_units_matches_allocations():
    """A stage of units [1, 4) (feed-forward half of layer 0, layer 1) holds
    shared + attn_unit + 2 ffn_unit bytes."""
    import torch

    import paper_2202_11836_amd as P
    c = synth.CONFIGS["bert_base_3"]
    print("case memory units bert_base_3 [1,4) bf16", flush=True)
    attn, ffn, shared = P.stage_memory_model_units(c.hidden, c.heads, c.ffn, c.batch, c.seq,
                                                   P.STAGE_BF16)
    st = P.Stage(None, c.hidden, c.heads, c.ffn, seed=1, dtype="bf16", first_unit=1, n_units=3)
    x = torch.zeros(c.batch, c.seq, c.hidden, dtype=torch.bfloat16, device="cuda")
    st.forward(x)
    torch.cuda.synchronize()
    assert st.device_bytes() == shared + attn + 2 * ffn
    st.close()
