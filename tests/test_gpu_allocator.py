"""The layer allocator (section IV-D, Algorithms 1 and 2) fed from this
device, as the paper's benchmark stage feeds it (section IV-B):

  * dt: the device's benchmark time, "the first few layers of the training
    model" run for tens of iterations: a 2-layer stage of the depth-sweep
    shape (h 1024, 16 heads, FFN 4096, B8 x S512, lengths in [128, 512]),
    forward + backward, median of 20 timed iterations with HIP events;
    heterogeneous devices are this device slowed by a factor 1 + slow_down,
    slow_down in [1, 7] (the paper's speed control, section VI-D);
  * lf: FLOPs of each allocation unit (half-layers here), from the
    per-token formula 3 [2 (4 h^2 + 2 h f) + 4 h S_k], split into its
    attention part 3 [8 h^2 + 4 h S_k] and feed-forward part 3 [4 h f];
  * lm: device bytes of each unit from stage_memory_model_units (the layer
    memory the benchmark stage estimates), checked against what a unit stage
    actually holds on this device;
  * ct: the time to copy one boundary tensor [B, S, h] bf16 on this device,
    as a stand-in for the communication latency between devices;
  * dm: device memories for a mix of large and small devices.

alloc_coarse then alloc_fine run through the C ABI on an 80-layer model
(160 units, the strong-scaling model of section VI-G) over 16 devices, and
must give exactly the oracle's partitions and round counts, with
alloc_workloads bit for bit.  The measured cost of the two unit kinds is
printed beside their FLOP ratio (the cost model of section IV-C assumes time
proportional to FLOPs), and the heuristic's largest workload beside even
allocation's and the exact optimum's."""
import random

import numpy as np
import pytest

import synth
from oracle import allocator as A

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


def _median_ms(fn, iters=20, warmup=3):
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    ts = []
    for _ in range(iters):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        fn()
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    return float(np.median(ts))


@pytest.mark.timeout(300)
def test_allocator_from_device_measurements():
    import torch
    import paper_2202_11836_amd as P
    from paper_2202_11836_amd import Stage

    cfg = synth.CONFIGS["deep_sweep"].with_(L=2)
    B, S, h, H, f = cfg.batch, cfg.seq, cfg.hidden, cfg.heads, cfg.ffn
    T = B * S
    inp = synth.make_inputs(cfg)
    x = torch.from_numpy(inp["x"].astype(np.float32)).to(torch.bfloat16).cuda()
    dy = torch.from_numpy(inp["dy"].astype(np.float32)).to(torch.bfloat16).cuda()
    mask = torch.from_numpy(inp["mask"]).cuda()

    # Benchmark stage: the first two layers, forward + backward.
    st = Stage(2, h, H, f, seed=cfg.seed, dtype="bf16")
    y, dx = torch.empty_like(x), torch.empty_like(x)

    def step(s=st):
        s.forward(x, mask, out=y)
        s.backward(dy, out=dx)
    t_bench = _median_ms(step)
    st.close()
    # Per unit kind: one attention unit, one feed-forward unit.
    t_unit = {}
    for name, first in (("attn", 0), ("ffn", 1)):
        u = Stage(None, h, H, f, seed=cfg.seed, dtype="bf16", first_unit=first, n_units=1)
        t_unit[name] = _median_ms(lambda u=u: step(u))
        held = u.device_bytes()
        u.close()
        t_unit[name + "_bytes"] = held
    # Boundary tensor copy.
    buf = torch.empty_like(x)
    t_copy = _median_ms(lambda: buf.copy_(x))
    _say(f"  benchmark: 2 layers fwd+bwd {t_bench:.3f} ms; attention unit {t_unit['attn']:.3f} ms, "
         f"feed-forward unit {t_unit['ffn']:.3f} ms; boundary copy {t_copy * 1e3:.1f} us")

    # Unit FLOPs (per step, valid keys) and unit memory.
    keys = float(inp["lengths"].astype(np.float64).sum()) * S  # sum over tokens of S_k
    lf_attn = 3.0 * (2.0 * T * 4 * h * h + 4.0 * h * keys)
    lf_ffn = 3.0 * (2.0 * T * 2 * h * f)
    a_b, f_b, shared = P.stage_memory_model_units(h, H, f, B, S, P.STAGE_BF16)
    assert t_unit["attn_bytes"] == a_b + shared and t_unit["ffn_bytes"] == f_b + shared
    _say(f"  cost model: time ratio attention/feed-forward {t_unit['attn'] / t_unit['ffn']:.3f}, "
         f"FLOP ratio {lf_attn / lf_ffn:.3f}; unit memory {a_b / 2**20:.1f} / {f_b / 2**20:.1f} MiB "
         f"(+ {shared / 2**20:.1f} MiB per stage)")

    # 80 encoder layers = 160 units over 16 devices.
    n_layers, D = 80, 16
    lf = [lf_attn if j % 2 == 0 else lf_ffn for j in range(2 * n_layers)]
    lm = [float(a_b) if j % 2 == 0 else float(f_b) for j in range(2 * n_layers)]
    rng = random.Random(7)
    slow = [min(7.0, max(1.0, rng.gauss(4.0, 1.5))) for _ in range(D)]
    dt = [t_bench * (1.0 + s) for s in slow]
    ct = [t_copy * (1.0 + 3.0 * rng.random()) for _ in range(D)]
    total = sum(lm)
    # every fourth device small: its even share does not fit, so Algorithm 1 moves layers
    dm = [total / D * (0.8 if i % 4 == 3 else 1.6) for i in range(D)]

    opi, osw, ok = A.coarse_allocation(lm, dm)
    assert ok
    pi, sweeps = P.alloc_coarse(lm, dm)
    assert (pi, sweeps) == (opi, osw)
    assert pi != A.equal_partition(len(lm), D), "memory limits should move the equal split"
    fpi, frounds = A.fine_allocation(dt, dm, ct, lf, lm, opi, 200)
    pi2, rounds = P.alloc_fine(dt, dm, ct, lf, lm, pi, 200)
    assert (pi2, rounds) == (fpi, frounds)
    for mode, per_layer in ((P.ALLOC_CT_PER_LAYER, True), (P.ALLOC_CT_PER_DEVICE, False)):
        w = P.alloc_workloads(dt, ct, lf, pi2, mode)
        assert w == [A.device_workload(dt, ct, lf, pi2, i, per_layer) for i in range(D)]
    assert A.memory_satisfied(lm, dm, pi2)
    heur = max(A.device_workload(dt, ct, lf, pi2, i) for i in range(D))
    best, bpi = A.optimal_partition(dt, dm, ct, lf, lm)
    even_pi = A.equal_partition(len(lm), D)
    even = max(A.device_workload(dt, ct, lf, even_pi, i) for i in range(D))
    _say(f"  allocation of 160 units over 16 devices: sweeps {sweeps}, rounds {rounds}; largest "
         f"workload even {even:.4g} (memory {'ok' if A.memory_satisfied(lm, dm, even_pi) else 'exceeded'}), "
         f"heuristic {heur:.4g} ({heur / best:.3f} x optimum), optimum {best:.4g}")
    assert best <= heur * (1 + 1e-12)
