"""Runs the host-only paths of the library under AddressSanitizer and
UndefinedBehaviorSanitizer (launched by test_sanitized_host.py with the
sanitizer runtime preloaded; argv[1] = the sanitized library).  No device is
touched and torch is not imported: the calls below either stay on the host
(the allocator, the dry-run memory model) or fail argument checks before any
HIP call.  Exits 0 when every result matches the oracle and every invalid
call is rejected; a sanitizer report aborts the process with its own
message."""
import ctypes
import os
import random
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))

from oracle import allocator as A  # noqa: E402
from test_memory_model import closed_form, closed_form_units  # noqa: E402

lib = ctypes.CDLL(sys.argv[1])
vp, i32, i64, u64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_uint64
dp, ip = ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i32)
lib.alloc_coarse.argtypes = [i32, i32, dp, dp, ip, ip]
lib.alloc_fine.argtypes = [i32, i32, dp, dp, dp, dp, dp, i32, ip, ip]
lib.alloc_workloads.argtypes = [i32, i32, dp, dp, dp, ip, i32, dp]
lib.stage_memory_model.argtypes = [i32, i32, i32, i32, i32, i32, ctypes.POINTER(i64),
                                   ctypes.POINTER(i64)]
lib.stage_memory_model_units.argtypes = [i32, i32, i32, i32, i32, i32, ctypes.POINTER(i64),
                                         ctypes.POINTER(i64), ctypes.POINTER(i64)]
lib.stage_init.argtypes = [i32, i32, i32, i32, u64, i32, vp, ctypes.POINTER(vp)]
lib.stage_init_units.argtypes = [i32, i32, i32, i32, i32, u64, i32, vp, ctypes.POINTER(vp)]
lib.stage_last_error.argtypes = [vp]
lib.stage_last_error.restype = ctypes.c_char_p
lib.stage_mfma_peak.argtypes = [vp, i32, dp, dp]
for name in ("stage_forward", "stage_backward", "stage_param", "stage_grad", "stage_set_param",
             "stage_read", "stage_trace_site", "stage_trace_mask", "stage_trace_read",
             "stage_device_bytes", "stage_set_stream", "stage_record_grads"):
    getattr(lib, name).restype = i32
OK, EINVAL, ENOFIT = 0, 1, 2


def dvec(v):
    return (ctypes.c_double * max(len(v), 1))(*[float(x) for x in v])


def ivec(v):
    return (i32 * max(len(v), 1))(*[int(x) for x in v])


def check(cond, what):
    if not cond:
        print("FAILED:", what, flush=True)
        sys.exit(1)


# Allocator: random instances against the oracle (same as the unsanitized test).
def random_instance(rng, L, D, tight):
    dt = [float(rng.randint(1, 7)) for _ in range(D)]
    ct = [rng.choice([0.0, 0.01, 0.5]) * rng.random() for _ in range(D)]
    lf = [rng.choice([0.05, 1.0, 3.0, 4.0]) * (0.5 + rng.random()) for _ in range(L)]
    lm = [0.5 + rng.random() for _ in range(L)]
    total = sum(lm)
    dm = [total / D * (0.6 + 1.2 * rng.random()) for _ in range(D)] if tight else [total] * D
    return dt, dm, ct, lf, lm


rng = random.Random(11)
for trial in range(150):
    L = rng.randint(1, 60)
    D = rng.randint(1, min(8, L))
    dt, dm, ct, lf, lm = random_instance(rng, L, D, trial % 2 == 0)
    opi, osw, ok = A.coarse_allocation(lm, dm)
    pi, sw = ivec([0] * (D + 1)), i32(0)
    st = lib.alloc_coarse(L, D, dvec(lm), dvec(dm), pi, ctypes.byref(sw))
    check(st == (OK if ok else ENOFIT) and list(pi)[:D + 1] == opi, f"alloc_coarse {trial}")
    if ok:
        check(sw.value == osw, f"alloc_coarse sweeps {trial}")
    else:
        opi, dm = A.equal_partition(L, D), [1e9] * D
    max_iter = rng.choice([0, 1, 3, 100])
    fpi, frounds = A.fine_allocation(dt, dm, ct, lf, lm, opi, max_iter)
    pi, rounds = ivec(opi), i32(0)
    st = lib.alloc_fine(L, D, dvec(dt), dvec(dm), dvec(ct), dvec(lf), dvec(lm), max_iter, pi,
                        ctypes.byref(rounds))
    check(st == OK and list(pi)[:D + 1] == fpi and rounds.value == frounds, f"alloc_fine {trial}")
    for mode, per_layer in ((0, True), (1, False)):
        out = (ctypes.c_double * D)()
        st = lib.alloc_workloads(L, D, dvec(dt), dvec(ct), dvec(lf), ivec(fpi), mode, out)
        want = [A.device_workload(dt, ct, lf, fpi, i, per_layer) for i in range(D)]
        check(st == OK and list(out) == want, f"alloc_workloads {trial}")

# Allocator: invalid arguments.
z = i32(0)
bad = [
    lambda: lib.alloc_coarse(1, 2, dvec([1.0]), dvec([1.0, 1.0]), ivec([0] * 3), ctypes.byref(z)),
    lambda: lib.alloc_coarse(0, 0, dvec([]), dvec([]), ivec([0]), ctypes.byref(z)),
    lambda: lib.alloc_coarse(2, 1, dvec([1.0, -1.0]), dvec([5.0]), ivec([0, 0]), ctypes.byref(z)),
    lambda: lib.alloc_coarse(2, 1, dvec([1.0, float("nan")]), dvec([5.0]), ivec([0, 0]),
                             ctypes.byref(z)),
    lambda: lib.alloc_coarse(2, 1, None, dvec([5.0]), ivec([0, 0]), ctypes.byref(z)),
    lambda: lib.alloc_fine(4, 2, dvec([1, 1]), dvec([9, 9]), dvec([0, 0]), dvec([1] * 4),
                           dvec([1] * 4), 5, ivec([0, 0, 4]), ctypes.byref(z)),
    lambda: lib.alloc_fine(4, 2, dvec([1, 1]), dvec([9, 9]), dvec([0, 0]), dvec([1] * 4),
                           dvec([1] * 4), 5, ivec([0, 1, 3]), ctypes.byref(z)),
    lambda: lib.alloc_fine(4, 2, dvec([1, 1]), dvec([9, 9]), dvec([0, 0]), dvec([1] * 4),
                           dvec([1] * 4), -1, ivec([0, 2, 4]), ctypes.byref(z)),
    lambda: lib.alloc_workloads(2, 1, dvec([1.0]), dvec([0.0]), dvec([1.0, 1.0]), ivec([0, 2]), 7,
                                (ctypes.c_double * 1)()),
]
for k, f in enumerate(bad):
    check(f() == EINVAL, f"allocator EINVAL case {k}")

# Memory model (dry-run stages: the allocation calls count bytes only).
for h, H, f_, B, S, bf16 in ((128, 2, 512, 2, 32, False), (768, 12, 3072, 16, 128, True),
                            (1024, 16, 4096, 32, 512, True), (1024, 16, 4096, 1, 384, True),
                            (1024, 16, 4096, 0, 512, True)):
    per, sh = i64(0), i64(0)
    check(lib.stage_memory_model(h, H, f_, B, S, int(bf16), ctypes.byref(per), ctypes.byref(sh)) == OK,
          "stage_memory_model")
    check(per.value == closed_form(h, H, f_, B, S, bf16), f"memory model {h} {B}x{S}")
    a, fu, sh2 = i64(0), i64(0), i64(0)
    check(lib.stage_memory_model_units(h, H, f_, B, S, int(bf16), ctypes.byref(a), ctypes.byref(fu),
                                       ctypes.byref(sh2)) == OK, "stage_memory_model_units")
    check((a.value, fu.value) == closed_form_units(h, H, f_, B, S, bf16) and sh2.value == sh.value,
          f"memory model units {h} {B}x{S}")
for args in [(100, 2, 512, 1, 8), (128, 3, 512, 1, 8), (128, 2, 500, 1, 8), (128, 2, 512, -1, 8)]:
    per, sh = i64(0), i64(0)
    check(lib.stage_memory_model(*args, 1, ctypes.byref(per), ctypes.byref(sh)) == EINVAL,
          f"memory model EINVAL {args}")
check(lib.stage_memory_model(128, 2, 512, 1, 8, 1, None, None) == EINVAL, "memory model null out")

# Stage arguments rejected before any device call.
out = vp()
for args in [(0, 128, 2, 512), (2, 100, 2, 512), (2, 128, 3, 512), (2, 128, 2, 500),
             (2, 4096, 64, 512)]:
    check(lib.stage_init(*args, 0, 1, None, ctypes.byref(out)) == EINVAL and not out.value,
          f"stage_init EINVAL {args}")
    check(len(lib.stage_last_error(None)) > 0, "stage_init message")
check(lib.stage_init(2, 128, 2, 512, 0, 7, None, ctypes.byref(out)) == EINVAL, "stage_init dtype")
check(lib.stage_init(2, 128, 2, 512, 0, 1, None, None) == EINVAL, "stage_init null out")
for args in [(-1, 2), (0, 0), (1 << 30, 1)]:
    check(lib.stage_init_units(*args, 128, 2, 512, 0, 1, None, ctypes.byref(out)) == EINVAL,
          f"stage_init_units EINVAL {args}")
t, g = ctypes.c_double(0), ctypes.c_double(0)
check(lib.stage_mfma_peak(None, 0, ctypes.byref(t), ctypes.byref(g)) == EINVAL, "peak iters")
check(lib.stage_mfma_peak(None, 10, None, ctypes.byref(g)) == EINVAL, "peak null")
# Calls on a null handle.
n = ctypes.c_int(0)
check(lib.stage_forward(None, None, None, 1, 1, None) == EINVAL, "forward null")
check(lib.stage_backward(None, None, None) == EINVAL, "backward null")
check(lib.stage_param(None, 0, 0, None, None, None) == EINVAL, "param null")
check(lib.stage_grad(None, 0, 0, None, None) == EINVAL, "grad null")
check(lib.stage_read(None, 0, 0, 0, None, 0) == EINVAL, "read null")
check(lib.stage_trace_read(None, ctypes.byref(n), None) == EINVAL, "trace null")
check(lib.stage_record_grads(None, 1) == EINVAL, "record null")
check(lib.stage_device_bytes(None, None) == EINVAL, "device bytes null")
lib.stage_destroy(None)
print("sanitized host paths: ok", flush=True)
