"""Host-path fuzz driver for a sanitizer build of libzeroshard (used by
tests/test_sanitizers_cpu.py).  Every zero_shard_step / zero_shard_apply call it
makes is invalid or empty, so it never needs a GPU: it exercises argument
validation, layout, accounting, the loss scaler and error reporting."""
import ctypes, sys, random
L = ctypes.CDLL(sys.argv[1])
class Layout(ctypes.Structure):
    _fields_ = [(k, ctypes.c_int64) for k in ("S", "off", "valid", "pad")]
class Scaler(ctypes.Structure):
    _fields_ = [("scale", ctypes.c_double), ("min_scale", ctypes.c_double), ("window", ctypes.c_int64), ("applied", ctypes.c_int64), ("good", ctypes.c_int64)]
P, i64, i32, dbl = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_double
L.zero_partition_layout.argtypes = [i64, i32, i32, ctypes.POINTER(Layout)]
L.zero_shard_step.argtypes = [P, P, P, P, P, i64, dbl, dbl, dbl, dbl, dbl, i64, dbl, dbl, P]
L.zero_shard_apply.argtypes = [P, P, P, P, P, i64, dbl, dbl, dbl, dbl, dbl, dbl, i64, dbl, dbl, P]
L.zero_shard_stats.argtypes = [P, i64, ctypes.POINTER(dbl), P]
L.zero_model_state_bytes.argtypes = [dbl, dbl, i32, dbl, ctypes.POINTER(dbl)]
L.zero_scaler_init.argtypes = [ctypes.POINTER(Scaler), dbl, i64, dbl]
L.zero_scaler_update.argtypes = [ctypes.POINTER(Scaler), i32]
L.zero_last_error.restype = ctypes.c_char_p
L.zero_profile_enable.argtypes = [i32]
r = random.Random(0)
lay = Layout()
for _ in range(20000):
    psi = r.choice([r.randrange(0, 100), r.randrange(0, 1 << 62), (1 << 62), -r.randrange(1, 5)])
    nd = r.choice([r.randrange(-2, 20), r.randrange(1, 1 << 31)])
    rank = r.randrange(-2, max(nd, 1) + 2)
    L.zero_partition_layout(psi, nd, rank, ctypes.byref(lay))
    L.zero_last_error()
out = dbl()
for st in range(-1, 6):
    L.zero_model_state_bytes(1e9, 4, st, 12, ctypes.byref(out))
L.zero_model_state_bytes(1e9, 4, 1, 12, None)
s = Scaler()
L.zero_scaler_init(ctypes.byref(s), 65536.0, 3, 1.0)
for _ in range(1000):
    L.zero_scaler_update(ctypes.byref(s), r.randrange(2))
L.zero_scaler_update(None, 0)
G = [0x10000000, 0x20000000, 0x30000000, 0x40000000, 0x50000000]
bad = 0
for _ in range(5000):
    ptrs = [p + r.choice([0, 0, 0, 1, 2, 8]) for p in G]
    if r.random() < 0.2: ptrs[r.randrange(5)] = 0
    n = r.choice([-5, 0, 10, (1 << 40) + 1])
    args = dict(lr=r.choice([1e-4, -1, float("nan")]), b1=r.choice([0.9, 1.0, -0.1]), b2=r.choice([0.999, 2.0]),
                eps=r.choice([1e-8, -1e-8]), wd=r.choice([0.0, float("inf")]), t=r.choice([1, 0, -3]),
                sc=r.choice([65536.0, 0.0, float("inf")]), clip=r.choice([1.0, float("nan"), -1]))
    rejected_or_empty = n <= 0 or args["lr"] != 1e-4 or args["b1"] != 0.9 or args["b2"] != 0.999 or args["eps"] != 1e-8 or args["wd"] != 0.0 or args["t"] != 1 or args["sc"] != 65536.0 or args["clip"] != 1.0 or 0 in ptrs or any(p % 2 for p in ptrs) or any(p % 4 for p in ptrs[1:4])
    if not rejected_or_empty:
        continue  # a valid call would launch kernels: no GPU here
    rc = L.zero_shard_step(*ptrs, n, args["lr"], args["b1"], args["b2"], args["eps"], args["wd"], args["t"], args["sc"], args["clip"], None)
    rc2 = L.zero_shard_apply(*ptrs, n, r.choice([-1.0, float("inf"), 1.0]), args["lr"], args["b1"], args["b2"], args["eps"], args["wd"], args["t"], args["sc"], args["clip"], None)
    L.zero_last_error()
    bad += 1
L.zero_shard_stats(None, 10, ctypes.byref(out), None)
L.zero_shard_stats(None, 0, ctypes.byref(out), None)
L.zero_profile_enable(-1); L.zero_profile_enable(0)
L.zero_shard_validate.argtypes = [P, P, P, P, P, i64]
for _ in range(2000):
    ptrs = [p + r.choice([0, 1, 2, 8]) for p in G]
    L.zero_shard_validate(*ptrs, r.choice([-1, 0, 10, 1 << 41]))
    L.zero_last_error()
L.zero_lamb_plan_create.argtypes = [P, i32, i64, ctypes.POINTER(P)]
L.zero_lamb_plan_destroy.argtypes = [P]
L.zero_lamb_step.argtypes = [P, P, P, P, P, P, dbl, dbl, dbl, dbl, dbl, i64, dbl, dbl, dbl, dbl, P]
L.zero_lamb_moments.argtypes = [P, P, P, P, P, dbl, dbl, dbl, dbl, dbl, i64, dbl, dbl, P, P]
L.zero_lamb_apply.argtypes = [P, P, P, P, P, dbl, P, dbl, dbl, dbl, dbl, dbl, i64, dbl, dbl, P]
plan = P()
for _ in range(3000):
    k = r.randrange(0, 6)
    offs = sorted(r.randrange(-2, 50) for _ in range(k + 1))
    if r.random() < 0.5 and offs:
        offs[0] = 0
    arr = (ctypes.c_int64 * max(1, len(offs)))(*offs) if offs else None
    n = offs[-1] if offs and r.random() < 0.7 else r.randrange(-3, 60)
    L.zero_lamb_plan_create(arr if r.random() < 0.95 else None, k, n, ctypes.byref(plan) if r.random() < 0.9 else None)
    L.zero_last_error()
L.zero_lamb_plan_destroy(None)
for _ in range(500):
    L.zero_lamb_step(None, *G, 1e-3, 0.9, 0.999, 1e-6, 0.0, 1, 65536.0, 1.0, 0.0, float("inf"), None)
    L.zero_lamb_moments(None, *G[:4], 1.0, 0.9, 0.999, 1e-6, 0.0, 1, 65536.0, 1.0, G[4], None)
    L.zero_lamb_apply(None, *G[1:], 1.0, G[0], 1e-3, 0.9, 0.999, 1e-6, 0.0, 1, 0.0, float("inf"), None)
    L.zero_last_error()
L.zero_shard_stats_async.argtypes = [P, i64, P, P]
L.zero_shard_apply_async.argtypes = [P, P, P, P, P, i64, P, dbl, dbl, dbl, dbl, dbl, i64, dbl, dbl, P, P]
for _ in range(2000):
    L.zero_shard_stats_async(G[0] + r.choice([0, 1]), r.choice([-1, 10, 1 << 41]), r.choice([None, G[1] + 4, G[0]]), None)
    L.zero_shard_apply_async(*G, r.choice([-1, 10]), r.choice([None, 0x60000004]), 1e-3, 0.9, 0.999, 1e-8, 0.0,
                             r.choice([0, -1]), 65536.0, 1.0, r.choice([None, 0x70000002]), None)
    L.zero_last_error()
L.zero_shard_step_resident.argtypes = [P, P, P, P, P, i64, P, P]
for _ in range(2000):
    ptrs = [p + r.choice([0, 1]) for p in G]
    L.zero_shard_step_resident(*ptrs, r.choice([-1, 10, 1 << 41]), r.choice([None, 0x60000004, G[1] + 8]), None)
    L.zero_last_error()
print("driver done", bad, "rejected or empty calls")
