"""The C-ABI library on the CPU: it loads, exports every symbol the header
declares, and its host-only entry points (layout, accounting, loss scaler,
argument validation) agree with the oracle.  No GPU work is launched here:
every zero_shard_step call below is rejected (or is a no-op) before any HIP
call is made."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "zero_shard.h")


@pytest.fixture(scope="module")
def zb():
    from paper_1910_02054_amd import build as b
    if b.is_stale():
        b.build()
    from paper_1910_02054_amd import binding
    return binding


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\**(zero_\w+)\s*\(", text, flags=re.M)))


def test_header_declares_the_boundary():
    names = _declared()
    for required in ("zero_partition_layout", "zero_shard_step", "zero_last_error"):
        assert required in names


def test_every_declared_symbol_is_exported(zb):
    names = _declared()
    lib = zb.raw_library()
    for name in names:
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", zb.LIB_PATH], stdout=subprocess.PIPE, check=True).stdout.decode()
    exported = set(re.findall(r"\bT (zero_\w+)", out))
    assert set(names) <= exported
    assert set(zb.EXPORTS) == set(names)


def test_layout_bitwise_vs_oracle(zb):
    for psi in list(range(0, 40)) + [4_194_304, 4_194_305, 1_500_000_000, 13_000_000_000, 6_250_000_000,
                                     62_500_000_000, (1 << 62)]:
        for nd in (1, 2, 3, 4, 7, 16, 25, 64, 1024):
            for rank in sorted({0, 1, nd // 2, nd - 1}):
                if rank >= nd:
                    continue
                lay = zb.zero_partition_layout(psi, nd, rank)
                assert (lay.shard_numel, lay.offset, lay.valid_numel, lay.padded_total) == oracle.layout(psi, nd, rank)


@pytest.mark.parametrize("psi,nd,rank", [(-1, 4, 0), (10, 0, 0), (10, 4, 4), (10, 4, -1), ((1 << 62) + 1, 2, 0)])
def test_layout_rejects(zb, psi, nd, rank):
    with pytest.raises(zb.ZeroError) as e:
        zb.zero_partition_layout(psi, nd, rank)
    assert e.value.code == zb.ZERO_EINVAL


def test_model_state_bytes_vs_oracle(zb):
    for psi in (7.5e9, 128e9, 1e12, 1.5e9, 1.0):
        for nd in (1, 4, 16, 64, 256, 1024):
            for stage in range(4):
                got = zb.zero_model_state_bytes(psi, nd, stage)
                assert got == pytest.approx(oracle.model_state_bytes(psi, nd, stage), rel=1e-15)
    with pytest.raises(zb.ZeroError):
        zb.zero_model_state_bytes(1e9, 4, 9)


def test_scaler_matches_oracle(zb):
    rng = np.random.default_rng(0)
    for window in (0, 1, 3, 1000):
        a = zb.Scaler(2.0 ** 16, window=window, min_scale=1.0)
        b = oracle.Scaler(2.0 ** 16, window=window, min_scale=1.0)
        for skipped in rng.integers(0, 2, size=60):
            assert a.t_next == b.t_next
            a.update(int(skipped))
            b.update(int(skipped))
            assert a.scale == b.scale.value and a.state.applied == b.applied.value and a.state.good == b.good.value


def _step_raw(zb, ptrs, n, **kw):
    args = dict(lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.0, step=1, scale=65536.0, clip=1.0)
    args.update(kw)
    lib = zb.raw_library()
    return lib.zero_shard_step(*ptrs, n, args["lr"], args["beta1"], args["beta2"], args["eps"], args["wd"],
                               args["step"], args["scale"], args["clip"], None)


# Fake, never-dereferenced addresses: validation must reject these calls before any HIP call.
GOOD = [0x10000000, 0x20000000, 0x30000000, 0x40000000, 0x50000000]


@pytest.mark.parametrize("kw,ptrs,n", [
    (dict(), GOOD, -1),
    (dict(), [0] + GOOD[1:], 10),
    (dict(), [GOOD[0] + 1] + GOOD[1:], 10),             # fp16 misaligned to 1 byte
    (dict(), GOOD[:1] + [GOOD[1] + 2] + GOOD[2:], 10),  # fp32 misaligned to 2 bytes
    (dict(), [GOOD[0], GOOD[1], GOOD[1] + 8] + GOOD[3:], 10),  # master and m overlap
    (dict(), [GOOD[0], GOOD[1], GOOD[2], GOOD[3], GOOD[0] + 4], 10),  # p16 overlaps grads
    (dict(beta1=1.0), GOOD, 10),
    (dict(beta2=-0.1), GOOD, 10),
    (dict(step=0), GOOD, 10),
    (dict(scale=0.0), GOOD, 10),
    (dict(scale=float("inf")), GOOD, 10),
    (dict(lr=float("nan")), GOOD, 10),
    (dict(lr=-1.0), GOOD, 10),
    (dict(eps=-1e-8), GOOD, 10),
    (dict(clip=float("nan")), GOOD, 10),
    (dict(wd=float("inf")), GOOD, 10),
    (dict(), GOOD, (1 << 40) + 1),
])
def test_step_rejects_invalid_arguments(zb, kw, ptrs, n):
    assert _step_raw(zb, ptrs, n, **kw) == zb.ZERO_EINVAL
    assert zb.zero_last_error() != ""


def test_step_with_zero_elements_is_a_noop(zb):
    assert _step_raw(zb, [0, 0, 0, 0, 0], 0) == zb.ZERO_OK
    st = zb.zero_shard_last_step_stats()
    assert st.n == 0 and st.skipped == 0


def _apply_raw(zb, ptrs, n, gsum, **kw):
    args = dict(lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.0, step=1, scale=65536.0, clip=1.0)
    args.update(kw)
    return zb.raw_library().zero_shard_apply(*ptrs, n, gsum, args["lr"], args["beta1"], args["beta2"], args["eps"],
                                             args["wd"], args["step"], args["scale"], args["clip"], None)


@pytest.mark.parametrize("kw,ptrs,n,gsum", [
    (dict(), GOOD, -1, 1.0),
    (dict(), [0] + GOOD[1:], 10, 1.0),
    (dict(), [GOOD[0], GOOD[1], GOOD[1] + 8] + GOOD[3:], 10, 1.0),
    (dict(step=0), GOOD, 10, 1.0),
    (dict(scale=-2.0), GOOD, 10, 1.0),
    (dict(), GOOD, 10, -1.0),
])
def test_apply_rejects_invalid_arguments(zb, kw, ptrs, n, gsum):
    assert _apply_raw(zb, ptrs, n, gsum, **kw) == zb.ZERO_EINVAL


def test_apply_overflow_and_empty_need_no_gpu(zb):
    # a non-finite global sum is the skip decision itself: nothing is launched
    assert _apply_raw(zb, GOOD, 10, float("inf")) == zb.ZERO_SKIPPED
    assert _apply_raw(zb, GOOD, 10, float("nan")) == zb.ZERO_SKIPPED
    assert _apply_raw(zb, [0, 0, 0, 0, 0], 0, 1.0) == zb.ZERO_OK


def test_stats_rejects_invalid_arguments(zb):
    lib = zb.raw_library()
    out = ctypes.c_double(7.0)
    assert lib.zero_shard_stats(None, 10, ctypes.byref(out), None) == zb.ZERO_EINVAL
    assert lib.zero_shard_stats(GOOD[0] + 1, 10, ctypes.byref(out), None) == zb.ZERO_EINVAL
    assert lib.zero_shard_stats(GOOD[0], -3, ctypes.byref(out), None) == zb.ZERO_EINVAL
    assert lib.zero_shard_stats(GOOD[0], 10, None, None) == zb.ZERO_EINVAL
    assert lib.zero_shard_stats(None, 0, ctypes.byref(out), None) == zb.ZERO_OK and out.value == 0.0


def test_profile_enable_rejects_negative(zb):
    assert zb.raw_library().zero_profile_enable(-1) == zb.ZERO_EINVAL
    assert zb.raw_library().zero_profile_enable(0) == zb.ZERO_OK


def test_validate_rejects_without_launching(zb):
    lib = zb.raw_library()
    lib.zero_shard_validate.argtypes = [ctypes.c_void_p] * 5 + [ctypes.c_int64]
    assert lib.zero_shard_validate(*GOOD, -1) == zb.ZERO_EINVAL
    assert lib.zero_shard_validate(GOOD[0] + 1, *GOOD[1:], 10) == zb.ZERO_EINVAL
    assert lib.zero_shard_validate(GOOD[0], GOOD[1], GOOD[1] + 8, *GOOD[3:], 10) == zb.ZERO_EINVAL  # no GPU memory
    assert lib.zero_shard_validate(0, *GOOD[1:], 10) == zb.ZERO_EINVAL
    assert lib.zero_shard_validate(0, 0, 0, 0, 0, 0) == zb.ZERO_OK
    # plausible addresses that are not GPU allocations (no GPU here at all): rejected
    assert lib.zero_shard_validate(*GOOD, 10) == zb.ZERO_EINVAL
    assert "GPU-accessible" in zb.zero_last_error()


def test_probe_copy_rejects_without_launching(zb):
    lib = zb.raw_library()
    lib.zero_probe_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
    assert lib.zero_probe_copy(GOOD[1], GOOD[2], 24, None) == zb.ZERO_EINVAL        # not a multiple of 16
    assert lib.zero_probe_copy(GOOD[1] + 4, GOOD[2], 32, None) == zb.ZERO_EINVAL    # misaligned
    assert lib.zero_probe_copy(GOOD[1], GOOD[1] + 16, 64, None) == zb.ZERO_EINVAL   # overlap
    assert lib.zero_probe_copy(GOOD[1], GOOD[2], 0, None) == zb.ZERO_OK
    # addresses outside any GPU allocation are refused before a launch
    assert lib.zero_probe_copy(GOOD[1], GOOD[2], 64, None) == zb.ZERO_EINVAL
    assert "GPU-accessible" in zb.zero_last_error()


def test_probe_adam_mix_rejects_without_launching(zb):
    lib = zb.raw_library()
    assert lib.zero_probe_adam_mix(*GOOD, -1, None) == zb.ZERO_EINVAL
    assert lib.zero_probe_adam_mix(0, *GOOD[1:], 10, None) == zb.ZERO_EINVAL                     # NULL
    assert lib.zero_probe_adam_mix(GOOD[0], GOOD[1] + 4, *GOOD[2:], 10, None) == zb.ZERO_EINVAL  # fp32 not 16-B
    assert "16-byte" in zb.zero_last_error()
    assert lib.zero_probe_adam_mix(GOOD[0] + 2, *GOOD[1:], 10, None) == zb.ZERO_EINVAL           # fp16 not 8-B
    assert "8-byte" in zb.zero_last_error()
    assert lib.zero_probe_adam_mix(GOOD[0], GOOD[1], GOOD[1] + 16, *GOOD[3:], 10, None) == zb.ZERO_EINVAL  # overlap
    assert lib.zero_probe_adam_mix(0, 0, 0, 0, 0, 0, None) == zb.ZERO_OK
    # addresses outside any GPU allocation are refused before a launch
    assert lib.zero_probe_adam_mix(*GOOD, 64, None) == zb.ZERO_EINVAL
    assert "GPU-accessible" in zb.zero_last_error()


def test_scaled_step_rejects_and_leaves_the_scaler_alone(zb):
    # the scaler-driven step: argument errors come back before any launch and never touch the
    # scaler; an empty shard is an applied step (t and the good count advance)
    lib = zb.raw_library()
    sc = zb.Scaler(2.0 ** 16, window=3)
    before = lambda: (sc.state.scale, sc.state.applied, sc.state.good)
    args = zb.StepArgs(*GOOD, 10, 1e-4, 0.9, 0.999, 1e-8, 0.0, 1.0, None)
    a = ctypes.addressof(args)
    assert lib.zero_shard_step_scaled(None, sc.addr) == zb.ZERO_EINVAL
    assert lib.zero_shard_step_scaled(a, None) == zb.ZERO_EINVAL
    for field, bad in (("beta1", 1.0), ("lr", float("nan")), ("n", -1), ("grad16", GOOD[0] + 1)):
        b = zb.StepArgs.from_buffer_copy(args)
        setattr(b, field, bad)
        s0 = before()
        assert lib.zero_shard_step_scaled(ctypes.addressof(b), sc.addr) == zb.ZERO_EINVAL, field
        assert before() == s0
    sc.state.applied = -1
    assert lib.zero_shard_step_scaled(a, sc.addr) == zb.ZERO_EINVAL
    sc.state.applied = 2 ** 63 - 1
    assert lib.zero_shard_step_scaled(a, sc.addr) == zb.ZERO_EINVAL
    assert sc.state.applied == 2 ** 63 - 1
    sc.state.applied = 0
    sc.state.scale = 0.0  # an invalid loss scale is the step's own check
    assert lib.zero_shard_step_scaled(a, sc.addr) == zb.ZERO_EINVAL and sc.state.applied == 0
    sc.state.scale = 2.0 ** 16
    empty = zb.StepArgs(0, 0, 0, 0, 0, 0, 1e-4, 0.9, 0.999, 1e-8, 0.0, 1.0, None)
    for k in range(3):
        assert lib.zero_shard_step_scaled(ctypes.addressof(empty), sc.addr) == zb.ZERO_OK
    assert sc.state.applied == 3 and sc.state.good == 0 and sc.state.scale == 2.0 ** 17  # grew at window 3


def test_lamb_plan_rejects_bad_tables_without_a_gpu(zb):
    lib = zb.raw_library()
    out = ctypes.c_void_p()

    def create(offs, n_seg, n, with_out=True):
        arr = (ctypes.c_int64 * len(offs))(*offs) if offs is not None else None
        return lib.zero_lamb_plan_create(arr, n_seg, n, ctypes.byref(out) if with_out else None)

    assert create([0, 5, 5, 10], 3, 10) == zb.ZERO_EINVAL      # not strictly rising
    assert create([0, 6, 4, 10], 3, 10) == zb.ZERO_EINVAL
    assert create([0, 5, 9], 2, 10) == zb.ZERO_EINVAL          # does not end at n
    assert create([1, 5, 10], 2, 10) == zb.ZERO_EINVAL         # does not start at 0
    assert create([0], 0, 10) == zb.ZERO_EINVAL                # n > 0 needs layers
    assert create([0, 1], 1, 0) == zb.ZERO_EINVAL              # n = 0 needs none
    assert create([0, 10], 1, -1) == zb.ZERO_EINVAL
    assert create([0, (1 << 40) + 1], 1, (1 << 40) + 1) == zb.ZERO_EINVAL
    assert create(None, 2, 10) == zb.ZERO_EINVAL
    assert create([0, 10], 1, 10, with_out=False) == zb.ZERO_EINVAL
    assert "seg_off" in zb.zero_last_error() or "out" in zb.zero_last_error()
    # a valid table gets as far as asking for the device
    assert create([0, 10], 1, 10) in (zb.ZERO_OK, zb.ZERO_EHIP)
    if out.value:
        assert lib.zero_lamb_plan_destroy(out) == zb.ZERO_OK
    assert lib.zero_lamb_plan_destroy(None) == zb.ZERO_OK


def test_lamb_calls_reject_a_null_plan(zb):
    lib = zb.raw_library()
    G = [0x10000000, 0x20000000, 0x30000000, 0x40000000, 0x50000000]
    assert lib.zero_lamb_step(None, *G, 1e-3, 0.9, 0.999, 1e-6, 0.0, 1, 65536.0, 1.0, 0.0, float("inf"),
                              None) == zb.ZERO_EINVAL
    assert lib.zero_lamb_moments(None, *G[:4], 1.0, 0.9, 0.999, 1e-6, 0.0, 1, 65536.0, 1.0, G[4],
                                 None) == zb.ZERO_EINVAL
    assert lib.zero_lamb_apply(None, *G[1:], 1.0, G[0], 1e-3, 0.9, 0.999, 1e-6, 0.0, 1, 0.0, float("inf"),
                               None) == zb.ZERO_EINVAL
    assert "NULL plan" in zb.zero_last_error()
    p = zb.LambProfile()
    assert lib.zero_lamb_profile_read(ctypes.byref(p)) == zb.ZERO_OK and p.steps == 0


def test_async_split_rejects_without_a_gpu(zb):
    lib = zb.raw_library()
    G = [0x10000000, 0x20000000, 0x30000000, 0x40000000, 0x50000000]
    assert lib.zero_shard_stats_async(G[0], 10, None, None) == zb.ZERO_EINVAL          # NULL sum
    assert lib.zero_shard_stats_async(G[0], 10, G[1] + 4, None) == zb.ZERO_EINVAL      # misaligned sum
    assert lib.zero_shard_stats_async(G[0] + 1, 10, G[1], None) == zb.ZERO_EINVAL      # misaligned grad
    assert lib.zero_shard_stats_async(G[0], -1, G[1], None) == zb.ZERO_EINVAL
    assert lib.zero_shard_stats_async(G[0], 10, G[0] + 8, None) == zb.ZERO_EINVAL      # sum inside grad16
    hp = (1e-3, 0.9, 0.999, 1e-8, 0.0, 1, 65536.0, 1.0)
    assert lib.zero_shard_apply_async(*G, 10, None, *hp, None, None) == zb.ZERO_EINVAL
    assert lib.zero_shard_apply_async(*G, 10, 0x60000000 + 4, *hp, None, None) == zb.ZERO_EINVAL
    assert lib.zero_shard_apply_async(*G, 10, 0x60000000, *hp, 0x70000000 + 2, None) == zb.ZERO_EINVAL
    assert lib.zero_shard_apply_async(*G, 10, G[1] + 8, *hp, None, None) == zb.ZERO_EINVAL  # sum inside master
    assert lib.zero_shard_apply_async(*G, 10, 0x60000000, 1e-3, 0.9, 0.999, 1e-8, 0.0, 0, 65536.0, 1.0, None,
                                      None) == zb.ZERO_EINVAL                                 # t = 0


def test_header_is_plain_c_and_links_from_c(zb, tmp_path):
    # The boundary is a C ABI: the header compiles as strict C99, a C program links every
    # declared entry point against the library and runs the host-only ones.
    import shutil
    if shutil.which("gcc") is None:
        pytest.skip("needs gcc")
    names = _declared()
    src = ["#include \"zero_shard.h\"", "#include <stdio.h>", "int main(void) {",
           "    typedef void (*fn_t)(void);",
           "    const fn_t f[] = {" + ", ".join("(fn_t)%s" % n for n in names) + "};",
           "    zero_layout_t lay; zero_scaler_t sc; double b = 0.0;",
           "    int rc = zero_partition_layout(62500000000LL, 1024, 1023, &lay);",
           "    rc |= zero_model_state_bytes(7.5e9, 64, ZERO_STAGE_OS_G, 12.0, &b);",
           "    rc |= zero_scaler_init(&sc, 65536.0, 1000, 1.0) | zero_scaler_update(&sc, 1);",
           "    if (zero_partition_layout(10, 0, 0, &lay) != ZERO_EINVAL || zero_last_error()[0] == 0) return 9;",
           "    zero_partition_layout(62500000000LL, 1024, 1023, &lay);",
           "    printf(\"%d %lld %lld %lld %lld %.1f %.1f %d\\n\", rc, (long long)lay.shard_numel, (long long)lay.offset,",
           "           (long long)lay.valid_numel, (long long)lay.padded_total, b, sc.scale, (int)(sizeof f / sizeof f[0]));",
           "    return rc;", "}"]
    c = tmp_path / "abi.c"
    c.write_text("\n".join(src) + "\n")
    exe = tmp_path / "abi"
    libdir = os.path.dirname(zb.LIB_PATH)
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic",
                    "-I", os.path.join(ROOT, "include"), str(c), "-L", libdir, "-lzeroshard",
                    "-Wl,-rpath," + libdir, "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], stdout=subprocess.PIPE, check=True).stdout.decode().split()
    S, off, valid, padded = oracle.layout(62_500_000_000, 1024, 1023)
    assert out[:5] == ["0", str(S), str(off), str(valid), str(padded)]
    assert float(out[5]) == pytest.approx(oracle.model_state_bytes(7.5e9, 64, oracle.STAGE_OS_G))
    assert float(out[6]) == 32768.0 and int(out[7]) == len(names)


def test_binding_structs_match_the_c_layout(zb, tmp_path):
    # every struct the binding mirrors has the header's size and field offsets
    import shutil
    if shutil.which("gcc") is None:
        pytest.skip("needs gcc")
    pairs = [("zero_layout_t", zb.Layout), ("zero_step_stats_t", zb.StepStats), ("zero_scaler_t", zb.ScalerState),
             ("zero_profile_t", zb.Profile), ("zero_lamb_profile_t", zb.LambProfile),
             ("zero_resident_state_t", zb.ResidentState), ("zero_step_args_t", zb.StepArgs)]
    text = open(HEADER).read()
    lines = ["#include \"zero_shard.h\"", "#include <stdio.h>", "#include <stddef.h>", "int main(void) {"]
    expect = []
    for cname, py in pairs:
        assert cname in text, cname
        lines.append('    printf("%%zu\\n", sizeof(%s));' % cname)
        expect.append(ctypes.sizeof(py))
        for fname, _ in py._fields_:
            lines.append('    printf("%%zu\\n", offsetof(%s, %s));' % (cname, fname))
            expect.append(getattr(py, fname).offset)
    lines += ["    return 0;", "}"]
    c = tmp_path / "layout.c"
    c.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"), str(c), "-o",
                    str(exe)], check=True)
    got = [int(x) for x in subprocess.run([str(exe)], stdout=subprocess.PIPE, check=True).stdout.split()]
    assert got == expect


def test_resident_step_rejects_without_a_gpu(zb):
    lib = zb.raw_library()
    G = [0x10000000, 0x20000000, 0x30000000, 0x40000000, 0x50000000]
    assert lib.zero_shard_step_resident(*G, 10, None, None) == zb.ZERO_EINVAL           # NULL state
    assert lib.zero_shard_step_resident(*G, 10, 0x60000004, None) == zb.ZERO_EINVAL     # misaligned state
    assert lib.zero_shard_step_resident(*G, 10, G[1] + 8, None) == zb.ZERO_EINVAL       # state inside master
    assert lib.zero_shard_step_resident(G[0] + 1, *G[1:], 10, 0x60000000, None) == zb.ZERO_EINVAL
    assert lib.zero_shard_step_resident(*G, -1, 0x60000000, None) == zb.ZERO_EINVAL
    assert "state" in zb.zero_last_error() or "n=" in zb.zero_last_error()


# ---------------------------------------------------------------------------
# The boundary's helper calls as the scope table declares them
# ---------------------------------------------------------------------------

def _table1_cells():
    gold = os.path.join(ROOT, "tests", "golden", "table1_memory.txt")
    models = [7.5e9, 128e9, 1e12]
    stages = [zb_stage for zb_stage in (1, 2, 3)]
    with open(gold) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                row = line.split()
                for j, printed in enumerate(row[1:]):
                    yield int(row[0]), models[j // 3], stages[j % 3], printed


def test_memory_bytes_on_every_table1_cell(zb):
    # Sec. 5.2, Table 1 (K = 12): each printed cell within one unit of its last digit, and
    # the value equal to the oracle's accounting
    cells = list(_table1_cells())
    assert len(cells) == 54
    for nd, psi, stage, printed in cells:
        got = zb.zero_memory_bytes(psi, nd, stage, 12)
        unit = 10.0 ** -len(printed.split(".")[1]) if "." in printed else 1.0
        assert abs(got / 1e9 - float(printed)) < unit, (nd, psi, stage, got, printed)
        assert got == oracle.model_state_bytes(psi, nd, stage)
    assert zb.zero_memory_bytes(7.5e9, 64, zb.ZERO_STAGE_DP, 12) == oracle.model_state_bytes(7.5e9, 64, 0)


def test_memory_bytes_rejects(zb):
    lib = zb.raw_library()
    out = ctypes.c_double()
    assert lib.zero_memory_bytes(1e9, 0, 1, 12, ctypes.byref(out)) == zb.ZERO_EINVAL
    assert lib.zero_memory_bytes(1e9, 4, 1, -1, ctypes.byref(out)) == zb.ZERO_EINVAL
    assert lib.zero_memory_bytes(-1.0, 4, 1, 12, ctypes.byref(out)) == zb.ZERO_EINVAL
    assert lib.zero_memory_bytes(float("nan"), 4, 1, 12, ctypes.byref(out)) == zb.ZERO_EINVAL
    assert lib.zero_memory_bytes(1e9, 4, 7, 12, ctypes.byref(out)) == zb.ZERO_EINVAL
    assert lib.zero_memory_bytes(1e9, 4, 1, 12, None) == zb.ZERO_EINVAL


def test_last_stats_three_pointer_form(zb):
    lib = zb.raw_library()
    # an empty step (no GPU work) sets the thread's statistics: norm 0, mult 1/scale, no overflow
    assert _step_raw(zb, [0, 0, 0, 0, 0], 0, scale=1024.0) == zb.ZERO_OK
    norm, mult, ovf = zb.zero_shard_last_stats()
    st = zb.zero_shard_last_step_stats()
    assert (norm, mult, ovf) == (0.0, np.float32(1.0 / 1024.0), 0)
    assert (norm, mult, ovf) == (st.norm, st.mult, st.overflow)
    only = ctypes.c_int(-1)
    assert lib.zero_shard_last_stats(None, None, ctypes.byref(only)) == zb.ZERO_OK and only.value == 0
    assert lib.zero_shard_last_stats(None, None, None) == zb.ZERO_EINVAL


def _exact_bias_correction_f32(beta, tmax):
    """fp32(1 - RN64(beta^t)) for t = 1..tmax from the exact power: beta is a dyadic
    rational, so beta^t is carried in 400-bit fixed point (truncation error below
    t * 2^-400) and rounded to the nearest double with the remainder as sticky bits
    (below 2^-60 the difference 1 - beta^t rounds to 1 whatever the power's bits)."""
    from fractions import Fraction
    prec = 400
    b = Fraction(beta)
    B = (b.numerator << prec) // b.denominator
    assert Fraction(B, 1 << prec) == b
    P = 1 << prec
    out = np.empty(tmax, np.float32)
    for t in range(1, tmax + 1):
        P = (P * B) >> prec
        if P.bit_length() <= prec - 60:   # beta^t < 2^-60: 1 - beta^t rounds to 1 in double
            out[t - 1] = np.float32(1.0)
            continue
        drop = P.bit_length() - 53
        mant, rem = P >> drop, P & ((1 << drop) - 1)
        half = 1 << (drop - 1)
        if rem > half or (rem == half and (mant & 1)):
            mant += 1
        out[t - 1] = np.float32(1.0 - float(np.ldexp(float(mant), drop - prec)))
    return out


@pytest.mark.parametrize("beta1,beta2", [(0.9, 0.98), (0.9, 0.999), (0.9, 0.9999), (0.95, 0.98), (0.95, 0.999),
                                         (0.95, 0.9999)])
def test_bias_corrections_match_the_exact_power_and_the_oracle(zb, beta1, beta2):
    # Adam's bias corrections 1 - beta^t (Kingma & Ba, cited in Sec. 3.1): the library's one
    # definition (the host calls and the resident kernel share it) against the exact power,
    # and against the oracle's C-library pow, for t = 1..20000
    tmax = 20000
    ex1, ex2 = _exact_bias_correction_f32(beta1, tmax), _exact_bias_correction_f32(beta2, tmax)
    lib = zb.raw_library()
    a, b = ctypes.c_float(), ctypes.c_float()
    for t in range(1, tmax + 1):
        assert lib.zero_bias_corrections(beta1, beta2, t, ctypes.byref(a), ctypes.byref(b)) == zb.ZERO_OK
        h = oracle.hyper(1e-4, beta1, beta2, 1e-8, 0.0, t)
        assert np.float32(a.value) == ex1[t - 1] == np.float32(h.bc1), (t, a.value, ex1[t - 1], h.bc1)
        assert np.float32(b.value) == ex2[t - 1] == np.float32(h.bc2), (t, b.value, ex2[t - 1], h.bc2)


def test_bias_corrections_rejects(zb):
    lib = zb.raw_library()
    a, b = ctypes.c_float(), ctypes.c_float()
    assert lib.zero_bias_corrections(1.0, 0.9, 1, ctypes.byref(a), ctypes.byref(b)) == zb.ZERO_EINVAL
    assert lib.zero_bias_corrections(0.9, -0.1, 1, ctypes.byref(a), ctypes.byref(b)) == zb.ZERO_EINVAL
    assert lib.zero_bias_corrections(0.9, 0.99, 0, ctypes.byref(a), ctypes.byref(b)) == zb.ZERO_EINVAL
    assert lib.zero_bias_corrections(0.9, 0.99, 1, None, ctypes.byref(b)) == zb.ZERO_EINVAL
    # beta = 0: 1 - 0^t = 1 at every t
    assert zb.zero_bias_corrections(0.0, 0.0, 7) == (1.0, 1.0)


def test_resident_state_init_checks_the_record(zb):
    ok = dict(lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0, clip=1.0, loss_scale=65536.0,
              min_scale=1.0, window=1000, t=1)
    st = zb.resident_state_record(**ok)
    assert (st.t, st.good, st.steps, st.skipped, st.loss_scale, st.window) == (1, 0, 0, 0, 65536.0, 1000)
    for bad in (dict(t=0), dict(beta1=1.0), dict(beta2=-0.5), dict(loss_scale=0.0), dict(loss_scale=float("inf")),
                dict(min_scale=0.0), dict(min_scale=float("nan")), dict(lr=-1.0), dict(eps=float("nan")),
                dict(clip=float("nan")), dict(weight_decay=float("inf"))):
        with pytest.raises(zb.ZeroError) as e:
            zb.resident_state_record(**dict(ok, **bad))
        assert e.value.code == zb.ZERO_EINVAL, bad
    assert zb.raw_library().zero_resident_state_init(None, 1e-4, 0.9, 0.999, 1e-8, 0.0, 1.0, 65536.0, 1.0, 1000,
                                                     1) == zb.ZERO_EINVAL


def test_workspace_count_without_a_gpu(zb):
    assert zb.zero_workspace_count() == (0, 0)
    assert zb.raw_library().zero_workspace_count(None, None) == zb.ZERO_EINVAL
    assert zb.raw_library().zero_resident_release(None) == zb.ZERO_EINVAL
