"""Pins of the oracle's model-state accounting against the numbers ZeRO prints.

Sec. 3.1 (16 bytes per parameter for mixed-precision Adam, K = 12), Sec. 5.1-5.3
(the three stages), Table 1 (Sec. 5.2), Table 2 (Sec. 7.1) and the prose
examples.  Nothing here retypes the formulas: each check compares the oracle
with a value printed in the paper, to within one unit of its last printed digit.
"""
import os
import re

import pytest

import oracle

GOLD = os.path.join(os.path.dirname(__file__), "golden")
STAGES = {"dp": oracle.STAGE_DP, "os": oracle.STAGE_OS, "os_g": oracle.STAGE_OS_G, "os_g_p": oracle.STAGE_OS_G_P}


def _rows(name):
    with open(os.path.join(GOLD, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                yield line.split()


def _last_digit_unit(s: str) -> float:
    return 10.0 ** -len(s.split(".")[1]) if "." in s else 1.0


def _table1_cases():
    models = [7.5e9, 128e9, 1e12]
    stages = [oracle.STAGE_OS, oracle.STAGE_OS_G, oracle.STAGE_OS_G_P]
    for row in _rows("table1_memory.txt"):
        nd = int(row[0])
        for j, printed in enumerate(row[1:]):
            yield nd, models[j // 3], stages[j % 3], printed


@pytest.mark.parametrize("nd,psi,stage,printed", list(_table1_cases()))
def test_table1_cell(nd, psi, stage, printed):
    gb = oracle.model_state_bytes(psi, nd, stage) / 1e9
    assert abs(gb - float(printed)) < _last_digit_unit(printed), (nd, psi, stage, gb, printed)


def test_table1_has_all_cells():
    assert len(list(_table1_cases())) == 54  # 6 rows x 9 columns


def test_baseline_dp_is_independent_of_nd():
    # Sec. 5.4: without ZeRO the per-device memory is Table 1's first row for any N_d.
    for nd in (1, 4, 64, 1024):
        assert oracle.model_state_bytes(7.5e9, nd, oracle.STAGE_DP) / 1e9 == pytest.approx(120.0)


def _parse_params(s: str) -> float:
    m = re.fullmatch(r"([0-9.]+)([BT])", s)
    return float(m.group(1)) * (1e9 if m.group(2) == "B" else 1e12), m.group(1)


def test_table2_max_theoretical_model_size():
    device_bytes = 32e9  # 32 GB V100, Sec. 10 / Table 1 caption
    rows = list(_rows("table2_max_model_size.txt"))
    stages = [oracle.STAGE_DP, oracle.STAGE_OS, oracle.STAGE_OS_G, oracle.STAGE_OS_G_P]
    first = {}
    for row in rows:
        mp, gpus = int(row[0]), int(row[1])
        nd = gpus // mp
        assert nd == 64
        for stage, cell in zip(stages, row[2:]):
            printed, digits = _parse_params(cell)
            per_param = oracle.model_state_bytes(1.0, nd, stage)
            exact = mp * device_bytes / per_param
            unit = _last_digit_unit(digits) * (1e9 if cell.endswith("B") else 1e12)
            if mp == 1:
                first[stage] = printed
                assert abs(exact - printed) <= unit / 2 + 1.0, (cell, exact)
            elif cell.endswith("T"):
                # Cells quoted in trillions (0.5T for 512B, 2T for 2048B) are coarse.
                assert abs(exact - printed) < unit, (mp, cell, exact)
            else:
                # Later rows scale the printed single-MP value, not the exact one.
                assert printed == pytest.approx(mp * first[stage], rel=1e-12), (mp, cell)
                assert abs(exact - printed) <= mp * 0.05e9 + 1.0, (mp, cell, exact)


def test_prose_examples():
    for label, psi, nd, stage, printed, *_cite in _rows("prose_memory.txt"):
        gb = oracle.model_state_bytes(float(psi), float(nd), STAGES[stage]) / 1e9
        assert abs(gb - float(printed)) < _last_digit_unit(printed), (label, gb, printed)


def test_sec54_largest_models_at_nd64():
    # Sec. 5.4: at N_d = 64 a 32 GB device holds up to 7.5B (P_os), 14B (P_os+g) and 128B
    # (P_os+g+p) parameters; one more "step" of model size in each case does not fit.
    cap = 32e9
    for stage, fits, too_big in ((oracle.STAGE_OS, 7.5e9, 8e9), (oracle.STAGE_OS_G, 14e9, 15e9),
                                 (oracle.STAGE_OS_G_P, 128e9, 129e9)):
        assert oracle.model_state_bytes(fits, 64, stage) <= cap
        assert oracle.model_state_bytes(too_big, 64, stage) > cap


def test_reductions_quoted_in_sec1():
    # Sec. 1: P_os gives ~4x, P_os+g ~8x, P_os+g+p N_d-x reduction for large N_d.
    psi, nd = 1e12, 1e9
    base = oracle.model_state_bytes(psi, nd, oracle.STAGE_DP)
    assert base / oracle.model_state_bytes(psi, nd, oracle.STAGE_OS) == pytest.approx(4.0, rel=1e-6)
    assert base / oracle.model_state_bytes(psi, nd, oracle.STAGE_OS_G) == pytest.approx(8.0, rel=1e-6)
    assert base / oracle.model_state_bytes(psi, 64, oracle.STAGE_OS_G_P) == pytest.approx(64.0)


def test_bad_arguments():
    with pytest.raises(ValueError):
        oracle.model_state_bytes(1e9, 0, oracle.STAGE_OS)
    with pytest.raises(ValueError):
        oracle.model_state_bytes(1e9, 4, 7)


def test_4psi_plus_12psi_over_nd_is_the_pos_stage():
    # 2*Psi + 2*Psi + 12*Psi/N_d is the P_os memory (Sec. 5.1: 31.4 GB at 7.5B, N_d = 64);
    # P_os+g is 2*Psi + 14*Psi/N_d (Sec. 5.2: 16.6 GB).  Only P_os matches the first form.
    psi, nd = 7.5e9, 64
    form = 2 * psi + 2 * psi + 12 * psi / nd
    assert oracle.model_state_bytes(psi, nd, oracle.STAGE_OS) == pytest.approx(form, rel=1e-15)
    assert oracle.model_state_bytes(psi, nd, oracle.STAGE_OS_G) / 1e9 == pytest.approx(16.640625)
    assert oracle.model_state_bytes(psi, nd, oracle.STAGE_OS_G) != pytest.approx(form, rel=1e-3)
