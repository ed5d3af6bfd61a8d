"""The C-ABI library loads and exports every entry point include/libecc.h
declares; host-only validation returns the documented status codes.  No GPU
call is made here."""
import os
import re

import numpy as np
import pytest

from paper_2203_17063_amd import capi as E

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    text = open(os.path.join(ROOT, "include", "libecc.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)        # drop comments
    names = re.findall(r"^[A-Za-z_][\w \*]*?\b(ecc_\w+)\s*\(", text, flags=re.M)
    return sorted(set(names))


def exported_symbols():
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only", E.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    return sorted(l.split()[-1] for l in out.splitlines() if " T ecc_" in l)


def test_library_loads_and_exports_header():
    E.lib()
    decl = header_functions()
    assert len(decl) >= 19
    exp = exported_symbols()
    assert decl == exp
    assert sorted(E.EXPORTED) == decl          # the binding covers every entry point
    assert E.ecc_abi_version() == 3


def header_constants():
    """Every integer constant the header defines: #define lines and the
    status enum."""
    text = open(os.path.join(ROOT, "include", "libecc.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    consts = {m.group(1): int(m.group(2), 0)
              for m in re.finditer(r"^#define\s+(ECC_\w+)\s+((?:0x)?[0-9a-fA-F]+)\s*$", text,
                                   flags=re.M)}
    consts.update({m.group(1): int(m.group(2))
                   for m in re.finditer(r"\b(ECC_(?:OK|ERR_\w+))\s*=\s*(\d+)", text)})
    return consts


def test_binding_constants_match_header():
    consts = header_constants()
    assert len(consts) >= 24
    for name, value in consts.items():
        assert getattr(E, name) == value, name


def test_status_strings():
    for code, name in E.STATUS_NAMES.items():
        assert E.lib().ecc_status_string(code).decode() == name


@pytest.mark.parametrize("P,counts,displs,S,expect", [
    (0, None, None, 0, E.ECC_ERR_ARG),                       # P < 1
    (3, None, None, -1, E.ECC_ERR_ARG),                      # negative staleness
    (3, None, None, 0, E.ECC_OK),                            # allreduce-only plan
    (3, [1, 2, 3], None, 0, E.ECC_ERR_ARG),                  # counts without displs
    (3, [1, -2, 3], [0, 1, 3], 0, E.ECC_ERR_ARG),            # negative count
    (3, [1, 2, 3], [0, -1, 3], 0, E.ECC_ERR_ARG),            # negative displacement
    (3, [2, 2, 2], [0, 1, 4], 0, E.ECC_ERR_OVERLAP),         # overlap
    (3, [2, 0, 2], [0, 1, 2], 0, E.ECC_OK),                  # empty block may sit anywhere
    (3, [2, 2, 2], [4, 0, 10], 0, E.ECC_OK),                 # unsorted with gaps
    (2, [1, 1], [0, 1 << 40], 0, E.ECC_ERR_RANGE),           # beyond 2^40
    (4, [5, 5, 5, 5], [0, 5, 10, 15], E.ECC_UNBOUNDED, E.ECC_OK),
])
def test_plan_validate(P, counts, displs, S, expect):
    assert E.ecc_plan_validate(P, counts, displs, S) == expect
    if expect != E.ECC_OK:
        assert E.ecc_last_error() != ""


def test_null_handles_are_rejected_without_device():
    L = E.lib()
    assert L.ecc_plan_reset(None) == E.ECC_ERR_ARG
    assert L.ecc_plan_destroy(None) == E.ECC_OK
    assert L.ecc_matrix_destroy(None) == E.ECC_OK
    assert L.ecc_partials_size(None) == 0
    assert L.ecc_allgatherv_assemble(None, None, None, None, None, None) == E.ECC_ERR_ARG
    assert L.ecc_residual(None, None, 1, 2, None, None) == E.ECC_ERR_ARG
    assert L.ecc_matrix_layout(None, None, None) == E.ECC_ERR_ARG


def test_product_path_does_not_touch_oracle():
    """The package and the HIP sources never import, link or call the oracle."""
    pkg = os.path.join(ROOT, "paper_2203_17063_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                for bad in ("import oracle", "from oracle", "liboracle", "orc_"):
                    assert bad not in text, (f, bad)


@pytest.mark.parametrize("P,m,slack,expect", [
    (0, 16, 0, E.ECC_ERR_ARG),                        # P < 1
    (3, 16, 0, E.ECC_ERR_ARG),                        # not a power of two
    (8192, 16, 0, E.ECC_ERR_ARG),                     # beyond 4096 processes
    (4, -1, 0, E.ECC_ERR_ARG),                        # negative length
    (4, 16, -1, E.ECC_ERR_ARG),                       # negative slack
    (4, (1 << 40) // 8 + 1, 0, E.ECC_ERR_RANGE),      # slots beyond 2^40 elements
    (1, 0x7fffffff * 64 + 1, 0, E.ECC_ERR_RANGE),     # beyond the grid's 64 elements per workgroup
])
def test_hypercube_create_checks_without_device(P, m, slack, expect):
    """Argument and range checks return before any device call."""
    with pytest.raises(E.EccError) as err:
        E.ecc_hypercube_create(P, m, slack)
    assert err.value.status == expect
