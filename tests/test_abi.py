"""The C-ABI library loads and exports every function include/epic.h declares
(CPU only: no device calls)."""
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared():
    src = open(os.path.join(ROOT, "include", "epic.h")).read()
    return sorted(set(re.findall(r"^\s*(?:epic_status|void|size_t|int32_t|const char\*)\s+(epic_\w+)\(", src, re.M)))


def test_header_declares_the_binding_functions():
    from paper_2606_00722_amd import epic

    assert declared() == sorted(epic.FUNCTIONS)


def test_library_exports_every_declared_symbol():
    from paper_2606_00722_amd import epic

    if not os.path.exists(epic.LIB_PATH):
        pytest.fail("libepic.so is not built; run __graft_entry__.build()")
    out = os.popen(f"nm -D --defined-only {epic.LIB_PATH}").read()
    names = set(re.findall(r" T (epic_\w+)$", out, re.M))
    for fn in declared():
        assert fn in names, fn


def test_status_strings():
    from paper_2606_00722_amd import epic

    lib = epic.lib()
    for code, text in epic.STATUS.items():
        assert lib.epic_status_string(code).decode() == text
