"""Helpers for tests that drive libqe.so."""
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_symbols():
    names = set()
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            text = open(os.path.join(ROOT, "include", fn)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names |= set(re.findall(r"\b(qe_[a-z0-9_]+)\s*\(", text))
    return sorted(names)


def need_lib():
    from paper_2609_23536_amd import qe
    if not os.path.exists(qe.LIB_PATH):
        pytest.fail("libqe.so is not built (run python -m paper_2609_23536_amd.build)")
    return qe
