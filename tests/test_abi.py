"""The C-ABI library loads and exports every function include/cf.h declares
(no compute call: this runs without a GPU)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cf.h")
LIB = os.path.join(ROOT, "paper_2512_14098_amd", "libcf.so")


def declared_functions():
    with open(HEADER) as fh:
        text = fh.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_][\w\s\*]*?\b(cf_\w+)\s*\(", text, flags=re.M)
    return sorted(set(names))


def test_header_declares_the_path():
    names = declared_functions()
    for f in ("cf_trace_gen", "cf_eval_coarse", "cf_select_topk", "cf_rate_grid", "cf_eval_fine", "cf_eval_mc", "cf_pareto",
              "cf_goodput_reduce", "cf_select_best"):
        assert f in names


def _comment_before(text, name):
    """The block comment that ends right before the declaration of name."""
    m = re.search(r"/\*((?:(?!\*/).)*?)\*/\s*(?:const\s+)?[A-Za-z_][\w\s\*]*?\b" + name + r"\s*\(", text, flags=re.S)
    assert m, name
    return m.group(1)


def test_path_calls_cite_the_passage_they_follow():
    """Each call of the hot path names the section, algorithm or equation it follows, and the
    capacity / flag contract of cf_eval_fine and cf_goodput_reduce is stated."""
    with open(HEADER) as fh:
        text = fh.read()
    cite = re.compile(r"Sec\. \d|Alg\. \d|Eq\. \(\d|Table \d")
    for f in ("cf_trace_gen", "cf_eval_coarse", "cf_select_topk", "cf_rate_grid", "cf_eval_fine",
              "cf_goodput_reduce", "cf_select_best"):
        assert cite.search(_comment_before(text, f)), f
    for flag in ("CF_FULL", "CF_DUMP_LAT", "CF_EARLY_EXIT"):
        assert re.search(r"#define " + flag + r"\b", text), flag
        assert flag in _comment_before(text, "cf_eval_fine"), flag
    assert "status" in _comment_before(text, "cf_goodput_reduce")


@pytest.mark.skipif(not os.path.exists(LIB), reason="libcf.so not built")
def test_library_exports_every_declared_function():
    lib = ctypes.CDLL(LIB)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


@pytest.mark.skipif(not os.path.exists(LIB), reason="libcf.so not built")
def test_binding_has_the_same_names():
    from paper_2512_14098_amd import cf
    for n in declared_functions():
        assert n in cf.EXPORTED
        if n not in ("cf_last_error", "cf_status_str", "cf_version"):
            assert callable(getattr(cf, n)), n


def test_product_path_does_not_import_the_oracle():
    pkg = os.path.join(ROOT, "paper_2512_14098_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                with open(os.path.join(dirpath, f)) as fh:
                    text = fh.read()
                assert "oracle" not in re.sub(r"#.*|//.*", "", text).lower() or f == "__init__.py", f
