"""The C-ABI library loads and exports every symbol include/eahr.h declares
(no GPU calls)."""
import os
import re

from paper_2608_07152_amd import eahr

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "eahr.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = re.findall(r"^(?!\s*typedef)\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\s*\*?\s*([a-z][a-z0-9_]*)\s*\(",
                       src, flags=re.M)
    return sorted(set(names))


def test_header_declares_the_boundary():
    names = _declared()
    for n in ("pvs_build", "pvs_open", "pvs_next", "eahr_topk", "pbm_build", "pbm_next"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = eahr.load()
    for n in _declared():
        assert hasattr(lib, n), n


def test_binding_covers_exactly_the_header():
    assert sorted(eahr.exported_symbols()) == _declared()


def test_last_error_is_a_string():
    lib = eahr.load()
    assert isinstance(lib.eahr_last_error(), bytes)
