"""Host-only checks of the C-ABI library: it loads, exports every function that
include/gorila.h declares, and its host-side sizing helpers agree with the
parameter layout.  No kernel is launched (no GPU here)."""
import ast
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gorila.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"\b(gorila_[a-z_]+)\s*\(", text)
    return sorted(set(names))


def test_library_exports_every_declared_function():
    import paper_1507_04296_amd as g
    L = g.lib()
    declared = _declared_functions()
    assert len(declared) >= 12
    for name in declared:
        assert hasattr(L, name), name
    assert sorted(g.EXPORTS) == declared


def test_param_count_matches_layout():
    import paper_1507_04296_amd as g
    from paper_1507_04296_amd import datagen
    for A in (1, 6, 18, 32):
        assert g.param_count(A) == datagen.param_count(A)
    assert g.param_count(18) == 1693362
    assert g.param_count(6) == 1687206
    assert g.param_count(0) == -1 and g.param_count(33) == -1


def test_param_layout_matches_oracle(oracle_mod):
    from paper_1507_04296_amd import datagen
    for A in (6, 18):
        off = oracle_mod.param_offsets(oracle_mod.Net(n_actions=A))
        sl = datagen.tensor_slices(A)
        assert [sl[n].start for n in ("W1", "b1", "W2", "b2", "W3", "b3", "W4", "b4", "W5", "b5")] \
            == off[:10]


def test_workspace_sizing_is_monotone():
    import paper_1507_04296_amd as g
    a = g.workspace_bytes(32, 18)
    b = g.workspace_bytes(512, 6)
    assert 0 < a < b
    assert g.workspace_bytes(0, 18) == 0
    assert g.workspace_bytes(8, 40) == 0
    assert g.workspace_bytes(8, 18, groups=16) > g.workspace_bytes(8, 18)
    # a context sized for a batch serves every smaller batch: small batches keep
    # several partial planes of the data gradients, so check every size across
    # the thresholds where the plane count changes
    for A in (6, 18):
        sizes = [g.workspace_bytes(b, A) for b in range(1, 300)]
        assert all(x <= y for x, y in zip(sizes, sizes[1:])), A


def test_strerror_names_every_code():
    import paper_1507_04296_amd as g
    for code in (0, -1, -2, -3, -4, -5):
        assert g.strerror(code)
    assert g.strerror(-99) == "unknown error"


def test_product_path_never_imports_the_oracle():
    pkg = os.path.join(ROOT, "paper_1507_04296_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            path = os.path.join(dirpath, f)
            if f.endswith(".py"):
                tree = ast.parse(open(path).read())
                for node in ast.walk(tree):
                    if isinstance(node, ast.Import):
                        assert all(not a.name.startswith("oracle") for a in node.names), path
                    if isinstance(node, ast.ImportFrom):
                        assert not (node.module or "").startswith("oracle"), path
            if f.endswith((".hip", ".h", ".cpp")):
                assert "gorila_oracle" not in open(path).read(), path


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    import paper_1507_04296_amd as g
    monkeypatch.setattr(g, "_lib", None)
    monkeypatch.setattr(g, "LIB_PATH", str(tmp_path / "libgorila.so"))
    with pytest.raises(RuntimeError, match="missing"):
        g.lib()


def test_epsilon_schedule_matches_oracle(oracle_mod):
    """gorila_epsilon is host arithmetic: equal to the oracle's schedule."""
    import paper_1507_04296_amd as g
    for u in (-3, 0, 1, 17, 250_000, 999_999, 1_000_000, 10**7):
        assert g.epsilon(u) == oracle_mod.epsilon(u)
    assert g.epsilon(5, 1.0, 0.3, 20) == oracle_mod.epsilon(5, 1.0, 0.3, 20)


def test_workspace_rejects_too_many_groups():
    import paper_1507_04296_amd as g
    assert g.workspace_bytes(64, 18, g.GORILA_BF16, 16) > 0
    assert g.workspace_bytes(64, 18, g.GORILA_BF16, 17) == 0
