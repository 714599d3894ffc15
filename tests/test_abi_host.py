"""The C-ABI library without a GPU: it loads, exports every function that
include/treelin.h declares, and its synchronous argument checks return the
documented codes before any device call (every case below fails a host
check, so nothing is launched)."""
import ctypes
import os
import re

import pytest

from paper_2608_01651_amd import treelin as tl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _lib_or_build():
    if not os.path.exists(tl._LIB_PATH):
        from paper_2608_01651_amd import build
        build.build()
    return tl.lib()


def _declared_functions():
    text = open(os.path.join(ROOT, "include", "treelin.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\s*\*?\s*([A-Za-z_][A-Za-z0-9_]*)\s*\(",
                       text, flags=re.M)
    return sorted(set(n for n in names if n not in ("if", "while", "return", "sizeof")))


def test_library_exports_every_declared_function():
    L = _lib_or_build()
    names = _declared_functions()
    assert {"tree_lin_attn_verify", "tl_workspace_bytes", "tree_state_commit", "tree_topology_export",
            "tree_state_commit_layers", "tree_accepted_path", "tree_conv_gates",
            "tree_conv_state_commit", "tree_budget_select",
            "tl_status_string", "tl_version"} <= set(names)
    for n in names:
        assert hasattr(L, n), f"{n} declared in include/treelin.h but not exported"


def test_status_strings_and_version():
    _lib_or_build()
    for code in range(6):
        assert tl.status_string(code).startswith(
            ("TL_OK", "TL_EINVAL", "TL_EBADTREE", "TL_EBADPATH", "TL_EUNSUPPORTED", "TL_EHIP"))
    assert "unknown" in tl.status_string(99)
    assert re.fullmatch(r"\d+\.\d+\.\d+", tl.version())


def test_missing_library_fails_loudly(monkeypatch):
    monkeypatch.setattr(tl, "_LIB_PATH", os.path.join(ROOT, "no_such_lib.so"))
    monkeypatch.setattr(tl, "_lib", None)
    with pytest.raises(RuntimeError, match="missing"):
        tl.lib()


# fake, never dereferenced device addresses (every case fails a host check first)
A16 = 0x10000
MIS = 0x10002


def _verify(prob, q=A16, k=A16, v=A16, g=A16, beta=None, state=A16, out=A16, offs=A16, par=A16,
            slot=None, err=None, ws=None, ws_bytes=0):
    return _lib_or_build().tree_lin_attn_verify(
        None if prob is None else ctypes.byref(prob), offs, par, q, k, v, g, beta, state, slot, out,
        err, ws, ws_bytes, None)


def _commit(prob, path_offsets=A16, path=A16, k=A16, v=A16, g=A16, beta=None, state=A16):
    return _lib_or_build().tree_state_commit(
        None if prob is None else ctypes.byref(prob), A16, A16, path_offsets, path, k, v, g, beta,
        state, None, None, None)


def _topology(prob, mask=A16, depth=A16):
    return _lib_or_build().tree_topology_export(
        None if prob is None else ctypes.byref(prob), A16, A16, mask, depth, None, None)


def _layers(prob, n, **kw):
    beta = A16 if prob.mode == tl.GDN else None
    f = dict(k=A16, v=A16, g=A16, beta=beta, state=A16)
    f.update(kw)
    return [tl.Layer(f["k"], f["v"], f["g"], f["beta"], f["state"]) for _ in range(n)]


def _commit_layers(prob, n=2, layers=None, terminal=A16, offs=A16, par=A16):
    table = _layers(prob, n) if layers is None and prob is not None else (layers or [])
    arr = (tl.Layer * max(1, len(table)))(*table)
    return _lib_or_build().tree_state_commit_layers(
        None if prob is None else ctypes.byref(prob), n, arr if layers != "null" else None,
        offs, par, terminal, None, None, None)


def _accepted_path(prob, terminal=A16, path_len=A16, path=A16):
    return _lib_or_build().tree_accepted_path(
        None if prob is None else ctypes.byref(prob), A16, A16, terminal, path_len, path, None, None)


def P(**kw):
    base = dict(batch=2, num_qk_heads=2, num_v_heads=4, d_k=64, d_v=64, max_nodes=64)
    base.update({k: v for k, v in kw.items() if k in base})
    extra = {k: v for k, v in kw.items() if k not in base}
    return tl.problem(**base, **extra)


@pytest.mark.parametrize("prob, code", [
    (None, tl.TL_EINVAL),
    (P(num_v_heads=3), tl.TL_EINVAL),            # Hv % Hk != 0
    (P(num_qk_heads=0), tl.TL_EINVAL),
    (P(batch=-1), tl.TL_EINVAL),
    (P(mode=7), tl.TL_EINVAL),
    (P(in_dtype=3), tl.TL_EINVAL),
    (P(d_k=48, d_v=48), tl.TL_EUNSUPPORTED),
    (P(d_k=256, d_v=256), tl.TL_EUNSUPPORTED),
    (P(d_v=32), tl.TL_EUNSUPPORTED),             # d_v != d_k
    (P(max_nodes=0), tl.TL_EUNSUPPORTED),
    (P(max_nodes=257), tl.TL_EUNSUPPORTED),
    (P(num_slots=0), tl.TL_EINVAL),
])
def test_problem_checks(prob, code):
    assert _budget(prob) == code
    assert _verify(prob) == code
    assert _commit(prob) == code
    assert _topology(prob) == code
    assert _commit_layers(prob) == code
    assert _accepted_path(prob) == code


def test_empty_batch_is_a_no_op():
    # nothing is launched and no pointer is needed
    prob = P(batch=0)
    assert _verify(prob, q=None, k=None, v=None, g=None, state=None, out=None, offs=None, par=None) == tl.TL_OK
    assert _commit(prob, path_offsets=None, path=None, k=None, v=None, g=None, state=None) == tl.TL_OK
    assert _topology(prob, mask=None, depth=None) == tl.TL_OK


@pytest.mark.parametrize("field", ["q", "k", "v", "g", "state", "out", "offs", "par"])
def test_verify_null_pointers(field):
    assert _verify(P(), **{field: None}) == tl.TL_EINVAL


@pytest.mark.parametrize("field", ["q", "k", "v", "state", "out"])
def test_verify_misaligned_pointers(field):
    assert _verify(P(), **{field: MIS}) == tl.TL_EINVAL


def test_beta_presence_must_match_the_rule():
    assert _verify(P(mode=tl.GLA), beta=A16) == tl.TL_EINVAL
    assert _verify(P(mode=tl.GDN), beta=None) == tl.TL_EINVAL
    assert _commit(P(mode=tl.GLA), beta=A16) == tl.TL_EINVAL
    assert _commit(P(mode=tl.GDN), beta=None) == tl.TL_EINVAL


def test_identity_slots_need_enough_slots():
    assert _verify(P(batch=4, num_slots=3)) == tl.TL_EINVAL


def test_commit_and_topology_pointer_checks():
    assert _commit(P(), path_offsets=None) == tl.TL_EINVAL
    assert _commit(P(), path_offsets=A16 + 2) == tl.TL_EINVAL
    assert _commit(P(), path=A16 + 2) == tl.TL_EINVAL
    assert _topology(P(), mask=None) == tl.TL_EINVAL
    assert _topology(P(), mask=A16 + 4) == tl.TL_EINVAL
    assert _topology(P(), depth=None) == tl.TL_EINVAL


def test_commit_layers_checks():
    L = _lib_or_build()
    assert _commit_layers(P(), n=tl.MAX_COMMIT_LAYERS + 1,
                          layers=_layers(P(), tl.MAX_COMMIT_LAYERS + 1)) == tl.TL_EINVAL
    assert _commit_layers(P(), n=-1, layers=[]) == tl.TL_EINVAL
    assert _commit_layers(P(), n=0, layers=[]) == tl.TL_OK            # nothing to do
    assert _commit_layers(P(batch=0)) == tl.TL_OK
    assert _commit_layers(P(), terminal=None) == tl.TL_EINVAL
    assert _commit_layers(P(), terminal=MIS) == tl.TL_EINVAL
    assert _commit_layers(P(), offs=None) == tl.TL_EINVAL
    assert L.tree_state_commit_layers(ctypes.byref(P()), 2, None, A16, A16, A16,
                                      None, None, None) == tl.TL_EINVAL
    # one bad layer anywhere in the table fails the whole call
    for field, val in (("state", None), ("k", None), ("v", MIS), ("state", MIS), ("g", None)):
        table = _layers(P(), 3)
        setattr(table[2], field, val)
        assert _commit_layers(P(), n=3, layers=table) == tl.TL_EINVAL, field
    assert _commit_layers(P(mode=tl.GLA), layers=_layers(P(mode=tl.GLA), 2, beta=A16)) == tl.TL_EINVAL
    assert _commit_layers(P(mode=tl.GDN), layers=_layers(P(mode=tl.GDN), 2, beta=None)) == tl.TL_EINVAL
    assert _commit_layers(P(batch=4, num_slots=3)) == tl.TL_EINVAL


def test_accepted_path_checks():
    for field in ("terminal", "path_len", "path"):
        assert _accepted_path(P(), **{field: None}) == tl.TL_EINVAL
        assert _accepted_path(P(), **{field: MIS}) == tl.TL_EINVAL
    assert _accepted_path(P(batch=0), terminal=None, path_len=None, path=None) == tl.TL_OK


def _conv(prob, width=4, eps=1e-6, **kw):
    gdn = prob is not None and prob.mode == tl.GDN
    f = dict(offs=A16, par=A16, x=A16, ga=A16, gb=A16 if gdn else None, w=A16, bias=A16, alog=A16,
             dtb=A16, cs=A16, slot=None, q=A16, k=A16, v=A16, g=A16, beta=A16 if gdn else None)
    f.update(kw)
    return _lib_or_build().tree_conv_gates(
        None if prob is None else ctypes.byref(prob), width, eps, f["offs"], f["par"], f["x"], f["ga"],
        f["gb"], f["w"], f["bias"], f["alog"], f["dtb"], f["cs"], f["slot"], f["q"], f["k"], f["v"],
        f["g"], f["beta"], None, None)


def _conv_commit(prob, width=4, **kw):
    f = dict(offs=A16, par=A16, term=A16, x=A16, cs=A16)
    f.update(kw)
    return _lib_or_build().tree_conv_state_commit(
        None if prob is None else ctypes.byref(prob), width, f["offs"], f["par"], f["term"], f["x"],
        f["cs"], None, None, None)


def test_conv_entry_points_checks():
    for mode in (tl.GLA, tl.GDN):
        assert _conv(P(mode=mode, batch=0)) == tl.TL_OK
    for width in (1, 5):
        assert _conv(P(), width=width) == tl.TL_EUNSUPPORTED
        assert _conv_commit(P(), width=width) == tl.TL_EUNSUPPORTED
    assert _conv(P(in_dtype=tl.F32)) == tl.TL_EUNSUPPORTED
    assert _conv_commit(P(in_dtype=tl.F32)) == tl.TL_EUNSUPPORTED
    assert _conv(P(), eps=-1.0) == tl.TL_EINVAL
    assert _conv(P(mode=tl.GLA), gb=A16) == tl.TL_EINVAL
    assert _conv(P(mode=tl.GLA), beta=A16) == tl.TL_EINVAL
    assert _conv(P(mode=tl.GDN), gb=None) == tl.TL_EINVAL
    assert _conv(P(mode=tl.GDN), beta=None) == tl.TL_EINVAL
    for field in ("offs", "par", "x", "ga", "w", "bias", "alog", "dtb", "cs", "q", "k", "v", "g"):
        assert _conv(P(), **{field: None}) == tl.TL_EINVAL, field
    for field in ("x", "cs", "q", "k", "v", "w", "bias"):
        assert _conv(P(), **{field: A16 + 4}) == tl.TL_EINVAL, field
    assert _conv(P(batch=4, num_slots=3)) == tl.TL_EINVAL
    for field in ("offs", "par", "term", "x", "cs"):
        assert _conv_commit(P(), **{field: None}) == tl.TL_EINVAL, field
    assert _conv_commit(P(), x=A16 + 4) == tl.TL_EINVAL
    assert _conv_commit(P(batch=0), offs=None) == tl.TL_OK


def _budget(prob, num_candidates=64, capacity=16, ws_bytes=1 << 20, **kw):
    f = dict(offs=A16, cpar=A16, cprob=A16, rho=A16, rank=A16, no=A16, par=A16, src=A16, ws=A16,
             err=None)
    f.update(kw)
    return _lib_or_build().tree_budget_select(
        None if prob is None else ctypes.byref(prob), num_candidates, capacity, f["offs"], f["cpar"],
        f["cprob"], f["rho"], f["rank"], f["no"], f["par"], f["src"], f["ws"], ws_bytes, f["err"], None)


def test_budget_select_checks():
    assert _budget(P(batch=0), offs=None, src=None, ws=None) == tl.TL_OK
    assert _budget(P(), num_candidates=-1) == tl.TL_EINVAL
    assert _budget(P(), capacity=-1) == tl.TL_EINVAL
    assert _budget(P(batch=1025)) == tl.TL_EUNSUPPORTED
    assert _budget(P(), num_candidates=32769) == tl.TL_EUNSUPPORTED
    for field in ("offs", "cpar", "cprob", "rho", "rank", "no", "par", "src", "ws"):
        assert _budget(P(), **{field: None}) == tl.TL_EINVAL, field
        assert _budget(P(), **{field: MIS}) == tl.TL_EINVAL, field
    assert _budget(P(), ws=A16 + 16) == tl.TL_EINVAL           # the workspace is 256-byte aligned
    assert _budget(P(), err=MIS) == tl.TL_EINVAL
    need = tl.budget_workspace_bytes(2, 64)
    assert need > 0 and need % 256 == 0
    assert _budget(P(), ws_bytes=need - 1) == tl.TL_EINVAL
    assert tl.budget_workspace_bytes(0, 64) == 0
    assert tl.budget_workspace_bytes(4, 64) > tl.budget_workspace_bytes(2, 64)


def test_verify_workspace():
    """The layer-local workspace of verify: its size query and the checks on
    the buffer a caller passes (§4.4's layer-local lifetime)."""
    L = _lib_or_build()
    for prob in (P(), P(mode=tl.GDN), P(max_nodes=256, d_k=128, d_v=128), P(batch=0), P(max_nodes=0)):
        assert tl.workspace_bytes(prob) == 0
    assert L.tl_workspace_bytes(None) == 0
    # a size of 0 needs no buffer; a buffer that is passed must be 256-byte aligned
    assert _verify(P(batch=0), q=None, k=None, v=None, g=None, state=None, out=None, offs=None,
                   par=None, ws=None, ws_bytes=0) == tl.TL_OK
    assert _verify(P(batch=0), ws=None, ws_bytes=256) == tl.TL_EINVAL
    assert _verify(P(batch=0), ws=A16 + 16, ws_bytes=256) == tl.TL_EINVAL
    assert _verify(P(batch=0), ws=0x100000, ws_bytes=256) == tl.TL_OK
    # the problem is still checked first
    assert _verify(P(num_v_heads=3), ws=0x100000, ws_bytes=256) == tl.TL_EINVAL


def _budget_noalloc(prob, num_candidates=64, capacity=16, **kw):
    f = dict(offs=A16, cpar=A16, cprob=A16, rho=A16, rank=A16, no=A16, par=A16, src=A16, err=None)
    f.update(kw)
    return _lib_or_build().tree_budget_select_noalloc(
        None if prob is None else ctypes.byref(prob), num_candidates, capacity, f["offs"], f["cpar"],
        f["cprob"], f["rho"], f["rank"], f["no"], f["par"], f["src"], f["err"], None)


def test_budget_select_noalloc_checks():
    """The allocation-free budget entry point: the same host checks as
    tree_budget_select, and a problem whose workspace exceeds the static
    buffer is refused before anything is enqueued."""
    assert _budget_noalloc(None) == tl.TL_EINVAL
    assert _budget_noalloc(P(batch=0), offs=None, src=None) == tl.TL_OK
    assert _budget_noalloc(P(), num_candidates=-1) == tl.TL_EINVAL
    assert _budget_noalloc(P(batch=1025)) == tl.TL_EUNSUPPORTED
    for field in ("offs", "cpar", "cprob", "rho", "rank", "no", "par", "src"):
        assert _budget_noalloc(P(), **{field: None}) == tl.TL_EINVAL, field
        assert _budget_noalloc(P(), **{field: MIS}) == tl.TL_EINVAL, field
    assert _budget_noalloc(P(), err=MIS) == tl.TL_EINVAL
    # the static buffer's bound: the largest shapes that fit, and the first that do not
    assert tl.budget_workspace_bytes(1024, 100) <= tl.BUDGET_NOALLOC_MAX_BYTES
    assert tl.budget_workspace_bytes(1024, 101) > tl.BUDGET_NOALLOC_MAX_BYTES
    assert tl.budget_workspace_bytes(407, 256) <= tl.BUDGET_NOALLOC_MAX_BYTES
    assert _budget_noalloc(P(batch=1024, max_nodes=101)) == tl.TL_EUNSUPPORTED
    assert _budget_noalloc(P(batch=408, max_nodes=256)) == tl.TL_EUNSUPPORTED
