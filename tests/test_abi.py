"""The C ABI library on the CPU: it loads, exports every symbol include/occam.h declares,
and rejects invalid arguments on the host before anything is enqueued.

No call here reaches a kernel launch: every case carries at least one invalid
argument, and validation runs before any HIP call.
"""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2605_29657_amd import build as occam_build
from paper_2605_29657_amd import occam

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "occam.h")
FAKE = 0x7f0000000000          # a 256-byte aligned, never-dereferenced "device" address


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(occam.LIB_PATH):
        occam_build.build()
    return occam.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(occam_[a-z_]+)\s*\(", text)))


def test_header_declares_the_five_steps_and_helpers():
    names = declared_functions()
    for fn in ("occam_score", "occam_threshold", "occam_select", "occam_gather", "occam_prune",
               "occam_workspace_size", "occam_status_string", "occam_version"):
        assert fn in names
    assert set(names) == set(occam.EXPORTS)


def test_library_exports_every_declared_symbol(L):
    out = subprocess.run(["nm", "-D", "--defined-only", occam.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (occam_\w+)", out))
    for fn in declared_functions():
        assert fn in exported, fn
        assert hasattr(L, fn)


def test_version_and_status_strings(L):
    assert L.occam_version() == 2
    for s in range(5):
        assert occam.status_string(s).startswith("OCCAM_")
    assert "unknown" in occam.status_string(77)


def good_problem(**kw):
    args = dict(batch=4, num_heads=16, num_kv_heads=16, head_dim=64, num_registers=4, rows=1,
                cands=576, dtype=occam.BF16)
    args.update(kw)
    return occam.Problem(**args)


def ws_size(p):
    return occam.workspace_size(p)


@pytest.mark.parametrize("kw", [
    dict(batch=0), dict(num_heads=0), dict(num_kv_heads=0), dict(num_heads=16, num_kv_heads=5),
    dict(head_dim=0), dict(head_dim=264), dict(num_registers=0), dict(num_registers=33),
    dict(rows=0), dict(cands=-1), dict(dtype=7), dict(softmax_scale=-1.0),
    dict(softmax_scale=float("inf")), dict(softmax_scale=float("nan")),
    dict(visual_row_reduce=2), dict(visual_row_reduce=-1),
])
def test_invalid_problems(L, kw):
    p = good_problem(**kw)
    assert ws_size(p) == 0
    st = L.occam_score(p.ref, FAKE, FAKE, None, FAKE, FAKE, 1 << 40, None)
    assert st == occam.ERR_INVALID_ARG


@pytest.mark.parametrize("kw", [
    dict(dtype=occam.F32, rows=8, num_heads=32, num_kv_heads=32, head_dim=128),   # f32 text rows
    dict(head_dim=6),                                                              # bf16 needs d % 8
    dict(dtype=occam.F32, head_dim=6),                                             # f32 needs d % 4
    dict(rows=64, head_dim=136),                                                   # text rows: d <= 128
])
def test_unsupported_shapes(L, kw):
    p = good_problem(**kw)
    assert ws_size(p) == 0
    st = L.occam_score(p.ref, FAKE, FAKE, None, FAKE, FAKE, 1 << 40, None)
    assert st == occam.ERR_UNSUPPORTED


def test_mutual_scoring_is_a_valid_problem(L):
    # Every token an anchor row, mean over rows (Eq. mutual_scoring).
    p = good_problem(rows=580, cands=576, visual_row_reduce=occam.ROWS_MEAN)
    assert ws_size(p) > 0
    # Partials per (sample, 128-row block[, head], key): the mean form keeps one per head
    # (column sums, 4 x 5 x 16 x 580 floats here), the max form one per row block.
    extra = ws_size(p) - ws_size(good_problem(rows=580, cands=576))
    want = 4 * 5 * (16 - 1) * 580 * 4
    assert want - 256 < extra < want + 256


def test_workspace_size_grows_with_the_batch(L):
    small = ws_size(good_problem(batch=1))
    big = ws_size(good_problem(batch=64))
    assert 0 < small < big
    txt = ws_size(good_problem(rows=128, num_heads=32, num_kv_heads=32, head_dim=128, cands=2880))
    assert txt > 0


def test_ragged_problem_needs_bounds(L):
    p = occam.Problem(4, 16, 16, 64, 4, q_offsets=FAKE, key_offsets=FAKE, max_rows=0,
                      max_cands=100, dtype=occam.BF16)
    assert ws_size(p) == 0
    p = occam.Problem(4, 16, 16, 64, 4, q_offsets=FAKE, key_offsets=FAKE, max_rows=1,
                      max_cands=100, dtype=occam.BF16)
    assert ws_size(p) > 0
    p = occam.Problem(4, 16, 16, 64, 4, q_offsets=FAKE + 2, key_offsets=FAKE, max_rows=1,
                      max_cands=100, dtype=occam.BF16)
    assert ws_size(p) == 0


def test_score_argument_checks(L):
    p = good_problem()
    n = ws_size(p)
    assert L.occam_score(p.ref, None, FAKE, None, FAKE, FAKE, n, None) == occam.ERR_INVALID_ARG
    assert L.occam_score(p.ref, FAKE + 8, FAKE, None, FAKE, FAKE, n, None) == occam.ERR_INVALID_ARG
    assert L.occam_score(p.ref, FAKE, FAKE, None, None, FAKE, n, None) == occam.ERR_INVALID_ARG
    assert L.occam_score(p.ref, FAKE, FAKE, None, FAKE, FAKE, n - 1, None) == occam.ERR_WORKSPACE
    assert L.occam_score(p.ref, FAKE, FAKE, None, FAKE, FAKE + 64, n, None) == occam.ERR_INVALID_ARG
    assert L.occam_score(None, FAKE, FAKE, None, FAKE, FAKE, n, None) == occam.ERR_INVALID_ARG


@pytest.mark.parametrize("lam", [-0.5, float("nan"), float("inf")])
def test_threshold_and_prune_reject_bad_lambda(L, lam):
    p = good_problem()
    assert L.occam_threshold(p.ref, FAKE, lam, 0, FAKE, None) == occam.ERR_INVALID_ARG
    st = L.occam_prune(p.ref, FAKE, FAKE, None, lam, 0, None, 0, None, None, None, FAKE, FAKE,
                       FAKE, FAKE, ws_size(p), None)
    assert st == occam.ERR_INVALID_ARG


def test_reduce_mode_is_checked(L):
    p = good_problem()
    for bad in (4, -1, 99):
        assert L.occam_threshold(p.ref, FAKE, 0.5, bad, FAKE, None) == occam.ERR_INVALID_ARG


def test_select_argument_checks(L):
    p = good_problem()
    n = ws_size(p)
    assert L.occam_select(p.ref, FAKE, FAKE, None, None, FAKE, FAKE, FAKE, n, None) == \
        occam.ERR_INVALID_ARG
    assert L.occam_select(p.ref, FAKE, FAKE, FAKE + 2, FAKE, FAKE, FAKE, FAKE, n, None) == \
        occam.ERR_INVALID_ARG
    assert L.occam_select(p.ref, FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, 16, None) == \
        occam.ERR_WORKSPACE


def rows_array(*items):
    arr = (occam._Rows * len(items))(*items)
    return arr


def test_gather_row_descriptor_checks(L):
    p = good_problem()
    ok = occam._Rows(FAKE, FAKE, 0, 0, 2048, 2048, 2048)
    bad_stride = occam._Rows(FAKE, FAKE, 0, 0, 1024, 2048, 2048)     # stride < row bytes
    bad_align = occam._Rows(FAKE + 2, FAKE, 0, 0, 2048, 2048, 2048)  # src not 4-byte aligned
    bad_len = occam._Rows(FAKE, FAKE, 0, 0, 2048, 2048, 2046)        # row bytes % 4
    neg_pad = occam._Rows(FAKE, FAKE, -1, 0, 2048, 2048, 2048)
    for r in (bad_stride, bad_align, bad_len, neg_pad):
        assert L.occam_gather(p.ref, 1, rows_array(r), FAKE, FAKE, None) == occam.ERR_INVALID_ARG
    assert L.occam_gather(p.ref, 9, rows_array(*([ok] * 9)), FAKE, FAKE, None) == \
        occam.ERR_INVALID_ARG
    assert L.occam_gather(p.ref, 1, None, FAKE, FAKE, None) == occam.ERR_INVALID_ARG
    assert L.occam_gather(p.ref, 1, rows_array(ok), None, FAKE, None) == occam.ERR_INVALID_ARG
    # n = 0 is a valid no-op that enqueues nothing.
    assert L.occam_gather(p.ref, 0, None, FAKE, FAKE, None) == occam.OK


def test_binding_raises_without_the_library(monkeypatch, tmp_path):
    monkeypatch.setattr(occam, "_lib", None)
    monkeypatch.setattr(occam, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError):
        occam.lib()


def test_register_redirect_validation(L):
    p = good_problem()
    ok = dict(h=FAKE, width=64, stride=128, ch=FAKE, n=4, slot=0)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        return L.occam_register_redirect(p.ref, a["h"], a["width"], a["stride"], a["ch"], a["n"],
                                         a["slot"], None)
    for bad in (dict(h=None), dict(h=FAKE + 1), dict(width=0), dict(stride=64),
                dict(stride=129), dict(ch=None), dict(ch=FAKE + 2), dict(n=-1), dict(n=1025),
                dict(slot=-1), dict(slot=4)):
        assert call(**bad) == occam.ERR_INVALID_ARG, bad
    assert L.occam_register_redirect(None, FAKE, 64, 128, FAKE, 4, 0, None) == occam.ERR_INVALID_ARG
    # n = 0 launches nothing and succeeds, even without a channel list or a GPU.
    assert call(ch=None, n=0) == occam.OK


def test_match_lambda_validation(L):
    p = good_problem()
    n = occam.workspace_size(p)
    ok = dict(sc=FAKE, red=occam.REG_MEAN, k=64.0, lam=FAKE, mk=FAKE, ws=FAKE, n=n)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        return L.occam_match_lambda(p.ref, a["sc"], a["red"], a["k"], a["lam"], a["mk"], a["ws"],
                                    a["n"], None)
    for bad in (dict(sc=None), dict(sc=FAKE + 2), dict(red=7), dict(k=-1.0), dict(k=float("nan")),
                dict(k=float("inf")), dict(lam=None), dict(lam=FAKE + 1), dict(mk=FAKE + 3)):
        assert call(**bad) == occam.ERR_INVALID_ARG, bad
    assert call(n=n - 1) == occam.ERR_WORKSPACE
    assert call(ws=None) == occam.ERR_INVALID_ARG
    assert L.occam_match_lambda(None, FAKE, 0, 1.0, FAKE, None, FAKE, n, None) == \
        occam.ERR_INVALID_ARG


def test_select_topk_validation(L):
    p = good_problem()
    n = occam.workspace_size(p)
    ok = dict(sc=FAKE, k=8, im=None, idx=FAKE, cnt=FAKE, off=FAKE, ws=FAKE, n=n)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        return L.occam_select_topk(p.ref, a["sc"], a["k"], a["im"], a["idx"], a["cnt"], a["off"],
                                   a["ws"], a["n"], None)
    for bad in (dict(sc=None), dict(sc=FAKE + 2), dict(k=-1), dict(im=FAKE + 1), dict(idx=None),
                dict(cnt=FAKE + 2), dict(off=None), dict(ws=None)):
        assert call(**bad) == occam.ERR_INVALID_ARG, bad
    assert call(n=n - 1) == occam.ERR_WORKSPACE


def test_mean_threshold_is_an_accepted_reduction(L):
    # OCCAM_REF_CAND_MEAN passes the reduction check (the null scores are what fail).
    p = good_problem()
    assert L.occam_threshold(p.ref, None, ctypes.c_float(1.0), occam.REF_CAND_MEAN, FAKE, None) == \
        occam.ERR_INVALID_ARG


def test_unsupported_batch_beyond_the_grid_limit(L):
    # The sample index sits in grid.y of several kernels (at most 65535).
    p = good_problem(batch=65536, cands=4)
    assert ws_size(p) == 0
    assert L.occam_score(p.ref, FAKE, FAKE, None, FAKE, FAKE, 1 << 40, None) == occam.ERR_UNSUPPORTED
    assert ws_size(good_problem(batch=65535, cands=4)) > 0


def test_prune_noalloc_validation(L):
    # Checks run before any HIP call, as in occam_prune; none of these reach a launch.
    p = good_problem()
    args = lambda **kw: dict(dict(q=FAKE, k=FAKE, lam=1.0, idx=FAKE, cnt=FAKE, off=FAKE), **kw)

    def call(prob, a):
        return L.occam_prune_noalloc(prob.ref, a["q"], a["k"], None, a["lam"], 0, None, 0, None,
                                     None, None, a["idx"], a["cnt"], a["off"], None)

    assert call(p, args(q=None)) == occam.ERR_INVALID_ARG
    assert call(p, args(k=FAKE + 8)) == occam.ERR_INVALID_ARG
    assert call(p, args(lam=-1.0)) == occam.ERR_INVALID_ARG
    assert call(p, args(off=None)) == occam.ERR_INVALID_ARG
    assert call(good_problem(batch=0), args()) == occam.ERR_INVALID_ARG
    assert call(good_problem(head_dim=6), args()) == occam.ERR_UNSUPPORTED
    # A problem whose workspace exceeds the built-in 32 MiB is refused, not truncated.
    big = good_problem(batch=1024, cands=4096)
    assert ws_size(big) > (32 << 20)
    assert call(big, args()) == occam.ERR_WORKSPACE
    assert L.occam_prune_noalloc(None, FAKE, FAKE, None, 1.0, 0, None, 0, None, None, None, FAKE,
                                 FAKE, FAKE, None) == occam.ERR_INVALID_ARG
