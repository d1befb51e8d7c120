"""The C-ABI library on the CPU: it loads, exports every declared symbol, and its host-only
helpers and argument validation behave as documented.  No kernel is launched: every call
below fails validation before any HIP call (the tests skip where a GPU is visible, so a
validation bug can never turn into a launch with a fake pointer)."""
import ctypes
import os
import re

import numpy as np
import pytest
import torch

from oracle import taskpress_oracle as o

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "taskpress.h")

from paper_2608_03276_amd import binding as B  # noqa: E402

lib = B.load()
no_gpu = pytest.mark.skipif(torch.cuda.device_count() > 0, reason="validation cases use fake device pointers")
FAKE = 0x10000  # 16-byte aligned, never dereferenced


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(tp_[a-z_0-9]+)\s*\(", src)))


def test_exports_every_declared_symbol():
    names = declared_functions()
    assert set(names) == set(B.EXPORTED)
    for n in names:
        assert hasattr(lib, n), n


def test_version_and_status_strings():
    assert "gfx950" in B.tp_version()
    for s, name in B._STATUS_NAMES.items():
        assert lib.tp_status_string(s).decode() == name


def test_keep_count_matches_oracle():
    rng = np.random.default_rng(3)
    for _ in range(2000):
        n = int(rng.integers(1, 300000))
        r = float(rng.choice([rng.random(), 0.1, 0.2, 0.25, 0.05, 1.0, 1e-7]))
        if r > 0:
            assert B.tp_keep_count(n, r, 0) == o.keep_count(n, keep_ratio=r)
        bud = int(rng.integers(1, 5000))
        assert B.tp_keep_count(n, 0.0, bud) == o.keep_count(n, keep_budget=bud)
    assert B.tp_keep_count(10, 0.5, 3) == -1  # both given
    assert B.tp_keep_count(10, 0.0, 0) == -1  # neither
    assert B.tp_keep_count(10, 1.5, 0) == -1
    assert B.tp_keep_count(0, 0.5, 0) == -1


def test_workspace_size():
    d = B.dims(32, 32, 8, 128)
    bt = B.Batch([0, 131072], [0, 64])
    ws = B.tp_workspace_size(B.TP_FN_GUIDE_SCORES, d, bt)
    rows = 32 * 32 * 64
    # at least: one (max, sum) pair per guide row and chunk, the row normalisers, the raw scores
    assert ws >= rows * 8 + rows * 4 + 32 * 8 * 131072 * 4
    assert B.tp_workspace_size(B.TP_FN_COMBINE_SELECT_TOPK, d, bt) >= 32 * 8 * 131072 * 4
    with pytest.raises(B.TaskPressError) as e:
        B.tp_workspace_size(7, d, bt)
    assert e.value.status == B.TP_ERR_PARAM


def _gs(d, bt, q=FAKE, k=FAKE, scale=0.125, pool=5, s=FAKE, ws=FAKE, wsb=1 << 40, kg=None):
    return lib.tp_guide_scores(ctypes.byref(d), ctypes.byref(bt.c) if bt is not None else None, q, k, kg, scale,
                               pool, s, ws, wsb, None)


@no_gpu
def test_guide_scores_validation():
    d = B.dims(2, 8, 2, 64)
    bt = B.Batch([0, 100, 300], [0, 16, 20])
    cases = [
        (dict(q=None), B.TP_ERR_NULL),
        (dict(k=None), B.TP_ERR_NULL),
        (dict(s=None), B.TP_ERR_NULL),
        (dict(scale=0.0), B.TP_ERR_PARAM),
        (dict(scale=-1.0), B.TP_ERR_PARAM),
        (dict(scale=float("inf")), B.TP_ERR_PARAM),
        (dict(pool=4), B.TP_ERR_PARAM),
        (dict(pool=0), B.TP_ERR_PARAM),
        (dict(ws=None), B.TP_ERR_WORKSPACE),
        (dict(wsb=100), B.TP_ERR_WORKSPACE),
        (dict(ws=FAKE + 16), B.TP_ERR_WORKSPACE),
        (dict(q=FAKE + 2), B.TP_ERR_PARAM),
        (dict(kg=FAKE + 8), B.TP_ERR_PARAM),
    ]
    for kw, want in cases:
        assert _gs(d, bt, **kw) == want, kw
        assert lib.tp_last_error().decode() != ""
    assert _gs(B.dims(2, 8, 3, 64), bt) == B.TP_ERR_SHAPE  # Hq % Hkv
    assert _gs(B.dims(2, 8, 2, 96), bt) == B.TP_ERR_UNSUPPORTED  # head_dim
    assert _gs(B.dims(0, 8, 2, 64), bt) == B.TP_ERR_SHAPE
    assert _gs(d, B.Batch([0, 100, 100], [0, 16, 20])) == B.TP_ERR_SHAPE  # empty sequence
    assert _gs(d, B.Batch([0, 100, 300], [0, 16, 16])) == B.TP_ERR_SHAPE  # empty guide
    assert _gs(d, B.Batch([1, 100, 300], [0, 16, 20])) == B.TP_ERR_SHAPE
    assert _gs(d, B.Batch([0, 100, 300])) == B.TP_ERR_NULL  # no guide offsets
    assert _gs(d, B.Batch(list(range(0, 66)), list(range(0, 66)))) == B.TP_ERR_UNSUPPORTED  # batch > 64
    assert lib.tp_guide_scores(None, ctypes.byref(bt.c), FAKE, FAKE, None, 0.1, 1, FAKE, FAKE, 1 << 40,
                               None) == B.TP_ERR_NULL


@no_gpu
def test_guide_scores_lse_validation():
    d = B.dims(2, 8, 2, 64)
    bt = B.Batch([0, 100, 300], [0, 16, 20])
    wsb = B.tp_workspace_size(B.TP_FN_GUIDE_SCORES, d, bt)

    def gl(lse=FAKE, scale=0.125, pool=5, ws=FAKE, nbytes=wsb, batch=bt):
        return lib.tp_guide_scores_lse(ctypes.byref(d), ctypes.byref(batch.c), FAKE, FAKE, lse, scale, pool, FAKE, ws,
                                       nbytes, None)

    assert gl(lse=None) == B.TP_ERR_NULL
    assert gl(lse=FAKE + 2) == B.TP_ERR_PARAM
    assert gl(scale=-1.0) == B.TP_ERR_PARAM
    assert gl(pool=4) == B.TP_ERR_PARAM
    assert gl(nbytes=wsb - 1) == B.TP_ERR_WORKSPACE
    assert gl(batch=B.Batch([0, 100, 300])) == B.TP_ERR_NULL  # guide offsets needed
    assert lib.tp_last_error().decode() != ""


@no_gpu
def test_compact_quantize_validation():
    d = B.dims(2, 8, 2, 64)
    bt = B.Batch([0, 100, 300])

    def cq(ko=(0, 25, 75), v=FAKE, vqo=FAKE, sco=FAKE, fmt=0, bits=8, kout=FAKE):
        return lib.tp_compact_quantize_kv(ctypes.byref(d), ctypes.byref(bt.c), B._i64_array(ko), FAKE, FAKE, v, fmt,
                                          bits, kout, vqo, sco, None)

    assert cq(v=None) == B.TP_ERR_NULL
    assert cq(vqo=None) == B.TP_ERR_NULL
    assert cq(sco=None) == B.TP_ERR_NULL
    assert cq(kout=None) == B.TP_ERR_NULL
    assert cq(v=FAKE + 8) == B.TP_ERR_PARAM
    assert cq(ko=(0, 101, 150)) == B.TP_ERR_SHAPE
    assert cq(bits=1) == B.TP_ERR_PARAM


@no_gpu
def test_quantize_validation():
    d = B.dims(2, 8, 2, 128)
    bt = B.Batch([0, 100])
    q = lambda fmt=0, bits=8, v=FAKE, s=FAKE, vq=FAKE: lib.tp_quantize_v_scales(
        ctypes.byref(d), ctypes.byref(bt.c), v, fmt, bits, s, vq, None)
    assert q(bits=1) == B.TP_ERR_PARAM
    assert q(bits=9) == B.TP_ERR_PARAM
    assert q(fmt=5) == B.TP_ERR_PARAM
    assert q(v=None) == B.TP_ERR_NULL
    assert q(s=None) == B.TP_ERR_NULL
    assert q(vq=FAKE + 4) == B.TP_ERR_PARAM


@no_gpu
def test_select_validation():
    d = B.dims(2, 8, 2, 64)
    bt = B.Batch([0, 100, 300])
    good = B.kept_offsets_for(bt, 0.25, 0)

    def sel(rule=0, ratio=0.25, budget=0, ko=good, kept=FAKE, s_out=FAKE, ws=None, wsb=0):
        return lib.tp_combine_select_topk(ctypes.byref(d), ctypes.byref(bt.c), FAKE, FAKE, rule, ratio, budget,
                                          B._i64_array(ko), kept, s_out, ws, wsb, None)

    assert sel(rule=4) == B.TP_ERR_PARAM
    assert sel(ratio=0.25, budget=10) == B.TP_ERR_PARAM
    assert sel(ratio=0.0, budget=0) == B.TP_ERR_PARAM
    assert sel(ratio=1.5) == B.TP_ERR_PARAM
    assert sel(ko=[0, 25, 74]) == B.TP_ERR_SHAPE
    assert sel(ko=[1, 26, 76]) == B.TP_ERR_SHAPE
    assert sel(kept=None) == B.TP_ERR_NULL
    assert sel(s_out=None) == B.TP_ERR_WORKSPACE  # no s_out and no workspace
    assert sel() == B.TP_ERR_WORKSPACE  # the workspace is required with s_out too
    ws = B.tp_workspace_size(B.TP_FN_COMBINE_SELECT_TOPK, d, bt)
    assert sel(ws=FAKE, wsb=ws - 1) == B.TP_ERR_WORKSPACE
    assert sel(ws=FAKE + 16, wsb=ws) == B.TP_ERR_WORKSPACE  # not 256-byte aligned


@no_gpu
def test_select_static_validation():
    """The no-allocation selection validates like tp_combine_select_topk and rejects, before
    any GPU call, a call whose combined scores exceed the static buffer."""
    assert B.TP_STATIC_SCRATCH_BYTES == 64 << 20

    def sel(d, bt, ko, rule=0, ratio=0.25, budget=0, kept=FAKE):
        return lib.tp_combine_select_topk_static(ctypes.byref(d), ctypes.byref(bt.c), FAKE, FAKE, rule, ratio, budget,
                                                 B._i64_array(ko), kept, None)

    d = B.dims(2, 8, 2, 64)
    bt = B.Batch([0, 100, 300])
    good = B.kept_offsets_for(bt, 0.25, 0)
    assert sel(d, bt, good, rule=4) == B.TP_ERR_PARAM
    assert sel(d, bt, good, ratio=0.25, budget=10) == B.TP_ERR_PARAM
    assert sel(d, bt, [0, 25, 74]) == B.TP_ERR_SHAPE
    assert sel(d, bt, good, kept=None) == B.TP_ERR_NULL
    # past the limit: the combined scores alone take 2^26 + 4 bytes
    d1 = B.dims(1, 1, 1, 64)
    n = (64 << 20) // 4 + 1
    bt1 = B.Batch([0, n])
    assert sel(d1, bt1, B.kept_offsets_for(bt1, 0.5, 0), ratio=0.5) == B.TP_ERR_WORKSPACE
    assert "static buffer" in lib.tp_last_error().decode()


@no_gpu
def test_guide_attention_validation():
    d = B.dims(2, 8, 2, 64)
    bt = B.Batch([0, 100, 300], [0, 16, 20])
    ws = B.tp_workspace_size(B.TP_FN_GUIDE_ATTENTION, d, bt)
    # at least a partial (max, sum) and output per guide row and slot (one chunk and the guide keys)
    assert ws >= 2 * 8 * 20 * 2 * (8 + 64 * 4)

    def att(q=FAKE, k=FAKE, v=FAKE, kg=None, vg=None, scale=0.125, o_=FAKE, lse=FAKE, w=FAKE, wsb=ws, batch=bt):
        return lib.tp_guide_attention(ctypes.byref(d), ctypes.byref(batch.c), q, k, v, kg, vg, scale, o_, lse, w,
                                      wsb, None)

    assert att(v=None) == B.TP_ERR_NULL
    assert att(lse=None) == B.TP_ERR_NULL
    assert att(kg=FAKE) == B.TP_ERR_NULL        # guide keys without their values
    assert att(vg=FAKE) == B.TP_ERR_NULL
    assert att(o_=FAKE + 4) == B.TP_ERR_PARAM   # not 16-byte aligned
    assert att(lse=FAKE + 2) == B.TP_ERR_PARAM
    assert att(scale=0.0) == B.TP_ERR_PARAM
    assert att(w=None) == B.TP_ERR_WORKSPACE
    assert att(wsb=ws - 1) == B.TP_ERR_WORKSPACE
    assert att(w=FAKE + 16) == B.TP_ERR_WORKSPACE
    assert att(batch=B.Batch([0, 100, 300])) == B.TP_ERR_NULL  # guide offsets required


@no_gpu
def test_guide_attention_quantize_validation():
    d = B.dims(2, 8, 2, 64)
    bt = B.Batch([0, 100, 300], [0, 16, 20])
    ws = B.tp_workspace_size(B.TP_FN_GUIDE_ATTENTION, d, bt)

    def attq(q=FAKE, k=FAKE, v=FAKE, kg=None, vg=None, scale=0.125, fmt=0, bits=8, o_=FAKE, lse=FAKE, sc=FAKE,
             vq=FAKE, w=FAKE, wsb=ws, batch=bt):
        return lib.tp_guide_attention_quantize(ctypes.byref(d), ctypes.byref(batch.c), q, k, v, kg, vg, scale, fmt,
                                               bits, o_, lse, sc, vq, w, wsb, None)

    assert attq(v=None) == B.TP_ERR_NULL
    assert attq(sc=None) == B.TP_ERR_NULL
    assert attq(vq=None) == B.TP_ERR_NULL       # the codes are always written
    assert attq(lse=None) == B.TP_ERR_NULL
    assert attq(kg=FAKE) == B.TP_ERR_NULL
    assert attq(fmt=3) == B.TP_ERR_PARAM
    assert attq(bits=1) == B.TP_ERR_PARAM
    assert attq(bits=9) == B.TP_ERR_PARAM
    assert attq(sc=FAKE + 4) == B.TP_ERR_PARAM
    assert attq(vq=FAKE + 8) == B.TP_ERR_PARAM
    assert attq(scale=-1.0) == B.TP_ERR_PARAM
    assert attq(wsb=ws - 1) == B.TP_ERR_WORKSPACE
    assert attq(batch=B.Batch([0, 100, 300])) == B.TP_ERR_NULL
    assert lib.tp_last_error().decode() != ""


@no_gpu
def test_compact_validation():
    d = B.dims(2, 8, 2, 64)
    bt = B.Batch([0, 100, 300])

    def cp(ko=(0, 25, 75), vq=FAKE, vqo=FAKE, sc=FAKE, sco=FAKE, fmt=0, bits=8):
        return lib.tp_compact_kv(ctypes.byref(d), ctypes.byref(bt.c), B._i64_array(ko), FAKE, FAKE, vq, sc, fmt, bits,
                                 FAKE, vqo, sco, None)

    assert cp(ko=(0, 101, 150)) == B.TP_ERR_SHAPE  # more kept than tokens
    assert cp(ko=(0, 30, 20)) == B.TP_ERR_SHAPE
    assert cp(vq=None) == B.TP_ERR_NULL
    assert cp(sco=None) == B.TP_ERR_NULL
    assert cp(bits=0) == B.TP_ERR_PARAM


def _ev(d, bt, **kw):
    a = dict(q=FAKE, k=FAKE, kg=None, lse=None, v=FAKE, scale=0.125, pool=5, qfmt=0, bits=8, rule=0, ratio=0.25, budget=0,
             ko=None, skey=FAKE, sc=FAKE, vq=FAKE, sout=FAKE, idx=FAKE, kout=FAKE, vqout=FAKE, scout=FAKE,
             ws=FAKE, wsb=1 << 40, prof=None)
    a.update(kw)
    if a["ko"] is None:
        a["ko"] = B.kept_offsets_for(bt, a["ratio"], a["budget"])
    ko = (ctypes.c_int64 * len(a["ko"]))(*a["ko"])
    prof = ctypes.byref(a["prof"]) if a["prof"] is not None else None
    return lib.tp_evict(ctypes.byref(d), ctypes.byref(bt.c), a["q"], a["k"], a["kg"], a["lse"], a["v"], a["scale"],
                        a["pool"],
                        a["qfmt"], a["bits"], a["rule"], a["ratio"], a["budget"], ko, a["skey"], a["sc"], a["vq"],
                        a["sout"], a["idx"], a["kout"], a["vqout"], a["scout"], a["ws"], a["wsb"], prof, None)


@no_gpu
def test_evict_validation():
    d = B.dims(2, 8, 2, 64)
    bt = B.Batch([0, 100, 300], [0, 16, 20])
    short_prof = B.TpProfile(3)
    null_prof = B.TpProfile(B.TP_EVICT_EVENTS)
    cases = [
        (dict(q=None), B.TP_ERR_NULL),
        # v = NULL: step 2 done beforehand, scales and codes are inputs and must be given
        (dict(v=None, vq=None), B.TP_ERR_NULL),
        (dict(v=None, vq=None, vqout=None), B.TP_ERR_NULL),
        (dict(v=None, sc=None), B.TP_ERR_NULL),
        (dict(v=None, vq=FAKE + 4), B.TP_ERR_PARAM),
        (dict(v=None, bits=9), B.TP_ERR_PARAM),
        (dict(v=None, qfmt=5), B.TP_ERR_PARAM),
        (dict(vq=None, vqout=None), B.TP_ERR_NULL),  # without v_q the kept rows are quantised: v_q_out needed
        (dict(vq=None, scout=None), B.TP_ERR_NULL),
        (dict(idx=None), B.TP_ERR_NULL),
        (dict(kout=None), B.TP_ERR_NULL),
        (dict(vqout=None), B.TP_ERR_NULL),
        (dict(scale=0.0), B.TP_ERR_PARAM),
        (dict(pool=2), B.TP_ERR_PARAM),
        (dict(qfmt=5), B.TP_ERR_PARAM),
        (dict(bits=9), B.TP_ERR_PARAM),
        (dict(rule=7), B.TP_ERR_PARAM),
        (dict(ratio=0.0, budget=0, ko=[0, 1, 2]), B.TP_ERR_PARAM),
        (dict(ko=[0, 25, 51]), B.TP_ERR_SHAPE),
        (dict(ws=None), B.TP_ERR_WORKSPACE),
        (dict(wsb=1024), B.TP_ERR_WORKSPACE),
        (dict(sout=None, wsb=B.tp_workspace_size(B.TP_FN_GUIDE_SCORES, d, bt)), B.TP_ERR_WORKSPACE),
        (dict(wsb=B.tp_workspace_size(B.TP_FN_EVICT, d, bt) - 1), B.TP_ERR_WORKSPACE),
        (dict(prof=short_prof), B.TP_ERR_PARAM),
        (dict(prof=null_prof), B.TP_ERR_NULL),
        (dict(k=FAKE + 8), B.TP_ERR_PARAM),
        (dict(kg=FAKE + 4), B.TP_ERR_PARAM),
        (dict(kg=FAKE, lse=FAKE), B.TP_ERR_PARAM),  # exclusive normaliser sources
        (dict(lse=FAKE + 2), B.TP_ERR_PARAM),
    ]
    for kw, want in cases:
        assert _ev(d, bt, **kw) == want, kw
        assert lib.tp_last_error().decode() != ""
    assert _ev(d, B.Batch([0, 100, 300])) == B.TP_ERR_NULL  # the score step needs guide offsets
    assert _ev(B.dims(2, 8, 2, 96), bt) == B.TP_ERR_UNSUPPORTED


def test_evict_workspace_size():
    d = B.dims(32, 32, 8, 128)
    bt = B.Batch([0, 131072], [0, 64])
    g = B.tp_workspace_size(B.TP_FN_GUIDE_SCORES, d, bt)
    s = B.tp_workspace_size(B.TP_FN_COMBINE_SELECT_TOPK, d, bt)
    assert B.tp_workspace_size(B.TP_FN_EVICT, d, bt) == g + s
    with pytest.raises(B.TaskPressError):
        B.tp_workspace_size(B.TP_FN_EVICT, d, B.Batch([0, 131072]))


def test_missing_library_fails_loudly(monkeypatch):
    """Without the built library the binding raises instead of falling back to anything."""
    monkeypatch.setattr(B, "_lib", None)
    monkeypatch.setattr(B, "LIB_PATH", os.path.join(ROOT, "no-such-dir", "libtaskpress.so"))
    with pytest.raises(ImportError, match="is missing"):
        B.load()
