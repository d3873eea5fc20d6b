"""Host-only checks of the C-ABI library: it loads, exports every symbol the
header declares, and its argument checking and model parsing work without
touching a GPU."""
import ctypes
import os
import re

import pytest

import paper_2111_00352_amd as gs
from conftest import ROOT

HEADER = os.path.join(ROOT, "include", "gnnspmm.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gs_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(gs.library_path()):
        from paper_2111_00352_amd import build
        build.build()
    return gs.lib()


def test_exports_every_declared_symbol(L):
    names = _declared()
    assert len(names) >= 18
    for n in names:
        assert hasattr(L, n), n


def test_abi_version_matches_header(L):
    m = re.search(r"#define GS_ABI_VERSION (\d+)", open(HEADER).read())
    assert L.gs_abi_version() == int(m.group(1))


def test_null_arguments_rejected_without_gpu(L):
    out = ctypes.c_void_p(123)
    assert L.gs_build_format(None, 1, None, None, ctypes.byref(out), None) == gs.ERR_INVALID_ARG
    assert out.value is None
    assert b"gs_coo" in L.gs_last_error()
    assert L.gs_spmm(None, None, 1, None, 1, 1, None) == gs.ERR_INVALID_ARG
    assert L.gs_spmm_noalloc(None, None, 1, None, 1, 1, None) == gs.ERR_INVALID_ARG
    assert L.gs_to_coo(None, None, None, None, None) == gs.ERR_INVALID_ARG
    assert L.gs_get_info(None, None) == gs.ERR_INVALID_ARG
    coo = gs._Coo(4, 4, 1, None, None, None)  # nnz > 0 with null arrays
    assert L.gs_build_format(ctypes.byref(coo), 1, None, None, ctypes.byref(out), None) == gs.ERR_INVALID_ARG
    coo = gs._Coo(-1, 4, 0, None, None, None)
    assert L.gs_build_format(ctypes.byref(coo), 1, None, None, ctypes.byref(out), None) == gs.ERR_INVALID_ARG
    coo = gs._Coo(1 << 31, 4, 0, None, None, None)
    assert L.gs_build_format(ctypes.byref(coo), 1, None, None, ctypes.byref(out), None) == gs.ERR_UNSUPPORTED
    coo = gs._Coo(4, 4, 0, None, None, None)
    assert L.gs_build_format(ctypes.byref(coo), 7, None, None, ctypes.byref(out), None) == gs.ERR_INVALID_ARG
    bad = gs._BuildOpts(65, 0, 0)
    assert L.gs_build_format(ctypes.byref(coo), 4, ctypes.byref(bad), None, ctypes.byref(out), None) == gs.ERR_INVALID_ARG


def _ctx(L, **kw):
    o = gs._SelOpts(kw.get("mode", 0), kw.get("fixed", 1), kw.get("path"), 0, kw.get("b", 16), 3, 0,
                    kw.get("mem_weight", 0.0))
    h = ctypes.c_void_p()
    rc = L.gs_ctx_create(ctypes.byref(o), ctypes.byref(h))
    return rc, h


def test_context_creation_and_builtin_model(L):
    rc, h = _ctx(L)
    assert rc == 0 and h.value
    st = gs._SelStats()
    assert L.gs_ctx_stats(h, ctypes.byref(st)) == 0
    L.gs_ctx_destroy(h)
    assert _ctx(L, mode=5)[0] == gs.ERR_INVALID_ARG
    assert _ctx(L, fixed=9)[0] == gs.ERR_INVALID_ARG
    assert _ctx(L, b=0)[0] == 0
    assert _ctx(L, b=99)[0] == gs.ERR_INVALID_ARG


MODEL_OK = """GSMODEL 1
nfeat 21
classes 2 1 3
min """ + " ".join(["0"] * 21) + """
max """ + " ".join(["1"] * 21) + """
base 0.5 0
ntrees 1
tree 1 3
12 0.9 1 2 0
-1 0 0 0 0
-1 0 0 0 1
"""


# the same model in version 2: hexadecimal reals, "L value" leaves
MODEL_OK_V2 = """GSMODEL 2
nfeat 21
classes 2 1 3
min """ + " ".join(["0x0.0p+0"] * 21) + """
max """ + " ".join(["0x1.0000000000000p+0"] * 21) + """
base 0x1.0000000000000p-1 0x0.0p+0
ntrees 1
tree 1 3
12 0x1.ccccccccccccdp-1 1 2
L 0x0.0p+0
L 0x1.0000000000000p+0
"""


@pytest.mark.parametrize("text,code", [
    (MODEL_OK, 0),
    (MODEL_OK_V2, 0),
    (MODEL_OK_V2.replace("0x1.ccccccccccccdp-1", "0.9"), gs.ERR_MODEL),            # decimal in version 2
    (MODEL_OK_V2.replace("0x1.ccccccccccccdp-1", "0x1.ccgp-1"), gs.ERR_MODEL),     # not a hex digit
    (MODEL_OK_V2.replace("0x1.ccccccccccccdp-1", "0x1.ccccccccccccdep-1"), gs.ERR_MODEL),  # 57 bits
    (MODEL_OK_V2.replace("L 0x1.0000000000000p+0", "L"), gs.ERR_MODEL),            # leaf without value
    (MODEL_OK_V2.replace("L 0x0.0p+0", "-1 0x0.0p+0 0 0"), gs.ERR_MODEL),         # leaf not marked
    ("", gs.ERR_MODEL),
    ("GSMODEL 2\n", gs.ERR_MODEL),
    (MODEL_OK.replace("nfeat 21", "nfeat 20"), gs.ERR_MODEL),
    (MODEL_OK.replace("classes 2 1 3", "classes 2 1 9"), gs.ERR_MODEL),
    (MODEL_OK.replace("12 0.9 1 2 0", "12 0.9 0 2 0"), gs.ERR_MODEL),   # child not after parent
    (MODEL_OK.replace("12 0.9 1 2 0", "30 0.9 1 2 0"), gs.ERR_MODEL),   # feature index
    (MODEL_OK.replace("tree 1 3", "tree 1 4"), gs.ERR_MODEL),           # short node list
])
def test_model_file_parsing(L, tmp_path, text, code):
    p = tmp_path / "m.gsm"
    p.write_text(text)
    rc, h = _ctx(L, path=str(p).encode())
    assert rc == code, L.gs_last_error()
    if rc == 0:
        L.gs_ctx_destroy(h)


def test_missing_model_file(L, tmp_path):
    rc, _ = _ctx(L, path=str(tmp_path / "absent.gsm").encode())
    assert rc == gs.ERR_MODEL
    # the profiling and fixed selectors never read a model
    for mode in (1, 2):
        rc, h = _ctx(L, mode=mode, path=str(tmp_path / "absent.gsm").encode())
        assert rc == 0, L.gs_last_error()
        L.gs_ctx_destroy(h)


def test_allocator_hooks_must_be_paired(L):
    a = gs._Allocator(gs._ALLOC_FN(lambda n, s, c: None), gs._FREE_FN(), None)
    assert L.gs_set_allocator(ctypes.byref(a)) == gs.ERR_INVALID_ARG
    assert L.gs_set_allocator(None) == 0


def test_shipped_trained_model_parses(L):
    from paper_2111_00352_amd.selector import MODEL_PATH
    assert os.path.exists(MODEL_PATH)
    rc, h = _ctx(L, path=MODEL_PATH.encode())
    assert rc == 0, L.gs_last_error()
    L.gs_ctx_destroy(h)


def test_trained_model_export_matches_sklearn(tmp_path):
    # re-train on the shipped profile data and check the exported trees
    # predict exactly what scikit-learn predicts (the library walks them)
    import numpy as np
    from paper_2111_00352_amd.selector import DATA_PATH, train
    X, T, groups, kinds = train.load(DATA_PATH)
    y = train.labels(T)
    mn, mx = X.min(axis=0), X.max(axis=0)
    Xn = train.normalise(X, mn, mx)
    clf = train.fit(Xn, y)
    trees, base, classes = train.export(clf, mn, mx, str(tmp_path / "m.gsm"))
    S = train.score_exported(trees, base, Xn)
    assert (np.array([classes[i] for i in S.argmax(axis=1)]) == clf.predict(Xn)).all()


def test_model_trained_for_a_weight_of_eq1(L, tmp_path):
    # a model trained on Eq. 1 labels for w = 0.25 records its w; a context
    # accepts it only with mem_weight = 0.75
    from paper_2111_00352_amd.selector import DATA_PATH, train
    X, T, _, _ = train.load(DATA_PATH)
    y = train.labels_eq1(T, train.footprints(DATA_PATH), 0.25)
    mn, mx = X.min(axis=0), X.max(axis=0)
    clf = train.fit(train.normalise(X, mn, mx), y)
    path = tmp_path / "w.gsm"
    train.export(clf, mn, mx, str(path), w=0.25)
    assert open(path).read().splitlines()[-1] == "w " + (0.25).hex()
    for mw, want in ((0.75, 0), (0.0, gs.ERR_MODEL), (0.5, gs.ERR_MODEL)):
        rc, h = _ctx(L, path=str(path).encode(), mem_weight=mw)
        assert rc == want, mw
        if rc == 0:
            L.gs_ctx_destroy(h)


def test_memory_weight_of_eq1(L, tmp_path):
    # mem_weight = 1 - w of Eq. 1: checked for [0, 1]; PROFILE takes any
    # weight; MODEL only the w its model file was trained for ("w" line, 1
    # when absent)
    for bad in (-0.1, 1.5, float("nan")):
        assert _ctx(L, mem_weight=bad)[0] == gs.ERR_INVALID_ARG
    rc, h = _ctx(L, mode=1, mem_weight=0.7)
    assert rc == 0
    L.gs_ctx_destroy(h)
    assert _ctx(L, mem_weight=0.5)[0] == gs.ERR_MODEL  # built-in model: w = 1
    from paper_2111_00352_amd.selector import MODEL_PATH
    text = open(MODEL_PATH).read()
    for line, mw, want in (("w 0x1.0000000000000p-1", 0.5, 0), ("w 0x1.0000000000000p-1", 0.0, gs.ERR_MODEL),
                           ("w 0x0.0p+0", 1.0, 0), ("w 0x1.8p+1", 0.0, gs.ERR_MODEL), ("w", 0.0, gs.ERR_MODEL)):
        p = tmp_path / "w.gsm"
        p.write_text(text + line + "\n")
        rc, h = _ctx(L, path=str(p).encode(), mem_weight=mw)
        assert rc == want, (line, mw)
        if rc == 0:
            L.gs_ctx_destroy(h)


def test_candidate_mask_is_checked(L):
    o = gs._SelOpts(0, 1, None, 0, 16, 3, 1 << 7, 0.0)  # bit 7 names no format
    h = ctypes.c_void_p()
    assert L.gs_ctx_create(ctypes.byref(o), ctypes.byref(h)) == gs.ERR_INVALID_ARG
    o = gs._SelOpts(0, 1, None, 0, 16, 3, (1 << 1) | (1 << 5), 0.0)  # CSR and CSC only
    assert L.gs_ctx_create(ctypes.byref(o), ctypes.byref(h)) == 0
    L.gs_ctx_destroy(h)


def test_eq1_labels_trade_time_for_memory():
    # Eq. 1 over min-max scaled time and memory: w = 1 picks the fastest
    # format, w = 0 the smallest, an infeasible (inf time) format never wins,
    # and near-equal objectives go to the earliest format in the tie order
    import numpy as np
    from paper_2111_00352_amd.selector import train
    inf = np.inf
    T = np.array([[2.0, 1.0, 3.0, inf, 4.0],     # fastest: coo (index 1)
                  [1.0, 1.0, 5.0, 6.0, 7.0]])    # csr and coo tie on time
    M = np.array([[5.0, 9.0, 1.0, 0.5, 8.0],     # smallest feasible: ell (the inf-time dia is out)
                  [3.0, 3.0, 9.0, 9.0, 9.0]])
    assert train.labels_eq1(T, M, 1.0).tolist() == [1, 0]
    assert train.labels_eq1(T, M, 0.0).tolist() == [2, 0]
    mid = train.labels_eq1(T, M, 0.5).tolist()
    assert mid[1] == 0 and mid[0] in (0, 1, 2)


def test_footprints_match_the_library_sizes():
    # M of Eq. 1 on the shipped profiles: the CSR and COO sizes follow from
    # the row and entry counts alone
    import numpy as np
    from paper_2111_00352_amd.selector import DATA_PATH, train
    M = train.footprints(DATA_PATH)
    assert M.shape[1] == 5 and np.all(M[:, 0] > 0)
    X, T, _, _ = train.load(DATA_PATH)
    R, Z = X[:, 0], X[:, 2]
    assert np.allclose(M[:, 0], 4 * (R + 1) + 8 * Z) and np.allclose(M[:, 1], 12 * Z)


def test_set_allocator_keeps_hooks_alive(L):
    # the binding keeps every installed hook set referenced: the caller may
    # drop its own callables at once, and a handle built with them can still
    # free its buffers through them later (no GPU needed: nothing allocates)
    import gc
    import weakref

    class Hook:
        def __call__(self, *args):
            return None

    a, f = Hook(), Hook()
    wa, wf = weakref.ref(a), weakref.ref(f)
    gs.set_allocator(a, f)
    del a, f
    gc.collect()
    assert wa() is not None and wf() is not None
    assert any(h[3] is wa() for h in gs._hooks_alive)
    with pytest.raises(ValueError):
        gs.set_allocator(lambda n, s: 0)
    gs.set_allocator()  # back to PyTorch's caching allocator
    assert gs._alloc_keep is not None
    gc.collect()
    assert wa() is not None  # still kept after the switch
