"""The C ABI library: exports and host-side argument validation (no GPU needed).

Every call here is rejected on the host before any device work, so it runs on
a machine without a GPU. Codes and conditions are those documented in
include/routebalance.h.
"""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2606_17949_amd as rb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "routebalance.h")
L = rb._lib
FAKE = ctypes.c_void_p(0x10000)        # never dereferenced: validation fails first
MISALIGNED = ctypes.c_void_p(0x10004)


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rb_[a-z_]+)\s*\(", text)))


def test_header_declares_and_library_exports_every_entry_point():
    decl = declared_functions()
    assert set(decl) == set(rb.EXPORTS), decl
    out = subprocess.run(["nm", "-D", "--defined-only", rb.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    syms = {line.split()[-1] for line in out.splitlines() if line.strip()}
    for name in decl:
        assert name in syms, f"{name} not exported"
        assert hasattr(L, name)


def test_status_strings():
    for code in range(-9, 1):
        assert rb.rb_status_string(code).startswith("RB_")
    assert "unknown" in rb.rb_status_string(5)


def test_header_constants_match_binding():
    text = open(HEADER).read()
    for name in ("RB_MAX_K", "RB_MAX_D", "RB_MAX_I", "RB_MAX_M"):
        v = int(re.search(rf"#define {name} (\d+)", text).group(1))
        assert v == getattr(rb, name)


def knn(q=FAKE, x=FAKE, norms=FAKE, dt=rb.RB_BF16, B=4, N=100, d=64, k=10, idx=FAKE, dist=None,
        ws=FAKE, ws_bytes=1 << 20):
    return L.rb_knn_topk(q, x, norms, dt, B, N, d, k, idx, dist, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,code", [
    (dict(k=0), rb.RB_ERR_DIMS), (dict(k=101), rb.RB_ERR_DIMS), (dict(k=65, N=1000), rb.RB_ERR_DIMS),
    (dict(B=-1), rb.RB_ERR_DIMS), (dict(N=0), rb.RB_ERR_DIMS), (dict(d=0), rb.RB_ERR_DIMS),
    (dict(d=60), rb.RB_ERR_DIMS), (dict(d=2056), rb.RB_ERR_DIMS),
    (dict(dt=rb.RB_F32, d=6), rb.RB_ERR_DIMS), (dict(dt=7), rb.RB_ERR_DTYPE),
    (dict(q=None), rb.RB_ERR_NULL), (dict(x=None), rb.RB_ERR_NULL), (dict(norms=None), rb.RB_ERR_NULL),
    (dict(idx=None), rb.RB_ERR_NULL), (dict(q=MISALIGNED), rb.RB_ERR_ALIGN),
    (dict(x=MISALIGNED), rb.RB_ERR_ALIGN),
])
def test_knn_validation(kw, code):
    assert knn(**kw) == code


def test_knn_empty_batch_is_a_no_op():
    assert knn(B=0, q=None, idx=None, ws=None, ws_bytes=0) == rb.RB_OK


def test_workspace_size_validation():
    n = ctypes.c_size_t(0)
    assert L.rb_workspace_size(4, 100, 64, rb.RB_BF16, 10, 4, None) == rb.RB_ERR_NULL
    assert L.rb_workspace_size(4, 100, 64, rb.RB_BF16, 0, 4, ctypes.byref(n)) == rb.RB_ERR_DIMS
    assert L.rb_workspace_size(4, 100, 64, rb.RB_BF16, 10, 0, ctypes.byref(n)) == rb.RB_ERR_DIMS
    assert L.rb_workspace_size(4, 100, 64, 3, 10, 4, ctypes.byref(n)) == rb.RB_ERR_DTYPE


def test_bank_norms_validation():
    assert L.rb_bank_norms(FAKE, rb.RB_BF16, 0, 64, FAKE, None) == rb.RB_ERR_DIMS
    assert L.rb_bank_norms(FAKE, rb.RB_BF16, 10, 12, FAKE, None) == rb.RB_ERR_DIMS
    assert L.rb_bank_norms(None, rb.RB_BF16, 10, 64, FAKE, None) == rb.RB_ERR_NULL
    assert L.rb_bank_norms(FAKE, rb.RB_BF16, 10, 64, None, None) == rb.RB_ERR_NULL
    assert L.rb_bank_norms(MISALIGNED, rb.RB_BF16, 10, 64, FAKE, None) == rb.RB_ERR_ALIGN
    assert L.rb_bank_norms(FAKE, 9, 10, 64, FAKE, None) == rb.RB_ERR_DTYPE


def test_predict_validation():
    args = lambda **kw: (kw.get("nbr", FAKE), None, kw.get("B", 4), kw.get("k", 10),
                         kw.get("wt", rb.RB_KNN_UNIFORM), kw.get("qual", FAKE), FAKE,
                         kw.get("N", 100), kw.get("M", 4), FAKE, FAKE, None)
    assert L.rb_predict(*args(wt=2)) == rb.RB_ERR_UNSUPPORTED
    assert L.rb_predict(*args(wt=rb.RB_KNN_INV_DIST)) == rb.RB_ERR_NULL   # needs nbr_dist
    assert L.rb_predict(*args(k=0)) == rb.RB_ERR_DIMS
    assert L.rb_predict(*args(k=65)) == rb.RB_ERR_DIMS
    assert L.rb_predict(*args(M=0)) == rb.RB_ERR_DIMS
    assert L.rb_predict(*args(nbr=None)) == rb.RB_ERR_NULL
    assert L.rb_predict(*args(qual=None)) == rb.RB_ERR_NULL
    assert L.rb_predict(*args(B=0, nbr=None)) == rb.RB_OK


def _inst(**kw):
    s = rb.rb_instances(*[FAKE] * 7)
    for f, v in kw.items():
        setattr(s, f, v)
    return s


W = rb.rb_weights(0.4, 0.3, 0.3)


@pytest.mark.parametrize("w", [(0.5, 0.5, 0.5), (-0.1, 0.6, 0.5), (float("nan"), 0.5, 0.5),
                               (float("inf"), 0, 0), (0.2, 0.2, 0.2)])
def test_score_and_assign_reject_off_simplex_weights(w):
    s = _inst()
    ww = rb.rb_weights(*w)
    assert L.rb_score(FAKE, FAKE, FAKE, 4, 4, ctypes.byref(s), 13, ww, FAKE, None) == rb.RB_ERR_WEIGHTS
    assert L.rb_assign(FAKE, FAKE, FAKE, 4, 4, ctypes.byref(s), 13, ww, FAKE, None, None,
                       None) == \
        rb.RB_ERR_WEIGHTS


def test_weights_accept_float32_thirds_and_corners():
    s = _inst()
    third = ctypes.c_float(1 / 3).value
    for w in [(third, third, third), (1, 0, 0), (0, 1, 0), (0, 0, 1)]:
        # B = 0 passes every check and enqueues nothing
        assert L.rb_score(None, None, None, 0, 4, ctypes.byref(s), 13, rb.rb_weights(*w), None,
                          None) == rb.RB_OK


def test_score_assign_instance_validation():
    assert L.rb_score(FAKE, FAKE, FAKE, 4, 4, None, 13, W, FAKE, None) == rb.RB_ERR_NULL
    for f in rb.DeviceInstances.FIELDS:
        s = _inst(**{f: None})
        assert L.rb_assign(FAKE, FAKE, FAKE, 4, 4, ctypes.byref(s), 13, W, FAKE, None, None,
                           None) == \
            rb.RB_ERR_NULL, f
    s = _inst()
    assert L.rb_score(FAKE, FAKE, FAKE, 4, 4, ctypes.byref(s), 0, W, FAKE, None) == rb.RB_ERR_DIMS
    assert L.rb_score(FAKE, FAKE, FAKE, 4, 4, ctypes.byref(s), 1025, W, FAKE, None) == \
        rb.RB_ERR_DIMS
    assert L.rb_score(FAKE, FAKE, FAKE, 4, 0, ctypes.byref(s), 13, W, FAKE, None) == rb.RB_ERR_DIMS
    assert L.rb_assign(FAKE, FAKE, FAKE, 4, 4, ctypes.byref(s), 13, W, None, None, None,
                       None) == \
        rb.RB_ERR_NULL


def test_route_batch_validation():
    s = _inst()

    def call(**kw):
        a = dict(q=FAKE, x=FAKE, n=FAKE, dt=rb.RB_BF16, B=4, N=100, d=64, k=10, qual=FAKE,
                 ln=FAKE, M=4, pl=FAKE, inst=ctypes.byref(s), I=13, w=W, asg=FAKE)
        a.update(kw)
        return L.rb_route_batch(a["q"], a["x"], a["n"], a["dt"], a["B"], a["N"], a["d"], a["k"],
                                a["qual"], a["ln"], a["M"], a["pl"], a["inst"], a["I"], a["w"],
                                a["asg"], None, None, None, None, None, None, FAKE, 1 << 20, None)
    assert call(k=11, N=10) == rb.RB_ERR_DIMS
    assert call(M=0) == rb.RB_ERR_DIMS
    assert call(I=0) == rb.RB_ERR_DIMS
    assert call(w=rb.rb_weights(1, 1, 0)) == rb.RB_ERR_WEIGHTS
    assert call(asg=None) == rb.RB_ERR_NULL
    assert call(qual=None) == rb.RB_ERR_NULL
    assert call(inst=None) == rb.RB_ERR_NULL
    assert call(q=MISALIGNED) == rb.RB_ERR_ALIGN
    assert call(B=0, q=None, asg=None, pl=None) == rb.RB_OK


def test_assign_ex_validation():
    s = _inst()

    def call(opts=None, **kw):
        a = dict(q=FAKE, B=4, M=4, inst=ctypes.byref(s), I=13, w=W, asg=FAKE)
        a.update(kw)
        o = None if opts is None else ctypes.byref(opts)
        return L.rb_assign_ex(a["q"], FAKE, FAKE, a["B"], a["M"], a["inst"], a["I"], a["w"], o,
                              a["asg"], None, None, None)
    assert call(rb.rb_options(2, 0, None, None, None)) == rb.RB_ERR_UNSUPPORTED
    assert call(rb.rb_options(0, 5, None, None, None)) == rb.RB_ERR_UNSUPPORTED
    assert call(rb.rb_options(-1, 0, None, None, None)) == rb.RB_ERR_UNSUPPORTED
    assert call(rb.rb_options(0, 0, None, None, None, rb.RB_FLAG_FROM_LISTS)) == \
        rb.RB_ERR_UNSUPPORTED   # a flag of rb_knn_predict only
    # LPT needs order_out
    assert call(rb.rb_options(rb.RB_ORDER_LPT, 0, None, None, None)) == rb.RB_ERR_NULL
    assert call(rb.rb_options(0, 0, None, None, None), asg=None) == rb.RB_ERR_NULL
    assert call(None, M=0) == rb.RB_ERR_DIMS
    assert call(None, I=1025) == rb.RB_ERR_DIMS
    assert call(None, w=rb.rb_weights(1, 1, 0)) == rb.RB_ERR_WEIGHTS
    assert call(rb.rb_options(rb.RB_ORDER_LPT, 0, None, None, None), B=0, q=None,
                asg=None) == rb.RB_OK


def test_route_batch_ex_validation():
    s = _inst()

    def call(opts, **kw):
        a = dict(q=FAKE, B=4, asg=FAKE)
        a.update(kw)
        return L.rb_route_batch_ex(a["q"], FAKE, FAKE, rb.RB_BF16, a["B"], 100, 64, 10, FAKE, FAKE,
                                   4, FAKE, ctypes.byref(s), 13, W,
                                   None if opts is None else ctypes.byref(opts), a["asg"], None,
                                   None, None, None, None, None, FAKE, 1 << 20, None)
    assert call(rb.rb_options(3, 0, None, None, None)) == rb.RB_ERR_UNSUPPORTED
    assert call(rb.rb_options(0, 3, None, None, None)) == rb.RB_ERR_UNSUPPORTED
    # the split-lookup flags belong to rb_knn_predict only
    for f in (rb.RB_FLAG_LISTS_ONLY, rb.RB_FLAG_FROM_LISTS):
        assert call(rb.rb_options(0, 0, None, None, None, f)) == rb.RB_ERR_UNSUPPORTED
    assert call(None, asg=None) == rb.RB_ERR_NULL
    assert call(None, q=MISALIGNED) == rb.RB_ERR_ALIGN
    assert call(rb.rb_options(rb.RB_ORDER_LPT, rb.RB_KNN_INV_DIST, None, None, None), B=0, q=None,
                asg=None) == rb.RB_OK


def test_knn_predict_validation():
    def call(opts=None, **kw):
        a = dict(q=FAKE, B=4, N=100, d=64, k=10, M=4, qual=FAKE, qh=FAKE, lh=FAKE, ws=FAKE)
        a.update(kw)
        return L.rb_knn_predict(a["q"], FAKE, FAKE, rb.RB_BF16, a["B"], a["N"], a["d"], a["k"],
                                a["qual"], FAKE, a["M"], None if opts is None else ctypes.byref(opts),
                                None, None, a["qh"], a["lh"], a["ws"], 1 << 20, None)
    assert call(k=0) == rb.RB_ERR_DIMS
    assert call(M=0) == rb.RB_ERR_DIMS
    assert call(d=60) == rb.RB_ERR_DIMS
    assert call(qh=None) == rb.RB_ERR_NULL
    assert call(lh=None) == rb.RB_ERR_NULL
    assert call(qual=None) == rb.RB_ERR_NULL
    assert call(q=MISALIGNED) == rb.RB_ERR_ALIGN
    assert call(rb.rb_options(0, 2, None, None, None, 0)) == rb.RB_ERR_UNSUPPORTED
    assert call(rb.rb_options(0, 0, None, None, None, 8)) == rb.RB_ERR_UNSUPPORTED   # unknown flag
    assert call(rb.rb_options(0, 0, None, None, None, rb.RB_FLAG_OVERLAP), B=0, q=None, qh=None,
                lh=None, ws=None) == rb.RB_OK
    # the split lookup: not both halves at once; the scan half needs no outputs,
    # the merge half no queries (both then stop at the device query or, with a
    # device, at the missing workspace: nothing is launched)
    both = rb.RB_FLAG_LISTS_ONLY | rb.RB_FLAG_FROM_LISTS
    assert call(rb.rb_options(0, 0, None, None, None, both)) == rb.RB_ERR_UNSUPPORTED
    lists = rb.rb_options(0, 0, None, None, None, rb.RB_FLAG_LISTS_ONLY)
    merge = rb.rb_options(0, 0, None, None, None, rb.RB_FLAG_FROM_LISTS)
    assert call(lists, q=None) == rb.RB_ERR_NULL
    assert call(merge, qh=None) == rb.RB_ERR_NULL
    assert call(lists, qh=None, lh=None, qual=None, ws=None) in (rb.RB_ERR_HIP,
                                                                 rb.RB_ERR_WORKSPACE)
    assert call(merge, q=None, ws=None) in (rb.RB_ERR_HIP, rb.RB_ERR_WORKSPACE)


def test_struct_layouts_match_the_header(tmp_path):
    # the C compiler's layout of the header's structs against the binding's
    src = tmp_path / "layout.c"
    src.write_text(
        '#include <stdio.h>\n#include <stddef.h>\n#include "routebalance.h"\n'
        'int main(void) {\n'
        '  printf("%zu %zu %zu %zu %zu %zu %zu\\n", sizeof(rb_options),\n'
        '         offsetof(rb_options, weighting), offsetof(rb_options, budget),\n'
        '         offsetof(rb_options, instance_mask), offsetof(rb_options, order_out),\n'
        '         offsetof(rb_options, flags), sizeof(rb_instances));\n'
        '  printf("%zu %zu\\n", sizeof(rb_weights), offsetof(rb_weights, w_cost));\n'
        '  return 0;\n}\n')
    exe = tmp_path / "layout"
    subprocess.check_call(["gcc", "-std=c11", "-I", os.path.dirname(HEADER), "-o", str(exe),
                           str(src)])
    lines = subprocess.run([str(exe)], capture_output=True, text=True,
                           check=True).stdout.split("\n")
    o = rb.rb_options
    assert list(map(int, lines[0].split())) == [ctypes.sizeof(o), o.weighting.offset,
                                                 o.budget.offset, o.instance_mask.offset,
                                                 o.order_out.offset, o.flags.offset,
                                                 ctypes.sizeof(rb.rb_instances)]
    assert list(map(int, lines[1].split())) == [ctypes.sizeof(rb.rb_weights),
                                                 rb.rb_weights.w_cost.offset]


def test_advance_validation():
    s = _inst()
    assert L.rb_advance_state(ctypes.byref(s), 13, -1.0, None) == rb.RB_ERR_DIMS
    assert L.rb_advance_state(ctypes.byref(s), 13, float("nan"), None) == rb.RB_ERR_DIMS
    assert L.rb_advance_state(ctypes.byref(s), 0, 1.0, None) == rb.RB_ERR_DIMS
    assert L.rb_advance_state(None, 13, 1.0, None) == rb.RB_ERR_NULL
