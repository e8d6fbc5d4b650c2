"""Property tests of the list validation in smat_plan_create and smat_merge_plan_create (host only,
no GPU): random tensor lists whose arrays are packed into a small address range, so that partial
overlaps, exact in-place aliases and overlaps across tensors are all common, against a plain pairwise
statement of the rules:

* within a tensor, no two of its arrays may overlap, except the buffer (merge: out) being exactly its
  theta0 (in place, equal dtypes);
* across tensors, an array that some operation writes (theta, the buffer, grad_theta; merge: out) may
  overlap nothing, while read-only arrays (theta0, grad_sim; merge: theta0 and the experts) may share
  memory."""
import ctypes

from hypothesis import given, settings, strategies as st

import paper_2609_33437_amd as smat
from paper_2609_33437_amd import _lib

BASE = 1 << 24
GRID = 64  # arrays start on multiples of this many bytes inside a window a few arrays wide


def overlaps(a, b):
    return a[0] < b[1] and b[0] < a[1]


@st.composite
def plan_lists(draw):
    count = draw(st.integers(1, 3))
    tensors = []
    for _ in range(count):
        n = draw(st.integers(1, 48))
        slot = st.integers(0, 240)
        arrays = {"theta": (draw(slot), 4 * n, True), "theta0": (draw(slot), 2 * n, False),
                  "out": (draw(slot), 2 * n, True), "grad_sim": (draw(slot), 2 * n, False),
                  "grad_theta": (draw(slot), 4 * n, True)}
        if draw(st.booleans()):  # in place: the buffer is theta0
            arrays["out"] = (arrays["theta0"][0], 2 * n, True)
        tensors.append((n, arrays))
    return tensors


def span(arr):
    lo = BASE + arr[0] * GRID
    return lo, lo + arr[1]


def plan_allowed(tensors):
    items = []
    for i, (_, arrays) in enumerate(tensors):
        inplace = arrays["out"][0] == arrays["theta0"][0]
        for name, a in arrays.items():
            if inplace and name == "theta0":
                continue  # held by the buffer
            items.append((i, name, span(a), a[2]))
    for x in range(len(items)):
        for y in range(x + 1, len(items)):
            i, _, sa, wa = items[x]
            j, _, sb, wb = items[y]
            if overlaps(sa, sb) and (i == j or wa or wb):
                return False
    return True


@settings(max_examples=400, deadline=None)
@given(plan_lists())
def test_plan_create_overlap_rules(tensors):
    lib = smat.lib()
    arr = (_lib.smat_tensor_desc * len(tensors))()
    for i, (n, a) in enumerate(tensors):
        d = arr[i]
        d.theta, d.theta0, d.out = span(a["theta"])[0], span(a["theta0"])[0], span(a["out"])[0]
        d.grad_sim, d.grad_theta = span(a["grad_sim"])[0], span(a["grad_theta"])[0]
        d.n, d.tensor_id = n, i
    p = ctypes.c_void_p()
    status = lib.smat_plan_create(arr, len(tensors), _lib.SMAT_BF16, _lib.SMAT_BF16, _lib.SMAT_BF16, 0,
                                  ctypes.byref(p))
    if status == _lib.SMAT_OK:
        assert lib.smat_plan_destroy(p) == 0
    assert status in (_lib.SMAT_OK, _lib.SMAT_ERR_INVALID)
    assert (status == _lib.SMAT_OK) == plan_allowed(tensors)


@st.composite
def merge_lists(draw):
    count = draw(st.integers(1, 3))
    nexp = draw(st.integers(1, 3))
    tensors = []
    for _ in range(count):
        n = draw(st.integers(1, 48))
        slot = st.integers(0, 30)
        t0 = draw(slot)
        out = t0 if draw(st.booleans()) else draw(slot)
        experts = [draw(slot) for _ in range(nexp)]
        tensors.append((n, t0, out, experts))
    return nexp, tensors


def merge_allowed(tensors):
    items = []
    for i, (n, t0, out, experts) in enumerate(tensors):
        items.append((i, "out", span((out, 2 * n)), True))
        if t0 != out:
            items.append((i, "theta0", span((t0, 2 * n)), False))
        items += [(i, f"expert{j}", span((e, 2 * n)), False) for j, e in enumerate(experts)]
    for x in range(len(items)):
        for y in range(x + 1, len(items)):
            i, na, sa, wa = items[x]
            j, nb, sb, wb = items[y]
            if not overlaps(sa, sb):
                continue
            # within a tensor only the output may not overlap its inputs; inputs may share memory
            if wa or wb:
                return False
    return True


@settings(max_examples=400, deadline=None)
@given(merge_lists())
def test_merge_plan_create_overlap_rules(case):
    nexp, tensors = case
    lib = smat.lib()
    D = _lib.smat_merge_desc
    arr = (D * len(tensors))(*[D(span((t0, 2 * n))[0], span((out, 2 * n))[0], n, i, 0, 0)
                               for i, (n, t0, out, _) in enumerate(tensors)])
    ptrs = (ctypes.c_void_p * (len(tensors) * nexp))(*[span((e, 0))[0] for *_, ex in tensors for e in ex])
    p = ctypes.c_void_p()
    status = lib.smat_merge_plan_create(arr, len(tensors), ptrs, nexp, _lib.SMAT_BF16, _lib.SMAT_BF16,
                                        _lib.SMAT_BF16, ctypes.byref(p))
    if status == _lib.SMAT_OK:
        assert lib.smat_merge_plan_destroy(p) == 0
    assert status in (_lib.SMAT_OK, _lib.SMAT_ERR_INVALID)
    assert (status == _lib.SMAT_OK) == merge_allowed(tensors)
