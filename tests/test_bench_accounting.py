"""The bench line's algorithmic counts of the batched products (the roofline's
work, issued MFMA flops and bytes) against an enumeration of the products one
outer step launches for each matrix: the polynomial iteration that replaces
the SVD of Algorithm 2 (a Gram, a polynomial and an update per step, and the
Gram of the final check), and the tall matrices' steps on n x n factors
(B = A M, A_k = M B, P = p_k(A_k), M <- M P, then X = X_first M once), each
product with its shape, its symmetry and the step whose arithmetic it takes.
The symmetric products count only their distinct output entries, enumerated
one by one on small shapes."""
import collections

import pytest

import bench

St = collections.namedtuple("St", "steps")

# kernels whose products take the early part count of the mixed precision
_UPDATE_KERNEL = {"AM", "upd"}


def _launches(m, n, s, window, check):
    """(product, rows, cols, K, symmetric, step) of every product of one m x n
    matrix (m >= n) that took s polar steps."""
    first, end = window
    fac = end > 0 and m >= 2 * n and s >= end
    out = []
    j = 0
    while j < s:
        out.append(("gram", n, n, m, True, j))  # A_j = X_j^T X_j
        if fac and j == first:
            out.append(("poly", n, n, n, True, j))  # M = p_first(A)
            for q in range(first + 1, end):
                out.append(("AM", n, n, n, False, q))  # B = A M
                out.append(("MB", n, n, n, True, q))  # A_q = M B (symmetric)
                out.append(("poly", n, n, n, True, q))  # P = p_q(A_q)
                out.append(("MP", n, n, n, True, q))  # M <- M P (symmetric)
            out.append(("upd", m, n, n, False, end - 1))  # X_end = X_first M
            j = end
        else:
            out.append(("poly", n, n, n, True, j))
            out.append(("upd", m, n, n, False, j))
            j += 1
    if check:
        out.append(("gram", n, n, m, True, s))  # Q^T Q
    return out


def _entries(rows, cols, symmetric):
    """Output entries a product computes: all of them, or those on and above
    the diagonal of a symmetric one (enumerated for small shapes)."""
    if not symmetric:
        return rows * cols
    if rows <= 64:
        return sum(1 for i in range(rows) for j in range(i, cols))
    return rows * (rows + 1) // 2


def _parts(precision, product, step):
    early, late = bench.PARTS[precision]
    return early if product in _UPDATE_KERNEL and step < bench.X6_STEPS else late


def _bytes(product, rows, cols, k):
    # each product reads its operands once and writes its output once (fp32)
    if product == "gram":
        return 4 * (k * rows + rows * cols)  # X (m x n), A (n x n)
    if product == "poly":
        return 4 * 2 * rows * cols  # A, P
    if product == "upd":
        return 4 * (2 * rows * cols + k * cols)  # X, X' (m x n), P (n x n)
    return 4 * 3 * rows * cols  # A M, M B, M P: two n x n operands, one n x n result


def _enumerated(layout, stats, check, precision, window):
    f = fm = b = 0
    for (_, r, c, kind), st in zip(layout, stats):
        if kind != 0:
            continue
        m, n = max(r, c), min(r, c)
        for prod, rows, cols, k, sym, step in _launches(m, n, st.steps, window, check):
            fl = 2 * _entries(rows, cols, sym) * k
            f += fl
            fm += fl * _parts(precision, prod, step)
            b += _bytes(prod, rows, cols, k)
    return f, fm, b


def _layout(shapes):
    lay, off = [], 0
    for r, c, kind in shapes:
        lay.append((off, r, c, kind))
        off += r * c
    return lay


SMALL = _layout([(6, 6, 0), (12, 5, 0), (5, 12, 0), (7, 3, 0), (9, 1, 1), (40, 8, 0)])


@pytest.mark.parametrize("precision", ["mixed", "bf16x3", "bf16x6", "fp32"])
@pytest.mark.parametrize("window", [(0, 0), (4, 7), (1, 7), (2, 5), (3, 9)])
@pytest.mark.parametrize("check", [True, False])
def test_small_shapes(precision, window, check):
    for steps in ([7, 7, 7, 7, 0, 7], [13, 9, 4, 10, 0, 16], [3, 5, 6, 8, 0, 21]):
        st = [St(s) for s in steps]
        f, fm, b = _enumerated(SMALL, st, check, precision, window)
        assert bench.gemm_flops_per_step(SMALL, st, check, precision, window) == (f, fm)
        if check:
            assert bench.gemm_bytes_per_step(SMALL, st, window) == b


@pytest.mark.parametrize("precision", ["mixed", "bf16x3"])
def test_workload_layouts(precision):
    """The three workloads' layouts with the step counts their bench lines
    reported, default window [4, 7]."""
    from workload import WORKLOADS, LLAMA_110M, LLAMA_341M, LLAMA_888M
    hist = {LLAMA_110M: {"tall": [7], "square": [13] * 44 + [16] * 4},
            LLAMA_341M: {"tall": [7] * 35 + [10] * 38, "square": [13] * 67 + [16] * 28 + [21]},
            LLAMA_888M: {"tall": [10], "square": [10, 13, 16]}}
    for name, h in hist.items():
        lay = WORKLOADS[name].layout
        st, it = [], {"tall": 0, "square": 0}
        for (_, r, c, kind) in lay:
            if kind != 0:
                st.append(St(0))
                continue
            cls = "tall" if max(r, c) >= 2 * min(r, c) else "square"
            seq = h[cls]
            st.append(St(seq[it[cls] % len(seq)]))
            it[cls] += 1
        f, fm, b = _enumerated(lay, st, True, precision, (4, 7))
        assert bench.gemm_flops_per_step(lay, st, True, precision, (4, 7)) == (f, fm)
        assert bench.gemm_bytes_per_step(lay, st, (4, 7)) == b


def test_default_workload_figures():
    """The 109.5M workload's step (37 matrices at 7 steps with the factored
    window [4, 7], 44 at 13 and 4 at 16): the fp32-equivalent flops and the
    algorithmic bytes the bench line and the profiles quote."""
    from workload import WORKLOADS, LLAMA_110M
    lay = WORKLOADS[LLAMA_110M].layout
    st, sq = [], 0
    for (_, r, c, kind) in lay:
        if kind != 0:
            st.append(St(0))
        elif max(r, c) >= 2 * min(r, c):
            st.append(St(7))
        else:
            st.append(St(16 if sq >= 44 else 13))
            sq += 1
    f, fm = bench.gemm_flops_per_step(lay, st, True, "mixed", (4, 7))
    assert f == 2424823676928
    assert bench.gemm_bytes_per_step(lay, st, (4, 7)) == 19680460800
