"""Pins for the CPU oracle: each check ties the oracle to something other
than itself (dense brute force, closed forms, exact special cases,
invariants, an independent selection method, a hand-worked greedy example),
so that a dropped term, a wrong sign or index, or a transposed operand fails
at least one of them. CPU only."""
import json
import os
import struct

import numpy as np
import pytest

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def dense(A, n_cols=None):
    n_cols = A.n if n_cols is None else n_cols
    M = np.zeros((A.n, n_cols), dtype=np.float64)
    for i in range(A.n):
        s, e = A.rowptr[i], A.rowptr[i + 1]
        M[i, A.col[s:e]] = A.val[s:e]
    return M


def key_of(q):
    """Key encoding written from its definition, independent of the oracle:
    NaN -> 0, else IEEE-754 bit pattern of the double plus one."""
    q = float(q)
    if q != q:
        return 0
    return struct.unpack("<Q", struct.pack("<d", q))[0] + 1


def ring(n, r_half):
    """r-regular circulant graph (each node linked to the r_half nearest on
    each side) with self-loops and GCN values fl32(1/(r+1))."""
    rows = []
    for i in range(n):
        nb = sorted({(i + o) % n for o in range(-r_half, r_half + 1)})
        rows.append(nb)
    rowptr = np.zeros(n + 1, np.int32)
    rowptr[1:] = np.cumsum([len(r) for r in rows])
    col = np.array([c for r in rows for c in r], np.int32)
    v = np.float32(1.0 / (2 * r_half + 1))
    val = np.full(len(col), v, np.float32)
    return synth.Csr(n, rowptr, col, val)


@pytest.fixture(scope="module")
def small_sym():
    A = synth.erdos_renyi(300, 0.05, seed=3)
    B = synth.dense_normal(300, 37, seed=4)
    return A, B


@pytest.fixture(scope="module")
def small_gen():
    """Non-symmetric, with empty rows, a hub row and negative values."""
    A = synth.random_csr(257, 190, 12, seed=5, hub_rows=2, hub_len=150, empty_frac=0.1)
    B = synth.dense_normal(190, 21, seed=6)
    return A, B


# ---------------------------------------------------------------- O0 / O1
def test_csr_check(small_gen):
    A, _ = small_gen
    assert oracle.check_csr(A.rowptr, A.col, A.n, 190) == 0
    bad = A.col.copy()
    i = int(np.argmax(np.diff(A.rowptr) > 1))
    bad[A.rowptr[i] + 1] = bad[A.rowptr[i]]          # duplicate column
    assert oracle.check_csr(A.rowptr, bad, A.n, 190) == 5
    bad = A.col.copy(); bad[0] = 190                 # out of range
    assert oracle.check_csr(A.rowptr, bad, A.n, 190) == 4
    bad = A.col.copy(); bad[0] = -1                  # negative column
    assert oracle.check_csr(A.rowptr, bad, A.n, 190) == 4
    rp = A.rowptr.copy(); rp[0] = 1                  # rowptr[0] != 0
    assert oracle.check_csr(rp, A.col, A.n, 190) == 2
    rp = A.rowptr.copy()
    i = int(np.argmax(rp > 0))                       # first row that starts past entry 0
    rp[i + 1] = rp[i] - 1                            # row i ends before it starts
    assert oracle.check_csr(rp, A.col, A.n, 190) == 3
    assert oracle.check_csr(A.rowptr, A.col, -1, 190) == 1
    assert oracle.check_csr(A.rowptr, A.col, A.n, -5) == 1


def test_gcn_values_closed_form_ring():
    # every node of a circulant graph with r = 4 neighbours has degree 5
    # (with the self-loop), so every value is fl32(1/sqrt(5*5)) = fl32(1/5)
    A = ring(50, 2)
    assert oracle.check_gcn_values(A.rowptr, A.col, A.val) == 0
    v = A.val.copy(); v[7] = np.nextafter(v[7], np.float32(1))
    assert oracle.check_gcn_values(A.rowptr, A.col, v) == 1
    # a structure without the self-loop (A instead of A + I) is not the operand
    keep = A.col != np.repeat(np.arange(A.n), np.diff(A.rowptr))
    rp = np.zeros(A.n + 1, np.int32); rp[1:] = np.cumsum(np.full(A.n, 4))
    noself = np.full(keep.sum(), np.float32(1.0 / 4.0), np.float32)
    assert oracle.check_gcn_values(rp, A.col[keep], noself) == A.n


def test_gcn_values_on_generated_graphs():
    for A in (synth.erdos_renyi(500, 0.02, seed=1), synth.make_graph("tiny", 0)):
        assert oracle.check_csr(A.rowptr, A.col, A.n, A.n) == 0
        assert oracle.check_gcn_values(A.rowptr, A.col, A.val) == 0
        D = dense(A)
        assert np.array_equal(D != 0, (D != 0).T)               # symmetric structure
        assert np.all(np.diag(D) != 0)                           # self-loops


# ---------------------------------------------------------------- O2
@pytest.mark.parametrize("which", ["small_sym", "small_gen"])
def test_spmm_dense_brute_force(which, request):
    A, B = request.getfixturevalue(which)
    n_cols = B.shape[0]
    Y, S = oracle.spmm(A.rowptr, A.col, A.val, B, with_mag=True)
    D = dense(A, n_cols)
    ref = D @ B.astype(np.float64)
    mag = np.abs(D) @ np.abs(B.astype(np.float64))
    # one fp32 rounding of an fp64 sum: |Y - ref| <= 2^-24 |ref| + fp64 noise
    assert np.all(np.abs(Y - ref) <= 2.0 ** -24 * np.abs(ref) + 1e-12 * mag + 1e-300)
    np.testing.assert_allclose(S, mag, rtol=1e-12, atol=0)


def test_spmm_identity_is_bitwise_dense(small_gen):
    A, _ = small_gen
    I = np.eye(190, dtype=np.float32)
    Y = oracle.spmm(A.rowptr, A.col, A.val, I)
    assert np.array_equal(Y, dense(A, 190).astype(np.float32))


def test_spmm_permutation_is_bitwise():
    rng = np.random.default_rng(0)
    n = 173
    p = rng.permutation(n).astype(np.int32)
    rowptr = np.arange(n + 1, dtype=np.int32)
    val = np.ones(n, np.float32)
    B = synth.dense_normal(n, 9, seed=2)
    Y = oracle.spmm(rowptr, p, val, B)
    assert np.array_equal(Y, B[p])


def test_spmm_row_subset_and_ld(small_gen):
    A, _ = small_gen
    B = synth.dense_normal(190, 21, seed=6, ld=24)       # padded leading dimension
    Yfull = oracle.spmm(A.rowptr, A.col, A.val, B, d=21)
    rows = np.array([0, 5, 256, 17, 5], np.int32)
    Ysub = oracle.spmm(A.rowptr, A.col, A.val, B, d=21, rows=rows)
    assert np.array_equal(Ysub, Yfull[rows])
    assert np.array_equal(Yfull, oracle.spmm(A.rowptr, A.col, A.val, B[:, :21].copy()))


def test_spmm_linearity(small_sym):
    A, B = small_sym
    B2 = synth.dense_normal(300, 37, seed=9)
    Y1, S1 = oracle.spmm(A.rowptr, A.col, A.val, B, with_mag=True)
    Y2, S2 = oracle.spmm(A.rowptr, A.col, A.val, B2, with_mag=True)
    Y12 = oracle.spmm(A.rowptr, A.col, A.val, (B + B2).astype(np.float32))
    assert np.all(np.abs(Y12 - (Y1.astype(np.float64) + Y2)) <= 1e-6 * (S1 + S2) + 1e-30)


# ---------------------------------------------------------------- O3 / O4
def test_col_sqnorms_closed_form_regular():
    # r-regular with self-loops, r + 1 = 7 <= 32: the sum of seven copies of
    # x^2 (x = fl32(1/7), x^2 exact in fp64) is exact, so cn2 = 7 x^2 bitwise
    A = ring(40, 3)
    AT = synth.transpose(A)
    cn2, colnnz = oracle.col_sqnorms(AT.rowptr, AT.val)
    x = float(np.float32(1.0 / 7.0))
    assert np.all(cn2 == 7.0 * x * x)
    assert np.all(colnnz == 7)


def test_col_sqnorms_dense(small_gen):
    A, _ = small_gen
    AT = synth.transpose(A, 190)
    cn2, colnnz = oracle.col_sqnorms(AT.rowptr, AT.val)
    D = dense(A, 190)
    np.testing.assert_allclose(cn2, (D ** 2).sum(axis=0), rtol=1e-14, atol=0)
    assert np.array_equal(colnnz, (D != 0).sum(axis=0))


def test_pair_keys_closed_forms():
    n, d = 6, 5
    B = np.zeros((n, d), np.float32)
    cs = np.float32([3.0, -0.5, 1e-20, 7.25, 0.0, 2.0 ** 60])
    for i in range(n):
        B[i, i % d] = cs[i]                                  # B[i,:] = c e_j
    cn2 = np.array([1.0, 2.0, 4.0, 0.5, 9.0, 1.0])
    out = oracle.pair_keys(cn2, B)
    assert np.array_equal(out["rn2"], cs.astype(np.float64) ** 2)   # exact
    assert np.array_equal(out["q"], cn2 * cs.astype(np.float64) ** 2)
    assert [int(k) for k in out["key"]] == [key_of(q) for q in out["q"]]
    assert out["key"][4] == 1                                # q = +0 -> key 1


def test_pair_keys_nan_inf_and_order():
    cn2 = np.array([1.0, 1.0, 0.0, 1.0, 2.0])
    B = np.ones((5, 3), np.float32)
    B[0, 1] = np.nan                                         # q NaN -> key 0
    B[1, 2] = np.inf                                         # q +Inf
    B[2, 0] = np.inf                                         # 0 * Inf = NaN
    out = oracle.pair_keys(cn2, B)
    assert out["key"][0] == 0 and out["key"][2] == 0
    assert out["key"][1] == key_of(np.inf)
    assert out["key"][1] > out["key"][4] > out["key"][3] > 0


def test_pair_keys_dense_and_cauchy_schwarz(small_sym):
    A, B = small_sym
    cn2, _ = oracle.col_sqnorms(A.rowptr, A.val)             # symmetric: A^T = A
    out = oracle.pair_keys(cn2, B)
    B64 = B.astype(np.float64)
    np.testing.assert_allclose(out["rn2"], (B64 ** 2).sum(axis=1), rtol=1e-14)
    # Eq. 3 written independently from dense norms
    D = dense(A)
    colnorm = np.linalg.norm(D, axis=0)
    rownorm = np.linalg.norm(B64, axis=1)
    p = colnorm * rownorm / np.sum(colnorm * rownorm)
    assert abs(p.sum() - 1.0) < 1e-12
    np.testing.assert_allclose(np.sqrt(out["q"]), colnorm * rownorm, rtol=1e-13)
    # ranking by p equals ranking by the key (continuous data: no ties)
    assert np.array_equal(np.argsort(-p, kind="stable"), oracle.rank_order(out["key"]))
    # normalised mass is at most 1 (Cauchy-Schwarz)
    assert np.sqrt(out["q"]).sum() <= np.sqrt(cn2.sum()) * np.sqrt(out["rn2"].sum()) * (1 + 1e-12)


# ---------------------------------------------------------------- O5
def topk_lexsort(key, k):
    """Independent selection: numpy lexsort on (~key, index); ~ reverses
    the order of unsigned integers."""
    order = np.lexsort((np.arange(len(key)), ~key.astype(np.uint64)))
    return np.sort(order[:k]).astype(np.int32)


def topk_partition(key, k):
    """Second independent route: threshold by partition, then a tie pass."""
    n = len(key)
    if k == 0:
        return np.zeros(0, np.int32)
    T = np.partition(key, n - k)[n - k]
    gt = np.nonzero(key > T)[0]
    eq = np.nonzero(key == T)[0][: k - len(gt)]
    return np.sort(np.concatenate([gt, eq])).astype(np.int32)


def mask_of(idx, n):
    m = np.zeros((n + 31) // 32, np.uint32)
    for i in idx:
        m[i >> 5] |= np.uint32(1 << (int(i) & 31))
    return m


@pytest.mark.parametrize("seed", range(4))
def test_topk_two_independent_methods(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 3000))
    # few distinct values -> many ties
    key = rng.integers(0, 40, size=n).astype(np.uint64) * np.uint64(1 << 40)
    for k in sorted({0, 1, n // 3, n // 2, n - 1, n}):
        if k < 0:
            continue
        idx, mask = oracle.topk(key, k)
        ref = topk_lexsort(key, k)
        assert np.array_equal(idx, ref)
        assert np.array_equal(idx, topk_partition(key, k))
        assert np.array_equal(mask, mask_of(ref, n))


def test_topk_special_cases():
    n = 100
    eq = np.full(n, 12345, np.uint64)
    assert np.array_equal(oracle.topk(eq, 37)[0], np.arange(37))
    dec = np.arange(n, 0, -1).astype(np.uint64)
    assert np.array_equal(oracle.topk(dec, 10)[0], np.arange(10))
    inc = np.arange(1, n + 1).astype(np.uint64)
    assert np.array_equal(oracle.topk(inc, 10)[0], np.arange(90, 100))
    assert len(oracle.topk(inc, 0)[0]) == 0 and not oracle.topk(inc, 0)[1].any()
    assert np.array_equal(oracle.topk(inc, n)[0], np.arange(n))
    # NaN (key 0) last, +Inf first
    q = np.array([1.0, np.nan, np.inf, 3.0, np.nan, np.inf])
    keys = np.array([key_of(x) for x in q], np.uint64)
    assert list(oracle.topk(keys, 2)[0]) == [2, 5]
    assert list(oracle.topk(keys, 5)[0]) == [0, 1, 2, 3, 5]


# ---------------------------------------------------------------- O6 / O7
def test_slice_identities(small_gen):
    A, B = small_gen
    n_cols = 190
    AT = synth.transpose(A, n_cols)
    _, colnnz = oracle.col_sqnorms(AT.rowptr, AT.val)
    rng = np.random.default_rng(1)
    D = dense(A, n_cols)
    for k in (0, 1, 50, 189, 190):
        idx = np.sort(rng.choice(n_cols, size=k, replace=False)).astype(np.int32)
        mask = mask_of(idx, n_cols)
        ro, co, vo = oracle.slice_csr(A.rowptr, A.col, A.val, mask)
        S = synth.Csr(A.n, ro, co, vo)
        keep = np.zeros(n_cols); keep[idx] = 1
        assert np.array_equal(dense(S, n_cols), D * keep[None, :])
        assert len(co) == int(colnnz[idx].sum())
        assert oracle.check_csr(ro, co, A.n, n_cols) == 0
        if k == 0:
            assert len(co) == 0 and not ro.any()
        if k == n_cols:
            assert np.array_equal(ro, A.rowptr) and np.array_equal(co, A.col)
            assert np.array_equal(vo.view(np.uint32), A.val.view(np.uint32))
        # O7: sampled product
        Ys = oracle.spmm(ro, co, vo, B)
        ref = D @ np.diag(keep) @ B.astype(np.float64)
        assert np.all(np.abs(Ys - ref) <= 2.0 ** -24 * np.abs(ref) + 1e-12 * (np.abs(D) @ np.abs(B)))
        # textbook column-row form: sum over kept i of A[:, i] B[i, :]
        cr = np.zeros((A.n, B.shape[1]))
        for i in idx:
            cr += np.outer(D[:, i], B[i].astype(np.float64))
        np.testing.assert_allclose(Ys, cr, rtol=1e-5, atol=1e-6)
        # complement: Y_S + Y_{S^c} = Y within rounding
        comp = mask_of(np.setdiff1d(np.arange(n_cols), idx), n_cols)
        rc, cc, vc = oracle.slice_csr(A.rowptr, A.col, A.val, comp)
        Yc = oracle.spmm(rc, cc, vc, B)
        Y, Smag = oracle.spmm(A.rowptr, A.col, A.val, B, with_mag=True)
        assert np.all(np.abs(Ys.astype(np.float64) + Yc - Y) <= 1e-6 * Smag + 1e-30)
        if k == n_cols:
            assert np.array_equal(Ys, Y)


# ---------------------------------------------------------------- O8
def test_k_from_fraction():
    assert oracle.k_from_fraction(4096, 50, 100) == 2048
    assert [oracle.k_from_fraction(232_965, p, 100) for p in (10, 30, 50)] == [23_296, 69_889, 116_482]
    assert oracle.k_from_fraction(2_449_029, 30, 100) == 734_708
    assert oracle.k_from_fraction(132_534, 30, 100) == 39_760
    assert oracle.k_from_fraction(7, 0, 1) == 0 and oracle.k_from_fraction(7, 1, 1) == 7


def _keys_from_scores(scores):
    return np.array([key_of(float(s) ** 2) for s in scores], np.uint64)


def test_greedy_hand_worked_example():
    g = json.load(open(os.path.join(GOLDEN, "greedy_hand_example.json")))
    keys = [_keys_from_scores(s) for s in g["scores"]]
    k, bud = oracle.greedy(keys, g["colnnz"], g["nnz"], g["d"], g["fro_a2"], g["fro_b2"],
                           tuple(g["C"]), tuple(g["alpha"]))
    assert k == g["expected_k"] and bud == g["expected_budget"]


def test_greedy_tie_goes_to_lower_layer_and_limits():
    scores = [5, 4, 3, 2, 1, 0]
    keys = [_keys_from_scores(scores)] * 2
    colnnz = [1] * 6
    # two identical layers: first shrink goes to layer 0, second to layer 1
    k, bud = oracle.greedy(keys, colnnz, 6, [1, 1], 1.0, [1.0, 1.0], (5, 6), (1, 6))
    assert k == [5, 5] and bud == 10
    # C = 1: already within budget, nothing shrinks
    k, bud = oracle.greedy(keys, colnnz, 6, [1, 1], 1.0, [1.0, 1.0], (1, 1), (1, 6))
    assert k == [6, 6] and bud == 12
    # C = 0: everything goes to zero, then the loop stops (no eligible layer)
    k, bud = oracle.greedy(keys, colnnz, 6, [1, 1], 1.0, [1.0, 1.0], (0, 1), (1, 3))
    assert k == [0, 0] and bud == 0


@pytest.mark.parametrize("C", [(1, 10), (3, 10), (1, 2)])
def test_greedy_invariants(C):
    A = synth.make_graph("tiny", 0)
    n = A.n
    cn2, colnnz = oracle.col_sqnorms(A.rowptr, A.val)
    keys, fro_b2, ds = [], [], [64, 16]
    for l, dl in enumerate(ds):
        out = oracle.pair_keys(cn2, synth.dense_normal(n, dl, seed=10 + l))
        keys.append(out["key"]); fro_b2.append(out["rn2"].sum())
    k, bud = oracle.greedy(keys, colnnz, A.nnz, ds, cn2.sum(), fro_b2, C, (2, 100))
    step = max(1, n * 2 // 100)
    total = A.nnz * sum(ds)
    assert bud * C[1] <= C[0] * total
    recomputed = 0
    for l in range(2):
        assert k[l] == 0 or (n - k[l]) % step == 0
        top = np.lexsort((np.arange(n), ~keys[l]))[: k[l]]
        recomputed += ds[l] * int(colnnz[top].sum())
    assert recomputed == bud
    assert C[0] == C[1] or any(k[l] < n for l in range(2))


def test_cache_policy():
    p = oracle.CachePolicy(10)
    seq = []
    for s in range(25):
        r = p.needs_refresh(s)
        seq.append(r)
        if r:
            p.refreshed(s)
    assert [i for i, r in enumerate(seq) if r] == [0, 10, 20]


# ---------------------------------------------------------------- SpMM_MEAN
def test_spmm_mean_appendix_example():
    g = json.load(open(os.path.join(GOLDEN, "spmm_mean_appendix_example.json")))
    Ad = np.array(g["A"], np.float32)
    rowptr = np.concatenate([[0], np.cumsum((Ad != 0).sum(axis=1))]).astype(np.int32)
    col = np.concatenate([np.nonzero(r)[0] for r in Ad]).astype(np.int32)
    val = Ad[Ad != 0].astype(np.float32)
    Y = oracle.spmm_mean(rowptr, col, val, np.array(g["H"], np.float32))
    assert np.array_equal(Y, np.array(g["expected_reading"], np.float32))
    # the printed example agrees with D^-1 A H on the row that has two entries
    assert np.array_equal(Y[2], np.array(g["printed"][2], np.float32))
    assert not np.array_equal(Y[:2], np.array(g["printed"][:2], np.float32))


def test_spmm_mean_dense_and_empty_rows(small_gen):
    A, B = small_gen
    Y = oracle.spmm_mean(A.rowptr, A.col, A.val, B)
    D = dense(A, 190)
    deg = (D != 0).sum(axis=1)
    ref = np.where(deg[:, None] > 0, (D @ B.astype(np.float64)) / np.maximum(deg, 1)[:, None], 0.0)
    mag = (np.abs(D) @ np.abs(B.astype(np.float64))) / np.maximum(deg, 1)[:, None]
    assert np.all(np.abs(Y - ref) <= 2.0 ** -24 * np.abs(ref) + 1e-12 * mag + 1e-300)
    assert np.all(Y[deg == 0] == 0)


# ---------------------------------------------------------------- randomized sampling
def test_splitmix64_reference_outputs():
    g = json.load(open(os.path.join(GOLDEN, "splitmix64_seed1234567.json")))
    assert [oracle.splitmix64(g["seed"], t) for t in range(len(g["outputs"]))] == [int(x) for x in g["outputs"]]


def _weight_bits(n):
    """Weight resolution S: 38 bits up to 2^24 pairs, then fewer, so that
    n * 2^S <= 2^62 and the int64 CDF cannot overflow."""
    return 38 if n <= 1 << 24 else 62 - (n - 1).bit_length()


def _weights_by_definition(key):
    """w_i = floor(sqrt(q_i) * 2^S / max_j sqrt(q_j)), written independently."""
    import math
    r = []
    for u in key:
        u = int(u)
        r.append(0.0 if u == 0 else math.sqrt(struct.unpack("<d", struct.pack("<Q", u - 1))[0]))
    m = max(r)
    scale = math.ldexp(1.0, _weight_bits(len(key))) / m
    return np.array([int(x * scale) for x in r], np.int64)


def test_sample_columns_counts_weights_and_scale():
    A = synth.make_graph("tiny", 0)
    cn2, _ = oracle.col_sqnorms(A.rowptr, A.val)
    key = oracle.pair_keys(cn2, synth.dense_normal(A.n, 16, seed=3))["key"]
    key[::50] = 0                                            # NaN pairs never drawn
    o = oracle.sample_columns(key, 1000, seed=7)
    assert o["count"].sum() == 1000
    assert np.array_equal(o["w"], _weights_by_definition(key))
    assert np.all(o["count"][::50] == 0)
    drawn = np.nonzero(o["count"])[0]
    assert np.array_equal(mask_of(drawn, A.n), o["mask"])
    total = float(o["w"].sum())
    want = o["count"][drawn] * total / (1000.0 * o["w"][drawn])
    assert np.array_equal(o["colw"][drawn], want) and not o["colw"][o["count"] == 0].any()


def test_sample_columns_single_weight_is_exact_slice():
    key = np.zeros(40, np.uint64)
    key[17] = key_of(2.5)
    o = oracle.sample_columns(key, 33, seed=1)
    assert o["count"][17] == 33 and o["count"].sum() == 33 and o["colw"][17] == 1.0


def test_sample_columns_infinite_scores_share_the_mass():
    """With +Inf scores present only those pairs can be drawn, uniformly
    (p = 1/2 each here), so colw = c / (k / 2)."""
    key = np.array([key_of(float(i)) for i in range(1, 41)], np.uint64)
    key[[7, 30]] = key_of(float("inf"))
    key[3] = 0
    k = 4000
    o = oracle.sample_columns(key, k, seed=5)
    assert o["count"][[7, 30]].sum() == k and o["count"].sum() == k
    assert abs(int(o["count"][7]) - k // 2) <= 5 * np.sqrt(k / 4)
    assert np.array_equal(o["colw"][[7, 30]], o["count"][[7, 30]] / (k / 2.0))


def test_sample_columns_frequencies():
    # 12 pairs with sqrt(q) = 1..12: p_i = i / 78
    key = np.array([key_of(float(i) ** 2) for i in range(1, 13)], np.uint64)
    k = 200_000
    o = oracle.sample_columns(key, k, seed=99)
    p = o["w"] / o["w"].sum()
    sd = np.sqrt(k * p * (1 - p))
    assert np.all(np.abs(o["count"] - k * p) <= 5 * sd)
    np.testing.assert_allclose(p, np.arange(1, 13) / 78.0, rtol=1e-9)


def boundary_case(S=38):
    """Two columns with weights (a, 2^S) and a seed whose first draw has
    u = floor(z * (a + 2^S) / 2^64) equal to a = W_0, a CDF boundary: the
    seed is the first whose first output z is below 2^51 (so a < 2^25 and
    sqrt(q_0) = a 2^-S is exact), a is the fixed point of that floor."""
    seed = next(s for s in range(1 << 22) if oracle.splitmix64(s, 0) < 1 << 51)
    z = oracle.splitmix64(seed, 0)
    a = (z << S) // ((1 << 64) - z)
    while (z * (a + (1 << S))) >> 64 > a:
        a += 1
    while (z * (a + (1 << S))) >> 64 < a:
        a -= 1
    assert (z * (a + (1 << S))) >> 64 == a and 0 < a < 1 << 25
    key = np.array([key_of((a * 2.0 ** -S) ** 2), key_of(1.0)], np.uint64)
    return key, seed, a


def test_sample_draw_on_a_cdf_boundary_goes_to_the_next_column():
    """With u uniform on the integers [0, total), column i must own exactly
    w_i of them for p_i = w_i / total (Eq. 3 up to the weights' rounding):
    [W_{i-1}, W_i). A draw with u = W_0 therefore lands on column 1; the rule
    'smallest i with W_i >= u' would give column 0 one value too many."""
    key, seed, a = boundary_case()
    assert np.array_equal(_weights_by_definition(key), [a, 1 << 38])
    o = oracle.sample_columns(key, 1, seed)
    assert list(o["w"]) == [a, 1 << 38]
    assert list(o["count"]) == [0, 1]


def test_slice_scaled_against_dense_definition(small_gen):
    """Scaled slice = dense(A) diag(mask * colw), each value rounded once to
    fp32; unit scales give the plain slice bit for bit, power-of-two scales
    are exact."""
    A, _ = small_gen
    n_cols = 190
    rng = np.random.default_rng(4)
    idx = np.sort(rng.choice(n_cols, size=70, replace=False)).astype(np.int32)
    mask = mask_of(idx, n_cols)
    ro, co, vo = oracle.slice_csr(A.rowptr, A.col, A.val, mask)
    r1, c1, v1 = oracle.slice_scaled(A.rowptr, A.col, A.val, mask, np.ones(n_cols))
    assert np.array_equal(r1, ro) and np.array_equal(c1, co) and np.array_equal(v1.view(np.uint32), vo.view(np.uint32))
    colw = rng.uniform(0.1, 9.0, n_cols)
    colw[::3] = 2.0 ** rng.integers(-4, 5, size=len(colw[::3]))
    rs, cs, vs = oracle.slice_scaled(A.rowptr, A.col, A.val, mask, colw)
    assert np.array_equal(rs, ro) and np.array_equal(cs, co)
    pow2 = (np.arange(n_cols) % 3 == 0)[cs]
    assert np.array_equal(vs[pow2].astype(np.float64), vo[pow2].astype(np.float64) * colw[cs[pow2]])
    keep = np.zeros(n_cols); keep[idx] = colw[idx]
    np.testing.assert_allclose(dense(synth.Csr(A.n, rs, cs, vs), n_cols), dense(A, n_cols) * keep[None, :],
                               rtol=2.0 ** -23, atol=0)


def test_sample_weight_resolution_keeps_cdf_in_range():
    """Above 2^24 pairs the weights lose bits so the CDF total stays below
    2^63: with equal scores every weight is exactly 2^S, and the scale of a
    column drawn c times is c n / k."""
    for n, bits in ((1 << 24, 38), ((1 << 24) + 1, 37)):
        assert _weight_bits(n) == bits
        key = np.full(n, key_of(3.0), np.uint64)
        o = oracle.sample_columns(key, 5000, seed=n)
        assert np.all(o["w"] == 1 << bits) and int(o["w"].sum()) == n << bits < 1 << 63
        drawn = np.nonzero(o["count"])[0]
        assert o["count"].sum() == 5000
        assert np.array_equal(o["colw"][drawn], o["count"][drawn] * float(n) / 5000.0)


def test_sampled_product_is_unbiased():
    """E[sum_i colw_i A[:, i] B[i, :]] = A B (Eq. 2 with s = 1/(k p)): the
    mean over many seeds converges to the exact product while one draw does
    not."""
    A = synth.random_csr(60, 50, 12, seed=8)
    B = synth.dense_normal(50, 6, seed=9)
    AT = synth.transpose(A, 50)
    cn2, _ = oracle.col_sqnorms(AT.rowptr, AT.val)
    key = oracle.pair_keys(cn2, B)["key"]
    exact = dense(A, 50) @ B.astype(np.float64)
    acc = np.zeros_like(exact)
    one = None
    seeds = 400
    for s in range(seeds):
        o = oracle.sample_columns(key, 10, seed=s)
        ro, co, vo = oracle.slice_scaled(A.rowptr, A.col, A.val, o["mask"], o["colw"])
        Y = oracle.spmm(ro, co, vo, B).astype(np.float64)
        acc += Y
        one = Y if one is None else one
    err_mean = np.linalg.norm(acc / seeds - exact)
    err_one = np.linalg.norm(one - exact)
    assert err_mean < 0.2 * err_one


# ---------------------------------------------------------------- GCN reference step
def _gcn_problem():
    A = synth.erdos_renyi(40, 0.15, seed=3)
    rng = np.random.default_rng(0)
    n, f, h, c = A.n, 5, 4, 3
    X = rng.standard_normal((n, f))
    W1, W2 = rng.standard_normal((f, h)), rng.standard_normal((h, c))
    Y = (rng.random((n, c)) < 0.5).astype(np.float64)
    return A, X, W1, W2, Y, [h, c]


def test_gcn_reference_gradients_are_the_loss_derivatives():
    """The reference step's exact backward (a refresh step) gives the
    derivatives of the loss its forward reports: central differences in fp64
    agree. A dropped term, a transposed operand or a wrong ReLU mask in the
    backward fails this; at zero logits the mean binary cross-entropy with
    logits is ln 2 whatever the labels."""
    from oracle.gcn_ref import RscReference
    A, X, W1, W2, Y, widths = _gcn_problem()

    def run(w1, w2):
        ref = RscReference(A.rowptr, A.col, A.val, A.n, widths, (1, 2), (1, 4), 10)
        return ref.step(X, w1, w2, Y, 0)

    out = run(W1, W2)
    assert out["mode"] == "score"
    eps = 1e-6
    for which, W in ((0, W1), (1, W2)):
        num = np.zeros_like(W)
        for ij in np.ndindex(W.shape):
            Wp, Wm = W.copy(), W.copy()
            Wp[ij] += eps
            Wm[ij] -= eps
            lp = run(Wp, W2)["loss"] if which == 0 else run(W1, Wp)["loss"]
            lm = run(Wm, W2)["loss"] if which == 0 else run(W1, Wm)["loss"]
            num[ij] = (lp - lm) / (2 * eps)
        np.testing.assert_allclose(out["gW1" if which == 0 else "gW2"], num, rtol=1e-5, atol=1e-9)
    assert abs(run(W1, np.zeros_like(W2))["loss"] - np.log(2.0)) < 1e-15


def test_gcn_reference_full_budget_slices_give_the_exact_backward():
    """With the budget C = 1 the greedy keeps every column (k_l = n), so the
    cached slices are the whole operand and a step between refreshes has the
    exact gradients."""
    from oracle.gcn_ref import RscReference
    A, X, W1, W2, Y, widths = _gcn_problem()
    ref = RscReference(A.rowptr, A.col, A.val, A.n, widths, (1, 1), (1, 4), 10)
    exact = ref.step(X, W1, W2, Y, 0)
    sampled = ref.step(X, W1, W2, Y, 1)
    assert exact["mode"] == "score" and sampled["mode"] == "sampled"
    assert exact["k"] == [A.n, A.n]
    for g in ("gW1", "gW2"):
        np.testing.assert_allclose(sampled[g], exact[g], rtol=1e-14, atol=0)


# ---------------------------------------------------------------- Eq. 4a normalisers
def test_sum_sequential_order_and_bound():
    """The Frobenius normalisers are plain left-to-right fp64 sums: the order
    shows where cancellation decides the result, and on positive data the
    sum stays within (n - 1) units of roundoff of the exact (correctly
    rounded) sum."""
    import math
    assert oracle.sum_sequential(np.array([1.0, 1e16, -1e16])) == 0.0   # 1 absorbed first
    assert oracle.sum_sequential(np.array([1e16, -1e16, 1.0])) == 1.0   # 1 added last
    assert oracle.sum_sequential(np.zeros(0)) == 0.0
    ints = np.arange(1, 100_001, dtype=np.float64)
    assert oracle.sum_sequential(ints) == 100_000 * 100_001 / 2         # exact below 2^53
    x = np.random.default_rng(4).random(200_001) ** 3 * 1e3
    exact = math.fsum(x)
    assert abs(oracle.sum_sequential(x) - exact) <= (len(x) - 1) * 2.0 ** -53 * exact
    assert np.isinf(oracle.sum_sequential(np.array([1.0, np.inf, 2.0])))


# ---------------------------------------------------------------- staleness (NEXT-4)
def _brute_auc(order, prev):
    pos = {int(i): p for p, i in enumerate(order)}
    sel = [i for i in range(len(order)) if i in prev]
    uns = [j for j in range(len(order)) if j not in prev]
    if not sel or not uns:
        return float("nan")
    good = sum(1 for i in sel for j in uns if pos[i] < pos[j])
    return good / (len(sel) * len(uns))


def _mask(idx, n):
    m = np.zeros((n + 31) // 32, np.uint32)
    for i in idx:
        m[i >> 5] |= np.uint32(1 << (i & 31))
    return m


@pytest.mark.parametrize("seed", range(6))
def test_selection_staleness_brute_force(seed):
    rng = np.random.default_rng(900 + seed)
    n = int(rng.integers(2, 180))
    key = rng.integers(1, 50, n).astype(np.uint64)          # many ties: rank by (key desc, index asc)
    order = oracle.rank_order(key)
    k_prev = int(rng.integers(0, n + 1))
    prev = set(int(i) for i in rng.choice(n, k_prev, replace=False))
    new = set(int(i) for i in rng.choice(n, int(rng.integers(0, n + 1)), replace=False))
    auc, overlap = oracle.selection_staleness(order, _mask(prev, n), _mask(new, n))
    want = _brute_auc(order, prev)
    assert (np.isnan(auc) and np.isnan(want)) or auc == want
    if prev:
        assert overlap == len(prev & new) / len(prev)
    else:
        assert overlap is None


def test_selection_staleness_special_cases():
    n = 100
    key = np.arange(n, 0, -1).astype(np.uint64)               # ranking 0, 1, ..., n-1
    order = oracle.rank_order(key)
    top = set(range(30))
    auc, ov = oracle.selection_staleness(order, _mask(top, n), _mask(top, n))
    assert auc == 1.0 and ov == 1.0                           # same ranking: the selection is still on top
    bottom = set(range(70, 100))
    auc, ov = oracle.selection_staleness(order, _mask(bottom, n), _mask(top, n))
    assert auc == 0.0 and ov == 0.0                           # ranked last now
    alt = set(range(0, n, 2))                                  # every other rank: above exactly half on average
    auc, _ = oracle.selection_staleness(order, _mask(alt, n))
    assert auc == sum(50 - i for i in range(50)) / (50 * 50)
    assert np.isnan(oracle.selection_staleness(order, _mask(set(), n))[0])
    assert np.isnan(oracle.selection_staleness(order, _mask(set(range(n)), n))[0])


def test_gcn_reference_staleness_record():
    """With tracking, each refresh after the first records per layer the AUC
    of the previous refresh's selection under the new keys and the overlap,
    and the k_l of every refresh (the Fig. 7 trace); the values equal the
    brute-force count on the keys the step scored."""
    from oracle.gcn_ref import RscReference
    A, X, W1, W2, Y, widths = _gcn_problem()
    ref = RscReference(A.rowptr, A.col, A.val, A.n, widths, (1, 3), (1, 10), 2, track_staleness=True)
    prev_idx, lr = None, 5.0
    for step in range(7):
        out = ref.step(X, W1, W2, Y, step)
        if out["mode"] == "score":
            rec = ref.history[-1]
            assert rec["step"] == step and rec["k"] == out["k"]
            if prev_idx is None:
                assert rec["auc"] == [] and rec["overlap"] == []
            else:
                for l in range(2):
                    order = oracle.rank_order(out["keys"][l])
                    assert rec["auc"][l] == _brute_auc(order, set(int(i) for i in prev_idx[l]))
                    inter = len(set(prev_idx[l].tolist()) & set(out["idx"][l].tolist()))
                    assert rec["overlap"][l] == inter / len(prev_idx[l])
            prev_idx = out["idx"]
        W1 = W1 - lr * out["gW1"]                               # the weights move between refreshes
        W2 = W2 - lr * out["gW2"]
    assert [r["step"] for r in ref.history] == [0, 2, 4, 6]
