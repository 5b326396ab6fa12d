"""Pins of the CPU oracle against what mathematics fixes (no GPU).

Each test ties one oracle step to something other than the oracle itself: a
closed form, an orthogonal-filter-bank invariant, a library routine applied to
an explicitly built input, or brute force on tiny inputs.  The paper prints no
worked numeric example for the filter path, so every pin here comes from the
definitions in Section 2.2 (eq. 5), Section 3 (eqs. 6-11) and the
cached-attention form of eq. 3.
"""
import itertools
import math

import numpy as np
import pytest
import scipy.special
import torch

import synth

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")


def _rng(seed):
    return np.random.default_rng(seed)


# ----------------------------------------------------------------- DWT (O1)

@pytest.mark.parametrize("levels", [1, 2, 3, 4, 5, 6])
def test_haar_closed_form(ref, levels):
    """Orthonormal Haar: A_J[j] = 2^{-J/2} * (sum of the 2^J tokens of block
    j) and D_j[n] = 2^{-j/2} * (first-half sum - second-half sum) of block n
    at level j.  Block j is exactly eq. 10's token range."""
    x = _rng(levels).standard_normal((128, 5))
    A, D = ref.dwt(x, levels, "haar", details=True)
    blk = 1 << levels
    want = x.reshape(-1, blk, 5).sum(axis=1) * 2.0 ** (-levels / 2)
    np.testing.assert_allclose(A, want, rtol=0, atol=1e-12)
    for j in range(1, levels + 1):
        b = x.reshape(-1, 1 << j, 5)
        h = 1 << (j - 1)
        want_d = (b[:, :h].sum(1) - b[:, h:].sum(1)) * 2.0 ** (-j / 2)
        np.testing.assert_allclose(D[j - 1], want_d, rtol=0, atol=1e-12)


def _analysis_matrix(ref, L, levels, wavelet, boundary):
    """Rows: the coefficients [A_J, D_J, ..., D_1] of each basis vector."""
    cols = []
    for i in range(L):
        e = np.zeros((L, 1))
        e[i] = 1.0
        A, D = ref.dwt(e, levels, wavelet, boundary, details=True)
        cols.append(np.concatenate([A[:, 0]] + [d[:, 0] for d in D[::-1]]))
    return np.stack(cols, axis=1)


@pytest.mark.parametrize("wavelet,boundary", [("haar", "symmetric"),
                                              ("haar", "periodic"),
                                              ("db2", "periodic")])
@pytest.mark.parametrize("levels", [1, 2, 3])
def test_orthogonal_filter_bank(ref, wavelet, boundary, levels):
    """An orthonormal filter bank with periodic extension is an orthogonal
    operator: M M^T = I.  That gives perfect reconstruction (x = M^T c) and
    Parseval (|x|^2 = |A_J|^2 + sum_j |D_j|^2)."""
    L = 32
    M = _analysis_matrix(ref, L, levels, wavelet, boundary)
    assert M.shape == (L, L)
    np.testing.assert_allclose(M @ M.T, np.eye(L), rtol=0, atol=1e-12)
    x = _rng(7).standard_normal((L, 3))
    A, D = ref.dwt(x, levels, wavelet, boundary, details=True)
    coeff = np.concatenate([A] + D[::-1], axis=0)
    np.testing.assert_allclose(M.T @ coeff, x, rtol=0, atol=1e-12)
    energy = (A ** 2).sum(0) + sum((d ** 2).sum(0) for d in D)
    np.testing.assert_allclose(energy, (x ** 2).sum(0), rtol=1e-12)


@pytest.mark.parametrize("wavelet,boundary", [("haar", "symmetric"),
                                              ("db2", "symmetric"),
                                              ("db2", "periodic")])
def test_constant_keys_have_no_detail(ref, wavelet, boundary):
    """Constant keys: every detail vanishes and A_J = 2^{J/2} c (the low-pass
    filter sums to sqrt 2, and both extensions keep a constant constant)."""
    c = np.array([0.75, -1.5, 3.0])
    x = np.tile(c, (256, 1))
    for levels in (1, 3, 6):
        A, D = ref.dwt(x, levels, wavelet, boundary, details=True)
        np.testing.assert_allclose(A, np.tile(c * 2 ** (levels / 2),
                                              (256 >> levels, 1)),
                                   rtol=1e-13, atol=1e-13)
        for d in D:
            np.testing.assert_allclose(d, 0.0, atol=1e-13)


def test_haar_piecewise_constant_blocks(ref):
    """Keys constant on each aligned 2^J block: Haar details D_1..D_J vanish."""
    J = 4
    vals = _rng(3).standard_normal((16, 6))
    x = np.repeat(vals, 1 << J, axis=0)
    A, D = ref.dwt(x, J, "haar", details=True)
    for d in D:
        np.testing.assert_allclose(d, 0.0, atol=1e-13)
    np.testing.assert_allclose(A, vals * 2 ** (J / 2), rtol=1e-13)


def _oracle_db2_filters(ref):
    """The oracle's own db2 analysis taps, read off its response to unit
    impulses (periodic, one level): A_1[0] = g_m, D_1[0] = h_m for x = e_m."""
    g, h = [], []
    for m in range(4):
        e = np.zeros((8, 1))
        e[m] = 1.0
        A, D = ref.dwt(e, 1, "db2", "periodic", details=True)
        g.append(A[0, 0])
        h.append(D[0][0, 0])
    return np.array(g), np.array(h)


def test_db2_filter_is_daubechies_d4(ref):
    """Daubechies' 4-tap filter is fixed by: sum g = sqrt 2, orthonormal
    to its even shifts (sum g^2 = 1, g0 g2 + g1 g3 = 0) and two vanishing
    moments of the high-pass (sum h = 0, sum m h_m = 0) with h_m =
    (-1)^m g_{3-m}.  Of its two mirror solutions the reading takes the one
    with g_0 < g_1."""
    g, h = _oracle_db2_filters(ref)
    assert abs(g.sum() - math.sqrt(2)) < 1e-14
    assert abs((g ** 2).sum() - 1) < 1e-14
    assert abs(g[0] * g[2] + g[1] * g[3]) < 1e-14
    assert abs(h.sum()) < 1e-14
    assert abs((np.arange(4) * h).sum()) < 1e-13
    np.testing.assert_allclose(h, [(-1) ** m * g[3 - m] for m in range(4)],
                               atol=1e-15)
    assert g[0] < g[1]


def test_db2_linear_ramp_interior_details_vanish(ref):
    """Two vanishing moments: db2 details of a linear ramp are zero at every
    coefficient whose support stays inside the sequence."""
    L, J = 256, 4
    t = np.arange(L, dtype=np.float64)
    x = np.stack([0.5 + 0.01 * t, -2.0 + 0.003 * t], axis=1)
    _, D = ref.dwt(x, J, "db2", "symmetric", details=True)
    for j in range(1, J + 1):
        n = np.arange(L >> j)
        inside = (1 << j) * n + 3 * ((1 << j) - 1) < L
        assert inside.sum() > 0
        np.testing.assert_allclose(D[j - 1][inside], 0.0, atol=1e-12)


@pytest.mark.parametrize("levels", [1, 2, 5])
def test_db2_symmetric_matches_correlate(ref, levels):
    """Each level equals numpy's correlation of the half-sample symmetric
    extension (y[N] = y[N-1], y[N+1] = y[N-2]) with the low/high-pass taps,
    kept at even offsets; the next level starts from the approximation."""
    g, h = _oracle_db2_filters(ref)
    x = _rng(11).standard_normal((128, 2))
    A, D = ref.dwt(x, levels, "db2", "symmetric", details=True)
    y = x.copy()
    for j in range(levels):
        N = y.shape[0]
        ext = np.concatenate([y, y[::-1][:2]], axis=0)
        a = np.stack([np.correlate(ext[:, c], g, "valid")[::2][:N // 2]
                      for c in range(2)], axis=1)
        dd = np.stack([np.correlate(ext[:, c], h, "valid")[::2][:N // 2]
                       for c in range(2)], axis=1)
        np.testing.assert_allclose(D[j], dd, rtol=0, atol=1e-12)
        y = a
    np.testing.assert_allclose(A, y, rtol=0, atol=1e-12)


def test_db2_symmetric_equals_periodic_away_from_the_end(ref):
    """The two extensions only differ on coefficients whose dependency cone
    reaches past the right end."""
    L, J = 256, 5
    x = _rng(5).standard_normal((L, 3))
    As, Ds = ref.dwt(x, J, "db2", "symmetric", details=True)
    Ap, Dp = ref.dwt(x, J, "db2", "periodic", details=True)
    n = np.arange(L >> J)
    inside = (1 << J) * n + 3 * ((1 << J) - 1) < L
    np.testing.assert_allclose(As[inside], Ap[inside], atol=1e-12)
    assert not np.allclose(As[~inside], Ap[~inside])
    for j in range(1, J + 1):
        n = np.arange(L >> j)
        inside = (1 << j) * n + 3 * ((1 << j) - 1) < L
        np.testing.assert_allclose(Ds[j - 1][inside], Dp[j - 1][inside],
                                   atol=1e-12)


# ----------------------------------------------------------- skim (O2, O3)

def test_skim_mass_and_uniform(ref):
    """Softmax rows sum to one, so sum_j W_j = B (eq. 8); with Q = 0 every
    perception weight is 1/n and W_j = B/n."""
    rng = _rng(1)
    Q = rng.standard_normal((7, 16))
    A = rng.standard_normal((40, 16))
    W = ref.skim(Q, A)
    assert abs(W.sum() - 7) < 1e-12
    np.testing.assert_allclose(ref.skim(np.zeros((5, 16)), A), 5 / 40,
                               rtol=1e-14)


def test_skim_two_regions_is_logistic(ref):
    """One query, two coarse rows: W_0 is the logistic function of the logit
    difference (eq. 7 with n = 2)."""
    Q = np.array([[1.3, -0.4]])
    A = np.array([[0.9, 0.0], [0.0, 2.5]])
    scale = 0.7
    W = ref.skim(Q, A, scale=scale)
    want0 = scipy.special.expit(scale * (1.3 * 0.9 - (-0.4) * 2.5))
    np.testing.assert_allclose(W, [want0, 1 - want0], rtol=1e-14)


@pytest.mark.parametrize("levels", [1, 3, 5])
def test_haar_skim_from_token_logits(ref, levels):
    """For Haar, <Q_i, A_J[j]> = 2^{-J/2} * sum over the block of
    <Q_i, K_t>: the skim logits recomputed from token-level logits."""
    rng = _rng(levels + 20)
    L, d, B = 256, 32, 6
    K = rng.standard_normal((L, d))
    Q = rng.standard_normal((B, d))
    scale = 1 / math.sqrt(d)
    W = ref.skim(Q, ref.dwt(K, levels, "haar"))
    tok_logit = scale * (Q @ K.T)
    s = tok_logit.reshape(B, -1, 1 << levels).sum(-1) * 2.0 ** (-levels / 2)
    want = scipy.special.softmax(s, axis=1).sum(axis=0)
    np.testing.assert_allclose(W, want, rtol=1e-12)


def test_single_query_skim_ranks_by_logit(ref):
    """With B = 1 the softmax is monotone: the top-S coarse regions are the
    top-S raw logits."""
    rng = _rng(9)
    Q = rng.standard_normal((1, 16))
    A = rng.standard_normal((64, 16))
    W = ref.skim(Q, A)
    raw = (Q @ A.T)[0]
    for S in (1, 5, 17):
        assert list(ref.topk(W, S)) == sorted(np.argsort(-raw)[:S].tolist())


def test_query_permutation_invariance(ref):
    """Permuting the query rows permutes nothing in W (a column sum)."""
    rng = _rng(4)
    Q = rng.standard_normal((12, 16))
    A = rng.standard_normal((50, 16))
    perm = rng.permutation(12)
    np.testing.assert_allclose(ref.skim(Q[perm], A), ref.skim(Q, A),
                               rtol=1e-13)


# ------------------------------------------------------------- top-k (O3/O6)

def _brute_force_topk(s, k):
    """The unique k-subset C with: x in C, y not in C => s_x > s_y, or
    s_x == s_y and x < y."""
    n = len(s)
    found = []
    for C in itertools.combinations(range(n), k):
        Cs = set(C)
        ok = all((s[x] > s[y]) or (s[x] == s[y] and x < y)
                 for x in Cs for y in range(n) if y not in Cs)
        if ok:
            found.append(list(C))
    assert len(found) == 1
    return found[0]


def test_topk_brute_force_with_ties(ref):
    rng = _rng(2)
    for trial in range(60):
        n = int(rng.integers(1, 9))
        s = rng.choice([0.1, 0.25, 0.5, 0.5, 1.0, 2.0], size=n)
        for k in range(1, n + 1):
            assert list(ref.topk(s, k)) == _brute_force_topk(s, k)


def test_topk_rejects_bad_k(ref):
    with pytest.raises(ValueError):
        ref.topk(np.ones(4), 5)
    with pytest.raises(ValueError):
        ref.topk(np.ones(4), 0)


# ----------------------------------------------------------- scan (O4-O6)

def test_scan_keep_all_returns_the_pool(ref):
    """With a budget at least the pool size, mu^0 is the whole pool: the
    union of eq. 10's token ranges of the kept regions."""
    rng = _rng(6)
    L, d, B, J = 512, 16, 4, 3
    K = rng.standard_normal((L, d))
    Q = rng.standard_normal((B, d))
    seg = np.array([0, 5, 6, 40, 63])
    Wp, tok = ref.scan(Q, K, seg, J, budget=10_000)
    want = np.concatenate([np.arange(8 * j, 8 * j + 8) for j in seg])
    assert list(tok) == list(want)
    assert abs(Wp.sum() - B) < 1e-12


def test_scan_single_query_ranks_by_token_logit(ref):
    rng = _rng(8)
    L, d, J = 256, 16, 2
    K = rng.standard_normal((L, d))
    Q = rng.standard_normal((1, d))
    seg = np.array([3, 9, 10, 30, 50])
    pool = np.concatenate([np.arange(4 * j, 4 * j + 4) for j in seg])
    raw = (Q @ K[pool].T)[0]
    _, tok = ref.scan(Q, K, seg, J, budget=7)
    assert list(tok) == sorted(pool[np.argsort(-raw)[:7]].tolist())


def test_constant_keys_select_the_first_regions(ref):
    """All scores tie: the lowest indices win at both stages."""
    L, d, B, J, S, k = 256, 8, 4, 3, 5, 20
    K = np.ones((L, d)) * 0.5
    V = _rng(0).standard_normal((L, d))
    Q = _rng(1).standard_normal((B, d))
    out = ref.filter_attend_unit(Q, K, V, J, S, k)
    assert list(out["seg"]) == list(range(S))
    assert list(out["tok"]) == list(range(k))


def test_scan_rejects_unsorted_regions(ref):
    K = np.zeros((64, 4))
    Q = np.zeros((1, 4))
    with pytest.raises(ValueError):
        ref.scan(Q, K, np.array([3, 1]), 2, 4)


# ------------------------------------------------------- attention (O7-O8)

def _sdpa(Q, Ks, Vs, scale):
    q = torch.from_numpy(Q)[None, None]
    k = torch.from_numpy(np.ascontiguousarray(Ks))[None, None]
    v = torch.from_numpy(np.ascontiguousarray(Vs))[None, None]
    o = torch.nn.functional.scaled_dot_product_attention(q, k, v, scale=scale)
    return o[0, 0].numpy()


def test_attention_matches_sdpa_with_tail(ref):
    rng = _rng(12)
    L, d, B, G = 300, 32, 9, 5
    K = rng.standard_normal((L, d))
    V = rng.standard_normal((L, d))
    Kg = rng.standard_normal((G, d))
    Vg = rng.standard_normal((G, d))
    Q = rng.standard_normal((B, d))
    tok = np.sort(rng.choice(L, 37, replace=False))
    O = ref.attend(Q, K, V, tok, Kg, Vg)
    want = _sdpa(Q, np.concatenate([K[tok], Kg]), np.concatenate([V[tok], Vg]),
                 1 / math.sqrt(d))
    np.testing.assert_allclose(O, want, rtol=0, atol=1e-12)


def test_attention_closed_forms(ref):
    rng = _rng(13)
    L, d = 64, 8
    K = rng.standard_normal((L, d))
    V = rng.standard_normal((L, d))
    tok = np.array([2, 9, 33, 60])
    # Q = 0: uniform weights, the mean of the selected values.
    O = ref.attend(np.zeros((3, d)), K, V, tok)
    np.testing.assert_allclose(O, np.tile(V[tok].mean(0), (3, 1)), atol=1e-14)
    # one key: the output is that key's value row.
    O = ref.attend(rng.standard_normal((2, d)), K, V, np.array([17]))
    np.testing.assert_allclose(O, np.tile(V[17], (2, 1)), atol=1e-14)


# ------------------------------------------------------------ end to end

@pytest.mark.parametrize("wavelet", ["haar", "db2"])
def test_keep_all_equals_dense_attention(ref, wavelet):
    """Keeping every region and every token turns the sparse cache into the
    full cache: O equals dense attention over all prompt keys plus the tail
    (eq. 3 form)."""
    rng = _rng(14)
    L, d, B, J, G = 256, 16, 6, 3, 4
    K = rng.standard_normal((L, d))
    V = rng.standard_normal((L, d))
    Q = rng.standard_normal((B, d))
    Kg = rng.standard_normal((G, d))
    Vg = rng.standard_normal((G, d))
    out = ref.filter_attend_unit(Q, K, V, J, L >> J, 10 * L, wavelet=wavelet,
                                 Kg=Kg, Vg=Vg)
    assert list(out["tok"]) == list(range(L))
    want = _sdpa(Q, np.concatenate([K, Kg]), np.concatenate([V, Vg]),
                 1 / math.sqrt(d))
    np.testing.assert_allclose(out["O"], want, rtol=0, atol=1e-12)


def test_batched_entry_matches_per_unit(ref):
    w = synth.WORKLOADS["tiny_scan"]
    Q, K, V = synth.make_inputs(w, workers=1)
    U = w.units
    O, tok = ref.filter_attend(Q.reshape(U, w.q_len, -1),
                               K.reshape(U, w.ctx_len, -1),
                               V.reshape(U, w.ctx_len, -1),
                               w.levels, w.segments, w.budget)
    for u in range(U):
        one = ref.filter_attend_unit(Q.reshape(U, w.q_len, -1)[u],
                                     K.reshape(U, w.ctx_len, -1)[u],
                                     V.reshape(U, w.ctx_len, -1)[u],
                                     w.levels, w.segments, w.budget)
        np.testing.assert_array_equal(one["tok"], tok[u])
        np.testing.assert_array_equal(one["O"], O[u])


def test_tiny_workload_finds_the_needle(ref):
    """On the tiny workload the kept tokens cover most of the planted needle
    span (a data-dependent sanity check of the input recipe, not a pin of the
    method: a needle that straddles a region border can lose its edge)."""
    w = synth.WORKLOADS["tiny"]
    Q, K, V = synth.make_inputs(w, workers=1)
    s = int(synth.needle_starts(w, 0, 0)[0])
    for h in range(w.heads):
        out = ref.filter_attend_unit(Q[0, h], K[0, h], V[0, h], w.levels,
                                     w.segments, w.budget)
        hit = set(range(s, s + synth.NEEDLE_LEN)) & set(out["tok"].tolist())
        assert len(hit) >= synth.NEEDLE_LEN // 2


# ------------------------------------------------------------- generator

def test_generator_is_deterministic():
    w = synth.small_variant(synth.WORKLOADS["tiny"], ctx_len=256)
    a = synth.unit_f64(w, 0, 0, 1)
    b = synth.unit_f64(w, 0, 0, 1)
    c = synth.unit_f64(w, 0, 0, 0)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)
    assert not np.array_equal(a[1], c[1])
    # keys have (roughly) the stated marginal variance 1 + 0.3^2 off-needle
    Q, K, V = synth.unit_f64(synth.WORKLOADS["layer8b"], 0, 0, 0)
    assert 0.8 < K[:1000].var() < 1.4


# ------------------------------------------------- recursion (R1, eqs. 9-11)

def _haar_recursion_numpy(Q, K, levels, props, scale):
    """The recursion with the Haar transform of each gathered sequence taken
    from its closed form (2^{-b/2} times sums of aligned 2^b runs of the
    gathered rows), eqs. 7-9 written out with numpy, and the count rule
    c = max(1, ceil(m n)).  Shares nothing with the oracle but the inputs."""
    L, d = K.shape
    mu = np.arange(L)
    for b in range(levels, 0, -1):
        run = 1 << b
        n = mu.size // run
        C = K[mu].reshape(n, run, d).sum(axis=1) * 2.0 ** (-b / 2)
        s = scale * (Q @ C.T)
        p = np.exp(s - s.max(axis=1, keepdims=True))
        W = (p / p.sum(axis=1, keepdims=True)).sum(axis=0)
        c = min(n, max(1, math.ceil(props[b - 1] * n)))
        order = np.lexsort((np.arange(n), -W))
        J = np.sort(order[:c])
        mu = mu.reshape(n, run)[J].reshape(-1)
    return mu


@pytest.mark.parametrize("levels,props", [
    (1, [0.3]), (2, [0.5, 0.4]), (3, [0.6, 0.5, 0.25]), (5, [0.9, 0.7, 0.5, 0.5, 0.2])])
def test_recursion_haar_matches_closed_form_route(ref, levels, props):
    """Haar: the transform of a gathered sequence is 2^{-b/2} times sums of
    its aligned runs, so a numpy recursion built on that closed form must pick
    the same positions at every scale."""
    rng = _rng(100 + levels)
    L, d, B = 256, 8, 5
    K = rng.standard_normal((L, d))
    Q = rng.standard_normal((B, d)) * 0.7
    tok, counts = ref.recursive_select(Q, K, levels, props, "haar")
    want = _haar_recursion_numpy(Q, K, levels, props, 1 / math.sqrt(d))
    np.testing.assert_array_equal(tok, want)
    assert tok.size == 2 * counts[0]
    assert np.all(np.diff(tok) > 0)


def test_recursion_counts_follow_the_proportions(ref):
    """c_b = max(1, ceil(m_b n_b)) with n_B = L / 2^B and n_b = 2 c_{b+1}."""
    rng = _rng(7)
    L, levels = 512, 4
    props = [0.3, 0.55, 0.01, 0.75]
    tok, counts = ref.recursive_select(rng.standard_normal((3, 4)),
                                       rng.standard_normal((L, 4)), levels,
                                       props)
    n = L >> levels
    want = {}
    for b in range(levels, 0, -1):
        c = min(n, max(1, math.ceil(props[b - 1] * n)))
        want[b] = c
        n = 2 * c
    assert [int(counts[b - 1]) for b in range(1, levels + 1)] == \
        [want[b] for b in range(1, levels + 1)]
    assert tok.size == 2 * want[1]
    assert ref.recursion_count(0.01, 64) == 1          # at least one
    assert ref.recursion_count(1.0, 64) == 64
    assert ref.recursion_count(0.5, 63) == 32          # rounds up


@pytest.mark.parametrize("wavelet,boundary", [("haar", "symmetric"),
                                              ("db2", "symmetric"),
                                              ("db2", "periodic")])
def test_recursion_keep_all_is_every_position(ref, wavelet, boundary):
    """All m_b = 1: every scale keeps every coefficient, so mu^0 is the whole
    prompt and the attention is dense attention."""
    rng = _rng(11)
    L, d, B = 128, 6, 4
    Q, K, V = (rng.standard_normal(s) for s in ((B, d), (L, d), (L, d)))
    tok, _ = ref.recursive_select(Q, K, 3, [1.0, 1.0, 1.0], wavelet, boundary)
    np.testing.assert_array_equal(tok, np.arange(L))
    O, toks = ref.filter_attend_recursive(Q[None], K[None], V[None], 3,
                                          [1.0] * 3, wavelet, boundary)
    s = Q @ K.T / math.sqrt(d)
    p = np.exp(s - s.max(axis=1, keepdims=True))
    dense = (p / p.sum(axis=1, keepdims=True)) @ V
    np.testing.assert_allclose(O[0], dense, rtol=0, atol=1e-12)


def test_recursion_constant_keys_keep_the_first_positions(ref):
    """Equal keys tie every weight at every scale; ties go to the lower
    index, so mu^0 is the first 2 c_1 positions."""
    L, levels = 256, 3
    K = np.full((L, 5), 0.25)
    Q = _rng(3).standard_normal((4, 5))
    props = [0.5, 0.25, 0.5]
    tok, counts = ref.recursive_select(Q, K, levels, props, "db2")
    np.testing.assert_array_equal(tok, np.arange(2 * counts[0]))


def test_recursion_single_query_ranks_by_block_logit(ref):
    """One query row: the softmax is monotone, so each scale keeps the c_b
    candidates of largest coarse logit <Q, C_b[j]>."""
    rng = _rng(21)
    L, d = 128, 7
    K = rng.standard_normal((L, d))
    q = rng.standard_normal((1, d))
    tok, counts = ref.recursive_select(q, K, 2, [0.5, 0.25], "haar")
    mu = np.arange(L)
    for b in (2, 1):
        n = mu.size >> b
        C = K[mu].reshape(n, 1 << b, d).sum(axis=1)  # positive rescaling
        s = (q @ C.T)[0]
        c = int(counts[b - 1])
        J = np.sort(np.argsort(-s, kind="stable")[:c])
        mu = mu.reshape(n, 1 << b)[J].reshape(-1)
    np.testing.assert_array_equal(tok, mu)


def test_recursion_query_permutation_invariance(ref):
    rng = _rng(5)
    Q = rng.standard_normal((6, 8))
    K = rng.standard_normal((256, 8))
    a, _ = ref.recursive_select(Q, K, 3, [0.5, 0.5, 0.25], "db2")
    b, _ = ref.recursive_select(Q[::-1].copy(), K, 3, [0.5, 0.5, 0.25], "db2")
    np.testing.assert_array_equal(a, b)


def test_recursion_db2_periodic_keep_all_matches_the_pyramid(ref):
    """With every scale keeping everything the gathered sequence at scale b is
    the whole prompt, so eq. 11's transform must equal the b-level transform
    of the prompt (a periodic db2 pyramid of the oracle's own O1, pinned
    above); checked through the first scale's ranking: a single query ranks
    the whole prompt by <q, A_B[j]>."""
    rng = _rng(9)
    L, d = 128, 5
    K = rng.standard_normal((L, d))
    q = rng.standard_normal((1, d))
    A = ref.dwt(K, 2, "db2", "periodic")
    c = ref.recursion_count(0.25, L >> 2)
    tok, _ = ref.recursive_select(q, K, 2, [1.0, 0.25], "db2", "periodic")
    J = np.sort(np.argsort(-(q @ A.T)[0], kind="stable")[:c])
    want = (J[:, None] * 4 + np.arange(4)).reshape(-1)
    np.testing.assert_array_equal(tok, want)


def test_recursion_db2_gathers_before_transforming(ref):
    """eq. 11 transforms the gathered keys as one sequence: for db2 the
    filter reads across the joins between kept regions, so the second scale
    is not the prompt's pyramid restricted to the kept regions.  With one
    query, the second scale's ranking follows <q, DWT(K[mu^1])>."""
    rng = _rng(13)
    L, d = 256, 4
    K = rng.standard_normal((L, d))
    q = rng.standard_normal((1, d))
    tok, counts = ref.recursive_select(q, K, 2, [0.25, 0.25], "db2")
    A2 = ref.dwt(K, 2, "db2")
    c2 = int(counts[1])
    J2 = np.sort(np.argsort(-(q @ A2.T)[0], kind="stable")[:c2])
    mu1 = (J2[:, None] * 4 + np.arange(4)).reshape(-1)
    C1 = ref.dwt(K[mu1], 1, "db2")                  # gathered, then transformed
    c1 = int(counts[0])
    J1 = np.sort(np.argsort(-(q @ C1.T)[0], kind="stable")[:c1])
    want = mu1.reshape(-1, 2)[J1].reshape(-1)
    np.testing.assert_array_equal(tok, want)
    # the pyramid restricted to the kept regions would rank differently here
    A1 = ref.dwt(K, 1, "db2")
    kept = mu1.reshape(-1, 2)[:, 0] // 2
    J1_pyr = np.sort(np.argsort(-(q @ A1[kept].T)[0], kind="stable")[:c1])
    assert not np.array_equal(J1_pyr, J1)


# --------------------------------------------- grouped query heads (GQA)

def test_grouped_heads_sum_of_weights_is_the_stacked_skim(ref):
    """W summed over the query heads that share a KV head equals the skim of
    the stacked query rows (eq. 8 is a column sum of row-wise softmaxes), so
    one selection per KV head is the selection of the stacked block."""
    rng = _rng(31)
    g, B, d, n = 4, 6, 8, 64
    A = rng.standard_normal((n, d))
    Qh = [rng.standard_normal((B, d)) for _ in range(g)]
    per_head = sum(ref.skim(q, A) for q in Qh)
    stacked = ref.skim(np.concatenate(Qh), A)
    np.testing.assert_allclose(stacked, per_head, rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(stacked.sum(), g * B, rtol=1e-12)


# ----------------------------------------- lengths not a multiple of 2^J

@pytest.mark.parametrize("levels,rem", [(3, 5), (4, 1), (2, 3)])
def test_remainder_is_kept_like_a_tail(ref, levels, rem):
    """A prompt of L = Lf + r positions (Lf a multiple of 2^J, 0 < r < 2^J):
    the first Lf are filtered and the last r always kept, which is the
    filtered path on the first Lf positions with those r rows placed in
    front of the generation tail (the tail path is pinned to SDPA above)."""
    rng = _rng(40 + levels)
    Lf, d, B, G = 256, 8, 5, 3
    L = Lf + rem
    Q = rng.standard_normal((B, d))
    K, V = rng.standard_normal((L, d)), rng.standard_normal((L, d))
    Kg, Vg = rng.standard_normal((G, d)), rng.standard_normal((G, d))
    S, k = 6, 20
    got = ref.filter_attend_unit(Q, K, V, levels, S, k, Kg=Kg, Vg=Vg)
    want = ref.filter_attend_unit(Q, K[:Lf], V[:Lf], levels, S, k,
                                  Kg=np.concatenate([K[Lf:], Kg]),
                                  Vg=np.concatenate([V[Lf:], Vg]))
    np.testing.assert_array_equal(got["tok"], want["tok"])
    np.testing.assert_array_equal(got["seg"], want["seg"])
    np.testing.assert_allclose(got["O"], want["O"], rtol=0, atol=1e-13)


def test_recursion_remainder_follows_mu0(ref):
    rng = _rng(77)
    Lf, rem, d = 256, 3, 6
    K = rng.standard_normal((Lf + rem, d))
    Q = rng.standard_normal((4, d))
    got, _ = ref.recursive_select(Q, K, 3, [0.5, 0.5, 0.25])
    base, _ = ref.recursive_select(Q, K[:Lf], 3, [0.5, 0.5, 0.25])
    np.testing.assert_array_equal(got, np.concatenate([base, np.arange(Lf, Lf + rem)]))


# ------------------------------------------------ layer-shared selection

def _shared_case(H, L=512, d=32, B=8, seed=7):
    rng = np.random.default_rng(seed)
    Q = rng.standard_normal((H, B, d)) / np.sqrt(d)
    K = rng.standard_normal((H, L, d)) * 0.3
    V = rng.standard_normal((H, L, d))
    return Q, K, V


def test_shared_selection_of_one_head_is_the_per_head_selection(ref):
    """H = 1: the shared path reduces to O1-O8 of that unit."""
    Q, K, V = _shared_case(1)
    sh = ref.filter_attend_shared(Q, K, V, 3, 10, 40)
    un = ref.filter_attend_unit(Q[0], K[0], V[0], 3, 10, 40)
    assert np.array_equal(sh["seg"], un["seg"]) and np.array_equal(sh["tok"], un["tok"])
    assert np.allclose(sh["W"], un["W"], rtol=1e-13, atol=0)
    assert np.allclose(sh["Wp"], un["Wp"], rtol=1e-13, atol=0)
    assert np.allclose(sh["O"][0], un["O"], rtol=0, atol=1e-13)


def test_shared_selection_of_identical_heads_is_each_heads_selection(ref):
    """H copies of one unit: the summed weights are H times the unit's, so
    the regions and tokens are the unit's and every head's output is its."""
    Q, K, V = _shared_case(1, seed=8)
    H = 4
    sh = ref.filter_attend_shared(np.repeat(Q, H, 0), np.repeat(K, H, 0),
                                     np.repeat(V, H, 0), 3, 12, 50)
    un = ref.filter_attend_unit(Q[0], K[0], V[0], 3, 12, 50)
    assert np.array_equal(sh["seg"], un["seg"]) and np.array_equal(sh["tok"], un["tok"])
    assert np.allclose(sh["W"], H * un["W"], rtol=1e-12, atol=0)
    for h in range(H):
        assert np.allclose(sh["O"][h], un["O"], rtol=0, atol=1e-13)


def test_shared_weights_are_the_heads_summed_softmax_column_sums(ref):
    """Haar W recomputed from scratch: A_J as 2^(-J/2) block sums, a
    row softmax per head, column sums added over the heads."""
    H, J = 3, 2
    Q, K, V = _shared_case(H, L=64, d=8, B=5, seed=9)
    sh = ref.filter_attend_shared(Q, K, V, J, 4, 8)
    W = np.zeros(64 >> J)
    for h in range(H):
        A = K[h].reshape(-1, 1 << J, 8).sum(1) * 2.0 ** (-J / 2)
        s = Q[h] @ A.T / np.sqrt(8)
        p = np.exp(s - s.max(1, keepdims=True))
        W += (p / p.sum(1, keepdims=True)).sum(0)
    assert np.allclose(sh["W"], W, rtol=1e-12, atol=0)
    # the pool weights the same way over the shared pool, at token level
    pool = (sh["seg"][:, None] * 4 + np.arange(4)).ravel()
    Wp = np.zeros(pool.size)
    for h in range(H):
        s = Q[h] @ K[h][pool].T / np.sqrt(8)
        p = np.exp(s - s.max(1, keepdims=True))
        Wp += (p / p.sum(1, keepdims=True)).sum(0)
    assert np.allclose(sh["Wp"], Wp, rtol=1e-12, atol=0)


def test_shared_selection_keeps_each_heads_needle(ref):
    """Head h's queries point at a needle only its own keys carry, in a
    block of its own: with S = H every needle block is kept, although no
    head alone scores the others' blocks."""
    H, L, d, B, J = 3, 256, 16, 4, 3
    rng = np.random.default_rng(11)
    K = rng.standard_normal((H, L, d)) * 0.1
    V = rng.standard_normal((H, L, d))
    Q = np.zeros((H, B, d))
    blocks = [5, 17, 26]
    for h in range(H):
        u = np.zeros(d)
        u[h] = 1.0
        K[h, blocks[h] * 8:(blocks[h] + 1) * 8] += 4 * u
        Q[h] = 4 * u + 0.01 * rng.standard_normal((B, d))
    sh = ref.filter_attend_shared(Q, K, V, J, H, 8 * H)
    assert sorted(sh["seg"].tolist()) == blocks
    assert np.array_equal(sh["tok"], np.concatenate([np.arange(b * 8, b * 8 + 8) for b in blocks]))
    # every head attends with its own keys and values at the shared tokens
    for h in range(H):
        s = Q[h] @ K[h][sh["tok"]].T / np.sqrt(d)
        p = np.exp(s - s.max(1, keepdims=True))
        O = (p / p.sum(1, keepdims=True)) @ V[h][sh["tok"]]
        assert np.allclose(sh["O"][h], O, rtol=0, atol=1e-12)
