"""Pins for the CPU oracle: each check is fixed by the mathematics, a library
routine or a published value -- never by re-typing the oracle's own formula.

Paper = "GaLore 2" (Su et al. 2025); Halko = Halko, Martinsson & Tropp 2011.
"""
import os

import numpy as np
import pytest

import galore_inputs as gi
from metrics import proj_dist

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
U64 = (1 << 64) - 1


# ---------------------------------------------------------------- Philox / sketch


def test_philox_known_answer(orc):
    """Published known-answer vector of Philox4x64-10 (Salmon et al. 2011)."""
    rows = [ln.split() for ln in open(os.path.join(GOLDEN, "philox4x64_10_kat.txt")) if ln.strip() and not ln.startswith("#")]
    assert rows
    for row in rows:
        v = [int(x, 16) for x in row]
        out = orc.philox4x64_10(v[0:4], v[4:6])
        assert [int(x) for x in out] == v[6:10]


@pytest.mark.parametrize("seed", [0, 1, 20250429, 2**63 + 12345])
def test_philox_matches_numpy_bit_generator(orc, seed):
    """numpy.random.Philox is Philox4x64-10; it increments the counter before each block."""
    rng = np.random.default_rng(seed)
    for _ in range(8):
        key = [int(x) for x in rng.integers(0, 2**63, size=2, dtype=np.int64)]
        ctr = [int(x) for x in rng.integers(0, 2**63, size=4, dtype=np.int64)]
        bg = np.random.Philox(key=np.array(key, dtype=np.uint64), counter=np.array(ctr, dtype=np.uint64))
        ref = bg.random_raw(8)
        c1 = [(ctr[0] + 1) & U64] + ctr[1:]
        c2 = [(ctr[0] + 2) & U64] + ctr[1:]
        got = np.concatenate([orc.philox4x64_10(c1, key), orc.philox4x64_10(c2, key)])
        assert np.array_equal(got.astype(np.uint64), ref.astype(np.uint64))


def test_box_muller_pair(orc):
    """The pair's radius is shared: z0^2 + z1^2 = -2 ln u1; u2 = 1/4 puts the
    whole radius in the sin member, u2 = 0 in the cos member."""
    r2 = -2.0 * np.log(2.0 ** -53)
    z0, z1 = orc.normal_pair_from_words(0, 1 << 62)          # u1 = 2^-53, u2 = 1/4
    assert abs(z0) < 1e-12 and abs(z1 - np.sqrt(r2)) < 1e-12
    z0, z1 = orc.normal_pair_from_words(0, 0)
    assert abs(z0 - np.sqrt(r2)) < 1e-12 and z1 == 0.0
    z0, z1 = orc.normal_pair_from_words(12345 << 11, 777 << 20)
    u1 = (12345 + 1) * 2.0 ** -53
    assert abs(z0 * z0 + z1 * z1 + 2.0 * np.log(u1)) < 1e-12


def test_box_muller_edges(orc):
    # u1 = 1 exactly (all top bits set) -> radius 0
    assert orc.normal_from_words(U64, 12345) == 0.0
    # u2 = 0 -> cos = 1 -> z = sqrt(-2 ln u1) > 0 ; smallest u1 = 2^-53 -> largest radius
    z = orc.normal_from_words(0, 0)
    assert abs(z - np.sqrt(2.0 * 53.0 * np.log(2.0))) < 1e-12
    # u2 = 1/2 -> cos = -1
    z = orc.normal_from_words(0, 1 << 63)
    assert abs(z + np.sqrt(2.0 * 53.0 * np.log(2.0))) < 1e-12


def test_sketch_is_standard_normal(orc):
    """Halko §4 needs i.i.d. N(0,1) entries: moments of 1e6 sketch entries, and a
    KS test of the normals before their bfloat16 rounding (the rounded values
    form a lattice, which a continuous KS test would reject by construction;
    the rounding moves each entry by at most 2^-8 of its magnitude)."""
    from scipy import stats
    om = orc.sketch(1000, 1000, seed=7, sketch_index=3)
    x = om.ravel()
    assert abs(x.mean()) < 5e-3
    assert abs(x.var() - 1.0) < 5e-3
    assert abs(stats.skew(x)) < 1e-2 and abs(stats.kurtosis(x)) < 2e-2
    rng = np.random.default_rng(8)
    z = np.array([orc.normal_from_words(int(a), int(b))
                  for a, b in rng.integers(0, 2 ** 63, size=(20000, 2), dtype=np.int64) * 2 + 1])
    assert stats.kstest(z, "norm").pvalue > 1e-3
    # independent columns / rows (including the rows of one Philox block: the
    # two members of a Box-Muller pair, and the two pairs)
    assert abs(np.corrcoef(om[:, 0], om[:, 1])[0, 1]) < 0.15
    assert abs(np.mean(om[:-1, :] * om[1:, :])) < 5e-3
    for a, b in ((0, 1), (2, 3), (0, 2), (1, 3)):
        assert abs(np.mean(om[a::4, :] * om[b::4, :])) < 1e-2


def test_round_bf16_ties_and_single_rounding(orc):
    """bfloat16 keeps 8 significant bits: near 1 the spacing is 2^-7. 1 + 2^-8 is
    a tie and goes to the even 1.0; 1 + 3 * 2^-8 goes to the even 1 + 2^-6; 1 +
    2^-8 + 2^-30 lies above the tie and rounds up (rounding through binary32
    first would lose the 2^-30 and round down); signs are symmetric."""
    assert orc.round_bf16(1 + 2.0 ** -8) == 1.0
    assert orc.round_bf16(1 + 3 * 2.0 ** -8) == 1 + 2.0 ** -6
    assert orc.round_bf16(1 + 2.0 ** -8 + 2.0 ** -30) == 1 + 2.0 ** -7
    assert orc.round_bf16(-(1 + 2.0 ** -8 + 2.0 ** -30)) == -(1 + 2.0 ** -7)
    assert orc.round_bf16(3.0) == 3.0 and orc.round_bf16(0.0) == 0.0


def test_sketch_structure(orc):
    a = orc.sketch(37, 9, seed=11, sketch_index=0)
    b = orc.sketch(37, 5, seed=11, sketch_index=0)
    assert np.array_equal(a[:, :5], b)                      # columns do not depend on k
    bits = a.astype(np.float32).view(np.uint32)
    assert np.array_equal(a.astype(np.float32).astype(np.float64), a) and not np.any(bits & 0xFFFF)   # bf16 values
    c = orc.sketch(37, 9, seed=11, sketch_index=1)
    d = orc.sketch(37, 9, seed=12, sketch_index=0)
    assert not np.any(a == c) or np.mean(a == c) < 0.05
    assert np.mean(a == d) < 0.05
    # entries (4 i4 + t, j) use counter j * ceil(l / 4) + i4, key (seed, 0):
    # words 0, 1 give rows 4 i4 and 4 i4 + 1 (cos and sin of one Box-Muller
    # pair), words 2, 3 rows 4 i4 + 2 and 4 i4 + 3; each rounded to bfloat16
    # (within half its spacing, at most 2^-8 relative)
    w = orc.philox4x64_10([4 * 10 + 2, 0, 0, 0], [11, 0])
    z = orc.normal_pair_from_words(int(w[0]), int(w[1])) + orc.normal_pair_from_words(int(w[2]), int(w[3]))
    assert z[0] == orc.normal_from_words(int(w[0]), int(w[1]))
    for t in range(4):
        assert a[8 + t, 4] == orc.round_bf16(z[t])
        assert abs(a[8 + t, 4] - z[t]) <= 2.0 ** -8 * abs(z[t])
    # the last row (l = 37 = 4 * 9 + 1) uses the cos member of its block's first pair
    w = orc.philox4x64_10([2 * 10 + 9, 0, 0, 0], [11, 0])
    assert a[36, 2] == orc.round_bf16(orc.normal_pair_from_words(int(w[0]), int(w[1]))[0])


# ---------------------------------------------------------------- Householder QR


@pytest.mark.parametrize("shape", [(50, 12), (12, 12), (300, 40), (7, 1)])
def test_householder_qr_against_lapack(orc, shape):
    rng = np.random.default_rng(sum(shape))
    Y = rng.standard_normal(shape)
    Q, R = orc.householder_qr(Y)
    k = shape[1]
    assert np.abs(Q.T @ Q - np.eye(k)).max() < 1e-13
    assert np.abs(Q @ R - Y).max() < 1e-13 * max(1.0, np.abs(Y).max())
    assert np.allclose(np.tril(R, -1), 0.0)
    Ql, Rl = np.linalg.qr(Y)
    assert np.abs(Q @ Q.T - Ql @ Ql.T).max() < 1e-12
    assert np.allclose(np.abs(np.diag(R)), np.abs(np.diag(Rl)), rtol=1e-12, atol=1e-13)


def test_householder_qr_degenerate(orc):
    Q, R = orc.householder_qr(np.zeros((9, 4)))
    assert np.array_equal(Q, np.eye(9)[:, :4]) and np.array_equal(R, np.zeros((4, 4)))
    rng = np.random.default_rng(5)
    x = rng.standard_normal((20, 2))
    Y = np.column_stack([x[:, 0], 2 * x[:, 0], x[:, 1], np.zeros(20)])   # rank 2
    Q, R = orc.householder_qr(Y)
    assert np.abs(Q.T @ Q - np.eye(4)).max() < 1e-13
    assert np.abs(Q @ R - Y).max() < 1e-13


# ---------------------------------------------------------------- Jacobi SVD


@pytest.mark.parametrize("shape", [(8, 20), (20, 20), (40, 688), (1, 5)])
def test_jacobi_against_lapack(orc, shape):
    rng = np.random.default_rng(shape[0] * 31 + shape[1])
    B = rng.standard_normal(shape)
    U, s, sw = orc.jacobi_left_svd(B)
    assert sw >= 0          # -1 would mean no convergence
    sl = np.linalg.svd(B, compute_uv=False)
    assert np.abs(s - sl).max() <= 1e-12 * sl[0]
    assert np.all(np.diff(s) <= 0)
    assert np.abs(U.T @ U - np.eye(shape[0])).max() < 1e-13
    # reconstruction: B = U diag(s) Vhat^T with Vhat = B^T U diag(1/s)
    Vh = (B.T @ U) / s
    assert np.abs(U @ np.diag(s) @ Vh.T - B).max() < 1e-12
    assert np.abs(Vh.T @ Vh - np.eye(shape[0])).max() < 1e-11
    Ul, _, _ = np.linalg.svd(B)
    for j in range(shape[0]):
        if j + 1 < shape[0] and (sl[j] - sl[j + 1]) < 1e-6 * sl[0]:
            continue
        if j > 0 and (sl[j - 1] - sl[j]) < 1e-6 * sl[0]:
            continue
        assert abs(abs(U[:, j] @ Ul[:, j]) - 1.0) < 1e-10


def test_jacobi_closed_forms(orc):
    d = np.array([0.5, -3.0, 2.0, 0.0])
    B = np.zeros((4, 6))
    B[np.arange(4), np.arange(4)] = d
    U, s, _ = orc.jacobi_left_svd(B)
    assert np.array_equal(s, np.array([3.0, 2.0, 0.5, 0.0]))
    assert np.array_equal(np.abs(U), np.eye(4)[:, [1, 2, 0, 3]])
    rng = np.random.default_rng(9)
    x, y = rng.standard_normal(5), rng.standard_normal(11)
    U, s, _ = orc.jacobi_left_svd(np.outer(x, y))
    assert abs(s[0] - np.linalg.norm(x) * np.linalg.norm(y)) < 1e-13 * s[0]
    assert np.all(s[1:] < 1e-13 * s[0])
    assert abs(abs(U[:, 0] @ x) / np.linalg.norm(x) - 1.0) < 1e-13


def test_canonical_signs(orc):
    P = np.array([[0.1, -0.9, 0.5], [-0.8, 0.2, -0.5], [0.3, 0.1, 0.1]])
    C = orc.canonical_signs(P)
    assert np.array_equal(C[:, 0], -P[:, 0])       # largest |.| is -0.8
    assert np.array_equal(C[:, 1], -P[:, 1])       # largest |.| is -0.9
    assert np.array_equal(C[:, 2], P[:, 2])        # tie 0.5/-0.5: lowest row (+) wins


# ---------------------------------------------------------------- randomized SVD


def test_rsvd_full_sketch_equals_exact_svd(orc):
    """k = min(r+p, s) = s: the sketch spans the whole range, so the rSVD is the
    exact SVD (textbook reduction)."""
    rng = np.random.default_rng(3)
    for (m, n, r, p) in [(6, 9, 4, 2), (9, 6, 3, 5), (8, 8, 5, 3)]:
        G = rng.standard_normal((m, n))
        P, sig, sw = orc.rsvd_update(G, r, p, 1, seed=5)
        u, ss, vt = np.linalg.svd(G)
        ref = u[:, :r] if m <= n else vt.T[:, :r]
        assert np.abs(sig - ss[:r]).max() < 1e-12 * ss[0]
        assert proj_dist(P, ref) < 1e-10
        for j in range(r):
            assert abs(abs(P[:, j] @ ref[:, j]) - 1.0) < 1e-10


@pytest.mark.parametrize("m,n,rank,r,p,q", [(256, 688, 32, 32, 8, 2), (256, 688, 36, 32, 8, 1),
                                             (688, 256, 20, 32, 8, 2), (64, 64, 10, 12, 4, 0)])
def test_rsvd_exact_recovery(orc, m, n, rank, r, p, q):
    """rank(G) <= k (noiseless): range(Y) = range(G), so the planted spectrum and
    the planted singular subspace are recovered exactly."""
    s = 10.0 * 0.85 ** np.arange(min(m, n))
    G = gi.planted_gradient(m, n, s, 0.0, seed=rank, rank=rank)
    P, sig, sw = orc.rsvd_update(G, r, p, q, seed=99)
    nr = min(r, rank)
    assert np.abs(sig[:nr] - s[:nr]).max() < 1e-12 * s[0]
    assert np.all(np.abs(sig[nr:]) < 1e-12 * s[0])
    u, ss, vt = np.linalg.svd(G)
    ref = (u if m <= n else vt.T)[:, :nr]
    assert proj_dist(P[:, :nr], ref) < 1e-10
    assert np.abs(P.T @ P - np.eye(r)).max() < 1e-12


def test_rsvd_zero_gradient(orc):
    P, sig, sw = orc.rsvd_update(np.zeros((20, 30)), 5, 3, 2, seed=1)
    assert np.array_equal(sig, np.zeros(5))
    assert np.array_equal(P, np.eye(20)[:, :5])


@pytest.mark.parametrize("q", [0, 1, 2])
def test_rsvd_invariants_and_halko_bound(orc, q):
    """Interlacing (B = Q^T G), orthonormal P, canonical signs, and the mean of
    ||(I - P P^T) A||_2 within Halko's average-case bound for the power scheme
    (their Cor. 10.10) plus the truncation term sigma_{r+1} (their §9.3)."""
    m, n, r, p = 120, 300, 10, 6
    s = 1.0 / (1.0 + np.arange(m)) ** 0.7
    G = gi.planted_gradient(m, n, s, 1e-3, seed=17)
    sg = np.linalg.svd(G, compute_uv=False)
    errs = []
    for seed in range(20):
        P, sig, sw = orc.rsvd_update(G, r, p, q, seed=seed)
        assert np.all(sig <= sg[:r] * (1 + 1e-12))
        assert np.abs(P.T @ P - np.eye(r)).max() < 1e-12
        idx = np.argmax(np.abs(P), axis=0)
        assert np.all(P[idx, np.arange(r)] > 0)
        errs.append(np.linalg.norm(G - P @ (P.T @ G), 2))
    kk = r
    pp = p
    tail = sg[kk:]
    e = np.e
    bound = ((1 + np.sqrt(kk / (pp - 1))) * sg[kk] ** (2 * q + 1)
             + e * np.sqrt(kk + pp) / pp * np.sqrt(np.sum(tail ** (2 * (2 * q + 1))))) ** (1.0 / (2 * q + 1))
    assert np.mean(errs) <= sg[r] + 2.0 * bound
    assert np.mean(errs) >= sg[r] * (1 - 1e-9)            # Eckart-Young lower bound


def test_rsvd_orientation(orc):
    """m > n uses the right singular vectors (rule of paper §3 / Alg. 1 applied to G^T)."""
    rng = np.random.default_rng(21)
    s = 2.0 * 0.6 ** np.arange(40)
    G = gi.planted_gradient(90, 40, s, 0.0, seed=4, rank=9)     # rank <= k: exact
    P1, s1, _ = orc.rsvd_update(G, 6, 4, 2, seed=8)
    P2, s2, _ = orc.rsvd_update(G.T.copy(), 6, 4, 2, seed=8)
    assert np.array_equal(P1, P2) and np.array_equal(s1, s2)
    u, ss, vt = np.linalg.svd(G)
    assert proj_dist(P1, vt.T[:, :6]) < 1e-9
    assert P1.shape == (40, 6)


def test_rsvd_planted_spectrum_weyl(orc):
    """c1-shaped case with noise: |sigma_i(G) - s_i| <= ||E||_2 (Weyl), and the
    rSVD values never exceed sigma_i(G)."""
    m, n = 256, 688
    s = gi.spectrum_geometric_cut(m)
    rng = np.random.default_rng(1)
    Ghaar = gi.planted_gradient(m, n, s, 0.0, seed=2)
    E = 1e-3 * rng.standard_normal((m, n))
    G = Ghaar + E
    P, sig, sw = orc.rsvd_update(G, 32, 8, 2, seed=20250429)
    sg = np.linalg.svd(G, compute_uv=False)
    e2 = np.linalg.norm(E, 2)
    assert np.all(np.abs(sg[:32] - s[:32]) <= e2 * (1 + 1e-9))
    assert np.all(sig <= sg[:32] * (1 + 1e-12))
    assert np.abs(sig - sg[:32]).max() < 5e-3 * sg[0]
    # residual of the rank-32 projection: Eckart-Young floor sigma_33 and a small excess
    res = np.linalg.norm(G - P @ (P.T @ G), 2)
    assert sg[32] * (1 - 1e-9) <= res <= 1.5 * sg[32]


# ---------------------------------------------------------------- per-step path


def test_adam_first_step_closed_form(orc):
    """t = 1 from zero moments: bias correction cancels (1-b1) and (1-b2), so
    N = R / (|R| + eps) exactly (paper Alg. 1)."""
    rng = np.random.default_rng(0)
    R = rng.standard_normal((3, 7)) * 1e-3
    b1, b2, eps = float(np.float32(0.9)), float(np.float32(0.999)), float(np.float32(1e-8))
    M, V, N = orc.adam(R, np.zeros_like(R), np.zeros_like(R), b1, b2, eps, 1)
    assert np.allclose(M, (1 - b1) * R, rtol=1e-15, atol=0)
    assert np.allclose(V, (1 - b2) * R * R, rtol=1e-15, atol=0)
    assert np.allclose(N, R / (np.abs(R) + eps), rtol=1e-13, atol=0)


def test_galore_two_steps_2x3(orc):
    """Hand-derivable 2x3 example: G1 = [[3,0,-4],[0,1,0]], r = 1, p = 1 (so the
    sketch is exact): sigma = 5, P = e1; two projected Adam steps."""
    b1, b2, eps, lr, al = 0.9, 0.999, 1e-8, 1e-3, 0.25
    G1 = np.array([[3.0, 0.0, -4.0], [0.0, 1.0, 0.0]])
    W0 = np.array([[0.01, -0.02, 0.03], [0.04, 0.05, -0.06]])
    P, sig, _ = orc.rsvd_update(G1, 1, 1, 2, seed=3)
    assert abs(sig[0] - 5.0) < 1e-14
    assert np.allclose(P, [[1.0], [0.0]], atol=1e-15)
    P = np.array([[1.0], [0.0]])
    R = orc.project(P, G1)
    assert np.array_equal(R, [[3.0, 0.0, -4.0]])
    M, V, N = orc.adam(R, np.zeros_like(R), np.zeros_like(R), b1, b2, eps, 1)
    assert np.allclose(N, [[3 / (3 + eps), 0.0, -4 / (4 + eps)]], rtol=1e-15)
    W1 = orc.project_back(P, N, W0, lr, al)
    assert np.allclose(W1[0], W0[0] - lr * al * N[0], rtol=0, atol=1e-18)
    assert np.array_equal(W1[1], W0[1])
    G2 = np.array([[1.0, 2.0, 0.0], [0.0, -1.0, 5.0]])
    R2 = orc.project(P, G2)
    assert np.array_equal(R2, [[1.0, 2.0, 0.0]])
    M2, V2, N2 = orc.adam(R2, M, V, b1, b2, eps, 2)
    # moments by hand: M = 0.9*0.1*R1 + 0.1*R2, V = 0.999*0.001*R1^2 + 0.001*R2^2
    assert np.allclose(M2, [[0.37, 0.2, -0.36]], rtol=1e-14)
    assert np.allclose(V2, [[0.009991, 0.004, 0.015984]], rtol=1e-13)
    # bias corrections 1-0.81 = 0.19 and 1-0.998001 = 0.001999
    want = (np.array([0.37, 0.2, -0.36]) / 0.19) / (np.sqrt(np.array([0.009991, 0.004, 0.015984]) / 0.001999) + eps)
    assert np.allclose(N2[0], want, rtol=1e-12)


def test_identity_projector_is_textbook_adam(orc):
    """P = I (r = m) reduces GaLore-Adam to plain Adam with step size lr*alpha
    (torch.optim.Adam on CPU fp64, weight_decay = 0)."""
    import torch
    rng = np.random.default_rng(4)
    m, n = 5, 8
    lr, al = 1e-2, 0.5
    b1, b2, eps = float(np.float32(0.9)), float(np.float32(0.999)), float(np.float32(1e-8))
    W0 = rng.standard_normal((m, n))
    grads = [rng.standard_normal((m, n)) for _ in range(4)]
    w = torch.tensor(W0.copy(), dtype=torch.float64, requires_grad=True)
    opt = torch.optim.Adam([w], lr=lr * al, betas=(b1, b2), eps=eps, weight_decay=0.0)
    P = np.eye(m)
    W = W0.copy()
    M = np.zeros((m, n))
    V = np.zeros((m, n))
    for t, g in enumerate(grads, start=1):
        w.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        R = orc.project(P, g)
        M, V, N = orc.adam(R, M, V, b1, b2, eps, t)
        W = orc.project_back(P, N, W, lr, al)
    assert np.abs(W - w.detach().numpy()).max() < 1e-14


def test_adam_sign_and_permutation_equivariance(orc):
    rng = np.random.default_rng(6)
    Rs = [rng.standard_normal((4, 6)) for _ in range(3)]
    def run(seq):
        M = np.zeros((4, 6)); V = np.zeros((4, 6)); N = None
        for t, R in enumerate(seq, start=1):
            M, V, N = orc.adam(R, M, V, 0.9, 0.999, 1e-8, t)
        return N
    N = run(Rs)
    assert np.array_equal(run([-R for R in Rs]), -N)
    perm = rng.permutation(4)
    assert np.array_equal(run([R[perm] for R in Rs]), N[perm])


@pytest.mark.parametrize("m,n", [(7, 13), (13, 7), (9, 9)])
def test_projection_and_back_projection(orc, m, n):
    rng = np.random.default_rng(m * n)
    s, l = min(m, n), max(m, n)
    r = 4
    G = rng.standard_normal((m, n))
    P = np.linalg.qr(rng.standard_normal((s, r)))[0]
    A = G if m <= n else G.T
    R = orc.project(P, G)
    assert np.abs(R - P.T @ A).max() < 1e-13
    # P = I gives R = A
    assert np.array_equal(orc.project(np.eye(s), G), A)
    # G = P X (left) / G = (P X)^T (right) is recovered: P R = A
    X = rng.standard_normal((r, l))
    Gx = P @ X if m <= n else (P @ X).T
    assert np.abs(P @ orc.project(P, Gx) - (P @ X)).max() < 1e-13
    # linearity
    G2 = rng.standard_normal((m, n))
    assert np.abs(orc.project(P, 2 * G - 3 * G2) - (2 * orc.project(P, G) - 3 * orc.project(P, G2))).max() < 1e-12
    N = rng.standard_normal((r, l))
    W = rng.standard_normal((m, n))
    Wn = orc.project_back(P, N, W, 1e-3, 0.25)
    upd = P @ N if m <= n else (P @ N).T
    assert np.abs(Wn - (W - 2.5e-4 * upd)).max() < 1e-15 * 10


def test_memory_accounting():
    """Paper §3: GaLore keeps mn + mr + 2nr numbers for an m x n layer (m <= n):
    the weight, P (m x r) and the two moments (r x n); plus nr for R."""
    m, n, r = 4096, 11008, 1024
    s, l = min(m, n), max(m, n)
    P_elems, MV_elems, R_elems = s * r, 2 * r * l, r * l
    assert m * n + P_elems + MV_elems == m * n + m * r + 2 * n * r
    assert R_elems == n * r


# ---------------------------------------------------------------- subspace switch


def _haar(rng, n, k):
    q, r = np.linalg.qr(rng.standard_normal((n, k)))
    return q * np.sign(np.diag(r))


def test_align_recovers_sign_flipped_projector(orc):
    """A new projector that differs from the old one only by column signs (the
    sign indeterminacy of paper §4.1.3) is mapped back onto the old one
    exactly, and the flips are exactly the negated columns."""
    rng = np.random.default_rng(21)
    P_old = _haar(rng, 120, 17)
    d = np.where(rng.random(17) < 0.5, -1.0, 1.0)
    P_new, flips, M_out = orc.align_projector(P_old, P_old * d)
    assert np.array_equal(P_new, P_old)
    assert np.array_equal(flips, (d < 0).astype(np.int32))
    assert M_out is None


def test_align_rotated_basis_invariants(orc):
    """For P_new = P_old Q (Q orthogonal r x r): every aligned column has a
    non-negative overlap with its predecessor, the aligned P_new spans the same
    space, and flipping changes nothing but signs."""
    rng = np.random.default_rng(22)
    s, r = 90, 12
    P_old = _haar(rng, s, r)
    Q = _haar(rng, r, r)
    P_raw = P_old @ Q
    P_new, flips, _ = orc.align_projector(P_old, P_raw)
    assert np.all(np.einsum("ij,ij->j", P_old, P_new) >= 0)
    assert np.allclose(np.abs(P_new), np.abs(P_raw), rtol=0, atol=0)
    assert np.allclose(P_new @ P_new.T, P_old @ P_old.T, atol=1e-12)
    # the flips are exactly the columns whose overlap (diag of Q) was negative
    assert np.array_equal(flips, (np.diag(Q) < 0).astype(np.int32))


def test_align_moment_reexpression_in_shared_span(orc):
    """Coordinates in the old basis, re-expressed with (P_new^T P_old), equal
    the coordinates in the new basis for any matrix inside the shared span:
    for G = P_old X, (P_new^T P_old)(P_old^T G) = P_new^T G. Identity when the
    projector does not change."""
    rng = np.random.default_rng(23)
    s, r, l = 70, 9, 31
    P_old = _haar(rng, s, r)
    P_raw = P_old @ _haar(rng, r, r)
    G = P_old @ rng.standard_normal((r, l))
    R_old = P_old.T @ G
    P_new, _, M_out = orc.align_projector(P_old, P_raw, R_old)
    assert np.allclose(M_out, P_new.T @ G, rtol=0, atol=1e-12)
    _, flips, M_same = orc.align_projector(P_old, P_old, R_old)
    assert not flips.any()
    assert np.allclose(M_same, R_old, rtol=0, atol=1e-12)


def test_align_zero_overlap_keeps_sign(orc):
    """A column orthogonal to its predecessor (overlap exactly 0) is kept."""
    P_old = np.zeros((4, 2))
    P_old[0, 0] = 1.0
    P_old[1, 1] = 1.0
    P_raw = np.zeros((4, 2))
    P_raw[2, 0] = -1.0
    P_raw[1, 1] = -1.0
    P_new, flips, _ = orc.align_projector(P_old, P_raw)
    assert list(flips) == [0, 1]
    assert P_new[2, 0] == -1.0 and P_new[1, 1] == 1.0


# ---------------------------------------------------------------- scheduled step (Alg. 1)


@pytest.mark.parametrize("m,n", [(6, 9), (9, 6)])
def test_step_full_rank_permutation_projector_is_adam(orc, m, n):
    """Gradients whose short-side singular vectors are the coordinate axes in a
    fixed non-sorted order give, at r = s, a projector that is a permutation
    matrix at every update; Adam commutes with row permutations, so the
    scheduled steps (updates every T = 2 steps, switch and re-expression on)
    equal torch.optim.Adam (CPU fp64) with step size lr*alpha from step 1 on:
    this fixes the schedule, the bias exponent tau + 1 and both orientations."""
    import torch
    rng = np.random.default_rng(31)
    s, l = min(m, n), max(m, n)
    d = np.array([3.0, 1.0, 5.0, 2.0, 4.0, 0.5, 6.0, 1.5, 2.5][:s])
    lr, al = 1e-2, 0.5
    b1, b2, eps = 0.9, 0.999, 1e-8
    W0 = rng.standard_normal((m, n))
    w = torch.tensor(W0.copy(), dtype=torch.float64, requires_grad=True)
    opt = torch.optim.Adam([w], lr=lr * al, betas=(b1, b2), eps=eps, weight_decay=0.0)
    W, P, M, V = W0.copy(), None, np.zeros((s, l)), np.zeros((s, l))
    for tau in range(5):
        Qrows = gi.haar_columns(rng, l, s).T                 # s x l, orthonormal rows
        A = d[:, None] * Qrows                                # A A^T = diag(d^2)
        G = A if m <= n else A.T
        w.grad = torch.tensor(G, dtype=torch.float64)
        opt.step()
        W, P, M, V = orc.galore_step(G, W, P, M, V, s, 2, 1, 7, tau, 2, beta1=b1, beta2=b2, eps=eps, lr=lr,
                                     alpha=al, align=True, reexpress=True)
        assert np.allclose(np.abs(P), np.eye(s)[:, np.argsort(-d)], atol=1e-12)
    assert np.abs(W - w.detach().numpy()).max() < 1e-11


def test_step_update_lies_in_last_projector_span(orc):
    """Every step moves W only inside the span of the projector computed at the
    last update step (tau mod T == 0), fixed by LAPACK's SVD of that step's
    gradient; each step's gradient has its own random singular vectors, so a
    projector refreshed at the wrong step moves W elsewhere."""
    rng = np.random.default_rng(32)
    m, n, r, T = 24, 40, 4, 3
    spec = gi.spectrum_gapped(gi.spectrum_geometric(m, 0.8), r)
    W, P, M, V = rng.standard_normal((m, n)), None, np.zeros((r, n)), np.zeros((r, n))
    basis = None
    for tau in range(7):
        G = gi.planted_gradient(m, n, spec, 1e-3, seed=900 + tau)
        if tau % T == 0:
            basis = np.linalg.svd(G)[0][:, :r]
        W1, P, M, V = orc.galore_step(G, W, P, M, V, r, 4, 2, 11, tau, T, align=True)
        dW = W1 - W
        W = W1
        assert np.linalg.norm(dW - basis @ (basis.T @ dW)) <= 1e-6 * np.linalg.norm(dW)
        assert np.linalg.norm(P @ P.T - basis @ basis.T) < 1e-6


# ---------------------------------------------------------------- low-bit projector


def test_quantize_hand_example_ties_to_even(orc):
    """Column 0 has max 127 * 2^-7, so its scale is exactly 2^-7 and the codes
    are P / 2^-7 rounded half to even: 2.5 -> 2, 3.5 -> 4, -2.5 -> -2,
    -0.5 -> 0. Column 1 (a single nonzero entry) gets the extreme code."""
    P = np.array([[127, 1], [2.5, 0], [3.5, 0], [-2.5, 0], [-0.5, 0]], dtype=np.float64) * 2.0 ** -7
    codes, scales = orc.quantize_projector(P, 8)
    assert codes[:, 0].tolist() == [127, 2, 4, -2, 0]
    assert codes[:, 1].tolist() == [127, 0, 0, 0, 0]
    assert scales[0] == np.float32(2.0 ** -7)
    codes4, scales4 = orc.quantize_projector(P, 4)
    assert scales4[0] == np.float32(127 * 2.0 ** -7 / 7)
    assert codes4[0, 0] == 7 and codes4[0, 1] == 7


@pytest.mark.parametrize("bits", [8, 4])
def test_quantize_exact_grid_and_zero_column(orc, bits):
    """A projector whose columns lie on a grid c * 2^-e with an entry of
    magnitude qmax * 2^-e is reproduced exactly (codes and scale); an all-zero
    column gets scale 0 and codes 0."""
    qmax = 2 ** (bits - 1) - 1
    rng = np.random.default_rng(41)
    s, r = 40, 6
    c0 = rng.integers(-qmax, qmax + 1, size=(s, r))
    c0[3, :] = np.where(rng.random(r) < 0.5, qmax, -qmax)
    e = rng.integers(3, 12, size=r)
    P = c0 * 2.0 ** -e.astype(np.float64)
    P[:, 4] = 0.0
    codes, scales = orc.quantize_projector(P, bits)
    want = c0.copy()
    want[:, 4] = 0
    assert np.array_equal(codes, want)
    assert scales[4] == 0.0
    keep = [j for j in range(r) if j != 4]
    assert np.array_equal(scales[keep], (2.0 ** -e[keep]).astype(np.float32) * np.float32(1.0))
    assert np.array_equal(orc.dequantize_projector(codes, scales), P)


@pytest.mark.parametrize("bits", [8, 4])
def test_quantize_error_bound_and_range(orc, bits):
    """For a Haar projector: every code lies in [-qmax, qmax], each column's
    largest-magnitude entry gets +-qmax, and the dequantised value is within
    half a quantisation step of P (up to the fp32 rounding of P / scale)."""
    qmax = 2 ** (bits - 1) - 1
    rng = np.random.default_rng(42)
    P = _haar(rng, 300, 20).astype(np.float32).astype(np.float64)
    codes, scales = orc.quantize_projector(P, bits)
    assert np.abs(codes).max() <= qmax
    imax = np.argmax(np.abs(P), axis=0)
    assert np.array_equal(codes[imax, np.arange(20)], (np.sign(P[imax, np.arange(20)]) * qmax).astype(np.int32))
    err = np.abs(orc.dequantize_projector(codes, scales) - P)
    assert np.all(err <= 0.5 * scales.astype(np.float64) * (1 + 2.0 ** -20))


def test_pack_codes_layout(orc):
    """8 bits: one two's-complement byte per code. 4 bits: column 2c in the low
    nibble, 2c + 1 in the high nibble; an odd last column leaves the high nibble
    zero: [1, -2, 7, -7, 3] -> 0xE1 0x97 0x03."""
    assert orc.pack_codes(np.array([[1, -2, 7, -7, 3]]), 4).tolist() == [[0xE1, 0x97, 0x03]]
    assert orc.pack_codes(np.array([[1, -2, 127, -127]]), 8).tolist() == [[0x01, 0xFE, 0x7F, 0x81]]


# ---------------------------------------------------------------- 8-bit Adam


def test_fp8_extreme_values(orc):
    """Values the OCP 8-bit floating point specification states for its two
    formats: E4M3 (bias 7) 1.0 = 0x38, largest finite 448 = 0x7E, smallest
    subnormal 2^-9 = 0x01, largest subnormal 7 * 2^-9 = 0x07, smallest normal
    2^-6 = 0x08; E5M2 (bias 15) 1.0 = 0x3C, largest finite 57344 = 0x7B,
    smallest subnormal 2^-16 = 0x01, smallest normal 2^-14 = 0x04."""
    e4 = {1.0: 0x38, 448.0: 0x7E, 2.0 ** -9: 0x01, 7 * 2.0 ** -9: 0x07, 2.0 ** -6: 0x08, -2.0: 0xC0}
    e5 = {1.0: 0x3C, 57344.0: 0x7B, 2.0 ** -16: 0x01, 2.0 ** -14: 0x04, -1.0: 0xBC}
    for fmt, table in ((orc.E4M3, e4), (orc.E5M2, e5)):
        vals = np.array(list(table), dtype=np.float64)
        codes = np.array(list(table.values()), dtype=np.uint8)
        assert np.array_equal(orc.fp8_encode(vals, fmt), codes)
        assert np.array_equal(orc.fp8_decode(codes, fmt), vals)
    assert orc.fp8_encode([1e9, -1e9], orc.E4M3).tolist() == [0x7E, 0xFE]      # saturation
    assert orc.fp8_encode([1e9], orc.E5M2).tolist() == [0x7B]


@pytest.mark.parametrize("fmt,top", [(0, 0x7E), (1, 0x7B)])
def test_fp8_round_trip_and_brute_force_rounding(orc, fmt, top):
    """Every finite code decodes to a strictly increasing magnitude and encodes
    back to itself; random binary32 values (and exact midpoints) encode to the
    nearest representable value by brute force, ties to the even code."""
    codes = np.arange(0, top + 1, dtype=np.uint8)
    vals = orc.fp8_decode(codes, fmt)
    assert np.all(np.diff(vals) > 0)
    assert np.array_equal(orc.fp8_encode(vals, fmt), codes)
    rng = np.random.default_rng(50 + fmt)
    mids = (vals[:-1] + vals[1:]) / 2
    ys = np.concatenate([np.exp(rng.uniform(np.log(vals[1] / 4), np.log(vals[-1]), 3000)), mids,
                         rng.uniform(0, vals[8], 200)]).astype(np.float32)
    got = orc.fp8_encode(ys, fmt)
    for y, c in zip(ys.astype(np.float64), got):
        d = np.abs(vals - y)
        best = np.flatnonzero(d == d.min())
        want = best[0] if len(best) == 1 else [b for b in best if b % 2 == 0][0]
        if y > vals[-1]:
            want = top
        assert c == want, (y, c, want)


def test_adam8_first_step_equals_adam(orc):
    """From the all-zero state the decoded moments are exactly zero, so the
    first 8-bit step's N equals the (pinned) fp64 Adam step's N."""
    rng = np.random.default_rng(51)
    R = rng.standard_normal((7, 700))
    count = R.size
    nb = (count + 2047) // 2048
    z8, zs = np.zeros(count, np.uint8), np.zeros(nb, np.float32)
    _, _, _, _, N, _, _ = orc.adam8(R, z8, zs, z8, zs, 0.9, 0.999, 1e-8, 1)
    _, _, Nref = orc.adam(R, np.zeros_like(R), np.zeros_like(R), 0.9, 0.999, 1e-8, 1)
    assert np.array_equal(N, Nref)


def test_adam8_grid_block_is_encoded_exactly(orc):
    """With beta1 = 0 the new first moment is the gradient itself; a block whose
    values are E4M3 values times 2^-5 with maximum 448 * 2^-5 has scale 2^-5
    and is encoded exactly (codes equal those values' own E4M3 codes)."""
    rng = np.random.default_rng(52)
    codes = rng.integers(0, 0x7F, size=2048).astype(np.uint8) | (rng.integers(0, 2, 2048) * 0x80).astype(np.uint8)
    codes[codes & 0x7F == 0x7F] = 0x7E
    codes[17] = 0x7E
    g = orc.fp8_decode(codes, orc.E4M3) * 2.0 ** -5
    M8, Ms, _, _, _, _, _ = orc.adam8(g, np.zeros(2048, np.uint8), np.zeros(1, np.float32), np.zeros(2048, np.uint8),
                                      np.zeros(1, np.float32), 0.0, 0.5, 1e-8, 1)
    assert Ms[0] == np.float32(2.0 ** -5)
    dec = orc.fp8_decode(M8, orc.E4M3)
    assert np.array_equal(dec, orc.fp8_decode(codes, orc.E4M3))


def test_adam8_quantisation_error_and_block_independence(orc):
    """Over three steps: each decoded moment is within half an E4M3 / E5M2 step
    of the binary32 moment that was encoded (relative 2^-4 / 2^-3 for normal
    values, half the subnormal spacing below), and changing the gradient in one
    block leaves every other block's codes and scales untouched; the last block
    is ragged (3 * 700 = 2100 elements = 2048 + 52)."""
    rng = np.random.default_rng(53)
    shape = (3, 700)
    count = 2100
    M8, V8 = np.zeros(count, np.uint8), np.zeros(count, np.uint8)
    Ms, Vs = np.zeros(2, np.float32), np.zeros(2, np.float32)
    for t in range(1, 4):
        R = rng.standard_normal(shape) * np.exp(rng.uniform(-3, 3, shape))
        M8, Ms, V8, Vs, N, m32, v32 = orc.adam8(R, M8, Ms, V8, Vs, 0.9, 0.999, 1e-8, t)
        blk = np.arange(count).reshape(shape) // 2048
        dm = orc.fp8_decode(M8, orc.E4M3) * Ms[blk]
        dv = orc.fp8_decode(V8, orc.E5M2) * Vs[blk]
        assert np.all(np.abs(dm - m32) <= np.maximum(2.0 ** -4 * np.abs(m32), 2.0 ** -10 * Ms[blk]) * (1 + 1e-6))
        assert np.all(np.abs(dv - v32) <= np.maximum(2.0 ** -3 * np.abs(v32), 2.0 ** -17 * Vs[blk]) * (1 + 1e-6))
    R2 = R.copy()
    R2.ravel()[2050] += 1.0                      # inside the second block
    a = orc.adam8(R, M8, Ms, V8, Vs, 0.9, 0.999, 1e-8, 4)
    b = orc.adam8(R2, M8, Ms, V8, Vs, 0.9, 0.999, 1e-8, 4)
    assert np.array_equal(a[0].ravel()[:2048], b[0].ravel()[:2048]) and a[1][0] == b[1][0]
    assert np.array_equal(a[2].ravel()[:2048], b[2].ravel()[:2048]) and a[3][0] == b[3][0]


@pytest.mark.parametrize("amax,k", [(448.0 * 2 ** -3, -3), (448.0 * 2 ** -3 * (1 + 2 ** -20), -2),
                                    (224.5 * 2 ** -3, -3), (224.0 * 2 ** -3, -4)])
def test_adam8_block_scale_is_smallest_power_of_two(orc, amax, k):
    """A block's M scale is the smallest 2^k with max |M| <= 448 * 2^k (the
    E4M3 largest finite value): exactly at 448 * 2^k it is 2^k, just above it
    2^(k+1), and at 224 * 2^k the next lower power already suffices."""
    g = np.zeros(2048)
    g[5] = -amax
    g[9] = amax / 3
    M8, Ms, V8, Vs, _, m32, v32 = orc.adam8(g, np.zeros(2048, np.uint8), np.zeros(1, np.float32),
                                            np.zeros(2048, np.uint8), np.zeros(1, np.float32), 0.0, 0.0, 1e-8, 1)
    assert Ms[0] == np.float32(2.0 ** k)
    vmax = np.float64(np.float32(amax) ** 2)
    kv = int(np.ceil(np.log2(vmax / 57344.0)))
    assert Vs[0] == np.float32(2.0 ** kv) and vmax <= 57344.0 * 2.0 ** kv and vmax > 57344.0 * 2.0 ** (kv - 1)
    assert orc.fp8_decode(M8[5], orc.E4M3) * Ms[0] == pytest.approx(-amax, rel=2 ** -4)
