/*
 * GaLore 2 hot path -- CPU oracle (TEST INFRASTRUCTURE ONLY).
 *
 * A plain, slow, fp64 implementation of what the GPU library computes. It is
 * used only by the test-suite, by the smoke check and by the CPU-baseline leg
 * of the benchmark. The product path never links, loads or calls it, and it
 * shares no source, header, table or constant generator with the HIP library.
 *
 * Every stored input is widened exactly to fp64 by the caller (fp32 -> fp64
 * and bf16 -> fp64 are exact), and scalar hyper-parameters arrive as the
 * widened fp32 values the GPU side receives, never as decimal literals.
 *
 * Paper: "GaLore 2: Large-Scale LLM Pre-Training by Gradient Low-Rank
 * Projection" (Su, Gu, Xu, Tian, Zhao, 2025). Sections cited as "paper §x",
 * the GaLore-Adam listing of appendix A as "paper Alg. 1".
 * The randomized SVD adopted in paper §4.1.2 is the one of Halko, Martinsson
 * and Tropp, "Finding structure with randomness", SIAM Review 53(2), 2011:
 * randomized subspace iteration (their Alg. 4.4) followed by the direct SVD of
 * the projected matrix (their Alg. 5.1).
 *
 * Layout: every matrix is row-major, leading dimension = row length.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>

#define ORC_API __attribute__((visibility("default")))

/* Threads the OpenMP loops of the oracle use (for reporting and timing). */
ORC_API int orc_num_threads(void) { return omp_get_max_threads(); }
ORC_API void orc_set_num_threads(int n) { if (n > 0) omp_set_num_threads(n); }

/* ------------------------------------------------------------------------ */
/* Philox4x64-10 counter-based generator (Salmon, Moraes, Dror, Shaw,        */
/* "Parallel random numbers: as easy as 1, 2, 3", SC 2011).                  */
/* Round: two 64x64->128 multiplies with the published multipliers, the      */
/* high halves xor-ed with the other counter words and the key; the key is   */
/* advanced by the published Weyl increments between rounds.                 */
/* ------------------------------------------------------------------------ */
static void mul_hi_lo_u64(uint64_t a, uint64_t b, uint64_t* hi, uint64_t* lo) {
    unsigned __int128 p = (unsigned __int128)a * (unsigned __int128)b;
    *hi = (uint64_t)(p >> 64);
    *lo = (uint64_t)p;
}

ORC_API void orc_philox4x64_10(const uint64_t ctr_in[4], const uint64_t key_in[2], uint64_t out[4]) {
    const uint64_t mult0 = 0xD2E7470EE14C6C93ULL, mult1 = 0xCA5A826395121157ULL;
    const uint64_t weyl0 = 0x9E3779B97F4A7C15ULL, weyl1 = 0xBB67AE8584CAA73BULL;
    uint64_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
    uint64_t k0 = key_in[0], k1 = key_in[1];
    for (int round = 0; round < 10; ++round) {
        uint64_t hi0, lo0, hi1, lo1;
        mul_hi_lo_u64(mult0, c0, &hi0, &lo0);
        mul_hi_lo_u64(mult1, c2, &hi1, &lo1);
        uint64_t n0 = hi1 ^ c1 ^ k0;
        uint64_t n2 = hi0 ^ c3 ^ k1;
        c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
        k0 += weyl0; k1 += weyl1;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* ------------------------------------------------------------------------ */
/* Gaussian sketch Omega (l x k) for the randomized range finder (Halko et   */
/* al. 2011, §4: an l x k matrix of i.i.d. standard normal entries).         */
/* Entry (i, j) has element index e = j*l + i (column-major in the index, so */
/* a column of Omega does not depend on k). Philox4x64-10 with key           */
/* (seed, 0) and counter (e, sketch_index, 0, 0) gives words x0, x1; their   */
/* top 53 bits give u1 in (0, 1] and u2 in [0, 1); Box-Muller (Box & Muller  */
/* 1958) gives z = sqrt(-2 ln u1) cos(2 pi u2) in fp64. The sketch is the    */
/* fp32 rounding of z, so it is a set of fp32 values that both sides share.  */
/* ------------------------------------------------------------------------ */
ORC_API double orc_normal_from_words(uint64_t x0, uint64_t x1) {
    const double two_pow_m53 = 1.0 / 9007199254740992.0; /* 2^-53 */
    double u1 = (double)((x0 >> 11) + 1) * two_pow_m53;
    double u2 = (double)(x1 >> 11) * two_pow_m53;
    const double two_pi = 6.283185307179586;
    return sqrt(-2.0 * log(u1)) * cos(two_pi * u2);
}

/* fp64 -> nearest bfloat16 value (8 significant bits, ties to even), rounded */
/* once from the fp64 value; finite nonzero inputs in bfloat16's normal range. */
ORC_API double orc_round_bf16(double z) {
    if (z == 0.0 || !isfinite(z)) return z;
    int e;
    const double m = frexp(z, &e);            /* |m| in [0.5, 1) */
    return ldexp(rint(ldexp(m, 8)), e - 8);   /* rint: round half to even */
}

/* Both normals of one Box-Muller pair (1958): radius sqrt(-2 ln u1) times   */
/* cos and sin of 2 pi u2, u1 and u2 from the top 53 bits of x0 and x1 as in */
/* orc_normal_from_words (which is the cos member).                           */
ORC_API void orc_normal_pair_from_words(uint64_t x0, uint64_t x1, double* z) {
    const double two_pow_m53 = 1.0 / 9007199254740992.0; /* 2^-53 */
    const double u1 = (double)((x0 >> 11) + 1) * two_pow_m53;
    const double u2 = (double)(x1 >> 11) * two_pow_m53;
    const double two_pi = 6.283185307179586;
    const double rad = sqrt(-2.0 * log(u1));
    z[0] = rad * cos(two_pi * u2);
    z[1] = rad * sin(two_pi * u2);
}

/* Entries (4 i4 + t, j), t = 0..3, of the l x k sketch share one Philox      */
/* block: counter (j * ceil(l / 4) + i4, sketch_index, 0, 0), key (seed, 0);  */
/* words 0, 1 give the Box-Muller pair of rows 4 i4 and 4 i4 + 1 (cos, sin)   */
/* and words 2, 3 the pair of rows 4 i4 + 2 and 4 i4 + 3. Each entry is its   */
/* normal rounded once to bfloat16.                                           */
ORC_API void orc_sketch(int64_t l, int64_t k, uint64_t seed, uint64_t sketch_index, double* omega) {
    const int64_t l4 = (l + 3) / 4;
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < l; ++i) {
        for (int64_t j = 0; j < k; ++j) {
            uint64_t ctr[4] = {(uint64_t)(j * l4 + i / 4), sketch_index, 0, 0};
            uint64_t key[2] = {seed, 0};
            uint64_t w[4];
            double z[2];
            orc_philox4x64_10(ctr, key, w);
            const int t = (int)(i % 4);
            if (t < 2)
                orc_normal_pair_from_words(w[0], w[1], z);
            else
                orc_normal_pair_from_words(w[2], w[3], z);
            omega[i * k + j] = orc_round_bf16(z[t % 2]);
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Plain matrix products, fp64.                                              */
/* ------------------------------------------------------------------------ */
/* C (m x n) = A (m x kk) * B (kk x n) */
static void mat_mul(const double* A, const double* B, double* C, int64_t m, int64_t kk, int64_t n) {
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < m; ++i) {
        double* c = C + i * n;
        for (int64_t j = 0; j < n; ++j) c[j] = 0.0;
        for (int64_t t = 0; t < kk; ++t) {
            double a = A[i * kk + t];
            const double* b = B + t * n;
            for (int64_t j = 0; j < n; ++j) c[j] += a * b[j];
        }
    }
}

/* C (m x n) = A^T * B where A is (kk x m) and B is (kk x n) */
static void mat_mul_tn(const double* A, const double* B, double* C, int64_t m, int64_t kk, int64_t n) {
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < m; ++i) {
        double* c = C + i * n;
        for (int64_t j = 0; j < n; ++j) c[j] = 0.0;
        for (int64_t t = 0; t < kk; ++t) {
            double a = A[t * m + i];
            const double* b = B + t * n;
            for (int64_t j = 0; j < n; ++j) c[j] += a * b[j];
        }
    }
}

static void transpose(const double* A, double* At, int64_t rows, int64_t cols) {
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < rows; ++i)
        for (int64_t j = 0; j < cols; ++j) At[j * rows + i] = A[i * cols + j];
}

/* ------------------------------------------------------------------------ */
/* Thin QR by Householder reflections (Golub & Van Loan, "Matrix            */
/* Computations", §5.2), with the LAPACK convention that a reflector whose  */
/* sub-column is exactly zero is the identity (tau = 0).                     */
/* Y is s x k with s >= k. Outputs Q (s x k, orthonormal columns) and R      */
/* (k x k upper triangular) with Y = Q R. Either output may be NULL.         */
/* ------------------------------------------------------------------------ */
ORC_API void orc_householder_qr(int64_t s, int64_t k, const double* Y, double* Q, double* R) {
    /* work on the transpose so that each column of Y is a contiguous row */
    double* a = (double*)malloc(sizeof(double) * (size_t)(s * k));   /* a[j*s + i] = Y[i][j] */
    double* tau = (double*)calloc((size_t)k, sizeof(double));
    transpose(Y, a, s, k);
    for (int64_t j = 0; j < k; ++j) {
        double* col = a + j * s;
        double alpha = col[j];
        double xnorm2 = 0.0;
        for (int64_t i = j + 1; i < s; ++i) xnorm2 += col[i] * col[i];
        if (xnorm2 == 0.0) {
            tau[j] = 0.0;                 /* H_j = I; R_jj = alpha */
            continue;
        }
        double beta = -copysign(sqrt(alpha * alpha + xnorm2), alpha);
        tau[j] = (beta - alpha) / beta;
        double scale = 1.0 / (alpha - beta);
        for (int64_t i = j + 1; i < s; ++i) col[i] *= scale;   /* v (v_j = 1 implicit) */
        col[j] = beta;
        /* apply H_j = I - tau v v^T to the remaining columns */
        #pragma omp parallel for schedule(static)
        for (int64_t c = j + 1; c < k; ++c) {
            double* y = a + c * s;
            double w = y[j];
            for (int64_t i = j + 1; i < s; ++i) w += col[i] * y[i];
            w *= tau[j];
            y[j] -= w;
            for (int64_t i = j + 1; i < s; ++i) y[i] -= w * col[i];
        }
    }
    if (R) {
        for (int64_t i = 0; i < k; ++i)
            for (int64_t j = 0; j < k; ++j) R[i * k + j] = (j >= i) ? a[j * s + i] : 0.0;
    }
    if (Q) {
        /* Q = H_0 H_1 ... H_{k-1} [I_k; 0], accumulated backwards */
        double* qt = (double*)calloc((size_t)(s * k), sizeof(double));   /* qt[c*s + i] = Q[i][c] */
        for (int64_t c = 0; c < k; ++c) qt[c * s + c] = 1.0;
        for (int64_t j = k - 1; j >= 0; --j) {
            if (tau[j] == 0.0) continue;
            const double* v = a + j * s;
            #pragma omp parallel for schedule(static)
            for (int64_t c = j; c < k; ++c) {
                double* y = qt + c * s;
                double w = y[j];
                for (int64_t i = j + 1; i < s; ++i) w += v[i] * y[i];
                w *= tau[j];
                y[j] -= w;
                for (int64_t i = j + 1; i < s; ++i) y[i] -= w * v[i];
            }
        }
        transpose(qt, Q, k, s);
        free(qt);
    }
    free(tau);
    free(a);
}

/* ------------------------------------------------------------------------ */
/* One-sided (Hestenes) Jacobi SVD, returning the LEFT singular vectors of a */
/* k x l matrix B (k <= l): the k rows of B are the columns of B^T; pairs of */
/* them are rotated until mutually orthogonal, and the rotations accumulate  */
/* in J (k x k, from the identity). Then B^T J = Vhat Sigma, i.e.            */
/* B = J Sigma Vhat^T, so the columns of J are B's left singular vectors and */
/* sigma_j is the norm of the j-th rotated row.                              */
/* Pair rotation: alpha = |b_i|^2, beta = |b_j|^2, gamma = b_i . b_j; rotate */
/* when |gamma| > tol sqrt(alpha beta), with zeta = (beta - alpha)/(2 gamma),*/
/* t = sign(zeta)/(|zeta| + sqrt(1 + zeta^2)) (sign(0) = +1),                */
/* c = 1/sqrt(1 + t^2), s = c t, b_i <- c b_i - s b_j, b_j <- s b_i + c b_j. */
/* Pairs are visited in the round-robin (Brent-Luk) parallel ordering; a     */
/* sweep visits each pair once; iteration stops after a sweep without any    */
/* rotation. Singular values are sorted descending, ties by index.           */
/* Returns the number of sweeps, or -1 if max_sweeps ran out.                */
/* U (k x k) receives the sorted left singular vectors, sigma (k) the values.*/
/* ------------------------------------------------------------------------ */
typedef struct { double v; int64_t idx; } val_idx;

static int cmp_val_idx(const void* pa, const void* pb) {
    const val_idx* a = (const val_idx*)pa;
    const val_idx* b = (const val_idx*)pb;
    if (a->v > b->v) return -1;
    if (a->v < b->v) return 1;
    return (a->idx < b->idx) ? -1 : (a->idx > b->idx);
}

ORC_API int orc_jacobi_left_svd(int64_t k, int64_t l, const double* B, double* U, double* sigma,
                                int max_sweeps) {
    double* b = (double*)malloc(sizeof(double) * (size_t)(k * l));
    double* jt = (double*)calloc((size_t)(k * k), sizeof(double));  /* jt[c*k + i] = J[i][c] */
    memcpy(b, B, sizeof(double) * (size_t)(k * l));
    for (int64_t c = 0; c < k; ++c) jt[c * k + c] = 1.0;
    const double tol = (double)l * 2.220446049250313e-16;

    /* round-robin tournament on an even number of slots (a phantom if k is odd) */
    int64_t slots = k + (k & 1);
    int64_t* ring = (int64_t*)malloc(sizeof(int64_t) * (size_t)(slots > 0 ? slots : 1));
    for (int64_t i = 0; i < slots; ++i) ring[i] = i;

    int sweeps = 0, converged = (k < 2);
    while (!converged && sweeps < max_sweeps) {
        int64_t rotations = 0;
        for (int64_t step = 0; step + 1 < slots; ++step) {
            #pragma omp parallel for schedule(dynamic, 1) reduction(+ : rotations)
            for (int64_t h = 0; h < slots / 2; ++h) {
                int64_t p = ring[h], q = ring[slots - 1 - h];
                if (p >= k || q >= k) continue;
                if (p > q) { int64_t t = p; p = q; q = t; }
                double* bp = b + p * l;
                double* bq = b + q * l;
                double alpha = 0.0, beta = 0.0, gamma = 0.0;
                for (int64_t x = 0; x < l; ++x) {
                    alpha += bp[x] * bp[x];
                    beta += bq[x] * bq[x];
                    gamma += bp[x] * bq[x];
                }
                if (!(fabs(gamma) > tol * sqrt(alpha * beta))) continue;
                double zeta = (beta - alpha) / (2.0 * gamma);
                double sgn = (zeta >= 0.0) ? 1.0 : -1.0;
                double t = sgn / (fabs(zeta) + sqrt(1.0 + zeta * zeta));
                double c = 1.0 / sqrt(1.0 + t * t);
                double s = c * t;
                for (int64_t x = 0; x < l; ++x) {
                    double u = bp[x], w = bq[x];
                    bp[x] = c * u - s * w;
                    bq[x] = s * u + c * w;
                }
                double* jp = jt + p * k;
                double* jq = jt + q * k;
                for (int64_t x = 0; x < k; ++x) {
                    double u = jp[x], w = jq[x];
                    jp[x] = c * u - s * w;
                    jq[x] = s * u + c * w;
                }
                rotations += 1;
            }
            /* rotate the ring, keeping slot 0 fixed */
            int64_t last = ring[slots - 1];
            for (int64_t i = slots - 1; i > 1; --i) ring[i] = ring[i - 1];
            ring[1] = last;
        }
        ++sweeps;
        if (rotations == 0) converged = 1;
    }

    val_idx* order = (val_idx*)malloc(sizeof(val_idx) * (size_t)(k > 0 ? k : 1));
    for (int64_t c = 0; c < k; ++c) {
        double nrm = 0.0;
        for (int64_t x = 0; x < l; ++x) nrm += b[c * l + x] * b[c * l + x];
        order[c].v = sqrt(nrm);
        order[c].idx = c;
    }
    qsort(order, (size_t)k, sizeof(val_idx), cmp_val_idx);
    for (int64_t j = 0; j < k; ++j) {
        sigma[j] = order[j].v;
        int64_t src = order[j].idx;
        for (int64_t i = 0; i < k; ++i) U[i * k + j] = jt[src * k + i];
    }
    free(order);
    free(ring);
    free(jt);
    free(b);
    return converged ? sweeps : -1;
}

/* ------------------------------------------------------------------------ */
/* Sign convention for singular vectors (paper §4.1.3 and its footnote: fix */
/* the sign of each component): in every column, the entry of largest       */
/* magnitude (lowest row index on exact ties) is made positive.              */
/* ------------------------------------------------------------------------ */
ORC_API void orc_canonical_signs(double* P, int64_t rows, int64_t cols) {
    for (int64_t j = 0; j < cols; ++j) {
        int64_t best = 0;
        double best_abs = -1.0;
        for (int64_t i = 0; i < rows; ++i) {
            double a = fabs(P[i * cols + j]);
            if (a > best_abs) { best_abs = a; best = i; }
        }
        if (P[best * cols + j] < 0.0)
            for (int64_t i = 0; i < rows; ++i) P[i * cols + j] = -P[i * cols + j];
    }
}

/* ------------------------------------------------------------------------ */
/* Subspace update (paper §3 and Alg. 1: SVD of the gradient, P = first r   */
/* left singular vectors when m <= n, the right ones otherwise; paper       */
/* §4.1.2: the SVD is the randomized one of Halko et al. 2011).              */
/*   orientation: A = G if m <= n, else A = G^T;  s = min(m,n), l = max(m,n) */
/*   k = min(r + p, s)                                                       */
/*   Omega (l x k) Gaussian;  Y = A Omega;  Q = qr(Y)                        */
/*   q times:  Z = A^T Q;  Z = qr(Z);  Y = A Z;  Q = qr(Y)                   */
/*   B = Q^T A (k x l);  B = U_B Sigma V^T (one-sided Jacobi)                */
/*   P = Q U_B[:, :r] (s x r), signs canonicalised;  sigma = Sigma[:r]       */
/* G is m x n (row-major). Returns the Jacobi sweep count, or -1 on         */
/* non-convergence.                                                          */
/* ------------------------------------------------------------------------ */
ORC_API int orc_rsvd_update(const double* G, int64_t m, int64_t n, int32_t r, int32_t p, int32_t q,
                            uint64_t seed, uint64_t sketch_index, double* P, double* sigma) {
    const int64_t s = (m <= n) ? m : n;
    const int64_t l = (m <= n) ? n : m;
    int64_t k = (int64_t)r + (int64_t)p;
    if (k > s) k = s;

    double* A = (double*)malloc(sizeof(double) * (size_t)(s * l));     /* s x l */
    if (m <= n) memcpy(A, G, sizeof(double) * (size_t)(s * l));
    else transpose(G, A, m, n);

    double* omega = (double*)malloc(sizeof(double) * (size_t)(l * k));
    double* Y = (double*)malloc(sizeof(double) * (size_t)(s * k));
    double* Qm = (double*)malloc(sizeof(double) * (size_t)(s * k));
    double* Z = (double*)malloc(sizeof(double) * (size_t)(l * k));
    double* Zq = (double*)malloc(sizeof(double) * (size_t)(l * k));

    orc_sketch(l, k, seed, sketch_index, omega);
    mat_mul(A, omega, Y, s, l, k);
    orc_householder_qr(s, k, Y, Qm, NULL);
    for (int32_t it = 0; it < q; ++it) {
        mat_mul_tn(A, Qm, Z, l, s, k);          /* Z = A^T Q */
        orc_householder_qr(l, k, Z, Zq, NULL);
        mat_mul(A, Zq, Y, s, l, k);             /* Y = A Z   */
        orc_householder_qr(s, k, Y, Qm, NULL);
    }
    double* Bm = (double*)malloc(sizeof(double) * (size_t)(k * l));
    mat_mul_tn(Qm, A, Bm, k, s, l);             /* B = Q^T A */
    double* UB = (double*)malloc(sizeof(double) * (size_t)(k * k));
    double* sig = (double*)malloc(sizeof(double) * (size_t)k);
    int sweeps = orc_jacobi_left_svd(k, l, Bm, UB, sig, 60);

    /* P = Q U_B[:, :r] */
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < s; ++i)
        for (int64_t j = 0; j < r; ++j) {
            double acc = 0.0;
            for (int64_t t = 0; t < k; ++t) acc += Qm[i * k + t] * UB[t * k + j];
            P[i * r + j] = acc;
        }
    orc_canonical_signs(P, s, r);
    for (int64_t j = 0; j < r; ++j) sigma[j] = sig[j];

    free(sig); free(UB); free(Bm); free(Zq); free(Z); free(Qm); free(Y); free(omega); free(A);
    return sweeps;
}

/* ------------------------------------------------------------------------ */
/* Projection R = P^T A (paper §3, R_t = P_t^T G_t; paper Alg. 1).          */
/* P is s x r, G is m x n; R is r x l. For m > n (right projector) this is  */
/* R = (G P)^T.                                                              */
/* ------------------------------------------------------------------------ */
ORC_API void orc_project(const double* P, const double* G, int64_t m, int64_t n, int32_t r, double* R) {
    const int64_t s = (m <= n) ? m : n;
    const int64_t l = (m <= n) ? n : m;
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < r; ++i) {
        for (int64_t j = 0; j < l; ++j) {
            double acc = 0.0;
            for (int64_t t = 0; t < s; ++t) {
                double a = (m <= n) ? G[t * n + j] : G[j * n + t];   /* A[t][j] */
                acc += P[t * r + i] * a;
            }
            R[i * l + j] = acc;
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Low-rank Adam (paper §3 moment equations and Alg. 1, with the bias       */
/* correction of Alg. 1 applied to temporaries; the stored moments stay     */
/* uncorrected, as in Adam of Kingma & Ba 2015):                            */
/*   M <- b1 M + (1 - b1) R ;  V <- b2 V + (1 - b2) R^2                      */
/*   N  = (M / (1 - b1^t)) / (sqrt(V / (1 - b2^t)) + eps)                    */
/* t >= 1 is the step number. N may alias R.                                 */
/* ------------------------------------------------------------------------ */
ORC_API void orc_adam(const double* R, double* M, double* V, double* N, int64_t count,
                      double beta1, double beta2, double eps, int64_t t) {
    const double bc1 = 1.0 - pow(beta1, (double)t);
    const double bc2 = 1.0 - pow(beta2, (double)t);
    for (int64_t i = 0; i < count; ++i) {
        double g = R[i];
        M[i] = beta1 * M[i] + (1.0 - beta1) * g;
        V[i] = beta2 * V[i] + (1.0 - beta2) * g * g;
        double mhat = M[i] / bc1;
        double vhat = V[i] / bc2;
        N[i] = mhat / (sqrt(vhat) + eps);
    }
}

/* ------------------------------------------------------------------------ */
/* Back-projection and weight update (paper §3: G~ = alpha P N,             */
/* W <- W + eta G~; paper Alg. 1). The library takes the autograd gradient  */
/* (+grad), so the update is W <- W - (lr alpha) P N for m <= n and         */
/* W <- W - (lr alpha) (P N)^T for m > n.  P: s x r, N: r x l, W: m x n.    */
/* ------------------------------------------------------------------------ */
ORC_API void orc_project_back(const double* P, const double* N, double* W, int64_t m, int64_t n,
                              int32_t r, double lr, double alpha) {
    const int64_t s = (m <= n) ? m : n;
    const int64_t l = (m <= n) ? n : m;
    const double c = lr * alpha;
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < s; ++i) {
        for (int64_t j = 0; j < l; ++j) {
            double acc = 0.0;
            for (int64_t t = 0; t < r; ++t) acc += P[i * r + t] * N[t * l + j];
            if (m <= n) W[i * n + j] -= c * acc;
            else W[j * n + i] -= c * acc;
        }
    }
}

/* ------------------------------------------------------------------------ */
/* Subspace switch (paper §4.1.3: singular vectors are defined only up to    */
/* sign, and the randomized SVD adds its own randomness, so consecutive      */
/* projectors can disagree in sign; paper Alg. 1 replaces P every T steps).  */
/* Column j of the new projector is negated when its overlap with column j  */
/* of the previous one, <p_old_j, p_new_j>, is negative (zero or NaN keeps   */
/* it). Optionally the first moment is re-expressed in the new basis:       */
/* M_out = (P_new^T P_old) M_in with the aligned P_new (r x r times r x l).  */
/* P_old, P_new: s x r; flips: r ints (1 = negated); M_in, M_out: r x l.     */
/* ------------------------------------------------------------------------ */
ORC_API void orc_align_projector(const double* P_old, double* P_new, int64_t s, int64_t r, int32_t* flips,
                                 const double* M_in, double* M_out, int64_t l) {
    for (int64_t j = 0; j < r; ++j) {
        double ov = 0.0;
        for (int64_t i = 0; i < s; ++i) ov += P_old[i * r + j] * P_new[i * r + j];
        flips[j] = (ov < 0.0) ? 1 : 0;
        if (flips[j])
            for (int64_t i = 0; i < s; ++i) P_new[i * r + j] = -P_new[i * r + j];
    }
    if (M_in == NULL || M_out == NULL) return;
    double* O = (double*)malloc(sizeof(double) * (size_t)(r * r));   /* O = P_new^T P_old */
    #pragma omp parallel for schedule(static)
    for (int64_t a = 0; a < r; ++a)
        for (int64_t b = 0; b < r; ++b) {
            double acc = 0.0;
            for (int64_t i = 0; i < s; ++i) acc += P_new[i * r + a] * P_old[i * r + b];
            O[a * r + b] = acc;
        }
    #pragma omp parallel for schedule(static)
    for (int64_t a = 0; a < r; ++a)
        for (int64_t c = 0; c < l; ++c) {
            double acc = 0.0;
            for (int64_t b = 0; b < r; ++b) acc += O[a * r + b] * M_in[b * l + c];
            M_out[a * l + c] = acc;
        }
    free(O);
}

/* ------------------------------------------------------------------------ */
/* Low-bit projector (paper §4.2: GaLore 2 supports low-bit projection      */
/* matrices, after Q-GaLore). Reading: symmetric per-column quantisation;   */
/* qmax = 2^(bits-1) - 1 (127 for 8 bits, 7 for 4 bits);                    */
/*   scale_j = max_i |P_ij| / qmax,  code_ij = round-half-even(P_ij/scale_j) */
/* clamped to [-qmax, qmax]; a zero column has scale 0 and codes 0. Every   */
/* step that decides a code is taken in binary32 (the precision P is held   */
/* in): the absolute maximum, the division giving the scale, the division   */
/* P/scale and its rounding. The dequantised projector is code * scale.     */
/* P: s x r (fp32 values in doubles); codes: s x r ints; scales: r floats.  */
/* ------------------------------------------------------------------------ */
ORC_API void orc_quantize_projector(const double* P, int64_t s, int64_t r, int32_t bits, int32_t* codes,
                                    float* scales) {
    const int32_t qmax = (1 << (bits - 1)) - 1;
    for (int64_t j = 0; j < r; ++j) {
        float amax = 0.0f;
        for (int64_t i = 0; i < s; ++i) {
            const float a = fabsf((float)P[i * r + j]);
            if (a > amax) amax = a;
        }
        const float scale = amax / (float)qmax;
        scales[j] = scale;
        for (int64_t i = 0; i < s; ++i) {
            int32_t c = 0;
            if (scale > 0.0f) {
                const float q = rintf((float)P[i * r + j] / scale);
                c = (q > (float)qmax) ? qmax : (q < (float)-qmax) ? -qmax : (int32_t)q;
            }
            codes[i * r + j] = c;
        }
    }
}

/* ------------------------------------------------------------------------ */
/* OCP 8-bit floating point (OCP 8-bit Floating Point Specification, 2023). */
/* E4M3: exponent bias 7, 3 mantissa bits, largest finite 448, no infinity. */
/* E5M2: exponent bias 15, 2 mantissa bits, largest finite 57344.           */
/* Encoding rounds a binary32 value half to even and saturates at the       */
/* largest finite value (never NaN or infinity); subnormals are kept.       */
/* ------------------------------------------------------------------------ */
static int orc_fp8_mbits(int32_t fmt) { return fmt == 0 ? 3 : 2; }
static int orc_fp8_bias(int32_t fmt) { return fmt == 0 ? 7 : 15; }
static int orc_fp8_maxcode(int32_t fmt) { return fmt == 0 ? 0x7E : 0x7B; }

ORC_API uint8_t orc_fp8_encode(float x, int32_t fmt) {
    const int mb = orc_fp8_mbits(fmt), bias = orc_fp8_bias(fmt), maxcode = orc_fp8_maxcode(fmt);
    const uint8_t sign = signbit(x) ? 0x80 : 0x00;
    const float y = fabsf(x);
    if (y == 0.0f) return sign;
    const int emin = 1 - bias;                 /* exponent of the smallest normal */
    int e2;
    frexpf(y, &e2);
    int E = e2 - 1;                            /* y in [2^E, 2^(E+1)) */
    if (E < emin) E = emin;
    if (E > 30) return (uint8_t)(sign | maxcode);
    float k = rintf(ldexpf(y, mb - E));        /* exact scaling by a power of two, then RNE */
    if (k == (float)(2 << mb)) {               /* rounded up into the next binade */
        E += 1;
        k = (float)(1 << mb);
    }
    const int ki = (int)k;
    if (ki < (1 << mb)) return (uint8_t)(sign | ki);    /* subnormal (E == emin) */
    int code = ((E + bias) << mb) | (ki - (1 << mb));
    if (code > maxcode) code = maxcode;
    return (uint8_t)(sign | code);
}

ORC_API double orc_fp8_decode(uint8_t c, int32_t fmt) {
    const int mb = orc_fp8_mbits(fmt), bias = orc_fp8_bias(fmt);
    const int mag = c & 0x7F, ef = mag >> mb, m = mag & ((1 << mb) - 1);
    const double v = (ef == 0) ? ldexp((double)m, 1 - bias - mb) : ldexp((double)((1 << mb) + m), ef - bias - mb);
    return (c & 0x80) ? -v : v;
}

/* ------------------------------------------------------------------------ */
/* 8-bit block-wise low-rank Adam (paper §4.2: GaLore 2 uses the 8-bit Adam  */
/* of bitsandbytes, after Dettmers et al.). Reading: the moments of each     */
/* matrix are stored in blocks of `block` consecutive elements of the        */
/* row-major r x l state, M as E4M3 codes of M / scale_M and V as E5M2 codes */
/* of V / scale_V. A block's scale is the smallest power of two 2^k with     */
/* block max |value| <= 2^k * (largest finite value of the format), so that  */
/* scaling is exact and only the format's own rounding decides a code (0    */
/* for an all-zero block, whose codes are 0). One step decodes the moments   */
/* exactly, runs the Adam step of orc_adam on them in fp64 (N from the fresh */
/* moments), rounds the new moments to binary32 and re-encodes them with the */
/* new block scales. Mnew/Vnew (optional) receive the binary32 moments.      */
/* ------------------------------------------------------------------------ */
static float orc_pow2_scale(float amax, float maxval) {
    if (!(amax > 0.0f)) return 0.0f;
    int e, em;
    const float f = frexpf(amax, &e), fm = frexpf(maxval, &em);
    return ldexpf(1.0f, e - em + (f > fm ? 1 : 0));
}

ORC_API void orc_adam8(const double* R, uint8_t* M8, float* Ms, uint8_t* V8, float* Vs, double* N, int64_t count,
                       int64_t block, double beta1, double beta2, double eps, int64_t t, float* Mnew,
                       float* Vnew) {
    const double bc1 = 1.0 - pow(beta1, (double)t);
    const double bc2 = 1.0 - pow(beta2, (double)t);
    const int64_t nb = (count + block - 1) / block;
    float* mf = (float*)malloc(sizeof(float) * (size_t)block);
    float* vf = (float*)malloc(sizeof(float) * (size_t)block);
    for (int64_t b = 0; b < nb; ++b) {
        const int64_t i0 = b * block, i1 = (i0 + block < count) ? i0 + block : count;
        float am = 0.0f, av = 0.0f;
        for (int64_t i = i0; i < i1; ++i) {
            const double m = orc_fp8_decode(M8[i], 0) * (double)Ms[b];
            const double v = orc_fp8_decode(V8[i], 1) * (double)Vs[b];
            const double g = R[i];
            const double m1 = beta1 * m + (1.0 - beta1) * g;
            const double v1 = beta2 * v + (1.0 - beta2) * g * g;
            N[i] = (m1 / bc1) / (sqrt(v1 / bc2) + eps);
            mf[i - i0] = (float)m1;
            vf[i - i0] = (float)v1;
            if (fabsf(mf[i - i0]) > am) am = fabsf(mf[i - i0]);
            if (fabsf(vf[i - i0]) > av) av = fabsf(vf[i - i0]);
        }
        const float sm = orc_pow2_scale(am, 448.0f), sv = orc_pow2_scale(av, 57344.0f);
        Ms[b] = sm;
        Vs[b] = sv;
        for (int64_t i = i0; i < i1; ++i) {
            M8[i] = (sm > 0.0f) ? orc_fp8_encode(mf[i - i0] / sm, 0) : 0;   /* exact division by 2^k */
            V8[i] = (sv > 0.0f) ? orc_fp8_encode(vf[i - i0] / sv, 1) : 0;
            if (Mnew) Mnew[i] = mf[i - i0];
            if (Vnew) Vnew[i] = vf[i - i0];
        }
    }
    free(mf);
    free(vf);
}
