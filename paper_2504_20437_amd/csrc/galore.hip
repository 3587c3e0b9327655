// Host side of the GaLore 2 library: argument validation, workspace carving and
// the launch sequence of each C-ABI entry point. Everything is enqueued on the
// caller's stream; nothing here allocates device memory or synchronises.
#include <math.h>
#include <string.h>

#include <algorithm>
#include <map>
#include <mutex>

#include "../../include/galore.h"

#include "common.hpp"

using namespace galore;

namespace {

constexpr int kMaxK = 4096;          // largest sketch width supported by the small-SVD kernels
constexpr int kMaxSweeps = 24;       // Jacobi sweep limit of the small SVD (k > 2048)
constexpr int kMaxSweepsSmall = 16;  // and for k <= 2048 (the workloads here converge in 6-10)

int jacobi_sweeps(int k) { return k <= 2048 ? kMaxSweepsSmall : kMaxSweeps; }
// relative off-diagonal below which a pair is orthogonal: well above the
// rounding of the pair Gram (fp32 plane products, about 1e-7), and small
// enough that the fp64 refinement step that follows, whose error is quadratic
// in what the sweeps leave, ends below the fp32 rounding of the projector
constexpr double kJacobiTol = 1e-5;
constexpr double kDeficTol = 1e-10;  // relative pivot below which a column is dependent
constexpr size_t kAlign = 256;

#define GALORE_TRY(expr)                                   \
    do {                                                   \
        hipError_t e_ = (expr);                            \
        if (e_ != hipSuccess) return GALORE_ERR_HIP;       \
    } while (0)

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
int64_t pad_elems(int64_t n) { return (n + 63) / 64 * 64; }   // per-matrix stride, 256-B multiple

struct Shape {
    int64_t m, n, s, l;
    int k;
    bool left;   // m <= n: A = G; otherwise A = G^T
};

Shape make_shape(int64_t m, int64_t n, int r, int p) {
    Shape sh;
    sh.m = m;
    sh.n = n;
    sh.left = (m <= n);
    sh.s = sh.left ? m : n;
    sh.l = sh.left ? n : m;
    int64_t k = static_cast<int64_t>(r) + p;
    if (k > sh.s) k = sh.s;
    sh.k = static_cast<int>(k);
    return sh;
}

// The exact Gram's kernel addresses one matrix's three int8 digit planes
// ((k padded) x (l padded) bytes each) with 32-bit offsets.
bool digits_fit(const Shape& sh) {
    return gram_i8_digit_bytes(static_cast<int>(sh.l), sh.k) <= static_cast<int64_t>(INT32_MAX);
}

// Workspace regions, each holding `batch` matrices at a fixed element stride.
struct Layout {
    int64_t strideL, strideS, strideKK, strideUr;
    size_t offL1, offL2, offS1, offS2, offC, offXinv, offRinv, offYt, offUr, offDef, offDiag0, offRot,
        offJexp, offTheta, offXb, offS, offGg, offLam, offFlags, offNorm, offPerm;
    int64_t strideTheta;
    // bf16-stored gradients only: transposed copy of G (n x ldgt) and three
    // bf16 planes of the split fp32 operand (k x ldpl each)
    bool bf16;
    int64_t ldgt, strideGt, ldpl, planeStride, stridePl;
    size_t offGt, offPl;
    // digit planes and column maxima of the exact int8 Gram
    int64_t strideQ, strideCM;
    size_t offQ, offCM;
    size_t total;
};

int64_t pad8(int64_t x) { return (x + 7) / 8 * 8; }

Layout make_layout(const Shape& sh, int r, int batch, bool bf16) {
    Layout L;
    const int64_t k = sh.k;
    L.strideL = pad_elems(sh.l * k);
    L.strideS = pad_elems(sh.s * k);
    L.strideKK = pad_elems(k * k);
    L.strideUr = pad_elems(k * r);
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t o = off;
        off = align_up(off + bytes, kAlign);
        return o;
    };
    const size_t B = static_cast<size_t>(batch);
    L.offL1 = take(B * L.strideL * sizeof(float));
    L.offL2 = take(B * L.strideL * sizeof(float));
    L.offS1 = take(B * L.strideS * sizeof(float));
    L.offS2 = take(B * L.strideS * sizeof(float));
    L.offC = take(B * L.strideKK * sizeof(double));
    L.offXinv = take(B * L.strideKK * sizeof(double));
    L.offRinv = take(B * L.strideKK * sizeof(float));
    L.offYt = take(B * L.strideKK * sizeof(float));
    L.offUr = take(B * L.strideUr * sizeof(float));
    L.offDef = take(B * static_cast<size_t>(pad_elems(k)) * sizeof(int));
    L.offDiag0 = take(B * static_cast<size_t>(pad_elems(k)) * sizeof(double));
    L.offRot = take(B * kMaxSweeps * sizeof(int));
    L.offJexp = take(B * sizeof(int));
    // fp64 refinement of the small SVD: a second fp32 k x k vector buffer, the
    // symmetric S and G, the Rayleigh quotients and the per-matrix flags (the
    // first vector buffer and T reuse the fp32 and fp64 inverse regions, free
    // after the last Cholesky)
    L.offXb = take(B * L.strideKK * sizeof(float));
    L.offS = take(B * L.strideKK * sizeof(double));
    L.offGg = take(B * L.strideKK * sizeof(double));
    L.offLam = take(B * static_cast<size_t>(k) * sizeof(double));
    L.offFlags = take(B * sizeof(int));
    L.offNorm = take(B * static_cast<size_t>(k) * sizeof(double));
    L.offPerm = take(B * static_cast<size_t>(k) * sizeof(int));
    // scratch of the orthonormal completion in the small-SVD finalize: 2k + r doubles
    L.strideTheta = 2 * pad_elems(2 * k + r);
    L.offTheta = take(B * L.strideTheta * sizeof(float));
    L.bf16 = bf16;
    L.ldgt = pad8(sh.m);
    L.strideGt = pad_elems(sh.n * L.ldgt);
    L.ldpl = pad8(sh.l);
    L.planeStride = pad_elems(k * L.ldpl);
    L.stridePl = 3 * L.planeStride;
    L.offGt = bf16 ? take(B * L.strideGt * sizeof(uint16_t)) : 0;
    L.offPl = bf16 ? take(B * L.stridePl * sizeof(uint16_t)) : 0;
    L.strideQ = static_cast<int64_t>(align_up(gram_i8_digit_bytes(static_cast<int>(sh.l), sh.k), kAlign));
    L.strideCM = pad_elems(k);
    L.offQ = take(B * L.strideQ);
    L.offCM = take(B * L.strideCM * sizeof(unsigned));
    L.total = off;
    return L;
}

bool finite_f(float x) { return isfinite(x) != 0; }

// The gradient operand of a GEMM: G itself or its transpose, in its storage dtype.
struct GradOp {
    const void* G;
    bool bf16;
    int64_t ldg, stride;
};

// Y (s x k, ld k) = A X, X (l x k, ld k)
hipError_t gemm_A_times(const Shape& sh, const GradOp& g, const float* X, int64_t strideX, float* Y,
                        int64_t strideY, int batch, hipStream_t st) {
    GemmArgs a{};
    a.A = g.G;
    a.lda = g.ldg;
    a.strideA = g.stride;
    a.B = X;
    a.ldb = sh.k;
    a.strideB = strideX;
    a.C = Y;
    a.ldc = sh.k;
    a.strideC = strideY;
    a.M = static_cast<int>(sh.s);
    a.N = sh.k;
    a.K = static_cast<int>(sh.l);
    a.alpha = 1.0f;
    a.beta = 0.0f;
    // left: A = G (s x l, K contiguous); right: A(i, kk) = G[kk][i] (M contiguous)
    return launch_gemm(sh.left ? ALayout::kKContig : ALayout::kMContig, BLayout::kNContig, g.bf16,
                       false, a, batch, st);
}

// Z (l x k, ld k) = A^T Q, Q (s x k, ld k)
hipError_t gemm_At_times(const Shape& sh, const GradOp& g, const float* Q, int64_t strideQ, float* Z,
                         int64_t strideZ, int batch, hipStream_t st) {
    GemmArgs a{};
    a.A = g.G;
    a.lda = g.ldg;
    a.strideA = g.stride;
    a.B = Q;
    a.ldb = sh.k;
    a.strideB = strideQ;
    a.C = Z;
    a.ldc = sh.k;
    a.strideC = strideZ;
    a.M = static_cast<int>(sh.l);
    a.N = sh.k;
    a.K = static_cast<int>(sh.s);
    a.alpha = 1.0f;
    a.beta = 0.0f;
    // left: A^T(i, kk) = G[kk][i] (M contiguous); right: A^T = G (K contiguous)
    return launch_gemm(sh.left ? ALayout::kMContig : ALayout::kKContig, BLayout::kNContig, g.bf16,
                       false, a, batch, st);
}

// The products of the subspace update with the gradient. For fp32 G they run
// on the fp32 matrix cores reading G in place; for bf16 G the fp32 operand is
// split into three bf16 planes and the product runs on the bf16 matrix cores
// (bf16x3.hip) with the rows of A (G or its transposed copy) K-contiguous.
struct Products {
    const Shape* sh;
    const Layout* L;
    GradOp g;
    uint16_t* gt;       // transposed copy of G, n x ldgt (bf16 path without direct loads)
    uint16_t* planes;   // split planes (bf16 path)
    bool direct;        // bf16: both products read G in place (direct-load kernel)
    int batch;
    hipStream_t st;
    unsigned* cmax;     // column maxima of the product for the next Gram (direct-load kernel only)
    int64_t strideCM;
};

// Zero the column-maximum buffer for a product that fills it; false when the
// product cannot (its Gram then takes the maxima itself).
bool cmax_prepare(const Products& P) {
    if (!P.direct || P.cmax == nullptr) return false;
    return launch_fill_u32(P.cmax, P.strideCM * P.batch, P.st) == hipSuccess;
}

// Three bf16 planes that a product's epilogue writes in place of its fp32
// output (the operand layout of the bf16 matrix-core products).
struct PlaneOut {
    uint16_t* planes;
    int64_t ldpl, planeStride, stridePl;
    int rows_pad;
};

// Out (rows x k) = In (rows x k) * Rinv (k x k), or, with po, only the three
// bf16 planes of that product
hipError_t gemm_right_tri(const float* In, float* Out, int64_t stride, int rows, int k,
                          const float* Rinv, int64_t strideKK, int batch, hipStream_t st,
                          const PlaneOut* po = nullptr) {
    GemmArgs a{};
    if (po != nullptr) {
        a.planes = po->planes;
        a.ldpl = po->ldpl;
        a.planeStride = po->planeStride;
        a.stridePl = po->stridePl;
        a.rows_pad = po->rows_pad;
    }
    a.A = In;
    a.lda = k;
    a.strideA = stride;
    a.B = Rinv;
    a.ldb = k;
    a.strideB = strideKK;
    a.C = Out;
    a.ldc = k;
    a.strideC = stride;
    a.M = rows;
    a.N = k;
    a.K = k;
    a.alpha = 1.0f;
    a.beta = 0.0f;
    a.b_upper = 1;
    return launch_gemm(ALayout::kKContig, BLayout::kNContig, false, false, a, batch, st);
}

struct Work {
    const Layout* L;
    char* base;
    float* f(size_t off) const { return reinterpret_cast<float*>(base + off); }
    double* d(size_t off) const { return reinterpret_cast<double*>(base + off); }
    int* i(size_t off) const { return reinterpret_cast<int*>(base + off); }
};

// Optional stage tracing of the subspace update: events recorded on the
// caller's stream around each stage instance (no-op when capacity is 0).
struct Tracer {
    hipEvent_t* events;
    int32_t* stages;
    int32_t capacity;
    int32_t count;
    hipStream_t stream;
    hipError_t begin(int stage) {
        if (count >= capacity) return hipSuccess;
        stages[count] = stage;
        return hipEventRecord(events[2 * count], stream);
    }
    hipError_t end() {
        if (count >= capacity) return hipSuccess;
        const hipError_t e = hipEventRecord(events[2 * count + 1], stream);
        ++count;
        return e;
    }
};

#define GALORE_TRACED(tr, stage, expr)                        \
    do {                                                      \
        if ((tr).begin(stage) != hipSuccess) return GALORE_ERR_HIP; \
        GALORE_TRY(expr);                                     \
        if ((tr).end() != hipSuccess) return GALORE_ERR_HIP;  \
    } while (0)

// Y (s x k) = A X, X (l x k). With planes1 (bf16 G only) X is not read: the
// planes already hold X^T as one bf16 plane (exact), two more zero planes when
// the product cannot read G in place.
int product_A(const Products& P, Tracer& tr, const float* X, int64_t strideX, float* Y, int64_t strideY,
              bool& cmax_ready, bool planes1 = false, bool planes_ready = false) {
    const Shape& sh = *P.sh;
    const Layout& L = *P.L;
    cmax_ready = false;
    if (!L.bf16) {
        GALORE_TRACED(tr, GALORE_STAGE_PRODUCT_A, gemm_A_times(sh, P.g, X, strideX, Y, strideY, P.batch, P.st));
        return GALORE_OK;
    }
    const int k = sh.k, s = static_cast<int>(sh.s), l = static_cast<int>(sh.l);
    if (!planes1 && !planes_ready)
        GALORE_TRACED(tr, GALORE_STAGE_OPERAND,
                      launch_split3_transpose(X, k, strideX, P.planes, L.ldpl, L.planeStride, L.stridePl, l, k,
                                              static_cast<int>(L.ldpl), P.batch, P.st));
    // left: A = G (K-contiguous); right: A = G^T, read in place (M-contiguous)
    // or from the transposed copy
    const bool inplace = sh.left || P.direct;
    const void* A = inplace ? P.g.G : static_cast<const void*>(P.gt);
    const int64_t lda = inplace ? P.g.ldg : L.ldgt;
    const int64_t strideA = inplace ? P.g.stride : L.strideGt;
    cmax_ready = cmax_prepare(P);
    GALORE_TRACED(tr, GALORE_STAGE_PRODUCT_A,
                  launch_gemm_bf16x3(A, lda, strideA, sh.left ? 0 : (P.direct ? 1 : 0), P.planes, L.ldpl,
                                     L.planeStride, L.stridePl, Y, k, strideY, 0, s, k, l, 1.0f, 0.0f, P.batch,
                                     P.st, cmax_ready ? P.cmax : nullptr, P.strideCM,
                                     (planes1 && P.direct) ? 1 : 3));
    return GALORE_OK;
}

// Z (l x k) = A^T Q, Q (s x k)
int product_At(const Products& P, Tracer& tr, const float* Q, int64_t strideQ, float* Z, int64_t strideZ,
               bool& cmax_ready, bool planes_ready = false) {
    const Shape& sh = *P.sh;
    const Layout& L = *P.L;
    cmax_ready = false;
    if (!L.bf16) {
        GALORE_TRACED(tr, GALORE_STAGE_PRODUCT_AT, gemm_At_times(sh, P.g, Q, strideQ, Z, strideZ, P.batch, P.st));
        return GALORE_OK;
    }
    const int k = sh.k, s = static_cast<int>(sh.s), l = static_cast<int>(sh.l);
    if (!planes_ready)
        GALORE_TRACED(tr, GALORE_STAGE_OPERAND,
                      launch_split3_transpose(Q, k, strideQ, P.planes, L.ldpl, L.planeStride, L.stridePl, s, k,
                                              static_cast<int>(pad8(s)), P.batch, P.st));
    // left: A^T = G^T, read in place (M-contiguous) or from the transposed
    // copy; right: A^T = G (K-contiguous)
    const bool inplace = !sh.left || P.direct;
    const void* At = inplace ? P.g.G : static_cast<const void*>(P.gt);
    const int64_t ldat = inplace ? P.g.ldg : L.ldgt;
    const int64_t strideAt = inplace ? P.g.stride : L.strideGt;
    cmax_ready = cmax_prepare(P);
    GALORE_TRACED(tr, GALORE_STAGE_PRODUCT_AT,
                  launch_gemm_bf16x3(At, ldat, strideAt, sh.left ? (P.direct ? 1 : 0) : 0, P.planes, L.ldpl,
                                     L.planeStride, L.stridePl, Z, k, strideZ, 0, l, k, s, 1.0f, 0.0f, P.batch,
                                     P.st, cmax_ready ? P.cmax : nullptr, P.strideCM));
    return GALORE_OK;
}

// Latency-bound stages (the small SVD's sweeps, the blocked Cholesky) can run
// the second half of the batch on a second stream supplied by the caller,
// forked from and joined back into the caller's main stream with events: the
// two halves' launch sequences then run side by side, so that one half's small
// or phase-bound launches overlap the other's (measured on 64 x 4096x11008:
// Jacobi 103 -> 95 ms, Cholesky 28 -> 25 ms). Without a second stream
// everything runs in order on the main stream. The library creates no stream;
// the two fork/join events of each device are created on first use and kept
// for the process, and the enqueue sequence holds a lock, so concurrent
// callers on one device cannot interleave their fork and join records.
struct ForkJoin {
    hipEvent_t fork = nullptr, join = nullptr;
};
std::mutex g_fj_mutex;
std::map<int, ForkJoin> g_fj;   // by device

// f(first, count, stream) enqueues the work of matrices [first, first + count)
template <typename F>
int on_two_streams(int batch, hipStream_t stream, hipStream_t aux, F&& f) {
    if (batch < 2 || aux == nullptr || aux == stream) return f(0, batch, stream);
    std::lock_guard<std::mutex> lock(g_fj_mutex);
    int dev = 0;
    GALORE_TRY(hipGetDevice(&dev));
    ForkJoin& fj = g_fj[dev];
    if (fj.fork == nullptr) {
        GALORE_TRY(hipEventCreateWithFlags(&fj.fork, hipEventDisableTiming));
        GALORE_TRY(hipEventCreateWithFlags(&fj.join, hipEventDisableTiming));
    }
    const int h1 = batch / 2;
    GALORE_TRY(hipEventRecord(fj.fork, stream));
    GALORE_TRY(hipStreamWaitEvent(aux, fj.fork, 0));
    int e = f(0, h1, stream);
    if (e == GALORE_OK) e = f(h1, batch - h1, aux);
    GALORE_TRY(hipEventRecord(fj.join, aux));
    GALORE_TRY(hipStreamWaitEvent(stream, fj.join, 0));
    return e;
}

int enqueue_jacobi_sweeps(float* Yt, int k, int64_t strideKK, int nb, int* rot, double* norms, int* jperm,
                          int batch, hipStream_t stream, hipStream_t aux) {
    return on_two_streams(batch, stream, aux, [&](int b0, int cnt, hipStream_t st) -> int {
        const int64_t ko = static_cast<int64_t>(b0) * k;
        for (int sw = 0; sw < jacobi_sweeps(k); ++sw) {
            GALORE_TRY(launch_jacobi_order(Yt + b0 * strideKK, k, strideKK, norms + ko, jperm + ko,
                                           rot + b0 * kMaxSweeps, kMaxSweeps, sw, cnt, st));
            for (int stp = 0; stp < nb - 1; ++stp)
                GALORE_TRY(launch_jacobi_step(Yt + b0 * strideKK, k, strideKK, nb, stp, sw, rot + b0 * kMaxSweeps,
                                              kMaxSweeps, kJacobiTol, jperm + ko, cnt, st));
        }
        return GALORE_OK;
    });
}

// Cholesky of the k x k Gram region (and, with rinv, the inverse of the factor)
int enqueue_cholesky(const Work& w, int k, bool with_inverse, int batch, hipStream_t stream, hipStream_t aux) {
    const Layout& L = *w.L;
    return on_two_streams(batch, stream, aux, [&](int b0, int cnt, hipStream_t st) -> int {
        const int64_t o = b0 * L.strideKK;
        GALORE_TRY(launch_cholesky(w.d(L.offC) + o, k, L.strideKK, with_inverse ? w.f(L.offRinv) + o : nullptr,
                                   w.d(L.offXinv) + o, L.strideKK, w.i(L.offDef) + static_cast<int64_t>(b0) * k,
                                   w.d(L.offDiag0) + static_cast<int64_t>(b0) * k, kDeficTol, cnt, st));
        return GALORE_OK;
    });
}

// C (the k x k Gram region) = X^T X for a rows x k panel X of the workspace
GramI8Args gram_args(const Work& w, const float* X, int64_t strideX, int rows, int k, bool cmax_ready) {
    const Layout& L = *w.L;
    GramI8Args g{};
    g.cmax_ready = cmax_ready ? 1 : 0;
    g.X = X;
    g.ldx = k;
    g.strideX = strideX;
    g.rows = rows;
    g.cols = k;
    g.cmax = reinterpret_cast<unsigned*>(w.base + L.offCM);
    g.strideCM = L.strideCM;
    g.D = reinterpret_cast<int8_t*>(w.base + L.offQ);
    g.strideD = L.strideQ;
    g.C = w.d(L.offC);
    g.ldc = k;
    g.strideC = L.strideKK;
    return g;
}

// One Cholesky-QR pass: Out = In R^-1 with R^T R = In^T In (exact Gram of the
// fixed-point image of In, fp64 factor);
// columns found dependent are replaced by generic unit vectors.
int orth_pass(const Work& w, const float* In, float* Out, int64_t stride, int rows, int k, int batch,
              hipStream_t st, hipStream_t aux, Tracer& tr, bool cmax_ready, const PlaneOut* po = nullptr) {
    const Layout& L = *w.L;
    GALORE_TRACED(tr, GALORE_STAGE_GRAM, launch_gram_i8(gram_args(w, In, stride, rows, k, cmax_ready), batch, st));
    if (tr.begin(GALORE_STAGE_CHOLESKY) != hipSuccess) return GALORE_ERR_HIP;
    {
        const int e = enqueue_cholesky(w, k, true, batch, st, aux);
        if (e != GALORE_OK) return e;
    }
    if (tr.end() != hipSuccess) return GALORE_ERR_HIP;
    GALORE_TRACED(tr, GALORE_STAGE_TRIANGULAR,
                  gemm_right_tri(In, Out, stride, rows, k, w.f(L.offRinv), L.strideKK, batch, st, po));
    if (po != nullptr)
        GALORE_TRACED(tr, GALORE_STAGE_OTHER,
                      launch_fill_deficient_planes(po->planes, po->ldpl, po->planeStride, po->stridePl, rows, k,
                                                   w.i(L.offDef), batch, st));
    else
        GALORE_TRACED(tr, GALORE_STAGE_OTHER, launch_fill_deficient(Out, rows, k, stride, w.i(L.offDef), batch, st));
    return GALORE_OK;
}

#define GALORE_CHECK(expr)               \
    do {                                 \
        const int st_ = (expr);          \
        if (st_ != GALORE_OK) return st_; \
    } while (0)

int rsvd_impl(const void* G, int32_t g_dtype, int64_t m, int64_t n, int64_t ldg, int64_t stride_g, int32_t r,
              int32_t p, int32_t q, uint64_t seed, uint64_t sketch_index0, float* P, int64_t ldp,
              int64_t stride_p, float* sigma, int64_t stride_sigma, int32_t* info, int32_t batch,
              void* workspace, size_t workspace_bytes, hipStream_t stream, hipStream_t aux, Tracer& tr) {
    if (G == nullptr || P == nullptr || workspace == nullptr) return GALORE_ERR_INVALID_ARG;
    if (g_dtype != GALORE_F32 && g_dtype != GALORE_BF16) return GALORE_ERR_INVALID_ARG;
    if (m < 1 || n < 1 || r < 1 || p < 0 || q < 0 || batch < 1) return GALORE_ERR_SHAPE;
    if (m > INT32_MAX || n > INT32_MAX) return GALORE_ERR_SHAPE;
    const Shape sh = make_shape(m, n, r, p);
    if (r > sh.s || static_cast<int64_t>(r) + p > kMaxK || !digits_fit(sh)) return GALORE_ERR_SHAPE;
    if (ldg < n || ldp < r) return GALORE_ERR_SHAPE;
    if (batch > 1 && (stride_g < m * ldg || stride_p < sh.s * ldp)) return GALORE_ERR_SHAPE;
    if (sigma != nullptr && batch > 1 && stride_sigma < r) return GALORE_ERR_SHAPE;
    const Layout L = make_layout(sh, r, batch, g_dtype == GALORE_BF16);
    if (workspace_bytes < L.total) return GALORE_ERR_WORKSPACE;
    if (reinterpret_cast<uintptr_t>(workspace) % kAlign != 0) return GALORE_ERR_WORKSPACE;

    Work w{&L, static_cast<char*>(workspace)};
    const GradOp gop{G, g_dtype == GALORE_BF16, ldg, stride_g};
    const int k = sh.k;
    const int s = static_cast<int>(sh.s);
    const int l = static_cast<int>(sh.l);
    float* L1 = w.f(L.offL1);
    float* L2 = w.f(L.offL2);
    float* Sa = w.f(L.offS1);
    float* Sb = w.f(L.offS2);

    Products prod{&sh, &L, gop, L.bf16 ? reinterpret_cast<uint16_t*>(w.base + L.offGt) : nullptr,
                  L.bf16 ? reinterpret_cast<uint16_t*>(w.base + L.offPl) : nullptr, false, batch, stream,
                  reinterpret_cast<unsigned*>(w.base + L.offCM), L.strideCM};
    bool ready = false;   // the last product left the column maxima of its output
    if (L.bf16) {
        // both products read G in place when the direct-load kernel takes them:
        // G rows are K-contiguous for one product and M-contiguous for the other
        const bool kc_ok = bf16x3_direct_ok(G, ldg, stride_g, prod.planes, L.ldpl, L.planeStride, L.stridePl,
                                            static_cast<int>(m), static_cast<int>(n), batch, 0);
        const bool mc_ok = bf16x3_direct_ok(G, ldg, stride_g, prod.planes, L.ldpl, L.planeStride, L.stridePl,
                                            static_cast<int>(n), static_cast<int>(m), batch, 1);
        prod.direct = kc_ok && mc_ok;
        if (!prod.direct)   // A^T (left) or A (right) as K-contiguous bf16 rows: G^T, n x m
            GALORE_TRACED(tr, GALORE_STAGE_OPERAND,
                          launch_transpose_bf16(G, ldg, stride_g, prod.gt, L.ldgt, L.strideGt, static_cast<int>(m),
                                                static_cast<int>(n), batch, stream));
    }

    // a1-a3: sketch, range sample, orthonormalise (a bf16 G takes the sketch as
    // the bf16 plane of its transpose: one exact bf16 product)
    if (L.bf16)
        GALORE_TRACED(tr, GALORE_STAGE_SKETCH,
                      launch_sketch_plane(prod.planes, L.ldpl, L.planeStride, L.stridePl, l, k, seed, sketch_index0,
                                          !prod.direct, batch, stream));
    else
        GALORE_TRACED(tr, GALORE_STAGE_SKETCH, launch_sketch(L1, l, k, L.strideL, seed, sketch_index0, batch, stream));
    GALORE_CHECK(product_A(prod, tr, L1, L.strideL, Sa, L.strideS, ready, L.bf16));
    float* Q = Sa;
    float* Qtmp = Sb;
    // with a bf16 G an orthonormal panel that only feeds the next product is
    // written by Y R^-1 straight as that product's three bf16 planes (the same
    // bits the split of its fp32 values gives), and never in fp32
    const PlaneOut po_s{prod.planes, L.ldpl, L.planeStride, L.stridePl, static_cast<int>(pad8(s))};
    const PlaneOut po_l{prod.planes, L.ldpl, L.planeStride, L.stridePl, static_cast<int>(L.ldpl)};
    bool q_planes = false;   // Q exists only as the planes of the next product
    auto orth_s = [&](int passes) -> int {
        for (int ps = 0; ps < passes; ++ps) {
            const bool to_planes = L.bf16 && passes == 1;
            const int e = orth_pass(w, Q, Qtmp, L.strideS, s, k, batch, stream, aux, tr, ps == 0 && ready,
                                    to_planes ? &po_s : nullptr);
            if (e != GALORE_OK) return e;
            q_planes = to_planes;
            float* t = Q;
            Q = Qtmp;
            Qtmp = t;
        }
        return GALORE_OK;
    };
    GALORE_CHECK(orth_s(q == 0 ? 2 : 1));
    // a4: power iterations with re-orthonormalisation after every product
    for (int it = 0; it < q; ++it) {
        GALORE_CHECK(product_At(prod, tr, Q, L.strideS, L1, L.strideL, ready, q_planes));
        GALORE_CHECK(orth_pass(w, L1, L2, L.strideL, l, k, batch, stream, aux, tr, ready, L.bf16 ? &po_l : nullptr));
        GALORE_CHECK(product_A(prod, tr, L2, L.strideL, Qtmp, L.strideS, ready, false, L.bf16));
        {
            float* t = Q;
            Q = Qtmp;
            Qtmp = t;
        }
        GALORE_CHECK(orth_s(it == q - 1 ? 2 : 1));
    }
    // a5: B^T = Z = A^T Q (l x k); its Gram B B^T = Z^T Z = R^T R (the last Q
    // came from two passes, in fp32)
    GALORE_CHECK(product_At(prod, tr, Q, L.strideS, L1, L.strideL, ready, q_planes));
    {
        GALORE_TRACED(tr, GALORE_STAGE_GRAM,
                      launch_gram_i8(gram_args(w, L1, L.strideL, l, k, ready), batch, stream));
        if (tr.begin(GALORE_STAGE_CHOLESKY) != hipSuccess) return GALORE_ERR_HIP;
        GALORE_CHECK(enqueue_cholesky(w, k, false, batch, stream, aux));
        if (tr.end() != hipSuccess) return GALORE_ERR_HIP;
    }
    // a6: one-sided Jacobi on the columns of Y = R^T: Y W = U Sigma, U = left
    // singular vectors of B
    float* Yt = w.f(L.offYt);
    int* rot = w.i(L.offRot);
    float* Ur = w.f(L.offUr);
    if (tr.begin(GALORE_STAGE_JACOBI) != hipSuccess) return GALORE_ERR_HIP;
    int* jexp = w.i(L.offJexp);
    GALORE_TRY(launch_jacobi_prepare(w.d(L.offC), k, L.strideKK, Yt, L.strideKK, rot, kMaxSweeps, w.d(L.offDiag0),
                                     jexp, batch, stream));
    const int nblk_real = (k + kJacobiBlock - 1) / kJacobiBlock;
    const int nb = nblk_real + (nblk_real & 1);
    GALORE_CHECK(enqueue_jacobi_sweeps(Yt, k, L.strideKK, nb, rot, w.d(L.offNorm), w.i(L.offPerm), batch, stream,
                                       aux));
    GALORE_TRY(launch_jacobi_finalize(Yt, k, L.strideKK, r, Ur, L.strideUr, sigma, stride_sigma, rot,
                                      kMaxSweeps, jacobi_sweeps(k), info, reinterpret_cast<double*>(w.f(L.offTheta)),
                                      L.strideTheta / 2, jexp, w.d(L.offNorm), w.i(L.offPerm), w.f(L.offRinv),
                                      w.i(L.offFlags), batch, stream));
    if (tr.end() != hipSuccess) return GALORE_ERR_HIP;
    // fp64 refinement of the vectors the fp32 sweeps produced
    GALORE_TRACED(tr, GALORE_STAGE_REFINE,
                  launch_refine(w.d(L.offC), L.strideKK, w.f(L.offRinv), w.f(L.offXb), L.strideKK, w.d(L.offXinv),
                                w.d(L.offS), w.d(L.offGg), L.strideKK, w.d(L.offLam), w.i(L.offPerm), k, r, Ur,
                                L.strideUr, sigma,
                                stride_sigma, w.i(L.offFlags), batch, stream));
    // a7: P = Q U_B[:, :r], canonical signs
    {
        GemmArgs a{};
        a.A = Q;
        a.lda = k;
        a.strideA = L.strideS;
        a.B = Ur;
        a.ldb = r;
        a.strideB = L.strideUr;
        a.C = P;
        a.ldc = ldp;
        a.strideC = stride_p;
        a.M = s;
        a.N = r;
        a.K = k;
        a.alpha = 1.0f;
        a.beta = 0.0f;
        // with the bf16 path's plane region (free once the last product has run)
        // Q is split by rows into three bf16 planes there and U_r^T into the
        // refinement's fp64 scratch (free after it), and the product runs on the
        // bf16 matrix cores as six plane products (k a multiple of 16); every
        // other case on the fp32 matrix cores
        uint16_t* qpl = L.bf16 ? reinterpret_cast<uint16_t*>(w.base + L.offPl) : nullptr;
        uint16_t* upl = reinterpret_cast<uint16_t*>(w.base + L.offS);
        const int64_t qps = static_cast<int64_t>(s) * k, ups = static_cast<int64_t>(r) * k;
        if (qpl != nullptr && k % 16 == 0 &&
            bf16x6_ok(qpl, k, qps, L.stridePl, upl, k, ups, 3 * ups, k, batch)) {
            GALORE_TRACED(tr, GALORE_STAGE_PROJECTOR,
                          launch_split3_rows(Q, k, L.strideS, qpl, k, qps, L.stridePl, s, k, k, batch, stream));
            GALORE_TRACED(tr, GALORE_STAGE_PROJECTOR,
                          launch_split3_transpose(Ur, r, L.strideUr, upl, k, ups, 3 * ups, k, r, k, batch, stream));
            GALORE_TRACED(tr, GALORE_STAGE_PROJECTOR,
                          launch_gemm_bf16x6(qpl, k, qps, L.stridePl, upl, k, ups, 3 * ups, P, ldp, stride_p, 0, 0, s,
                                             r, k, 1.0f, 0.0f, batch, stream));
        } else {
            GALORE_TRACED(tr, GALORE_STAGE_PROJECTOR,
                          launch_gemm(ALayout::kKContig, BLayout::kNContig, false, false, a, batch, stream));
        }
    }
    GALORE_TRACED(tr, GALORE_STAGE_OTHER, launch_sign_fix(P, s, r, ldp, stride_p, batch, stream));
    return GALORE_OK;
}

// First moment in the new basis: O^T = P_old^T P_new (r x r per matrix, into
// Ot), then M_out = O M_in = (O^T)^T M_in, both on the fp32 matrix cores.
int reexpress_moment(const float* P_old, int64_t ldo, int64_t so, const float* P_new, int64_t ldn, int64_t sn,
                     int64_t s, int r, const float* M_in, int64_t ldmi, int64_t smi, float* M_out, int64_t ldmo,
                     int64_t smo, int64_t l, float* Ot, int batch, hipStream_t stream) {
    const int64_t strideO = pad_elems(static_cast<int64_t>(r) * r);
    {
        GemmArgs a{};
        a.A = P_old;        // A(i, kk) = P_old[kk][i]: M contiguous
        a.lda = ldo;
        a.strideA = so;
        a.B = P_new;
        a.ldb = ldn;
        a.strideB = sn;
        a.C = Ot;
        a.ldc = r;
        a.strideC = strideO;
        a.M = r;
        a.N = r;
        a.K = static_cast<int>(s);
        a.alpha = 1.0f;
        a.beta = 0.0f;
        GALORE_TRY(launch_gemm(ALayout::kMContig, BLayout::kNContig, false, false, a, batch, stream));
    }
    {
        GemmArgs a{};
        a.A = Ot;           // A(i, kk) = O^T[kk][i] = O[i][kk]: M contiguous
        a.lda = r;
        a.strideA = strideO;
        a.B = M_in;
        a.ldb = ldmi;
        a.strideB = smi;
        a.C = M_out;
        a.ldc = ldmo;
        a.strideC = smo;
        a.M = r;
        a.N = static_cast<int>(l);
        a.K = r;
        a.alpha = 1.0f;
        a.beta = 0.0f;
        GALORE_TRY(launch_gemm(ALayout::kMContig, BLayout::kNContig, false, false, a, batch, stream));
    }
    return GALORE_OK;
}

// ---- the no-allocation projection's scratch ----------------------------------
// galore_project_noalloc keeps the three bf16 planes of P^T in this file-scope
// device array instead of a caller workspace. Every device the library runs on
// holds its own copy for the life of the process. Host code never uses the
// array's name as an address: the device address of each device's copy is
// looked up once (hipGetSymbolAddress, with that device current) and kept.
constexpr size_t kStaticScratchBytes = size_t(64) << 20;
__device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

std::mutex g_scratch_mutex;
std::map<int, void*> g_scratch_ptr;   // by device

// the current device's copy of `scratch` (nullptr if the lookup failed)
void* scratch_on_current_device() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    auto it = g_scratch_ptr.find(dev);
    if (it != g_scratch_ptr.end()) return it->second;
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return nullptr;
    g_scratch_ptr[dev] = ptr;
    return ptr;
}

}  // namespace

extern "C" {

const char* galore_status_string(int status) {
    switch (status) {
        case GALORE_OK: return "GALORE_OK";
        case GALORE_ERR_INVALID_ARG: return "GALORE_ERR_INVALID_ARG";
        case GALORE_ERR_SHAPE: return "GALORE_ERR_SHAPE";
        case GALORE_ERR_WORKSPACE: return "GALORE_ERR_WORKSPACE";
        case GALORE_ERR_HIP: return "GALORE_ERR_HIP";
        default: return "GALORE_UNKNOWN_STATUS";
    }
}

int galore_version(void) { return 200; }

int galore_sketch(float* omega, int64_t l, int64_t k, uint64_t seed, uint64_t sketch_index,
                  hipStream_t stream) {
    if (omega == nullptr) return GALORE_ERR_INVALID_ARG;
    if (l < 1 || k < 1) return GALORE_ERR_SHAPE;
    GALORE_TRY(launch_sketch(omega, l, k, l * k, seed, sketch_index, 1, stream));
    return GALORE_OK;
}

size_t galore_rsvd_workspace_size(int64_t m, int64_t n, int32_t r, int32_t p, int32_t batch, int32_t g_dtype) {
    if (m < 1 || n < 1 || r < 1 || p < 0 || batch < 1) return 0;
    if (g_dtype != GALORE_F32 && g_dtype != GALORE_BF16) return 0;
    if (m > INT32_MAX || n > INT32_MAX) return 0;
    const Shape sh = make_shape(m, n, r, p);
    if (r > sh.s || static_cast<int64_t>(r) + p > kMaxK || !digits_fit(sh)) return 0;
    return make_layout(sh, r, batch, g_dtype == GALORE_BF16).total;
}

int galore_rsvd_update(const void* G, int32_t g_dtype, int64_t m, int64_t n, int64_t ldg,
                       int64_t stride_g, int32_t r, int32_t p, int32_t q, uint64_t seed,
                       uint64_t sketch_index0, float* P, int64_t ldp, int64_t stride_p,
                       float* sigma, int64_t stride_sigma, int32_t* info, int32_t batch,
                       void* workspace, size_t workspace_bytes, hipStream_t stream, hipStream_t aux_stream) {
    Tracer tr{nullptr, nullptr, 0, 0, stream};
    return rsvd_impl(G, g_dtype, m, n, ldg, stride_g, r, p, q, seed, sketch_index0, P, ldp, stride_p, sigma,
                     stride_sigma, info, batch, workspace, workspace_bytes, stream, aux_stream, tr);
}

int galore_rsvd_update_traced(const void* G, int32_t g_dtype, int64_t m, int64_t n, int64_t ldg,
                              int64_t stride_g, int32_t r, int32_t p, int32_t q, uint64_t seed,
                              uint64_t sketch_index0, float* P, int64_t ldp, int64_t stride_p,
                              float* sigma, int64_t stride_sigma, int32_t* info, int32_t batch,
                              void* workspace, size_t workspace_bytes, hipStream_t stream, hipStream_t aux_stream,
                              hipEvent_t* events, int32_t* stages, int32_t capacity, int32_t* count) {
    if (capacity < 0 || (capacity > 0 && (events == nullptr || stages == nullptr)) || count == nullptr)
        return GALORE_ERR_INVALID_ARG;
    for (int32_t i = 0; i < 2 * capacity; ++i)
        if (events[i] == nullptr) return GALORE_ERR_INVALID_ARG;
    Tracer tr{events, stages, capacity, 0, stream};
    const int st = rsvd_impl(G, g_dtype, m, n, ldg, stride_g, r, p, q, seed, sketch_index0, P, ldp, stride_p,
                             sigma, stride_sigma, info, batch, workspace, workspace_bytes, stream, aux_stream, tr);
    *count = tr.count;
    return st;
}

size_t galore_svd_workspace_size(int64_t m, int64_t n, int32_t r, int32_t batch, int32_t g_dtype) {
    if (m < 1 || n < 1 || r < 1 || std::min(m, n) > kMaxK) return 0;
    return galore_rsvd_workspace_size(m, n, r, static_cast<int32_t>(std::min(m, n) - r), batch, g_dtype);
}

int galore_svd_update(const void* G, int32_t g_dtype, int64_t m, int64_t n, int64_t ldg, int64_t stride_g, int32_t r,
                      float* P, int64_t ldp, int64_t stride_p, float* sigma, int64_t stride_sigma, int32_t* info,
                      int32_t batch, void* workspace, size_t workspace_bytes, hipStream_t stream,
                      hipStream_t aux_stream) {
    if (m < 1 || n < 1 || r < 1 || std::min(m, n) > kMaxK || r > std::min(m, n)) return GALORE_ERR_SHAPE;
    // k = s: the sketch spans the whole short side, so no power iteration is needed
    Tracer tr{nullptr, nullptr, 0, 0, stream};
    return rsvd_impl(G, g_dtype, m, n, ldg, stride_g, r, static_cast<int32_t>(std::min(m, n) - r), 0, 0, 0, P, ldp,
                     stride_p, sigma, stride_sigma, info, batch, workspace, workspace_bytes, stream, aux_stream, tr);
}

// Workspace of the projection with a bf16 gradient: the three bf16 planes of
// P^T (r x pad8(s) each) per matrix.
struct ProjLayout {
    int64_t ldpl, planeStride, stridePl;
    size_t total;
};

ProjLayout make_proj_layout(const Shape& sh, int r, int batch) {
    ProjLayout pl;
    pl.ldpl = pad8(sh.s);
    pl.planeStride = pad_elems(static_cast<int64_t>(r) * pl.ldpl);
    pl.stridePl = 3 * pl.planeStride;
    pl.total = align_up(static_cast<size_t>(batch) * pl.stridePl * sizeof(uint16_t), kAlign);
    return pl;
}

size_t galore_project_workspace_size(int64_t m, int64_t n, int32_t r, int32_t batch, int32_t g_dtype) {
    if (m < 1 || n < 1 || r < 1 || batch < 1 || m > INT32_MAX || n > INT32_MAX) return 0;
    if (g_dtype != GALORE_BF16) return 0;
    const Shape sh = make_shape(m, n, r, 0);
    if (r > sh.s) return 0;
    return make_proj_layout(sh, r, batch).total;
}

int galore_project(const float* P, int64_t ldp, int64_t stride_p, const void* G, int32_t g_dtype,
                   int64_t m, int64_t n, int64_t ldg, int64_t stride_g, int32_t r, float* R,
                   int64_t ldr, int64_t stride_r, int32_t batch, void* workspace, size_t workspace_bytes,
                   hipStream_t stream) {
    if (P == nullptr || G == nullptr || R == nullptr) return GALORE_ERR_INVALID_ARG;
    if (g_dtype != GALORE_F32 && g_dtype != GALORE_BF16) return GALORE_ERR_INVALID_ARG;
    if (m < 1 || n < 1 || r < 1 || batch < 1 || m > INT32_MAX || n > INT32_MAX) return GALORE_ERR_SHAPE;
    const Shape sh = make_shape(m, n, r, 0);
    if (r > sh.s || ldp < r || ldg < n || ldr < sh.l) return GALORE_ERR_SHAPE;
    if (batch > 1 && (stride_p < sh.s * ldp || stride_g < m * ldg || stride_r < r * ldr))
        return GALORE_ERR_SHAPE;
    if (workspace != nullptr && (reinterpret_cast<uintptr_t>(workspace) % kAlign) != 0) return GALORE_ERR_WORKSPACE;
    if (g_dtype == GALORE_BF16 && workspace != nullptr) {
        const ProjLayout pl = make_proj_layout(sh, r, batch);
        if (workspace_bytes < pl.total) return GALORE_ERR_WORKSPACE;
        uint16_t* planes = static_cast<uint16_t*>(workspace);
        // R^T (l x r) = A^T P on the bf16 matrix cores, stored transposed into R:
        // left: A^T = G^T (G read M-contiguous); right: A^T = G (K-contiguous)
        const int a_mc = sh.left ? 1 : 0;
        if (bf16x3_direct_ok(G, ldg, stride_g, planes, pl.ldpl, pl.planeStride, pl.stridePl,
                             static_cast<int>(sh.l), static_cast<int>(sh.s), batch, a_mc)) {
            GALORE_TRY(launch_split3_transpose(P, ldp, (batch > 1) ? stride_p : sh.s * ldp, planes, pl.ldpl,
                                               pl.planeStride, pl.stridePl, static_cast<int>(sh.s), r,
                                               static_cast<int>(pl.ldpl), batch, stream));
            GALORE_TRY(launch_gemm_bf16x3(G, ldg, stride_g, a_mc, planes, pl.ldpl, pl.planeStride, pl.stridePl, R,
                                          ldr, stride_r, 1, static_cast<int>(sh.l), r, static_cast<int>(sh.s),
                                          1.0f, 0.0f, batch, stream));
            return GALORE_OK;
        }
    }
    GemmArgs a{};
    // R (r x l) = P^T A : A-operand P^T (P[kk][i], M contiguous), B-operand A
    a.A = P;
    a.lda = ldp;
    a.strideA = stride_p;
    a.B = G;
    a.ldb = ldg;
    a.strideB = stride_g;
    a.C = R;
    a.ldc = ldr;
    a.strideC = stride_r;
    a.M = r;
    a.N = static_cast<int>(sh.l);
    a.K = static_cast<int>(sh.s);
    a.alpha = 1.0f;
    a.beta = 0.0f;
    // left: A = G (K x N rows, N contiguous); right: A(kk, j) = G[j][kk] (K contiguous)
    GALORE_TRY(launch_gemm(ALayout::kMContig, sh.left ? BLayout::kNContig : BLayout::kKContig, false,
                           g_dtype == GALORE_BF16, a, batch, stream));
    return GALORE_OK;
}

size_t galore_project_noalloc_max_bytes(void) { return kStaticScratchBytes; }

int galore_project_noalloc(const float* P, int64_t ldp, int64_t stride_p, const void* G, int32_t g_dtype, int64_t m,
                           int64_t n, int64_t ldg, int64_t stride_g, int32_t r, float* R, int64_t ldr,
                           int64_t stride_r, int32_t batch, hipStream_t stream) {
    // the arguments galore_project validates, checked before any device call
    if (P == nullptr || G == nullptr || R == nullptr) return GALORE_ERR_INVALID_ARG;
    if (g_dtype != GALORE_F32 && g_dtype != GALORE_BF16) return GALORE_ERR_INVALID_ARG;
    if (m < 1 || n < 1 || r < 1 || batch < 1 || m > INT32_MAX || n > INT32_MAX) return GALORE_ERR_SHAPE;
    const Shape sh = make_shape(m, n, r, 0);
    if (r > sh.s || ldp < r || ldg < n || ldr < sh.l) return GALORE_ERR_SHAPE;
    if (batch > 1 && (stride_p < sh.s * ldp || stride_g < m * ldg || stride_r < r * ldr)) return GALORE_ERR_SHAPE;
    if (g_dtype == GALORE_F32)   // the fp32 path needs no scratch
        return galore_project(P, ldp, stride_p, G, g_dtype, m, n, ldg, stride_g, r, R, ldr, stride_r, batch, nullptr,
                              0, stream);
    const size_t need = make_proj_layout(sh, r, batch).total;
    if (need > kStaticScratchBytes) return GALORE_ERR_WORKSPACE;
    void* ws = scratch_on_current_device();
    if (ws == nullptr) return GALORE_ERR_HIP;
    return galore_project(P, ldp, stride_p, G, g_dtype, m, n, ldg, stride_g, r, R, ldr, stride_r, batch, ws, need,
                          stream);
}

size_t galore_align_workspace_size(int32_t r, int32_t batch) {
    if (r < 1 || batch < 1) return 0;
    return align_up(static_cast<size_t>(batch) * pad_elems(static_cast<int64_t>(r) * r) * sizeof(float), kAlign);
}

int galore_align_projector(const float* P_old, int64_t ld_old, int64_t stride_old, float* P_new, int64_t ld_new,
                           int64_t stride_new, int64_t s, int32_t r, int32_t* flips, const float* M_in,
                           float* M_out, int64_t ldm, int64_t stride_m, int64_t l, int32_t batch,
                           void* workspace, size_t workspace_bytes, hipStream_t stream) {
    if (P_old == nullptr || P_new == nullptr) return GALORE_ERR_INVALID_ARG;
    if ((M_in == nullptr) != (M_out == nullptr)) return GALORE_ERR_INVALID_ARG;
    if (s < 1 || r < 1 || r > s || s > INT32_MAX || batch < 1) return GALORE_ERR_SHAPE;
    if (ld_old < r || ld_new < r) return GALORE_ERR_SHAPE;
    if (batch > 1 && (stride_old < s * ld_old || stride_new < s * ld_new)) return GALORE_ERR_SHAPE;
    const int64_t so = (batch > 1) ? stride_old : s * ld_old;
    const int64_t sn = (batch > 1) ? stride_new : s * ld_new;
    const bool reexpress = (M_in != nullptr);
    int64_t sm = 0;
    if (reexpress) {
        if (l < 1 || l > INT32_MAX || ldm < l) return GALORE_ERR_SHAPE;
        if (batch > 1 && stride_m < r * ldm) return GALORE_ERR_SHAPE;
        sm = (batch > 1) ? stride_m : r * ldm;
        // M_out must not overlap M_in (the product reads all of M_in)
        const char* a0 = reinterpret_cast<const char*>(M_in);
        const char* a1 = a0 + ((batch - 1) * sm + (r - 1) * ldm + l) * sizeof(float);
        const char* b0 = reinterpret_cast<const char*>(M_out);
        const char* b1 = b0 + ((batch - 1) * sm + (r - 1) * ldm + l) * sizeof(float);
        if (a0 < b1 && b0 < a1) return GALORE_ERR_INVALID_ARG;
        if (workspace == nullptr || (reinterpret_cast<uintptr_t>(workspace) % kAlign) != 0) return GALORE_ERR_WORKSPACE;
        if (workspace_bytes < galore_align_workspace_size(r, batch)) return GALORE_ERR_WORKSPACE;
    }
    GALORE_TRY(launch_align(P_old, ld_old, so, P_new, ld_new, sn, static_cast<int>(s), r, flips, batch, stream));
    if (!reexpress) return GALORE_OK;
    return reexpress_moment(P_old, ld_old, so, P_new, ld_new, sn, s, r, M_in, ldm, sm, M_out, ldm, sm, l,
                            static_cast<float*>(workspace), batch, stream);
}

int galore_lowrank_adam_step(const float* R, float* M, float* V, float* N, int64_t rows,
                             int64_t cols, int64_t ld, int64_t stride, int32_t batch, float beta1,
                             float beta2, float eps, int64_t t, hipStream_t stream) {
    if (R == nullptr || M == nullptr || V == nullptr || N == nullptr) return GALORE_ERR_INVALID_ARG;
    if (!finite_f(beta1) || !finite_f(beta2) || !finite_f(eps)) return GALORE_ERR_INVALID_ARG;
    if (beta1 < 0.0f || beta1 >= 1.0f || beta2 < 0.0f || beta2 >= 1.0f || eps <= 0.0f || t < 1)
        return GALORE_ERR_INVALID_ARG;
    if (rows < 1 || cols < 1 || ld < cols || batch < 1) return GALORE_ERR_SHAPE;
    if (batch > 1 && stride < rows * ld) return GALORE_ERR_SHAPE;
    // bias terms in fp64 from the fp32 betas, rounded once to fp32
    const double bc1 = 1.0 - pow(static_cast<double>(beta1), static_cast<double>(t));
    const double bc2 = 1.0 - pow(static_cast<double>(beta2), static_cast<double>(t));
    if (!(bc1 > 0.0) || !(bc2 > 0.0)) return GALORE_ERR_INVALID_ARG;
    const int64_t st = (batch > 1) ? stride : rows * ld;
    GALORE_TRY(launch_adam(R, M, V, N, rows, cols, ld, st, batch, beta1, beta2, eps,
                           static_cast<float>(bc1), static_cast<float>(bc2), stream));
    return GALORE_OK;
}

// Workspace of the back-projection: three bf16 planes of P (s x pad8(r) each)
// and of N^T (l x pad8(r) each) per matrix.
struct BackLayout {
    int64_t ldr, planeP, planeN;
    size_t offN, total;
};

BackLayout make_back_layout(const Shape& sh, int r, int batch) {
    BackLayout bl;
    bl.ldr = pad8(r);
    bl.planeP = pad_elems(sh.s * bl.ldr);
    bl.planeN = pad_elems(sh.l * bl.ldr);
    bl.offN = align_up(static_cast<size_t>(batch) * 3 * bl.planeP * sizeof(uint16_t), kAlign);
    bl.total = bl.offN + align_up(static_cast<size_t>(batch) * 3 * bl.planeN * sizeof(uint16_t), kAlign);
    return bl;
}

size_t galore_project_back_workspace_size(int64_t m, int64_t n, int32_t r, int32_t batch) {
    if (m < 1 || n < 1 || r < 1 || batch < 1 || m > INT32_MAX || n > INT32_MAX) return 0;
    const Shape sh = make_shape(m, n, r, 0);
    if (r > sh.s) return 0;
    return make_back_layout(sh, r, batch).total;
}

int galore_project_back(const float* P, int64_t ldp, int64_t stride_p, const float* N,
                        int64_t ldn, int64_t stride_n, float* W, int64_t m, int64_t n,
                        int64_t ldw, int64_t stride_w, int32_t r, float lr, float alpha,
                        int32_t batch, void* workspace, size_t workspace_bytes, hipStream_t stream) {
    if (P == nullptr || N == nullptr || W == nullptr) return GALORE_ERR_INVALID_ARG;
    if (!finite_f(lr) || !finite_f(alpha)) return GALORE_ERR_INVALID_ARG;
    if (m < 1 || n < 1 || r < 1 || batch < 1 || m > INT32_MAX || n > INT32_MAX) return GALORE_ERR_SHAPE;
    const Shape sh = make_shape(m, n, r, 0);
    if (r > sh.s || ldp < r || ldn < sh.l || ldw < n) return GALORE_ERR_SHAPE;
    if (batch > 1 && (stride_p < sh.s * ldp || stride_n < r * ldn || stride_w < m * ldw))
        return GALORE_ERR_SHAPE;
    if (workspace != nullptr) {
        if ((reinterpret_cast<uintptr_t>(workspace) % kAlign) != 0) return GALORE_ERR_WORKSPACE;
        const BackLayout bl = make_back_layout(sh, r, batch);
        if (workspace_bytes < bl.total) return GALORE_ERR_WORKSPACE;
        uint16_t* ppl = static_cast<uint16_t*>(workspace);
        uint16_t* npl = reinterpret_cast<uint16_t*>(static_cast<char*>(workspace) + bl.offN);
        if (bf16x6_ok(ppl, bl.ldr, bl.planeP, 3 * bl.planeP, npl, bl.ldr, bl.planeN, 3 * bl.planeN, r, batch)) {
            // C = P N (s x l) on the bf16 matrix cores, P and N^T split into three
            // planes each; W += -(lr alpha) C, or its transpose for m > n
            GALORE_TRY(launch_split3_rows(P, ldp, (batch > 1) ? stride_p : sh.s * ldp, ppl, bl.ldr, bl.planeP,
                                          3 * bl.planeP, static_cast<int>(sh.s), r, static_cast<int>(bl.ldr), batch,
                                          stream));
            GALORE_TRY(launch_split3_transpose(N, ldn, (batch > 1) ? stride_n : r * ldn, npl, bl.ldr, bl.planeN,
                                               3 * bl.planeN, r, static_cast<int>(sh.l), static_cast<int>(bl.ldr),
                                               batch, stream));
            GALORE_TRY(launch_gemm_bf16x6(ppl, bl.ldr, bl.planeP, 3 * bl.planeP, npl, bl.ldr, bl.planeN,
                                          3 * bl.planeN, W, ldw, stride_w, sh.left ? 0 : 1, 0,
                                          static_cast<int>(sh.s), static_cast<int>(sh.l), r, -(lr * alpha), 1.0f,
                                          batch, stream));
            return GALORE_OK;
        }
    }
    GemmArgs a{};
    a.C = W;
    a.ldc = ldw;
    a.strideC = stride_w;
    a.K = r;
    a.alpha = -(lr * alpha);
    a.beta = 1.0f;
    if (sh.left) {
        // W (s x l) -= c * P N : A = P (K contiguous), B = N (N contiguous)
        a.A = P;
        a.lda = ldp;
        a.strideA = stride_p;
        a.B = N;
        a.ldb = ldn;
        a.strideB = stride_n;
        a.M = static_cast<int>(sh.s);
        a.N = static_cast<int>(sh.l);
        GALORE_TRY(launch_gemm(ALayout::kKContig, BLayout::kNContig, false, false, a, batch, stream));
    } else {
        // W (l x s) -= c * N^T P^T : A(i, kk) = N[kk][i] (M contiguous), B(kk, j) = P[j][kk]
        a.A = N;
        a.lda = ldn;
        a.strideA = stride_n;
        a.B = P;
        a.ldb = ldp;
        a.strideB = stride_p;
        a.M = static_cast<int>(sh.l);
        a.N = static_cast<int>(sh.s);
        GALORE_TRY(launch_gemm(ALayout::kMContig, BLayout::kKContig, false, false, a, batch, stream));
    }
    return GALORE_OK;
}

// ---- measurement helper -----------------------------------------------------

int galore_probe_mfma_bf16(int64_t iterations, int32_t blocks, float* sink, double* flops, hipStream_t stream) {
    if (sink == nullptr || flops == nullptr) return GALORE_ERR_INVALID_ARG;
    if (iterations < 1 || blocks < 1) return GALORE_ERR_SHAPE;
    // four waves per block, four chains per wave, 32 x 32 x 16 x 2 flop per MFMA
    *flops = static_cast<double>(blocks) * 4.0 * 4.0 * static_cast<double>(iterations) * 32768.0;
    GALORE_TRY(launch_mfma_probe(iterations, blocks, sink, stream));
    return GALORE_OK;
}

int galore_probe_copy(const void* src, void* dst, size_t bytes, hipStream_t stream) {
    if (src == nullptr || dst == nullptr) return GALORE_ERR_INVALID_ARG;
    if (bytes == 0 || bytes % 16 != 0) return GALORE_ERR_SHAPE;
    if ((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) % 16 != 0) return GALORE_ERR_INVALID_ARG;
    const char* s0 = static_cast<const char*>(src);
    const char* d0 = static_cast<const char*>(dst);
    if (s0 < d0 + bytes && d0 < s0 + bytes) return GALORE_ERR_INVALID_ARG;
    GALORE_TRY(launch_copy_probe(src, dst, static_cast<int64_t>(bytes / 16), stream));
    return GALORE_OK;
}

// ---- 8-bit Adam -------------------------------------------------------------

int64_t galore_adam8_scale_count(int64_t rows, int64_t cols) {
    if (rows < 1 || cols < 1) return 0;
    return adam8_block_count(rows, cols);
}

int galore_lowrank_adam8_step(const float* R, float* N, int64_t ld, int64_t stride, uint8_t* M8, float* Ms,
                              uint8_t* V8, float* Vs, int64_t rows, int64_t cols, int32_t batch, float beta1,
                              float beta2, float eps, int64_t t, hipStream_t stream) {
    if (R == nullptr || N == nullptr || M8 == nullptr || Ms == nullptr || V8 == nullptr || Vs == nullptr)
        return GALORE_ERR_INVALID_ARG;
    if (!finite_f(beta1) || !finite_f(beta2) || !finite_f(eps)) return GALORE_ERR_INVALID_ARG;
    if (beta1 < 0.0f || beta1 >= 1.0f || beta2 < 0.0f || beta2 >= 1.0f || eps <= 0.0f || t < 1)
        return GALORE_ERR_INVALID_ARG;
    if (rows < 1 || cols < 1 || ld < cols || batch < 1) return GALORE_ERR_SHAPE;
    if (batch > 1 && stride < rows * ld) return GALORE_ERR_SHAPE;
    const double bc1 = 1.0 - pow(static_cast<double>(beta1), static_cast<double>(t));
    const double bc2 = 1.0 - pow(static_cast<double>(beta2), static_cast<double>(t));
    if (!(bc1 > 0.0) || !(bc2 > 0.0)) return GALORE_ERR_INVALID_ARG;
    GALORE_TRY(launch_adam8(R, N, ld, (batch > 1) ? stride : rows * ld, M8, Ms, V8, Vs, rows, cols, batch, beta1,
                            beta2, eps, static_cast<float>(bc1), static_cast<float>(bc2), stream));
    return GALORE_OK;
}

// ---- low-bit projector ------------------------------------------------------

bool codes_shape_ok(int64_t s, int32_t r, int32_t bits, int64_t ldq) {
    return ldq >= ((bits == 8) ? r : (static_cast<int64_t>(r) + 1) / 2) && s <= INT32_MAX;
}

int galore_quantize_projector(const float* P, int64_t ldp, int64_t stride_p, int64_t s, int32_t r, int32_t bits,
                              uint8_t* Q, int64_t ldq, int64_t stride_q, float* scales, int64_t stride_scales,
                              int32_t batch, hipStream_t stream) {
    if (P == nullptr || Q == nullptr || scales == nullptr) return GALORE_ERR_INVALID_ARG;
    if (bits != 8 && bits != 4) return GALORE_ERR_INVALID_ARG;
    if (s < 1 || r < 1 || r > s || batch < 1 || ldp < r || !codes_shape_ok(s, r, bits, ldq)) return GALORE_ERR_SHAPE;
    if (batch > 1 && (stride_p < s * ldp || stride_q < s * ldq || stride_scales < r)) return GALORE_ERR_SHAPE;
    GALORE_TRY(launch_quantize(P, ldp, (batch > 1) ? stride_p : s * ldp, static_cast<int>(s), r, bits, Q, ldq,
                               (batch > 1) ? stride_q : s * ldq, scales, (batch > 1) ? stride_scales : r, batch,
                               stream));
    return GALORE_OK;
}

// Workspace of the low-bit projection and back-projection: the bf16 plane of
// the codes (and, for the back-projection, three bf16 planes of the
// scale-folded N^T), or the fp32 dequantised projector on the fp32 path; one
// region serves whichever path runs.
struct QuantLayout {
    int64_t ldpl, plane, planeN, strideT;
    size_t offN, total;
};

QuantLayout make_quant_layout(const Shape& sh, int r, int batch, bool back) {
    QuantLayout q{};
    q.strideT = pad_elems(sh.s * r);
    const size_t fp32_path = align_up(static_cast<size_t>(batch) * q.strideT * sizeof(float), kAlign);
    if (back) {
        q.ldpl = pad8(r);
        q.plane = pad_elems(sh.s * q.ldpl);
        q.planeN = pad_elems(sh.l * q.ldpl);
        q.offN = align_up(static_cast<size_t>(batch) * q.plane * sizeof(uint16_t), kAlign);
        q.total = std::max(fp32_path, q.offN + align_up(static_cast<size_t>(batch) * 3 * q.planeN * sizeof(uint16_t),
                                                        kAlign));
    } else {
        q.ldpl = pad8(sh.s);
        q.plane = pad_elems(static_cast<int64_t>(r) * q.ldpl);
        q.total = std::max(fp32_path, align_up(static_cast<size_t>(batch) * q.plane * sizeof(uint16_t), kAlign));
    }
    return q;
}

size_t galore_project_quantized_workspace_size(int64_t m, int64_t n, int32_t r, int32_t batch) {
    if (m < 1 || n < 1 || r < 1 || batch < 1 || m > INT32_MAX || n > INT32_MAX || r > std::min(m, n)) return 0;
    return make_quant_layout(make_shape(m, n, r, 0), r, batch, false).total;
}

size_t galore_project_back_quantized_workspace_size(int64_t m, int64_t n, int32_t r, int32_t batch) {
    if (m < 1 || n < 1 || r < 1 || batch < 1 || m > INT32_MAX || n > INT32_MAX || r > std::min(m, n)) return 0;
    return make_quant_layout(make_shape(m, n, r, 0), r, batch, true).total;
}

int galore_project_quantized(const uint8_t* Q, int64_t ldq, int64_t stride_q, const float* scales,
                             int64_t stride_scales, int32_t bits, const void* G, int32_t g_dtype, int64_t m, int64_t n,
                             int64_t ldg, int64_t stride_g, int32_t r, float* R, int64_t ldr, int64_t stride_r,
                             int32_t batch, void* workspace, size_t workspace_bytes, hipStream_t stream) {
    if (Q == nullptr || scales == nullptr || G == nullptr || R == nullptr) return GALORE_ERR_INVALID_ARG;
    if (bits != 8 && bits != 4) return GALORE_ERR_INVALID_ARG;
    if (g_dtype != GALORE_F32 && g_dtype != GALORE_BF16) return GALORE_ERR_INVALID_ARG;
    if (m < 1 || n < 1 || r < 1 || batch < 1 || m > INT32_MAX || n > INT32_MAX) return GALORE_ERR_SHAPE;
    const Shape sh = make_shape(m, n, r, 0);
    if (r > sh.s || ldg < n || ldr < sh.l || !codes_shape_ok(sh.s, r, bits, ldq)) return GALORE_ERR_SHAPE;
    if (batch > 1 && (stride_q < sh.s * ldq || stride_scales < r || stride_g < m * ldg || stride_r < r * ldr))
        return GALORE_ERR_SHAPE;
    if (workspace == nullptr || (reinterpret_cast<uintptr_t>(workspace) % kAlign) != 0) return GALORE_ERR_WORKSPACE;
    const QuantLayout ql = make_quant_layout(sh, r, batch, false);
    if (workspace_bytes < ql.total) return GALORE_ERR_WORKSPACE;
    const int64_t sq = (batch > 1) ? stride_q : sh.s * ldq;
    const int64_t ss = (batch > 1) ? stride_scales : r;
    if (g_dtype == GALORE_BF16) {
        uint16_t* plane = static_cast<uint16_t*>(workspace);
        const int a_mc = sh.left ? 1 : 0;
        if (bf16x3_direct_ok(G, ldg, stride_g, plane, ql.ldpl, 0, ql.plane, static_cast<int>(sh.l),
                             static_cast<int>(sh.s), batch, a_mc)) {
            // R^T (l x r) = A^T (codes^T)^T on the bf16 matrix cores, one plane of
            // exact codes, each column of R^T (row of R) times its scale
            GALORE_TRY(launch_codes_plane(Q, ldq, sq, bits, static_cast<int>(sh.s), r, plane, ql.ldpl, ql.plane,
                                          static_cast<int>(ql.ldpl), true, batch, stream));
            GALORE_TRY(launch_gemm_bf16x3(G, ldg, stride_g, a_mc, plane, ql.ldpl, 0, ql.plane, R, ldr, stride_r, 1,
                                          static_cast<int>(sh.l), r, static_cast<int>(sh.s), 1.0f, 0.0f, batch,
                                          stream, nullptr, 0, 1, scales, ss));
            return GALORE_OK;
        }
    }
    float* Pt = static_cast<float*>(workspace);
    GALORE_TRY(launch_dequantize(Q, ldq, sq, bits, scales, ss, static_cast<int>(sh.s), r, Pt, r, ql.strideT, batch,
                                 stream));
    return galore_project(Pt, r, ql.strideT, G, g_dtype, m, n, ldg, stride_g, r, R, ldr, stride_r, batch, nullptr, 0,
                          stream);
}

int galore_project_back_quantized(const uint8_t* Q, int64_t ldq, int64_t stride_q, const float* scales,
                                  int64_t stride_scales, int32_t bits, const float* N, int64_t ldn, int64_t stride_n,
                                  float* W, int64_t m, int64_t n, int64_t ldw, int64_t stride_w, int32_t r, float lr,
                                  float alpha, int32_t batch, void* workspace, size_t workspace_bytes,
                                  hipStream_t stream) {
    if (Q == nullptr || scales == nullptr || N == nullptr || W == nullptr) return GALORE_ERR_INVALID_ARG;
    if (bits != 8 && bits != 4) return GALORE_ERR_INVALID_ARG;
    if (!finite_f(lr) || !finite_f(alpha)) return GALORE_ERR_INVALID_ARG;
    if (m < 1 || n < 1 || r < 1 || batch < 1 || m > INT32_MAX || n > INT32_MAX) return GALORE_ERR_SHAPE;
    const Shape sh = make_shape(m, n, r, 0);
    if (r > sh.s || ldn < sh.l || ldw < n || !codes_shape_ok(sh.s, r, bits, ldq)) return GALORE_ERR_SHAPE;
    if (batch > 1 && (stride_q < sh.s * ldq || stride_scales < r || stride_n < r * ldn || stride_w < m * ldw))
        return GALORE_ERR_SHAPE;
    if (workspace == nullptr || (reinterpret_cast<uintptr_t>(workspace) % kAlign) != 0) return GALORE_ERR_WORKSPACE;
    const QuantLayout ql = make_quant_layout(sh, r, batch, true);
    if (workspace_bytes < ql.total) return GALORE_ERR_WORKSPACE;
    const int64_t sq = (batch > 1) ? stride_q : sh.s * ldq;
    const int64_t ss = (batch > 1) ? stride_scales : r;
    uint16_t* plane = static_cast<uint16_t*>(workspace);
    uint16_t* npl = reinterpret_cast<uint16_t*>(static_cast<char*>(workspace) + ql.offN);
    if (bf16x3_direct_ok(plane, ql.ldpl, ql.plane, npl, ql.ldpl, ql.planeN, 3 * ql.planeN, static_cast<int>(sh.s), r,
                         batch, 0)) {
        // W (s x l, or its transpose) += -(lr alpha) codes (diag(scale) N): one
        // exact plane of codes against three planes of the scale-folded N^T
        GALORE_TRY(launch_codes_plane(Q, ldq, sq, bits, static_cast<int>(sh.s), r, plane, ql.ldpl, ql.plane,
                                      static_cast<int>(ql.ldpl), false, batch, stream));
        GALORE_TRY(launch_split3_transpose(N, ldn, (batch > 1) ? stride_n : r * ldn, npl, ql.ldpl, ql.planeN,
                                           3 * ql.planeN, r, static_cast<int>(sh.l), static_cast<int>(ql.ldpl), batch,
                                           stream, scales, ss));
        GALORE_TRY(launch_gemm_bf16x3(plane, ql.ldpl, ql.plane, 0, npl, ql.ldpl, ql.planeN, 3 * ql.planeN, W, ldw,
                                      (batch > 1) ? stride_w : m * ldw, sh.left ? 0 : 1, static_cast<int>(sh.s),
                                      static_cast<int>(sh.l), r, -(lr * alpha), 1.0f, batch, stream));
        return GALORE_OK;
    }
    float* Pt = static_cast<float*>(workspace);
    GALORE_TRY(launch_dequantize(Q, ldq, sq, bits, scales, ss, static_cast<int>(sh.s), r, Pt, r, ql.strideT, batch,
                                 stream));
    return galore_project_back(Pt, r, ql.strideT, N, ldn, stride_n, W, m, n, ldw, stride_w, r, lr, alpha, batch,
                               nullptr, 0, stream);
}

// Workspace of one scheduled step. Region X holds the subspace update's
// workspace, reused after it for the projected gradient R (= N, packed
// r x l) and the projection and back-projection planes; region Y holds what
// lives across the update: sigma, the previous projector and the previous
// first moment (for the switch) and the switch's overlap matrices.
struct StepLayout {
    size_t offR, offPws, offBws, pwsBytes, bwsBytes;
    size_t offSigma, offPold, offMold, offAws, awsBytes, total;
    int64_t strideR, stridePold, strideMold;
};

StepLayout make_step_layout(const Shape& sh, int r, int p, int batch, int32_t g_dtype, int32_t flags) {
    StepLayout sl{};
    const size_t rs = galore_rsvd_workspace_size(sh.m, sh.n, r, p, batch, g_dtype);
    sl.strideR = static_cast<int64_t>(r) * sh.l;     // packed: Adam's one-pass kernel applies to contiguous M, V
    sl.offR = 0;
    sl.pwsBytes = galore_project_workspace_size(sh.m, sh.n, r, batch, g_dtype);
    sl.bwsBytes = galore_project_back_workspace_size(sh.m, sh.n, r, batch);
    sl.offPws = align_up(static_cast<size_t>(batch) * sl.strideR * sizeof(float), kAlign);
    sl.offBws = sl.offPws + align_up(sl.pwsBytes, kAlign);
    const size_t x = std::max(rs, sl.offBws + align_up(sl.bwsBytes, kAlign));
    sl.offSigma = align_up(x, kAlign);
    size_t off = sl.offSigma + align_up(static_cast<size_t>(batch) * r * sizeof(float), kAlign);
    sl.stridePold = pad_elems(sh.s * r);
    sl.strideMold = pad_elems(static_cast<int64_t>(r) * sh.l);
    sl.offPold = off;
    if (flags & GALORE_STEP_ALIGN) off += align_up(static_cast<size_t>(batch) * sl.stridePold * sizeof(float), kAlign);
    sl.offMold = off;
    sl.offAws = off;
    if (flags & GALORE_STEP_REEXPRESS) {
        off += align_up(static_cast<size_t>(batch) * sl.strideMold * sizeof(float), kAlign);
        sl.offAws = off;
        sl.awsBytes = galore_align_workspace_size(r, batch);
        off += align_up(sl.awsBytes, kAlign);
    }
    sl.total = off;
    return sl;
}

bool step_sizes_ok(int64_t m, int64_t n, int32_t r, int32_t p, int32_t q, int32_t batch, int32_t g_dtype) {
    if (m < 1 || n < 1 || r < 1 || p < 0 || q < 0 || batch < 1 || m > INT32_MAX || n > INT32_MAX) return false;
    if (g_dtype != GALORE_F32 && g_dtype != GALORE_BF16) return false;
    return r <= std::min(m, n) && static_cast<int64_t>(r) + p <= kMaxK && digits_fit(make_shape(m, n, r, p));
}

size_t galore_step_workspace_size(int64_t m, int64_t n, int32_t r, int32_t p, int32_t batch, int32_t g_dtype,
                                  int32_t flags) {
    if (!step_sizes_ok(m, n, r, p, 0, batch, g_dtype)) return 0;
    if ((flags & ~(GALORE_STEP_ALIGN | GALORE_STEP_REEXPRESS)) != 0) return 0;
    if ((flags & GALORE_STEP_REEXPRESS) && !(flags & GALORE_STEP_ALIGN)) return 0;
    return make_step_layout(make_shape(m, n, r, p), r, p, batch, g_dtype, flags).total;
}

int galore_step(const void* G, int32_t g_dtype, int64_t m, int64_t n, int64_t ldg, int64_t stride_g, float* W,
                int64_t ldw, int64_t stride_w, float* P, int64_t ldp, int64_t stride_p, float* M, float* V,
                int64_t ldm, int64_t stride_m, int32_t r, int32_t p, int32_t q, uint64_t seed,
                uint64_t sketch_index0, int64_t tau, int32_t T, float beta1, float beta2, float eps, float lr,
                float alpha, int32_t flags, int32_t* info, int32_t batch, void* workspace, size_t workspace_bytes,
                hipStream_t stream, hipStream_t aux_stream) {
    if (G == nullptr || W == nullptr || P == nullptr || M == nullptr || V == nullptr) return GALORE_ERR_INVALID_ARG;
    if (g_dtype != GALORE_F32 && g_dtype != GALORE_BF16) return GALORE_ERR_INVALID_ARG;
    if (tau < 0 || T < 1) return GALORE_ERR_INVALID_ARG;
    if ((flags & ~(GALORE_STEP_ALIGN | GALORE_STEP_REEXPRESS)) != 0) return GALORE_ERR_INVALID_ARG;
    if ((flags & GALORE_STEP_REEXPRESS) && !(flags & GALORE_STEP_ALIGN)) return GALORE_ERR_INVALID_ARG;
    if (!finite_f(beta1) || !finite_f(beta2) || !finite_f(eps) || !finite_f(lr) || !finite_f(alpha))
        return GALORE_ERR_INVALID_ARG;
    if (beta1 < 0.0f || beta1 >= 1.0f || beta2 < 0.0f || beta2 >= 1.0f || eps <= 0.0f) return GALORE_ERR_INVALID_ARG;
    const double bc1 = 1.0 - pow(static_cast<double>(beta1), static_cast<double>(tau + 1));
    const double bc2 = 1.0 - pow(static_cast<double>(beta2), static_cast<double>(tau + 1));
    if (!(bc1 > 0.0) || !(bc2 > 0.0)) return GALORE_ERR_INVALID_ARG;
    if (!step_sizes_ok(m, n, r, p, q, batch, g_dtype)) return GALORE_ERR_SHAPE;
    const Shape sh = make_shape(m, n, r, p);
    if (ldg < n || ldw < n || ldp < r || ldm < sh.l) return GALORE_ERR_SHAPE;
    if (batch > 1 && (stride_g < m * ldg || stride_w < m * ldw || stride_p < sh.s * ldp || stride_m < r * ldm))
        return GALORE_ERR_SHAPE;
    const int64_t sg = (batch > 1) ? stride_g : m * ldg;
    const int64_t sw = (batch > 1) ? stride_w : m * ldw;
    const int64_t sp = (batch > 1) ? stride_p : sh.s * ldp;
    const int64_t sm = (batch > 1) ? stride_m : r * ldm;
    const StepLayout sl = make_step_layout(sh, r, p, batch, g_dtype, flags);
    if (workspace == nullptr || (reinterpret_cast<uintptr_t>(workspace) % kAlign) != 0) return GALORE_ERR_WORKSPACE;
    if (workspace_bytes < sl.total) return GALORE_ERR_WORKSPACE;
    char* ws = static_cast<char*>(workspace);
    float* R = reinterpret_cast<float*>(ws + sl.offR);
    float* sigma = reinterpret_cast<float*>(ws + sl.offSigma);

    // Alg. 1: a new projector from the gradient of every T-th step
    if (tau % T == 0) {
        const bool align = (flags & GALORE_STEP_ALIGN) && tau > 0;
        const bool reexpress = align && (flags & GALORE_STEP_REEXPRESS);
        float* Pold = reinterpret_cast<float*>(ws + sl.offPold);
        float* Mold = reinterpret_cast<float*>(ws + sl.offMold);
        if (align)
            GALORE_TRY(launch_copy_rows(P, ldp, sp, Pold, r, sl.stridePold, static_cast<int>(sh.s), r, batch,
                                        stream));
        if (reexpress)
            GALORE_TRY(launch_copy_rows(M, ldm, sm, Mold, sh.l, sl.strideMold, r, static_cast<int>(sh.l), batch,
                                        stream));
        int st = galore_rsvd_update(G, g_dtype, m, n, ldg, sg, r, p, q, seed, sketch_index0, P, ldp, sp, sigma, r,
                                    info, batch, ws, sl.offSigma, stream, aux_stream);
        if (st != GALORE_OK) return st;
        if (align)
            GALORE_TRY(launch_align(Pold, r, sl.stridePold, P, ldp, sp, static_cast<int>(sh.s), r, nullptr, batch,
                                    stream));
        if (reexpress) {
            st = reexpress_moment(Pold, r, sl.stridePold, P, ldp, sp, sh.s, r, Mold, sh.l, sl.strideMold, M, ldm, sm,
                                  sh.l, reinterpret_cast<float*>(ws + sl.offAws), batch, stream);
            if (st != GALORE_OK) return st;
        }
    }
    // R = P^T A; Adam on (M, V) writes N over R; W -= lr alpha P N
    int st = galore_project(P, ldp, sp, G, g_dtype, m, n, ldg, sg, r, R, sh.l, sl.strideR, batch,
                            sl.pwsBytes ? ws + sl.offPws : nullptr, sl.pwsBytes, stream);
    if (st != GALORE_OK) return st;
    GALORE_TRY(launch_adam2(R, R, sh.l, sl.strideR, M, V, ldm, sm, r, sh.l, batch, beta1, beta2, eps,
                            static_cast<float>(bc1), static_cast<float>(bc2), stream));
    return galore_project_back(P, ldp, sp, R, sh.l, sl.strideR, W, m, n, ldw, sw, r, lr, alpha, batch,
                               ws + sl.offBws, sl.bwsBytes, stream);
}

}  // extern "C"
