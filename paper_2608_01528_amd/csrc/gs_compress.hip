// Gram-Space compression on the GPU: block Gram-Schmidt with
// re-orthogonalisation and a relative rank threshold, in fp64.
//
// The paper builds the basis U and the Gram-loc codebook T = U^T W by
// Gram-Schmidt at initialisation (Sec. 3.3), with k the algebraic rank of the
// codebook (Sec. 3.2).  Codebook rows are taken in panels of PB rows, in index
// order.  For each panel W (pb x D):
//
//  1. first pass against the basis Q built from earlier panels (r_old rows):
//     H1 = W Q^T (its coefficients, into R), W -= H1 Q, in two parts: first
//     against the vectors of the panels before the previous one, then
//     against the previous panel's (block modified Gram-Schmidt over the two
//     parts).  The first part needs nothing of the previous panel, so it
//     runs while that panel is factored (on a second stream when one is
//     given, otherwise before it on the same stream; the results are the
//     same bit for bit);
//  2. the rows of the panel are orthogonalised among themselves in the small
//     space of the panel's triangular factor: W^T = Q_t R_t by a tree of
//     Householder factorisations (TSQR), so the columns a_i of R_t have the
//     inner products of the rows w_i.  Modified Gram-Schmidt runs on those
//     32-entry columns in index order, with a second projection for a column
//     that lost most of its norm; row i is dependent when the norm of what
//     is left of it is <= tol * ||c_i||, otherwise it adds a basis vector.
//     Each new basis vector is a combination of the panel's rows: V = X1 W;
//  3. second pass on the new vectors (where the first can have left them
//     measurably off the earlier span): H2 = V Q^T, V -= H2 Q, then V is
//     re-orthonormalised within itself (Cholesky of its Gram matrix, which is
//     the identity up to rounding at this point): Q_new = L^-1 V;
//  4. R of the panel's rows: R[i, old] = H1 + C1 H2 and R[i, new] = C1 L, with
//     C1 the small-space coefficients of step 2 (C1[i][k] = <w_i, v_k>).
//
// The result is the unique factorisation of the row-wise rules (rows in index
// order, first occurrence of a direction kept, positive pivots), so it is the
// one a Householder factorisation with column skipping returns.  The products
// with the basis run on fp64 matrix cores (v_mfma_f64_16x16x4f64).  The
// running rank lives on the device (rank_after[i] = rank once row i is
// done), so no launch waits on the host; grids are sized for the largest rank
// possible at that point and surplus work-groups exit.  Every reduction has a
// fixed order (no atomics), so results are bitwise reproducible.
#include <utility>

#include "gs_internal.h"

namespace gs {
namespace {

constexpr int PB = 32;        // panel rows
constexpr int NT = 256;       // threads of the panel kernels
constexpr int TCH = 256;      // rows of a TSQR node: panel columns of a leaf, or 8 stacked factors
constexpr int TFAN = TCH / PB;
constexpr int BK = 512;       // D-chunk of the split products W Q^T
constexpr int BK_PREV = 128;  // D-chunk of the product with the previous panel's vectors (short: two K-steps)
constexpr int KS = 64;        // K-step staged in LDS by the matrix-core products
constexpr int BN = 64;        // basis vectors (dots) or columns (update) per work-group
constexpr int LDK = KS + 1;   // LDS row stride (odd in doubles)

typedef double d4 __attribute__((ext_vector_type(4)));

// Row-count sources of the panel kernels: the panel's rows, the basis rows
// built before the panel, or the new basis vectors of the panel.
// The earlier basis splits for the first pass: ROWS_OLD_A, the vectors of
// the panels before the previous one; ROWS_OLD_B, the previous panel's.
enum Rows { ROWS_PANEL = 0, ROWS_OLD = 1, ROWS_NEW = 2, ROWS_OLD_PASS2 = 3, ROWS_OLD_A = 4, ROWS_OLD_B = 5 };

// Second pass against the earlier basis: needed only where the first pass
// can have left the new vectors measurably off orthogonal to it.  A new
// vector v = sum_i X1[i] w_i inherits each w_i's rounding-level component
// along the earlier basis (about eps ||c_i||) weighted by |X1[i]|, so the
// pass runs when some sum_i |X1[i]| ||c_i|| exceeds PASS2_WEIGHT (a vector
// made from rows that were each at least about 1/PASS2_WEIGHT of their norm
// away from the earlier span needs none).
constexpr double PASS2_WEIGHT = 8.0;

struct WsLayout {
    size_t qm, wp, wp_next, w2, hc, h2, g2, part, part_next, part_prev, gpart, tsq0, tsq1, x1, c1, lx, cn,
        rank_after, kept, flag, pass2, total;
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

int64_t leaf_count(int64_t D) { return (D + TCH - 1) / TCH; }
int64_t chunk_count(int64_t D, int64_t bk = BK) { return (D + bk - 1) / bk; }

WsLayout layout(int64_t M, int64_t D) {
    WsLayout L;
    const int64_t nch = chunk_count(D), nl = leaf_count(D);
    size_t o = 0;
    L.qm = o;    o = align256(o + sizeof(double) * M * D);
    L.wp = o;    o = align256(o + sizeof(double) * PB * D);
    L.wp_next = o; o = align256(o + sizeof(double) * PB * D);
    L.w2 = o;    o = align256(o + sizeof(double) * PB * D);
    L.hc = o;    o = align256(o + sizeof(double) * M * M);
    L.h2 = o;    o = align256(o + sizeof(double) * PB * M);
    L.g2 = o;    o = align256(o + sizeof(double) * PB * PB);
    L.part = o;  o = align256(o + sizeof(double) * nch * PB * (M > PB ? M : PB));
    L.part_next = o; o = align256(o + sizeof(double) * nch * PB * (M > PB ? M : PB));
    L.part_prev = o; o = align256(o + sizeof(double) * chunk_count(D, BK_PREV) * PB * PB);
    L.gpart = o; o = align256(o + sizeof(double) * ((D + BN - 1) / BN) * PB * PB);
    L.tsq0 = o;  o = align256(o + sizeof(double) * nl * PB * PB);
    L.tsq1 = o;  o = align256(o + sizeof(double) * nl * PB * PB);
    L.x1 = o;    o = align256(o + sizeof(double) * PB * PB);
    L.c1 = o;    o = align256(o + sizeof(double) * PB * PB);
    L.lx = o;    o = align256(o + sizeof(double) * 2 * PB * PB);
    L.cn = o;    o = align256(o + sizeof(double) * M);
    L.rank_after = o; o = align256(o + sizeof(int32_t) * M);
    L.kept = o;  o = align256(o + sizeof(int32_t) * M);
    L.flag = o;  o = align256(o + sizeof(int32_t));
    L.pass2 = o; o = align256(o + sizeof(int32_t));
    L.total = o;
    return L;
}

// Device view of the panel being processed.
struct Panel {
    int64_t i0;                 // first codebook row of the panel
    int pb;                     // rows in the panel
    const int32_t *rank_after;  // running rank
    const int32_t *pass2;       // set by the rank decisions: the second pass is needed
};

__device__ __forceinline__ int rank_before(const int32_t *rank_after, int64_t row) {
    return row == 0 ? 0 : rank_after[row - 1];
}

// Rank before the previous panel (0 for the first two panels).
__device__ __forceinline__ int rank_before_prev(const Panel &p) {
    return p.i0 >= PB ? rank_before(p.rank_after, p.i0 - PB) : 0;
}

__device__ __forceinline__ int rows_of(const Panel &p, int which) {
    const int r_old = rank_before(p.rank_after, p.i0);
    if (which == ROWS_PANEL) return p.pb;
    if (which == ROWS_OLD) return r_old;
    if (which == ROWS_OLD_PASS2) return *p.pass2 ? r_old : 0;
    if (which == ROWS_OLD_A) return rank_before_prev(p);
    if (which == ROWS_OLD_B) return r_old - rank_before_prev(p);
    return p.rank_after[p.i0 + p.pb - 1] - r_old;   // ROWS_NEW: valid after the panel's rank decisions
}

// First basis row of a set of basis rows (ROWS_OLD_B starts past ROWS_OLD_A).
__device__ __forceinline__ int rows_first(const Panel &p, int which) {
    return which == ROWS_OLD_B ? rank_before_prev(p) : 0;
}

template <typename T> __device__ __forceinline__ double ld_f64(const T *p, int64_t i);
template <> __device__ __forceinline__ double ld_f64<float>(const float *p, int64_t i) { return (double)p[i]; }
template <> __device__ __forceinline__ double ld_f64<double>(const double *p, int64_t i) { return p[i]; }
template <> __device__ __forceinline__ double ld_f64<bf16_t>(const bf16_t *p, int64_t i) {
    return (double)bf16_to_f32(p[i].bits);
}

// Sum of v over the work-group in a fixed order; result valid in thread 0.
__device__ double block_sum(double v, double *red) {
    const int t = threadIdx.x;
    for (int off = 32; off > 0; off >>= 1) v += __shfl_down(v, off);
    if ((t & 63) == 0) red[t >> 6] = v;
    __syncthreads();
    double s = 0.0;
    if (t == 0)
        for (int w = 0; w < NT / 64; ++w) s += red[w];
    __syncthreads();
    return s;
}

// Cross-lane moves of a double within a row of 16 lanes by DPP (no LDS
// round trip): the two 32-bit halves move alike.
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
    const long long b = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_update_dpp(0, (int)(b & 0xffffffffLL), CTRL, 0xf, 0xf, false);
    const int hi = __builtin_amdgcn_update_dpp(0, (int)(b >> 32), CTRL, 0xf, 0xf, false);
    return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}

// The panel factorisation and the small-space steps are chains of dependent
// steps on a few work-groups, and the next panel's products may share their
// CUs; their waves take instruction-issue precedence over those.
__device__ __forceinline__ void raise_wave_priority() { __builtin_amdgcn_s_setprio(3); }

__global__ void k_init(double *hc, int64_t nhc, int32_t *kept, int32_t *rank_after, int64_t M,
                       int32_t *flag) {
    const int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * NT;
    for (int64_t e = i; e < nhc; e += stride) hc[e] = 0.0;
    for (int64_t e = i; e < M; e += stride) { kept[e] = -1; rank_after[e] = 0; }
    if (i == 0) *flag = 0;
}

// Norms of the codebook rows (the rank threshold is relative to them) and
// the check for non-finite entries.  One work-group per row.
template <typename T>
__global__ void __launch_bounds__(NT) k_norms(const T *C, int64_t ldc, int64_t D, double *cn, int32_t *flag) {
    __shared__ double red[NT / 64];
    const int64_t i = blockIdx.x;
    double s = 0.0;
    bool bad = false;
    for (int64_t d = threadIdx.x; d < D; d += NT) {
        const double v = ld_f64<T>(C, i * ldc + d);
        bad |= !isfinite(v);
        s += v * v;
    }
    if (bad) *flag = 1;
    s = block_sum(s, red);
    if (threadIdx.x == 0) cn[i] = sqrt(s);
}

// Copy the panel's rows to fp64.  Grid: (rows, column blocks of 8 NT).
template <typename T>
__global__ void __launch_bounds__(NT) k_load_panel(const T *C, int64_t ldc, int64_t D, int64_t i0, double *wp) {
    const int64_t i = blockIdx.x;
    const int64_t d0 = (int64_t)blockIdx.y * NT * 8 + threadIdx.x;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        const int64_t d = d0 + u * NT;
        if (d < D) wp[i * D + d] = ld_f64<T>(C, (i0 + i) * ldc + d);
    }
}

// ---------------------------------------------------------------- products with the basis
//
// Matrix-core fp64 tiles: a work-group of four waves computes a 32 x 64
// block; wave w owns columns 16w .. 16w + 15 as two 16 x 16 blocks (rows
// 0..15 and 16..31).  For v_mfma_f64_16x16x4f64, lane l supplies A[l % 16][l / 16]
// and B[l / 16][l % 16], and holds D[l / 16 + 4 j][l % 16] in element j.

// part[c][i][kb + n] = sum over the c-th D-chunk (bk columns, a multiple of
// KS) of S[i][d] * Qb[kb + n][d] (i < rows(sw), kb + n < rows(qw)).  Grid:
// (basis blocks of 64, D-chunks).
__global__ void __launch_bounds__(NT) k_bdots(const double *S, int sw, const double *Qb, int qw, int64_t D,
                                              int64_t bk, Panel p, double *part, int64_t ldp) {
    __shared__ double Ss[PB * LDK];
    __shared__ double Qs[BN * LDK];
    const int ns = rows_of(p, sw), nq = rows_of(p, qw);
    const int kb = blockIdx.x * BN;
    if (kb >= nq || ns == 0) return;
    Qb += (int64_t)rows_first(p, qw) * D;
    const int64_t c = blockIdx.y;
    const int64_t d_lo = c * bk, d_hi = (d_lo + bk < D) ? d_lo + bk : D;
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    // staging: element u of a thread is row (t + 256 u) / 64, column t % 64,
    // so the 64 lanes of a wave read 64 consecutive doubles of one row
    const int col = t & 63, row0 = t >> 6;
    double sreg[8], qreg[16];
    auto fetch = [&](int64_t d0) {
        const int64_t d = d0 + col;
        const bool din = d < d_hi;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int r = row0 + 4 * u;
            sreg[u] = (r < ns && din) ? S[(int64_t)r * D + d] : 0.0;
        }
#pragma unroll
        for (int u = 0; u < 16; ++u) {
            const int r = row0 + 4 * u;
            qreg[u] = (kb + r < nq && din) ? Qb[(int64_t)(kb + r) * D + d] : 0.0;
        }
    };
    auto stash = [&]() {
#pragma unroll
        for (int u = 0; u < 8; ++u) Ss[(row0 + 4 * u) * LDK + col] = sreg[u];
#pragma unroll
        for (int u = 0; u < 16; ++u) Qs[(row0 + 4 * u) * LDK + col] = qreg[u];
    };
    d4 acc0 = {0, 0, 0, 0}, acc1 = {0, 0, 0, 0};
    fetch(d_lo);
    stash();
    __syncthreads();
    for (int64_t d0 = d_lo; d0 < d_hi; d0 += KS) {
        const bool more = d0 + KS < d_hi;
        if (more) fetch(d0 + KS);
#pragma unroll
        for (int s = 0; s < KS / 4; ++s) {
            const int kk = 4 * s + (lane >> 4);
            const double b = Qs[(16 * w + (lane & 15)) * LDK + kk];
            const double a0 = Ss[(lane & 15) * LDK + kk];
            const double a1 = Ss[(16 + (lane & 15)) * LDK + kk];
            acc0 = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b, acc0, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b, acc1, 0, 0, 0);
        }
        __syncthreads();
        if (more) {
            stash();
            __syncthreads();
        }
    }
    const int n = 16 * w + (lane & 15);
    if (kb + n < nq) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int i = (lane >> 4) + 4 * j;
            part[(c * PB + i) * ldp + kb + n] = acc0[j];
            part[(c * PB + 16 + i) * ldp + kb + n] = acc1[j];
        }
    }
}

// Sum of the n values p[0], p[st], ..., p[(n - 1) st] in a fixed order:
// eight running sums (terms 8 m + j, in order of m), so that eight loads are
// in flight at a time, added pairwise.
__device__ __forceinline__ double strided_sum(const double *p, int64_t n, int64_t st) {
    double s[8] = {0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0};
    int64_t c = 0;
    for (; c + 8 <= n; c += 8) {
#pragma unroll
        for (int j = 0; j < 8; ++j) s[j] += p[(c + j) * st];
    }
    for (int j = 0; c < n; ++c, ++j) s[j] += p[c * st];
    return ((s[0] + s[1]) + (s[2] + s[3])) + ((s[4] + s[5]) + (s[6] + s[7]));
}

// out[i][k] (leading dimension ldo) = sum over the chunks c of part[c][i][k],
// for i < rows(sw), k < rows(qw).  A work-group of 256 threads for 64
// entries, each quarter of the threads summing a quarter of the chunks,
// quarters added in order.
__global__ void __launch_bounds__(NT) k_breduce(const double *part, int64_t nch, int64_t ldp, int sw, int qw,
                                                Panel p, double *out, int64_t ldo) {
    __shared__ double red[4][64];
    const int ns = rows_of(p, sw), nq = rows_of(p, qw);
    const int t = threadIdx.x, qt = t >> 6;
    const int64_t e = (int64_t)blockIdx.x * 64 + (t & 63);
    const int i = (int)(e / ldp), k = (int)(e % ldp);
    const bool live = i < ns && k < nq;
    if (blockIdx.x * (int64_t)64 >= (int64_t)ns * ldp) return;     // the whole group is past the rows
    const int64_t c0 = nch * qt / 4, c1 = nch * (qt + 1) / 4;
    red[qt][t & 63] = live ? strided_sum(part + (c0 * PB + i) * ldp + k, c1 - c0, (int64_t)PB * ldp) : 0.0;
    __syncthreads();
    if (qt == 0 && live)
        out[rows_first(p, qw) + (int64_t)i * ldo + k] = (red[0][t] + red[1][t]) + (red[2][t] + red[3][t]);
}

// G[i][j] = sum over the column blocks b (in a fixed order) of
// gpart[b][i][j]: work-group of 256 threads for 64 entries, each quarter of
// the threads summing a quarter of the blocks, quarters added in order.
__global__ void __launch_bounds__(NT) k_gram_reduce(const double *gpart, int64_t nblk, double *G) {
    __shared__ double red[4][64];
    const int t = threadIdx.x, e = blockIdx.x * 64 + (t & 63), qt = t >> 6;
    const int64_t b0 = nblk * qt / 4, b1 = nblk * (qt + 1) / 4;
    red[qt][t & 63] = strided_sum(gpart + b0 * PB * PB + e, b1 - b0, (int64_t)PB * PB);
    __syncthreads();
    if (qt == 0) G[e] = (red[0][t] + red[1][t]) + (red[2][t] + red[3][t]);
}

// S[i][d] -= sum over k < rows(qw) of H[i][k] * Qb[k][d], for i < rows(sw).
// Grid: column blocks of 64.  With gpart, also the block's share of the
// Gram matrix of the updated rows: gpart[blk][i][j] = sum over the block's
// columns of S[i][d] S[j][d] (rows(qw) may then be 0: only the Gram part).
__global__ void __launch_bounds__(NT) k_bupdate(double *S, int sw, const double *H, int64_t ldh,
                                                const double *Qb, int qw, int64_t D, Panel p, double *gpart) {
    __shared__ double Hs[PB * LDK];
    __shared__ double Qs[KS * LDK];
    const int ns = rows_of(p, sw), nq = rows_of(p, qw);
    if (ns == 0 || (nq == 0 && !gpart)) return;
    const int q0 = rows_first(p, qw);
    H += q0;
    Qb += (int64_t)q0 * D;
    const int64_t d0 = (int64_t)blockIdx.x * BN;
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    // staging: element u of a thread is row (t + 256 u) / 64, column t % 64
    // (H tile 32 x 64 over k; Q tile 64 (k) x 64 (d)): 64 consecutive
    // doubles of one row per wave
    const int scol = t & 63, row0 = t >> 6;
    double hreg[8], qreg[16];
    auto fetch = [&](int k0) {
        const int k = k0 + scol;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int r = row0 + 4 * u;
            hreg[u] = (r < ns && k < nq) ? H[(int64_t)r * ldh + k] : 0.0;
        }
        const int64_t d = d0 + scol;
#pragma unroll
        for (int u = 0; u < 16; ++u) {
            const int r = row0 + 4 * u;
            qreg[u] = (k0 + r < nq && d < D) ? Qb[(int64_t)(k0 + r) * D + d] : 0.0;
        }
    };
    auto stash = [&]() {
#pragma unroll
        for (int u = 0; u < 8; ++u) Hs[(row0 + 4 * u) * LDK + scol] = hreg[u];
#pragma unroll
        for (int u = 0; u < 16; ++u) Qs[(row0 + 4 * u) * LDK + scol] = qreg[u];
    };
    d4 acc0 = {0, 0, 0, 0}, acc1 = {0, 0, 0, 0};
    if (nq > 0) {
        fetch(0);
        stash();
        __syncthreads();
    }
    for (int k0 = 0; k0 < nq; k0 += KS) {
        const bool more = k0 + KS < nq;
        if (more) fetch(k0 + KS);
#pragma unroll
        for (int s = 0; s < KS / 4; ++s) {
            const int kk = 4 * s + (lane >> 4);
            const double b = Qs[kk * LDK + 16 * w + (lane & 15)];
            const double a0 = Hs[(lane & 15) * LDK + kk];
            const double a1 = Hs[(16 + (lane & 15)) * LDK + kk];
            acc0 = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b, acc0, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b, acc1, 0, 0, 0);
        }
        __syncthreads();
        if (more) {
            stash();
            __syncthreads();
        }
    }
    const int col = 16 * w + (lane & 15);
    const int64_t d = d0 + col;
    double nv[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int i = (lane >> 4) + 4 * j;
        nv[j] = (i < ns && d < D) ? S[(int64_t)i * D + d] - acc0[j] : 0.0;
        nv[4 + j] = (16 + i < ns && d < D) ? S[(int64_t)(16 + i) * D + d] - acc1[j] : 0.0;
        if (i < ns && d < D) S[(int64_t)i * D + d] = nv[j];
        if (16 + i < ns && d < D) S[(int64_t)(16 + i) * D + d] = nv[4 + j];
    }
    if (!gpart) return;
    // the updated 32 x 64 block through LDS, then its Gram share
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int i = (lane >> 4) + 4 * j;
        Hs[i * LDK + col] = nv[j];
        Hs[(16 + i) * LDK + col] = nv[4 + j];
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < (PB * PB) / NT; ++u) {
        const int e = t + u * NT;
        const int i = e / PB, j = e % PB;
        double g0 = 0.0, g1 = 0.0;
#pragma unroll 8
        for (int c = 0; c < BN; c += 2) {
            g0 += Hs[i * LDK + c] * Hs[j * LDK + c];
            g1 += Hs[i * LDK + c + 1] * Hs[j * LDK + c + 1];
        }
        gpart[((int64_t)blockIdx.x * PB + i) * PB + j] = g0 + g1;
    }
}

// ---------------------------------------------------------------- panel factor (TSQR)
//
// Triangular factor R (PB x PB, upper) of a tall matrix T (TCH x PB) by
// Householder reflections, T = Q R.  Leaf: T[t][i] = S[i][TCH c + t], the
// panel's rows (i < rows(sw)) over D-chunk c.  Node: T stacks up to TFAN
// factors of the previous level.  Thread (k, g) = (t / TG, t % TG) holds
// column k of T in registers, rows g + TG q (q < TR), so the rows above a
// reflection (j < PB = 2 TG) are the first two of every lane's rows and the
// other rows need no masking; only the current reflector goes through LDS.
// Signs of R's rows are whatever the reflections give: only the inner
// products of R's columns (those of the panel's rows) are used.
//
// Reflection j: with x the part of column j from row j down, alpha = x_j,
// beta = -sign(alpha) ||x|| and v = x - beta e_j, H = I - v v^T / (beta
// (beta - alpha)) maps x to beta e_j.  The two factors are applied one after
// the other, (w / beta) / (beta - alpha) for w = <v, a>, each as a
// reciprocal: their product underflows for columns of norm below about
// 1e-154, the rounding residue that a rank-deficient panel leaves, and its
// reciprocal would overflow.  The loop over j is a loop (not unrolled), so the
// kernel's code stays small.

constexpr int TG = 16;              // lanes per column (one DPP row)
constexpr int TR = TCH / TG;        // rows of T held per lane
constexpr int TSQR_NT = PB * TG;    // threads of the TSQR kernel
// LDS stride of a lane's entries of the reflector: 16-byte reads of the 16
// lanes of a column start at 36 g mod 64 banks, all distinct
constexpr int VST = TR + 2;
static_assert(PB == 2 * TG, "rows above a reflection: the first two of each lane");

// Sum over the 16 lanes of a DPP row; every lane gets the same value (each
// pairing adds the same two operands on both lanes).
__device__ __forceinline__ double group16_sum(double v) {
    v += dpp_f64<0xB1>(v);     // quad_perm [1, 0, 3, 2]
    v += dpp_f64<0x4E>(v);     // quad_perm [2, 3, 0, 1]
    v += dpp_f64<0x141>(v);    // row_half_mirror
    v += dpp_f64<0x140>(v);    // row_mirror
    return v;
}

__global__ void __launch_bounds__(TSQR_NT) k_tsqr(const double *S, int sw, int64_t D, const double *Rin,
                                                  int64_t nin, double *Rout, Panel p) {
    __shared__ __attribute__((aligned(16))) double vbuf[2][VST * TG];
    __shared__ double coefs[2][2];
    raise_wave_priority();
    const int t = threadIdx.x;
    const int k = t / TG, g = t % TG;
    const int64_t c = blockIdx.x;
    double a[TR];
    if (S) {
        const int ns = rows_of(p, sw);
#pragma unroll
        for (int q = 0; q < TR; ++q) {
            const int64_t d = c * TCH + g + TG * q;
            a[q] = (k < ns && d < D) ? S[(int64_t)k * D + d] : 0.0;
        }
    } else {
#pragma unroll
        for (int q = 0; q < TR; ++q) {
            const int row = g + TG * q;                // row of the stack
            const int64_t f = c * TFAN + row / PB;     // factor index
            a[q] = (f < nin) ? Rin[(f * PB + (row % PB)) * PB + k] : 0.0;
        }
    }
    double diag = 0.0;                  // R[k][k], set at reflection k
#pragma unroll 1
    for (int j = 0; j < PB; ++j) {
        const int buf = j & 1;
        if (k == j) {
            // ||x below row j||^2 and alpha = T[j][j], on all 16 lanes
            const double t0 = (g > j) ? a[0] : 0.0, t1 = (g + TG > j) ? a[1] : 0.0;
            double s4[4] = {t0 * t0, t1 * t1, 0.0, 0.0};
#pragma unroll
            for (int q = 2; q < TR; ++q) s4[q & 3] += a[q] * a[q];
            const double al = (g == (j & (TG - 1))) ? (j < TG ? a[0] : a[1]) : 0.0;
            const double sg = group16_sum((s4[0] + s4[1]) + (s4[2] + s4[3]));
            const double alpha = group16_sum(al);
            double beta = alpha, c1 = 0.0, c2 = 0.0;
            if (sg != 0.0) {
                const double nrm = sqrt(alpha * alpha + sg);
                beta = (alpha <= 0.0) ? nrm : -nrm;
                c1 = 1.0 / beta;
                c2 = 1.0 / (beta - alpha);
            }
            vbuf[buf][VST * g] = (g > j) ? a[0] : (g == j ? alpha - beta : 0.0);
            vbuf[buf][VST * g + 1] = (g + TG > j) ? a[1] : (g + TG == j ? alpha - beta : 0.0);
#pragma unroll
            for (int q = 2; q < TR; ++q) vbuf[buf][VST * g + q] = a[q];
            if (g == 0) {
                coefs[buf][0] = c1;
                coefs[buf][1] = c2;
            }
            diag = beta;
        }
        __syncthreads();
        if (k > j) {
            const double c1 = coefs[buf][0], c2 = coefs[buf][1];
            double vr[TR];
#pragma unroll
            for (int q = 0; q < TR; ++q) vr[q] = vbuf[buf][VST * g + q];
            double w4[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
            for (int q = 0; q < TR; ++q) w4[q & 3] += vr[q] * a[q];
            const double wsum = (group16_sum((w4[0] + w4[1]) + (w4[2] + w4[3])) * c1) * c2;
#pragma unroll
            for (int q = 0; q < TR; ++q) a[q] -= wsum * vr[q];
        }
    }
    // upper triangle of the first PB rows: R[i][k] for i < k from the
    // registers, R[k][k] = beta of reflection k
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const int i = g + TG * q;
        Rout[(c * PB + i) * PB + k] = (i < k) ? a[q] : (i == k ? diag : 0.0);
    }
}

// ---------------------------------------------------------------- small-space steps (one wave)

// v of lane `lane` (a compile-time constant in the unrolled loops), on every lane.
__device__ __forceinline__ double lane_value(double v, int lane) {
    const long long b = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_readlane((int)(b & 0xffffffffLL), lane);
    const int hi = __builtin_amdgcn_readlane((int)(b >> 32), lane);
    return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}

// Rank decisions of the panel, in the panel's small space: column a_i of the
// factor R_t stands for row w_i (same inner products).  Rows are taken in
// index order by modified Gram-Schmidt, right-looking: lane j holds a_j in
// registers; when row i adds a vector z (its residual a_i / rho), the lanes
// of the later rows project it out of their columns at once (local dot
// products, one LDS broadcast of z per kept row).  Row i is dependent when the
// norm rho left is <= tol * ||c_i||.  Where the projections took away most of
// a_i (rho below REORTH of its norm), a_i is projected against all the kept
// vectors once more (classical Gram-Schmidt) before the decision, so the kept
// vectors stay orthogonal to working precision.  Outputs: X1[l][i] (new
// vector l = sum_i X1[l][i] w_i), C1[i][l] = <w_i, v_l> summed over the
// projections (the pivot for the row that made v_l), rank_after and kept for
// the panel's rows, vectors in the order they were kept.  One wave; lanes
// 0..31 are panel rows (columns of R_t) or vector entries.
constexpr int LP = PB + 2;         // LDS row stride of the small-space matrices (16-byte aligned rows)
constexpr double REORTH = 0.5;     // second projection when rho < REORTH * ||a_i||

// Column c of the inverse of the lower-triangular matrix Ck (nk x nk) whose
// row r is C[krow[r]][0 .. r] (the coefficients of the r-th kept row on the
// vectors up to its own, the pivot last): y[r] for r < nk, zero above c and
// past nk; rinv[r] = 1 / pivot r.  Rows are compile-time, so y stays in
// registers.
template <int... I>
__device__ __forceinline__ void tri_inverse_column(double (&y)[PB], int c, int nk, const double (*C)[LP],
                                                   const int *krow, const double *rinv,
                                                   std::integer_sequence<int, I...>) {
    auto row = [&](auto ic) {
        constexpr int r = decltype(ic)::value;
        const double *cr = C[krow[r]];
        double s0 = (r == c) ? 1.0 : 0.0, s1 = 0.0;
#pragma unroll
        for (int q = 0; q + 1 < r; q += 2) {
            s0 -= cr[q] * y[q];
            s1 -= cr[q + 1] * y[q + 1];
        }
        if constexpr (r % 2 == 1) s0 -= cr[r - 1] * y[r - 1];
        y[r] = (r >= c && r < nk) ? (s0 + s1) * rinv[r] : 0.0;
    };
    (row(std::integral_constant<int, I>{}), ...);
}

__global__ void __launch_bounds__(64) k_small_rank(const double *Rt, const double *cn, double tol, Panel p,
                                                   int32_t *rank_after, int32_t *kept, double *X1, double *C1,
                                                   int32_t *pass2_out) {
    __shared__ __attribute__((aligned(16))) double C1s[PB][LP];  // C1s[i][k]: coefficient of row i on vector k
    __shared__ __attribute__((aligned(16))) double XT[PB][LP];   // XT[i][k]: weight of row i in vector k
    __shared__ __attribute__((aligned(16))) double P[PB][LP];    // second projection: h_k z_k[e]
    __shared__ __attribute__((aligned(16))) double zb[PB];       // the vector broadcast
    __shared__ __attribute__((aligned(16))) double tb[PB];
    __shared__ double thr[PB], thr_cn[PB];
    __shared__ int kidx[PB];                                     // kept index of each row (-1: dependent)
    __shared__ int krow[PB];                                     // row that made each kept vector
    __shared__ double rinv[PB];                                  // 1 / pivot of each kept vector
    raise_wave_priority();
    const int l = threadIdx.x;
    const bool act = l < PB;
    const bool row_l = l < p.pb;       // lane l is a row of this panel
    const int r_old = rank_before(p.rank_after, p.i0);
    if (row_l) {
        thr_cn[l] = cn[p.i0 + l];
        thr[l] = tol * thr_cn[l];
    }
    if (act) {
        kidx[l] = -1;
        krow[l] = 0;
    }
    for (int e = l; e < PB * LP; e += 64) {
        (&C1s[0][0])[e] = 0.0;
        (&XT[0][0])[e] = 0.0;
    }
    // lane l: column l of R_t (zero for lanes past the panel)
    double a[PB];
#pragma unroll
    for (int e = 0; e < PB; ++e) a[e] = row_l ? Rt[e * PB + l] : 0.0;
    auto sumsq = [&]() {
        double q0 = 0.0, q1 = 0.0, q2 = 0.0, q3 = 0.0;
#pragma unroll
        for (int e = 0; e < PB; e += 4) {
            q0 += a[e] * a[e]; q1 += a[e + 1] * a[e + 1]; q2 += a[e + 2] * a[e + 2]; q3 += a[e + 3] * a[e + 3];
        }
        return (q0 + q1) + (q2 + q3);
    };
    const double n0 = sqrt(sumsq());
    __syncthreads();
    int nk = 0;
    for (int i = 0; i < p.pb; ++i) {
        double rho = sqrt(lane_value(sumsq(), i));
        if (nk > 0 && rho < REORTH * lane_value(n0, i)) {
            // a_i -= sum over kept k of <a_i, z_k> z_k; kept lanes k < i hold z_k
            if (l == i) {
#pragma unroll
                for (int e = 0; e < PB; ++e) zb[e] = a[e];
            }
            __syncthreads();
            const bool holds_z = act && l < i && kidx[l] >= 0;
            double h = 0.0;
            if (holds_z) {
                double h0 = 0.0, h1 = 0.0, h2 = 0.0, h3 = 0.0;
#pragma unroll
                for (int e = 0; e < PB; e += 4) {
                    h0 += zb[e] * a[e]; h1 += zb[e + 1] * a[e + 1]; h2 += zb[e + 2] * a[e + 2]; h3 += zb[e + 3] * a[e + 3];
                }
                h = (h0 + h1) + (h2 + h3);
                C1s[i][kidx[l]] += h;
            }
            if (act) {
#pragma unroll
                for (int e = 0; e < PB; ++e) P[l][e] = holds_z ? h * a[e] : 0.0;
            }
            __syncthreads();
            if (act) {
                double t0 = 0.0, t1 = 0.0;           // entry l of sum_k h_k z_k, rows in order
#pragma unroll
                for (int k = 0; k < PB; k += 2) { t0 += P[k][l]; t1 += P[k + 1][l]; }
                tb[l] = t0 + t1;
            }
            __syncthreads();
            if (l == i) {
#pragma unroll
                for (int e = 0; e < PB; ++e) a[e] -= tb[e];
            }
            rho = sqrt(lane_value(sumsq(), i));
        }
        const bool keep = rho > thr[i];
        if (keep) {
            // lane i: z = a_i / rho; the later rows project it out
            if (l == i) {
                const double inv = 1.0 / rho;
#pragma unroll
                for (int e = 0; e < PB; ++e) {
                    a[e] *= inv;
                    zb[e] = a[e];
                }
                C1s[i][nk] = rho;
                kidx[i] = nk;
                rinv[nk] = inv;
            }
            __syncthreads();
            if (row_l && l > i) {
                double d0 = 0.0, d1 = 0.0, d2 = 0.0, d3 = 0.0;
#pragma unroll
                for (int e = 0; e < PB; e += 4) {
                    d0 += zb[e] * a[e]; d1 += zb[e + 1] * a[e + 1]; d2 += zb[e + 2] * a[e + 2]; d3 += zb[e + 3] * a[e + 3];
                }
                const double d = (d0 + d1) + (d2 + d3);
#pragma unroll
                for (int e = 0; e < PB; ++e) a[e] -= d * zb[e];
                C1s[l][nk] = d;
            }
            if (l == 0) {
                kept[r_old + nk] = (int32_t)(p.i0 + i);
                krow[nk] = i;
            }
            ++nk;
            __syncthreads();
        }
        if (l == 0) rank_after[p.i0 + i] = r_old + nk;
    }
    __syncthreads();
    // weights of the new vectors: with Ck the coefficients of the kept rows on
    // the new vectors (lower triangular, pivots on the diagonal), the kept
    // rows are Ck times the new vectors, so X1 = Ck^-1 on the kept rows'
    // columns.  Lane c: column c, written to XT[row of c][k]
    if (act && l < nk) {
        double y[PB];
        tri_inverse_column(y, l, nk, C1s, krow, rinv, std::make_integer_sequence<int, PB>{});
        const int ir = krow[l];
#pragma unroll
        for (int k = 0; k < PB; ++k)
            if (k < nk) XT[ir][k] = y[k];
    }
    __syncthreads();
    // outputs; and the largest combination weight sum_i |X1[k][i]| ||c_i||
    // over the new vectors (lane k: vector k)
    for (int e = l; e < PB * PB; e += 64) {
        const int i = e / PB, k = e % PB;           // C1[i][k]
        C1[e] = (i < p.pb && k < nk) ? C1s[i][k] : 0.0;
        const int kx = e / PB, ix = e % PB;         // X1[kx][ix]
        X1[e] = (kx < nk && ix < p.pb) ? XT[ix][kx] : 0.0;
    }
    double wk = 0.0;
    if (act && l < nk)
        for (int i = 0; i < p.pb; ++i) wk += fabs(XT[i][l]) * thr_cn[i];
    for (int off = 32; off > 0; off >>= 1) wk = fmax(wk, __shfl_xor(wk, off));
    if (l == 0) *pass2_out = (wk > PASS2_WEIGHT) ? 1 : 0;
}

// Cholesky factor L of the Gram matrix G (n x n, n = new vectors; the
// vectors are orthonormal up to rounding) and its inverse.  LX[0] = L (lower),
// LX[1] = L^-1.  A pivot that is not positive sets flag 2.  One wave,
// right-looking: lane l holds column l of the trailing matrix in registers;
// step j broadcasts column j through LDS, and every later lane subtracts its
// outer-product share (entries at or above j of a lane's column are no
// longer read and are left as they come).
template <int... I>
__device__ __forceinline__ void inv_rows(double (&y)[PB], int c, const double (*L)[PB + 1], const double *rd,
                                         std::integer_sequence<int, I...>) {
    // y[i] = (delta_ic - sum_{k<i} L[i][k] y[k]) / L[i][i], rows in order, two running sums
    auto row = [&](auto ic) {
        constexpr int i = decltype(ic)::value;
        double s0 = (i == c) ? 1.0 : 0.0, s1 = 0.0;
#pragma unroll
        for (int k = 0; k + 1 < i; k += 2) {
            s0 -= L[i][k] * y[k];
            s1 -= L[i][k + 1] * y[k + 1];
        }
        if constexpr (i % 2 == 1) s0 -= L[i][i - 1] * y[i - 1];
        y[i] = (i >= c) ? (s0 + s1) * rd[i] : 0.0;
    };
    (row(std::integral_constant<int, I>{}), ...);
}

__global__ void __launch_bounds__(64) k_small_chol(const double *G, Panel p, double *LX, int32_t *flag) {
    __shared__ double L[PB][PB + 1];
    __shared__ __attribute__((aligned(16))) double zb[PB];
    __shared__ double rd[PB];          // 1 / L[j][j]
    raise_wave_priority();
    const int l = threadIdx.x;
    const bool act = l < PB;
    const int n = rows_of(p, ROWS_NEW);
    for (int e = l; e < PB * (PB + 1); e += 64) (&L[0][0])[e] = 0.0;
    double a[PB];
#pragma unroll
    for (int e = 0; e < PB; ++e) a[e] = (act && l < n && e < n) ? G[e * PB + l] : 0.0;
    bool bad = false;
    for (int j = 0; j < n; ++j) {
        if (l == j) {
#pragma unroll
            for (int e = 0; e < PB; ++e) zb[e] = a[e];
        }
        __syncthreads();
        const double piv = zb[j];
        if (!(piv > 0.0)) bad = true;
        const double d = sqrt(piv > 0.0 ? piv : 1.0);
        const double inv = 1.0 / d;
        if (act && l >= j && l < n) L[l][j] = (l == j) ? d : zb[l] * inv;
        if (l == j) rd[j] = inv;
        if (act && l > j && l < n) {
            const double f = zb[l] * inv * inv;    // L[l][j] / L[j][j]
#pragma unroll
            for (int e = 0; e < PB; ++e) a[e] -= f * zb[e];
        }
        __syncthreads();
    }
    // identity padding beyond n keeps the inverse finite
    if (act && l >= n) {
        L[l][l] = 1.0;
        rd[l] = 1.0;
    }
    __syncthreads();
    double y[PB];
    if (act) inv_rows(y, l, L, rd, std::make_integer_sequence<int, PB>{});
#pragma unroll
    for (int i = 0; i < PB; ++i)
        if (act) LX[PB * PB + i * PB + l] = (l < n && i < n) ? y[i] : 0.0;
    for (int e = l; e < PB * PB; e += 64) {
        const int i = e / PB, k = e % PB;
        LX[e] = (i < n && k < n) ? L[i][k] : 0.0;
    }
    if (bad && l == 0) *flag |= 2;
}

// dst[o][d] = sum over i < rows(sw) of X[o][i] * src[i][d], for o < rows(ow);
// with at_new, dst starts at row r_old (the panel's new basis rows).  Grid:
// column blocks of 64; thread (column t % 64, output group t / 64) forms the
// outputs o = t / 64 + 4 m.
__global__ void __launch_bounds__(NT) k_combine(const double *X, int ow, const double *src, int sw, double *dst,
                                                bool at_new, int64_t D, Panel p) {
    __shared__ double Xs[PB * PB];
    const int no = rows_of(p, ow), ns = rows_of(p, sw);
    if (no == 0) return;
    if (at_new) dst += (int64_t)rank_before(p.rank_after, p.i0) * D;
    for (int e = threadIdx.x; e < PB * PB; e += NT) Xs[e] = X[e];
    __syncthreads();
    const int64_t d = (int64_t)blockIdx.x * 64 + (threadIdx.x & 63);
    const int og = threadIdx.x >> 6;
    if (d >= D) return;
    double sv[PB];
#pragma unroll
    for (int i = 0; i < PB; ++i) sv[i] = (i < ns) ? src[(int64_t)i * D + d] : 0.0;
#pragma unroll
    for (int m = 0; m < PB / 4; ++m) {
        const int o = og + 4 * m;
        if (o < no) {
            double a0 = 0.0, a1 = 0.0;
#pragma unroll
            for (int i = 0; i < PB; i += 2) {
                a0 += Xs[o * PB + i] * sv[i];
                a1 += Xs[o * PB + i + 1] * sv[i + 1];
            }
            dst[(int64_t)o * D + d] = a0 + a1;
        }
    }
}

// Coefficients of the panel's rows: R[i0 + i][k] += sum_l C1[i][l] H2[l][k]
// (k < r_old, second pass) and R[i0 + i][r_old + l] = sum_m C1[i][m] L[m][l].
// One thread per (row, column); grid: (column blocks of 256, panel rows).
__global__ void __launch_bounds__(NT) k_coef(const double *C1, const double *H2, int64_t ldh, bool pass2,
                                             const double *LX, double *hc, int64_t M, Panel p) {
    __shared__ double c[PB];
    const int r_old = rank_before(p.rank_after, p.i0);
    const int nn = rows_of(p, ROWS_NEW);
    const int i = blockIdx.y;
    if (threadIdx.x < PB) c[threadIdx.x] = C1[i * PB + threadIdx.x];
    __syncthreads();
    const int64_t k = (int64_t)blockIdx.x * NT + threadIdx.x;
    if (k < r_old && pass2 && *p.pass2) {
        double s = 0.0;
#pragma unroll 8
        for (int l = 0; l < nn; ++l) s += c[l] * H2[(int64_t)l * ldh + k];
        hc[(p.i0 + i) * M + k] += s;
    } else if (k >= r_old && k < r_old + nn) {
        const int l = (int)(k - r_old);
        double s = 0.0;
        for (int m = l; m < nn; ++m) s += c[m] * LX[m * PB + l];
        hc[(p.i0 + i) * M + k] = s;
    }
}

template <typename TQ, typename TR>
__global__ void k_outputs(const double *qm, const double *hc, const double *cnd,
                          const int32_t *rank_after, const int32_t *kept_ws, int64_t M, int64_t D,
                          TQ *Q, int64_t ldq, TR *R, int64_t ldr, int32_t *kept, float *cnorm, int64_t row_base) {
    const int r = rank_after[M - 1];
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    for (int64_t e = i0; e < M * D; e += stride) {
        const int64_t k = e / D, d = e % D;
        const double v = (k < r) ? qm[e] : 0.0;
        if constexpr (sizeof(TQ) == 8) Q[k * ldq + d] = v;
        else if constexpr (sizeof(TQ) == 4) Q[k * ldq + d] = (float)v;
        else Q[k * ldq + d].bits = f64_to_bf16(v);
    }
    for (int64_t e = i0; e < M * M; e += stride) {
        const int64_t i = e / M, k = e % M;
        const double v = (k < r) ? hc[e] : 0.0;
        if constexpr (sizeof(TR) == 8) R[i * ldr + k] = v;
        else if constexpr (sizeof(TR) == 4) R[i * ldr + k] = (float)v;
        else R[i * ldr + k].bits = f64_to_bf16(v);
    }
    for (int64_t e = i0; e < M; e += stride) {
        if (kept) kept[e] = (e < r) ? (int32_t)(kept_ws[e] + row_base) : -1;
        if (cnorm) cnorm[e] = (float)cnd[e];
    }
}

template <typename TQ, typename TR>
hipError_t launch_outputs(const WsLayout &L, char *ws, int64_t M, int64_t D, void *Q, int64_t ldq,
                          void *R, int64_t ldr, int32_t *kept, float *cnorm, int64_t row_base, hipStream_t s) {
    hipLaunchKernelGGL((k_outputs<TQ, TR>), dim3(1024), dim3(NT), 0, s,
                       (const double *)(ws + L.qm), (const double *)(ws + L.hc),
                       (const double *)(ws + L.cn), (const int32_t *)(ws + L.rank_after),
                       (const int32_t *)(ws + L.kept), M, D, (TQ *)Q, ldq, (TR *)R, ldr, kept, cnorm, row_base);
    return hipGetLastError();
}

template <typename TQ>
hipError_t outputs_r(gs_dtype rt, const WsLayout &L, char *ws, int64_t M, int64_t D, void *Q,
                     int64_t ldq, void *R, int64_t ldr, int32_t *kept, float *cnorm, int64_t row_base,
                     hipStream_t s) {
    if (rt == GS_F64) return launch_outputs<TQ, double>(L, ws, M, D, Q, ldq, R, ldr, kept, cnorm, row_base, s);
    if (rt == GS_F32) return launch_outputs<TQ, float>(L, ws, M, D, Q, ldq, R, ldr, kept, cnorm, row_base, s);
    return launch_outputs<TQ, bf16_t>(L, ws, M, D, Q, ldq, R, ldr, kept, cnorm, row_base, s);
}

template <typename T>
hipError_t launch_load(const void *C, int64_t ldc, int64_t D, int64_t i0, int pb, double *wp, hipStream_t s) {
    hipLaunchKernelGGL((k_load_panel<T>), dim3(pb, (unsigned)((D + NT * 8 - 1) / (NT * 8))), dim3(NT), 0, s,
                       (const T *)C, ldc, D, i0, wp);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_norms(const void *C, int64_t ldc, int64_t M, int64_t D, double *cn, int32_t *flag,
                        hipStream_t s) {
    hipLaunchKernelGGL((k_norms<T>), dim3((unsigned)M), dim3(NT), 0, s, (const T *)C, ldc, D, cn, flag);
    return hipGetLastError();
}

#define GS_TRY(x) do { hipError_t e_ = (x); if (e_ != hipSuccess) return e_; } while (0)

// One pass of the block projection: H = S Qb^T (split over D-chunks of bk
// columns, reduced in a fixed order into out, leading dimension ldo), then
// S -= H Qb (with gpart, also the column blocks' shares of the Gram matrix
// of the updated S).  part holds chunk_count(D, bk) x PB x ldp partial sums.
hipError_t block_pass(double *S, int sw, const double *Qb, int qw, int64_t max_q, int64_t D, int64_t bk,
                      const Panel &p, double *part, int64_t ldp, double *out, int64_t ldo, double *gpart,
                      hipStream_t s) {
    const int64_t nch = chunk_count(D, bk);
    const dim3 gd((unsigned)((max_q + BN - 1) / BN), (unsigned)nch);
    hipLaunchKernelGGL(k_bdots, gd, dim3(NT), 0, s, (const double *)S, sw, Qb, qw, D, bk, p, part, ldp);
    const unsigned gr = (unsigned)((PB * ldp + 63) / 64);
    hipLaunchKernelGGL(k_breduce, dim3(gr), dim3(NT), 0, s, (const double *)part, nch, ldp, sw, qw, p, out, ldo);
    if (!gpart) {
        hipLaunchKernelGGL(k_bupdate, dim3((unsigned)((D + BN - 1) / BN)), dim3(NT), 0, s, S, sw,
                           (const double *)out, ldo, Qb, qw, D, p, (double *)nullptr);
    } else {
        hipLaunchKernelGGL(k_bupdate, dim3((unsigned)((D + BN - 1) / BN)), dim3(NT), 0, s, S, sw,
                           (const double *)out, ldo, Qb, qw, D, p, gpart);
    }
    return hipGetLastError();
}

// Triangular factor of the panel held in S (rows(sw) rows): leaves, then
// nodes until one factor remains.  Returns the buffer holding it.
hipError_t panel_factor(const double *S, int sw, int64_t D, const Panel &p, double *b0, double *b1,
                        double **out, hipStream_t s) {
    int64_t n = leaf_count(D);
    hipLaunchKernelGGL(k_tsqr, dim3((unsigned)n), dim3(TSQR_NT), 0, s, S, sw, D, (const double *)nullptr, (int64_t)0,
                       b0, p);
    double *cur = b0, *nxt = b1;
    while (n > 1) {
        const int64_t m = (n + TFAN - 1) / TFAN;
        hipLaunchKernelGGL(k_tsqr, dim3((unsigned)m), dim3(TSQR_NT), 0, s, (const double *)nullptr, 0, D,
                           (const double *)cur, n, nxt, p);
        double *tmp = cur; cur = nxt; nxt = tmp;
        n = m;
    }
    *out = cur;
    return hipGetLastError();
}

}  // namespace

size_t compress_workspace(int64_t M, int64_t D) { return layout(M, D).total; }

hipError_t run_compress(const void *C, gs_dtype ct, int64_t M, int64_t D, int64_t ldc, double tol,
                        void *Q, gs_dtype qt, int64_t ldq, void *R, gs_dtype rt, int64_t ldr,
                        int32_t *kept, float *cnorm, int32_t *rank, int *nonfinite, void *ws_,
                        hipStream_t s, int64_t row_base, const CompressOverlap *ov) {
    const WsLayout L = layout(M, D);
    char *ws = static_cast<char *>(ws_);
    double *qm = (double *)(ws + L.qm), *w2 = (double *)(ws + L.w2);
    double *wbuf[2] = {(double *)(ws + L.wp), (double *)(ws + L.wp_next)};
    double *hc = (double *)(ws + L.hc), *h2 = (double *)(ws + L.h2), *g2 = (double *)(ws + L.g2);
    double *part = (double *)(ws + L.part), *part_next = (double *)(ws + L.part_next);
    double *part_prev = (double *)(ws + L.part_prev);
    double *tsq0 = (double *)(ws + L.tsq0), *tsq1 = (double *)(ws + L.tsq1);
    double *gpart = (double *)(ws + L.gpart);
    const int64_t nblk = (D + BN - 1) / BN;
    double *x1 = (double *)(ws + L.x1), *c1 = (double *)(ws + L.c1), *lx = (double *)(ws + L.lx);
    double *cn = (double *)(ws + L.cn);
    int32_t *rank_after = (int32_t *)(ws + L.rank_after), *kept_ws = (int32_t *)(ws + L.kept);
    int32_t *flag = (int32_t *)(ws + L.flag), *pass2 = (int32_t *)(ws + L.pass2);
    const int64_t ldp = M > PB ? M : PB;
    const int64_t npanels = (M + PB - 1) / PB;
    auto panel = [&](int64_t q) {
        const int64_t i0 = q * PB;
        return Panel{i0, (int)((M - i0 < PB) ? (M - i0) : PB), rank_after, pass2};
    };
    // Panel q's rows into its buffer, and the first part of its first pass:
    // against the vectors of the panels before q - 1 (coefficients into R).
    // Reads only what panels up to q - 2 produced.
    auto stage = [&](int64_t q, hipStream_t st) -> hipError_t {
        const Panel pn = panel(q);
        double *w = wbuf[q & 1];
        if (ct == GS_F32) GS_TRY(launch_load<float>(C, ldc, D, pn.i0, pn.pb, w, st));
        else if (ct == GS_F64) GS_TRY(launch_load<double>(C, ldc, D, pn.i0, pn.pb, w, st));
        else GS_TRY(launch_load<bf16_t>(C, ldc, D, pn.i0, pn.pb, w, st));
        if (pn.i0 >= 2 * PB)
            GS_TRY(block_pass(w, ROWS_PANEL, qm, ROWS_OLD_A, pn.i0 - PB, D, BK, pn, part_next, ldp, hc + pn.i0 * M,
                              M, nullptr, st));
        return hipSuccess;
    };

    hipLaunchKernelGGL(k_init, dim3(1024), dim3(NT), 0, s, hc, M * M, kept_ws, rank_after, M, flag);
    GS_TRY(hipGetLastError());
    if (ct == GS_F32) GS_TRY(launch_norms<float>(C, ldc, M, D, cn, flag, s));
    else if (ct == GS_F64) GS_TRY(launch_norms<double>(C, ldc, M, D, cn, flag, s));
    else GS_TRY(launch_norms<bf16_t>(C, ldc, M, D, cn, flag, s));
    GS_TRY(stage(0, s));

    for (int64_t q = 0; q < npanels; ++q) {
        const Panel p = panel(q);
        const int64_t i0 = p.i0;
        double *wp = wbuf[q & 1];
        // 1. the rest of the first pass: against the previous panel's vectors
        if (q > 0) {
            if (ov) GS_TRY(hipStreamWaitEvent(s, ov->join, 0));
            GS_TRY(block_pass(wp, ROWS_PANEL, qm, ROWS_OLD_B, PB, D, BK_PREV, p, part_prev, PB, hc + i0 * M, M,
                              nullptr, s));
        }
        // the next panel's rows and the first part of its first pass, beside
        // this panel's factorisation (they touch none of its buffers)
        if (q + 1 < npanels) {
            if (ov) {
                GS_TRY(hipEventRecord(ov->fork, s));
                GS_TRY(hipStreamWaitEvent(ov->aux, ov->fork, 0));
                GS_TRY(stage(q + 1, ov->aux));
                GS_TRY(hipEventRecord(ov->join, ov->aux));
            } else {
                GS_TRY(stage(q + 1, s));
            }
        }
        // 2. rank decisions in the panel's small space; first-round new vectors
        double *rt_ = nullptr;
        GS_TRY(panel_factor(wp, ROWS_PANEL, D, p, tsq0, tsq1, &rt_, s));
        hipLaunchKernelGGL(k_small_rank, dim3(1), dim3(64), 0, s, (const double *)rt_, (const double *)cn, tol, p,
                           rank_after, kept_ws, x1, c1, pass2);
        hipLaunchKernelGGL(k_combine, dim3((unsigned)nblk), dim3(NT), 0, s, (const double *)x1,
                           (int)ROWS_NEW, (const double *)wp, (int)ROWS_PANEL, w2, false, D, p);
        GS_TRY(hipGetLastError());
        // 3. second pass on the new vectors, with their Gram matrix, and its
        // Cholesky factor
        if (i0 > 0) {
            GS_TRY(block_pass(w2, ROWS_NEW, qm, ROWS_OLD_PASS2, i0, D, BK, p, part, ldp, h2, M, gpart, s));
        } else {
            hipLaunchKernelGGL(k_bupdate, dim3((unsigned)nblk), dim3(NT), 0, s, w2, (int)ROWS_NEW,
                               (const double *)h2, M, (const double *)qm, (int)ROWS_OLD, D, p, gpart);
        }
        hipLaunchKernelGGL(k_gram_reduce, dim3(PB * PB / 64), dim3(NT), 0, s, (const double *)gpart, nblk, g2);
        GS_TRY(hipGetLastError());
        hipLaunchKernelGGL(k_small_chol, dim3(1), dim3(64), 0, s, (const double *)g2, p, lx, flag);
        // final basis vectors Q_new = L^-1 V, and the panel's coefficients
        hipLaunchKernelGGL(k_combine, dim3((unsigned)nblk), dim3(NT), 0, s,
                           (const double *)(lx + PB * PB), (int)ROWS_NEW, (const double *)w2, (int)ROWS_NEW,
                           qm, true, D, p);
        GS_TRY(hipGetLastError());
        hipLaunchKernelGGL(k_coef, dim3((unsigned)((i0 + PB + NT - 1) / NT), (unsigned)p.pb), dim3(NT), 0, s,
                           (const double *)c1,
                           (const double *)h2, M, i0 > 0, (const double *)lx, hc, M, p);
        GS_TRY(hipGetLastError());
    }

    if (qt == GS_F64) GS_TRY(outputs_r<double>(rt, L, ws, M, D, Q, ldq, R, ldr, kept, cnorm, row_base, s));
    else if (qt == GS_F32) GS_TRY(outputs_r<float>(rt, L, ws, M, D, Q, ldq, R, ldr, kept, cnorm, row_base, s));
    else GS_TRY(outputs_r<bf16_t>(rt, L, ws, M, D, Q, ldq, R, ldr, kept, cnorm, row_base, s));

    int32_t host[2] = {0, 0};
    GS_TRY(hipMemcpyAsync(&host[0], rank_after + (M - 1), sizeof(int32_t), hipMemcpyDeviceToHost, s));
    GS_TRY(hipMemcpyAsync(&host[1], flag, sizeof(int32_t), hipMemcpyDeviceToHost, s));
    GS_TRY(hipStreamSynchronize(s));
    *rank = host[0];
    *nonfinite = host[1];
    return hipSuccess;
}

namespace {

// Fill a rows x cols matrix (leading dimension ld, element size es) with
// zero bits, or int32 matrices with fill_i32.
__global__ void k_fill(char *base, int64_t rows, int64_t cols, int64_t ld, int es, int32_t fill_i32) {
    const int64_t n = rows * cols;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += stride) {
        const int64_t i = e / cols, k = e % cols;
        char *p = base + (i * ld + k) * es;
        if (es == 8) *reinterpret_cast<double *>(p) = 0.0;
        else if (es == 4) *reinterpret_cast<int32_t *>(p) = fill_i32;
        else *reinterpret_cast<uint16_t *>(p) = 0;
    }
}

size_t esz(gs_dtype t) { return t == GS_F64 ? 8 : (t == GS_F32 ? 4 : 2); }

// The augmented codebook of the padded basis, fp64: rows 0 .. M-1 the
// codebook, rows M .. M + k - 1 the unit vectors e_0 .. e_{k-1}.
template <typename T>
__global__ void k_augment(const T *C, int64_t ldc, int64_t M, int64_t D, int64_t k, double *A) {
    const int64_t n = (M + k) * D;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += stride) {
        const int64_t i = e / D, d = e % D;
        A[e] = (i < M) ? ld_f64<T>(C, i * ldc + d) : ((d == i - M) ? 1.0 : 0.0);
    }
}

// out = op(A) op(B) in fp64 for small sizes (m x n, inner dimension kk):
// A is m x kk (lda); B is kk x n (ldb), or n x kk read transposed when
// b_trans.  16 x 16 tiles through LDS, one output per thread.
__global__ void __launch_bounds__(256) k_dgemm(const double *A, int64_t lda, const double *B, int64_t ldb,
                                               bool b_trans, double *out, int64_t ldo, int64_t m, int64_t n,
                                               int64_t kk) {
    __shared__ double As[16][17], Bs[16][17];
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    const int64_t i = (int64_t)blockIdx.y * 16 + ty, j = (int64_t)blockIdx.x * 16 + tx;
    double acc = 0.0;
    for (int64_t t0 = 0; t0 < kk; t0 += 16) {
        As[ty][tx] = (i < m && t0 + tx < kk) ? A[i * lda + t0 + tx] : 0.0;
        const int64_t bt = t0 + ty;
        double bv = 0.0;
        if (bt < kk && j < n) bv = b_trans ? B[j * ldb + bt] : B[bt * ldb + j];
        Bs[ty][tx] = bv;
        __syncthreads();
#pragma unroll
        for (int q = 0; q < 16; ++q) acc += As[ty][q] * Bs[q][tx];
        __syncthreads();
    }
    if (i < m && j < n) out[i * ldo + j] = acc;
}

// Store an fp64 matrix (rows x cols, leading dimension lds) as type T.
template <typename T>
__global__ void k_store(const double *src, int64_t lds, T *dst, int64_t ldd, int64_t rows, int64_t cols) {
    const int64_t n = rows * cols;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += stride) {
        const int64_t i = e / cols, c = e % cols;
        const double v = src[i * lds + c];
        if constexpr (sizeof(T) == 8) dst[i * ldd + c] = v;
        else if constexpr (sizeof(T) == 4) dst[i * ldd + c] = (float)v;
        else dst[i * ldd + c].bits = f64_to_bf16(v);
    }
}

hipError_t store_as(gs_dtype t, const double *src, int64_t lds, void *dst, int64_t ldd, int64_t rows, int64_t cols,
                    hipStream_t s) {
    if (t == GS_F64) hipLaunchKernelGGL((k_store<double>), dim3(1024), dim3(NT), 0, s, src, lds, (double *)dst, ldd, rows, cols);
    else if (t == GS_F32) hipLaunchKernelGGL((k_store<float>), dim3(1024), dim3(NT), 0, s, src, lds, (float *)dst, ldd, rows, cols);
    else hipLaunchKernelGGL((k_store<bf16_t>), dim3(1024), dim3(NT), 0, s, src, lds, (bf16_t *)dst, ldd, rows, cols);
    return hipGetLastError();
}

struct PadLayout { size_t aug, qa, ra, qh, rh, kept, cn, cws, total; };

PadLayout pad_layout(int64_t M, int64_t D, int64_t k) {
    PadLayout L;
    const int64_t Ma = M + k;
    size_t o = 0;
    L.aug = o;  o = align256(o + sizeof(double) * Ma * D);
    L.qa = o;   o = align256(o + sizeof(double) * Ma * D);
    L.ra = o;   o = align256(o + sizeof(double) * Ma * Ma);
    L.qh = o;   o = align256(o + sizeof(double) * k * D);
    L.rh = o;   o = align256(o + sizeof(double) * M * k);
    L.kept = o; o = align256(o + sizeof(int32_t) * Ma);
    L.cn = o;   o = align256(o + sizeof(float) * Ma);
    L.cws = o;  o = align256(o + compress_workspace(Ma, D));
    L.total = o;
    return L;
}

// Copy n int32 / float values (4-byte elements).
__global__ void k_copy4(const int32_t *src, int32_t *dst, int64_t n, int64_t valid) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e < n) dst[e] = (e < valid) ? src[e] : -1;
}

}  // namespace

size_t compress_padded_workspace(int64_t M, int64_t D, int64_t k) { return pad_layout(M, D, k).total; }

hipError_t run_compress_padded(const void *C, gs_dtype ct, int64_t M, int64_t D, int64_t ldc, double tol,
                               int64_t k, const double *H, int64_t ldh, void *Q, gs_dtype qt, int64_t ldq,
                               void *R, gs_dtype rt, int64_t ldr, int32_t *kept, float *cnorm, int32_t *rank,
                               int *nonfinite, void *ws_, hipStream_t s, const CompressOverlap *ov) {
    const PadLayout L = pad_layout(M, D, k);
    char *ws = static_cast<char *>(ws_);
    double *aug = (double *)(ws + L.aug), *qa = (double *)(ws + L.qa), *ra = (double *)(ws + L.ra);
    int32_t *kept_a = (int32_t *)(ws + L.kept);
    float *cn_a = (float *)(ws + L.cn);
    const int64_t Ma = M + k;
    if (ct == GS_F32) hipLaunchKernelGGL((k_augment<float>), dim3(1024), dim3(NT), 0, s, (const float *)C, ldc, M, D, k, aug);
    else if (ct == GS_F64) hipLaunchKernelGGL((k_augment<double>), dim3(1024), dim3(NT), 0, s, (const double *)C, ldc, M, D, k, aug);
    else hipLaunchKernelGGL((k_augment<bf16_t>), dim3(1024), dim3(NT), 0, s, (const bf16_t *)C, ldc, M, D, k, aug);
    GS_TRY(hipGetLastError());
    // the augmented codebook, codebook rows first: its first basis vectors and
    // the codebook's coordinates are those of the plain compression, and the
    // unit rows then complete the basis (its rank is at least k)
    int32_t ra_rank = 0;
    GS_TRY(run_compress(aug, GS_F64, Ma, D, D, tol, qa, GS_F64, D, ra, GS_F64, Ma, kept_a, cn_a, &ra_rank,
                        nonfinite, ws + L.cws, s, 0, ov));
    // rank of the codebook itself: the kept rows below M (kept is in index order)
    int32_t r = 0;
    GS_TRY(hipMemcpyAsync(&r, ws + L.cws + layout(Ma, D).rank_after + sizeof(int32_t) * (M - 1), sizeof(int32_t),
                          hipMemcpyDeviceToHost, s));
    const double *qk = qa, *rk = ra;     // first k basis vectors; the codebook rows' coordinates on them
    int64_t ldqk = D, ldrk = Ma;
    if (H) {
        double *qh = (double *)(ws + L.qh), *rh = (double *)(ws + L.rh);
        hipLaunchKernelGGL(k_dgemm, dim3((unsigned)((D + 15) / 16), (unsigned)((k + 15) / 16)), dim3(256), 0, s,
                           H, ldh, (const double *)qa, D, false, qh, D, k, D, k);
        hipLaunchKernelGGL(k_dgemm, dim3((unsigned)((k + 15) / 16), (unsigned)((M + 15) / 16)), dim3(256), 0, s,
                           (const double *)ra, Ma, H, ldh, true, rh, k, M, k, k);
        GS_TRY(hipGetLastError());
        qk = qh; rk = rh; ldrk = k;
    }
    GS_TRY(store_as(qt, qk, ldqk, Q, ldq, k, D, s));
    GS_TRY(store_as(rt, rk, ldrk, R, ldr, M, k, s));
    GS_TRY(hipStreamSynchronize(s));      // r is on the host now
    if (kept)
        hipLaunchKernelGGL(k_copy4, dim3((unsigned)((M + NT - 1) / NT)), dim3(NT), 0, s, (const int32_t *)kept_a,
                           kept, M, (int64_t)r);
    if (cnorm)
        hipLaunchKernelGGL(k_copy4, dim3((unsigned)((M + NT - 1) / NT)), dim3(NT), 0, s, (const int32_t *)cn_a,
                           (int32_t *)cnorm, M, M);
    GS_TRY(hipGetLastError());
    GS_TRY(hipStreamSynchronize(s));
    *rank = r;
    (void)ra_rank;
    return hipSuccess;
}

hipError_t run_compress_partitioned(const void *C, gs_dtype ct, int64_t M, int64_t D, int64_t ldc, double tol,
                                    int64_t subset, void *Q, gs_dtype qt, int64_t ldq, void *R, gs_dtype rt,
                                    int64_t ldr, int32_t *kept, float *cnorm, int32_t *ranks, int32_t *total,
                                    int *nonfinite, void *ws, hipStream_t s, const CompressOverlap *ov) {
    // R's capacity starts at zero: each subset writes its own block only
    hipLaunchKernelGGL(k_fill, dim3(1024), dim3(NT), 0, s, (char *)R, M, M, ldr, (int)esz(rt), 0);
    GS_TRY(hipGetLastError());
    int64_t o = 0, end = 0;
    *nonfinite = 0;
    for (int64_t m0 = 0, g = 0; m0 < M; m0 += subset, ++g) {
        const int64_t mg = (M - m0 < subset) ? M - m0 : subset;
        int32_t rg = 0;
        int nf = 0;
        GS_TRY(run_compress(static_cast<const char *>(C) + m0 * ldc * (int64_t)esz(ct), ct, mg, D, ldc, tol,
                            static_cast<char *>(Q) + o * ldq * (int64_t)esz(qt), qt, ldq,
                            static_cast<char *>(R) + (m0 * ldr + o) * (int64_t)esz(rt), rt, ldr,
                            kept ? kept + o : nullptr, cnorm ? cnorm + m0 : nullptr, &rg, &nf, ws, s, m0, ov));
        ranks[g] = rg;
        *nonfinite |= nf;
        end = o + mg;         // rows o .. o + mg - 1 of Q / entries of kept were written
        o += rg;
    }
    // capacity past the last subset's frame: zero rows of Q, kept entries -1
    if (end < M) {
        hipLaunchKernelGGL(k_fill, dim3(1024), dim3(NT), 0, s, static_cast<char *>(Q) + end * ldq * (int64_t)esz(qt),
                           M - end, D, ldq, (int)esz(qt), 0);
        if (kept)
            hipLaunchKernelGGL(k_fill, dim3(64), dim3(NT), 0, s, (char *)(kept + end), (int64_t)1, M - end, M - end,
                               4, -1);
        GS_TRY(hipGetLastError());
        GS_TRY(hipStreamSynchronize(s));
    }
    *total = (int32_t)o;
    return hipSuccess;
}

}  // namespace gs
