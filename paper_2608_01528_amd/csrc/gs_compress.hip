// Gram-Space compression on the GPU: blocked modified Gram-Schmidt with one
// re-orthogonalisation pass and a relative rank threshold, in fp64.
//
// The paper builds the basis U and the Gram-loc codebook T = U^T W by
// Gram-Schmidt at initialisation (Sec. 3.3), with k the algebraic rank of the
// codebook (Sec. 3.2).  Here codebook rows are processed in panels of PB rows.
// Each panel is first orthogonalised against every basis vector built from
// earlier panels (two block passes: coefficients H = W_p Q^T, then
// W_p -= H Q), then row by row against the basis vectors created inside the
// panel (two passes each).  A row whose remaining norm is <= tol * ||c_i||
// after both passes is dependent; otherwise it is normalised into the next
// basis vector.  The coefficients of both passes are summed into R, which
// gives R[i, k] = <c_i, q_k> and a positive pivot for kept rows.
//
// The running rank lives on the device (rank_after[i] = rank once row i is
// done), so no launch waits on the host; grids are sized for the largest rank
// possible at that point and surplus work-groups exit.  Every reduction has a
// fixed order (no atomics), so results are bitwise reproducible.
#include "gs_internal.h"

namespace gs {
namespace {

constexpr int PB = 32;        // panel rows
constexpr int DCH = 512;      // D-chunk of a panel coefficient work-group
constexpr int ICH = 1024;     // D-chunk of the in-panel kernels (256 thr x 4)
constexpr int NT = 256;

struct WsLayout {
    size_t qm, wp, hc, hb, part, part2, part3, cn, rank_after, kept, flag, total;
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

WsLayout layout(int64_t M, int64_t D) {
    WsLayout L;
    const int64_t nch = (D + DCH - 1) / DCH, nch2 = (D + ICH - 1) / ICH;
    size_t o = 0;
    L.qm = o;    o = align256(o + sizeof(double) * M * D);
    L.wp = o;    o = align256(o + sizeof(double) * PB * D);
    L.hc = o;    o = align256(o + sizeof(double) * M * M);
    L.hb = o;    o = align256(o + sizeof(double) * PB * M);
    L.part = o;  o = align256(o + sizeof(double) * nch * PB * M);
    L.part2 = o; o = align256(o + sizeof(double) * nch2 * PB);
    L.part3 = o; o = align256(o + sizeof(double) * nch2);
    L.cn = o;    o = align256(o + sizeof(double) * M);
    L.rank_after = o; o = align256(o + sizeof(int32_t) * M);
    L.kept = o;  o = align256(o + sizeof(int32_t) * M);
    L.flag = o;  o = align256(o + sizeof(int32_t));
    L.total = o;
    return L;
}

__device__ __forceinline__ int rank_before(const int32_t *rank_after, int64_t row) {
    return row == 0 ? 0 : rank_after[row - 1];
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

__global__ void k_init(double *hc, int64_t nhc, int32_t *kept, int32_t *rank_after, int64_t M,
                       int32_t *flag) {
    const int64_t i = (int64_t)blockIdx.x * NT + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * NT;
    for (int64_t e = i; e < nhc; e += stride) hc[e] = 0.0;
    for (int64_t e = i; e < M; e += stride) { kept[e] = -1; rank_after[e] = 0; }
    if (i == 0) *flag = 0;
}

// Copy panel rows to fp64 and record their norms.  One work-group per row.
template <typename T>
__global__ void __launch_bounds__(NT) k_load_panel(const T *C, int64_t ldc, int64_t D, int64_t i0,
                                                   double *wp, double *cn, int32_t *flag) {
    __shared__ double red[NT / 64];
    const int64_t i = blockIdx.x;
    double s = 0.0;
    bool bad = false;
    for (int64_t d = threadIdx.x; d < D; d += NT) {
        const double v = ld_f64<T>(C, (i0 + i) * ldc + d);
        bad |= !isfinite(v);
        wp[i * D + d] = v;
        s += v * v;
    }
    if (bad) *flag = 1;
    s = block_sum(s, red);
    if (threadIdx.x == 0) cn[i0 + i] = sqrt(s);
}

// part[c][i][k] = sum over D-chunk c of W_p[i, d] * Q[k, d], for the basis
// vectors k < rank at panel start.  Work-group (kb, c): 32 basis vectors x 32
// panel rows; thread t owns row t / 8 and basis vectors 4 (t % 8) + 0..3.
__global__ void __launch_bounds__(NT) k_panel_dots(const double *wp, const double *qm, int64_t D,
                                                   int pb, int64_t i0, const int32_t *rank_after,
                                                   double *part, int64_t M) {
    constexpr int DT = 32;
    __shared__ double ws[PB][DT + 1];
    __shared__ double qs[32][DT + 1];
    const int r = rank_before(rank_after, i0);
    const int kb = blockIdx.x * 32;
    if (kb >= r) return;
    const int64_t c = blockIdx.y;
    const int64_t d_lo = c * DCH, d_hi = (d_lo + DCH < D) ? d_lo + DCH : D;
    const int t = threadIdx.x;
    const int i = t >> 3, kq = 4 * (t & 7);
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    for (int64_t d0 = d_lo; d0 < d_hi; d0 += DT) {
        for (int e = t; e < 32 * DT; e += NT) {
            const int rr = e / DT, dd = e % DT;
            const int64_t d = d0 + dd;
            ws[rr][dd] = (rr < pb && d < d_hi) ? wp[rr * D + d] : 0.0;
            qs[rr][dd] = (kb + rr < r && d < d_hi) ? qm[(int64_t)(kb + rr) * D + d] : 0.0;
        }
        __syncthreads();
#pragma unroll 8
        for (int dd = 0; dd < DT; ++dd) {
            const double w = ws[i][dd];
#pragma unroll
            for (int q = 0; q < 4; ++q) acc[q] += w * qs[kq + q][dd];
        }
        __syncthreads();
    }
    if (i < pb)
#pragma unroll
        for (int q = 0; q < 4; ++q)
            if (kb + kq + q < r) part[(c * PB + i) * M + kb + kq + q] = acc[q];
}

// h[i][k] = sum_c part[c][i][k] (chunk order); R[i0 + i, k] += h.
__global__ void k_panel_reduce(const double *part, int64_t nch, int pb, int64_t i0,
                               const int32_t *rank_after, double *hc, double *hb, int64_t M) {
    const int r = rank_before(rank_after, i0);
    const int64_t e = (int64_t)blockIdx.x * NT + threadIdx.x;
    const int i = (int)(e / M), k = (int)(e % M);
    if (i >= pb || k >= r) return;
    double s = 0.0;
    for (int64_t c = 0; c < nch; ++c) s += part[(c * PB + i) * M + k];
    hb[(int64_t)i * M + k] = s;
    hc[(i0 + i) * M + k] += s;
}

// W_p[i, d] -= sum_k h[i][k] Q[k, d] over k < rank at panel start.
// Work-group: 64 columns x 32 rows; thread t owns row t / 8, columns
// 8 (t % 8) + 0..7.
__global__ void __launch_bounds__(NT) k_panel_update(double *wp, const double *qm, const double *hb,
                                                     int64_t D, int pb, int64_t i0,
                                                     const int32_t *rank_after, int64_t M) {
    constexpr int KT = 32, DC = 64;
    __shared__ double hs[PB][KT + 1];
    __shared__ double qs[KT][DC + 1];
    const int r = rank_before(rank_after, i0);
    const int64_t d0 = (int64_t)blockIdx.x * DC;
    const int t = threadIdx.x;
    const int i = t >> 3, cb = 8 * (t & 7);
    double acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int k0 = 0; k0 < r; k0 += KT) {
        for (int e = t; e < PB * KT; e += NT) {
            const int rr = e / KT, kk = e % KT;
            hs[rr][kk] = (rr < pb && k0 + kk < r) ? hb[(int64_t)rr * M + k0 + kk] : 0.0;
        }
        for (int e = t; e < KT * DC; e += NT) {
            const int kk = e / DC, dd = e % DC;
            qs[kk][dd] = (k0 + kk < r && d0 + dd < D) ? qm[(int64_t)(k0 + kk) * D + d0 + dd] : 0.0;
        }
        __syncthreads();
#pragma unroll 4
        for (int kk = 0; kk < KT; ++kk) {
            const double h = hs[i][kk];
#pragma unroll
            for (int j = 0; j < 8; ++j) acc[j] += h * qs[kk][cb + j];
        }
        __syncthreads();
    }
    if (i < pb)
#pragma unroll
        for (int j = 0; j < 8; ++j)
            if (d0 + cb + j < D) wp[i * D + d0 + cb + j] -= acc[j];
}

// In-panel pass for row i: partial dots of W_p[i] with the basis vectors made
// earlier in this panel (at most PB - 1 of them), per D-chunk of ICH.
__global__ void __launch_bounds__(NT) k_intra_dots(const double *wp, const double *qm, int64_t D,
                                                   int64_t i0, int i, const int32_t *rank_after,
                                                   double *part2) {
    __shared__ double red[NT / 64][PB];
    const int rb = rank_before(rank_after, i0);
    const int nb = rank_before(rank_after, i0 + i) - rb;
    if (nb == 0) return;
    const int64_t c = blockIdx.x;
    const int t = threadIdx.x;
    double s[PB];
#pragma unroll
    for (int j = 0; j < PB; ++j) s[j] = 0.0;
    for (int q = 0; q < ICH / NT; ++q) {
        const int64_t d = c * ICH + q * NT + t;
        if (d < D) {
            const double w = wp[(int64_t)i * D + d];
#pragma unroll
            for (int j = 0; j < PB; ++j)
                if (j < nb) s[j] += w * qm[(int64_t)(rb + j) * D + d];
        }
    }
#pragma unroll
    for (int j = 0; j < PB; ++j) {
        double v = s[j];
        for (int off = 32; off > 0; off >>= 1) v += __shfl_down(v, off);
        if ((t & 63) == 0) red[t >> 6][j] = v;
    }
    __syncthreads();
    if (t < nb) {
        double v = 0.0;
        for (int w = 0; w < NT / 64; ++w) v += red[w][t];
        part2[c * PB + t] = v;
    }
}

// Finish the pass for row i: reduce the chunk partials to coefficients g_j,
// W_p[i] -= sum_j g_j q_{rb+j}, accumulate g into R, and emit per-chunk
// partial sums of the updated row's squares.
__global__ void __launch_bounds__(NT) k_intra_update(double *wp, const double *qm, double *hc,
                                                     int64_t D, int64_t i0, int i,
                                                     const int32_t *rank_after, const double *part2,
                                                     int64_t nch2, double *part3, int64_t M) {
    __shared__ double g[PB];
    __shared__ double red[NT / 64];
    const int rb = rank_before(rank_after, i0);
    const int nb = rank_before(rank_after, i0 + i) - rb;
    const int t = threadIdx.x;
    if (t < nb) {
        double v = 0.0;
        for (int64_t c = 0; c < nch2; ++c) v += part2[c * PB + t];
        g[t] = v;
        if (blockIdx.x == 0) hc[(i0 + i) * M + rb + t] += v;
    }
    __syncthreads();
    const int64_t c = blockIdx.x;
    double s = 0.0;
    for (int q = 0; q < ICH / NT; ++q) {
        const int64_t d = c * ICH + q * NT + t;
        if (d < D) {
            double w = wp[(int64_t)i * D + d];
            for (int j = 0; j < nb; ++j) w -= g[j] * qm[(int64_t)(rb + j) * D + d];
            wp[(int64_t)i * D + d] = w;
            s += w * w;
        }
    }
    s = block_sum(s, red);
    if (t == 0) part3[c] = s;
}

// Rank decision for row i after both passes; normalise it into the next basis
// vector if it is independent.
__global__ void __launch_bounds__(NT) k_intra_finalize(const double *wp, double *qm, double *hc,
                                                       int64_t D, int64_t i0, int i,
                                                       int32_t *rank_after, const double *part3,
                                                       int64_t nch2, const double *cn, double tol,
                                                       int32_t *kept, int64_t M) {
    const int r = rank_before(rank_after, i0 + i);
    double s = 0.0;
    for (int64_t c = 0; c < nch2; ++c) s += part3[c];
    const double rho = sqrt(s);
    const bool keep = rho > tol * cn[i0 + i];
    const int64_t c = blockIdx.x;
    if (keep) {
        for (int q = 0; q < ICH / NT; ++q) {
            const int64_t d = c * ICH + q * NT + threadIdx.x;
            if (d < D) qm[(int64_t)r * D + d] = wp[(int64_t)i * D + d] / rho;
        }
    }
    if (c == 0 && threadIdx.x == 0) {
        rank_after[i0 + i] = r + (keep ? 1 : 0);
        if (keep) {
            hc[(i0 + i) * M + r] = rho;
            kept[r] = (int32_t)(i0 + i);
        }
    }
}

template <typename TQ, typename TR>
__global__ void k_outputs(const double *qm, const double *hc, const double *cnd,
                          const int32_t *rank_after, const int32_t *kept_ws, int64_t M, int64_t D,
                          TQ *Q, int64_t ldq, TR *R, int64_t ldr, int32_t *kept, float *cnorm) {
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
        if (kept) kept[e] = (e < r) ? kept_ws[e] : -1;
        if (cnorm) cnorm[e] = (float)cnd[e];
    }
}

template <typename TQ, typename TR>
hipError_t launch_outputs(const WsLayout &L, char *ws, int64_t M, int64_t D, void *Q, int64_t ldq,
                          void *R, int64_t ldr, int32_t *kept, float *cnorm, hipStream_t s) {
    hipLaunchKernelGGL((k_outputs<TQ, TR>), dim3(1024), dim3(NT), 0, s,
                       (const double *)(ws + L.qm), (const double *)(ws + L.hc),
                       (const double *)(ws + L.cn), (const int32_t *)(ws + L.rank_after),
                       (const int32_t *)(ws + L.kept), M, D, (TQ *)Q, ldq, (TR *)R, ldr, kept, cnorm);
    return hipGetLastError();
}

template <typename TQ>
hipError_t outputs_r(gs_dtype rt, const WsLayout &L, char *ws, int64_t M, int64_t D, void *Q,
                     int64_t ldq, void *R, int64_t ldr, int32_t *kept, float *cnorm, hipStream_t s) {
    if (rt == GS_F64) return launch_outputs<TQ, double>(L, ws, M, D, Q, ldq, R, ldr, kept, cnorm, s);
    if (rt == GS_F32) return launch_outputs<TQ, float>(L, ws, M, D, Q, ldq, R, ldr, kept, cnorm, s);
    return launch_outputs<TQ, bf16_t>(L, ws, M, D, Q, ldq, R, ldr, kept, cnorm, s);
}

template <typename T>
hipError_t launch_load(const void *C, int64_t ldc, int64_t D, int64_t i0, int pb, double *wp,
                       double *cn, int32_t *flag, hipStream_t s) {
    hipLaunchKernelGGL((k_load_panel<T>), dim3(pb), dim3(NT), 0, s, (const T *)C, ldc, D, i0, wp, cn, flag);
    return hipGetLastError();
}

}  // namespace

size_t compress_workspace(int64_t M, int64_t D) { return layout(M, D).total; }

#define GS_TRY(x) do { hipError_t e_ = (x); if (e_ != hipSuccess) return e_; } while (0)

hipError_t run_compress(const void *C, gs_dtype ct, int64_t M, int64_t D, int64_t ldc, double tol,
                        void *Q, gs_dtype qt, int64_t ldq, void *R, gs_dtype rt, int64_t ldr,
                        int32_t *kept, float *cnorm, int32_t *rank, int *nonfinite, void *ws_,
                        hipStream_t s) {
    const WsLayout L = layout(M, D);
    char *ws = static_cast<char *>(ws_);
    double *qm = (double *)(ws + L.qm), *wp = (double *)(ws + L.wp), *hc = (double *)(ws + L.hc);
    double *hb = (double *)(ws + L.hb), *part = (double *)(ws + L.part);
    double *part2 = (double *)(ws + L.part2), *part3 = (double *)(ws + L.part3);
    double *cn = (double *)(ws + L.cn);
    int32_t *rank_after = (int32_t *)(ws + L.rank_after), *kept_ws = (int32_t *)(ws + L.kept);
    int32_t *flag = (int32_t *)(ws + L.flag);
    const int64_t nch = (D + DCH - 1) / DCH, nch2 = (D + ICH - 1) / ICH;

    hipLaunchKernelGGL(k_init, dim3(1024), dim3(NT), 0, s, hc, M * M, kept_ws, rank_after, M, flag);
    GS_TRY(hipGetLastError());

    for (int64_t i0 = 0; i0 < M; i0 += PB) {
        const int pb = (int)((M - i0 < PB) ? (M - i0) : PB);
        if (ct == GS_F32) GS_TRY(launch_load<float>(C, ldc, D, i0, pb, wp, cn, flag, s));
        else if (ct == GS_F64) GS_TRY(launch_load<double>(C, ldc, D, i0, pb, wp, cn, flag, s));
        else GS_TRY(launch_load<bf16_t>(C, ldc, D, i0, pb, wp, cn, flag, s));
        if (i0 > 0) {
            const dim3 gd((unsigned)((i0 + 31) / 32), (unsigned)nch);
            const unsigned gr = (unsigned)((pb * M + NT - 1) / NT);
            const unsigned gu = (unsigned)((D + 63) / 64);
            for (int pass = 0; pass < 2; ++pass) {
                hipLaunchKernelGGL(k_panel_dots, gd, dim3(NT), 0, s, wp, qm, D, pb, i0, rank_after, part, M);
                hipLaunchKernelGGL(k_panel_reduce, dim3(gr), dim3(NT), 0, s, part, nch, pb, i0, rank_after, hc, hb, M);
                hipLaunchKernelGGL(k_panel_update, dim3(gu), dim3(NT), 0, s, wp, qm, hb, D, pb, i0, rank_after, M);
                GS_TRY(hipGetLastError());
            }
        }
        for (int i = 0; i < pb; ++i) {
            for (int pass = 0; pass < 2; ++pass) {
                if (i > 0)
                    hipLaunchKernelGGL(k_intra_dots, dim3((unsigned)nch2), dim3(NT), 0, s, wp, qm, D, i0, i, rank_after, part2);
                hipLaunchKernelGGL(k_intra_update, dim3((unsigned)nch2), dim3(NT), 0, s, wp, qm, hc, D, i0, i, rank_after, part2, nch2, part3, M);
            }
            hipLaunchKernelGGL(k_intra_finalize, dim3((unsigned)nch2), dim3(NT), 0, s, wp, qm, hc, D, i0, i, rank_after, part3, nch2, cn, tol, kept_ws, M);
            GS_TRY(hipGetLastError());
        }
    }

    if (qt == GS_F64) GS_TRY(outputs_r<double>(rt, L, ws, M, D, Q, ldq, R, ldr, kept, cnorm, s));
    else if (qt == GS_F32) GS_TRY(outputs_r<float>(rt, L, ws, M, D, Q, ldq, R, ldr, kept, cnorm, s));
    else GS_TRY(outputs_r<bf16_t>(rt, L, ws, M, D, Q, ldq, R, ldr, kept, cnorm, s));

    int32_t host[2] = {0, 0};
    GS_TRY(hipMemcpyAsync(&host[0], rank_after + (M - 1), sizeof(int32_t), hipMemcpyDeviceToHost, s));
    GS_TRY(hipMemcpyAsync(&host[1], flag, sizeof(int32_t), hipMemcpyDeviceToHost, s));
    GS_TRY(hipStreamSynchronize(s));
    *rank = host[0];
    *nonfinite = host[1];
    return hipSuccess;
}

}  // namespace gs
