// Probability vectorisation of sparse probability rows on Gram-loc
// (Sec. 2.2, Sec. 3.1): t_b = sum over the stored entries (j, p) of row b of
// p R_j, rows given in compressed sparse row form.  One wave per row; lane l
// accumulates the coordinates l + 64 u of the current column chunk, reading
// each stored entry's row of R (coalesced, mostly from L2: R is M x r and is
// shared by every row of the batch).  Entries are summed in their stored
// order; stored column indices outside [0, M) and pointer ranges outside
// [0, nnz] are skipped, so malformed input cannot read out of bounds.
#include "gs_internal.h"

namespace gs {
namespace {

constexpr int SP_WAVES = 4;             // rows per work-group
constexpr int SP_U = 4;                 // accumulators per lane: chunks of 256 coordinates

template <typename TV, typename TT>
__global__ void __launch_bounds__(64 * SP_WAVES) sparse_p2v_kernel(SparseArgs a) {
    const int lane = threadIdx.x & 63;
    const int64_t b = (int64_t)blockIdx.x * SP_WAVES + (threadIdx.x >> 6);
    if (b >= a.B) return;
    const TV *vals = static_cast<const TV *>(a.vals);
    const TV *R = static_cast<const TV *>(a.R);
    TT *T = static_cast<TT *>(a.T);
    int64_t e0 = a.rowptr[b], e1 = a.rowptr[b + 1];
    e0 = e0 < 0 ? 0 : (e0 > a.nnz ? a.nnz : e0);
    e1 = e1 < e0 ? e0 : (e1 > a.nnz ? a.nnz : e1);
    for (int64_t c0 = 0; c0 < a.r; c0 += 64 * SP_U) {
        float acc[SP_U];
#pragma unroll
        for (int u = 0; u < SP_U; ++u) acc[u] = 0.f;
        // stored entries four at a time: their indices and values, then the
        // rows of R, are requested before any is used; sums stay in order
        for (int64_t e = e0; e < e1; e += 4) {
            int64_t j[4];
            float pv[4];
            bool ok[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const bool in = e + q < e1;
                j[q] = in ? (int64_t)a.cols[e + q] : -1;
                pv[q] = in ? ld_f32<TV>(vals, e + q) : 0.f;
                ok[q] = j[q] >= 0 && j[q] < a.M;
            }
            float rv[4][SP_U];
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int u = 0; u < SP_U; ++u) {
                    const int64_t c = c0 + lane + 64 * u;
                    rv[q][u] = (ok[q] && c < a.r) ? ld_f32<TV>(R, j[q] * a.ldr + c) : 0.f;
                }
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if (ok[q])
#pragma unroll
                    for (int u = 0; u < SP_U; ++u) acc[u] += pv[q] * rv[q][u];
        }
#pragma unroll
        for (int u = 0; u < SP_U; ++u) {
            const int64_t c = c0 + lane + 64 * u;
            if (c < a.r) st_f32<TT>(T, b * a.ldt + c, acc[u]);
        }
    }
}

template <typename TV, typename TT>
hipError_t launch(const SparseArgs &a, hipStream_t s) {
    const dim3 grid((unsigned)((a.B + SP_WAVES - 1) / SP_WAVES)), block(64 * SP_WAVES);
    hipLaunchKernelGGL((sparse_p2v_kernel<TV, TT>), grid, block, 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_sparse_prob2vec(gs_dtype tv, gs_dtype tt, const SparseArgs &a, hipStream_t s) {
    if (a.B == 0) return hipSuccess;
    if (tv == GS_F32 && tt == GS_F32) return launch<float, float>(a, s);
    if (tv == GS_F32 && tt == GS_BF16) return launch<float, bf16_t>(a, s);
    if (tv == GS_BF16 && tt == GS_F32) return launch<bf16_t, float>(a, s);
    if (tv == GS_BF16 && tt == GS_BF16) return launch<bf16_t, bf16_t>(a, s);
    return hipErrorInvalidValue;
}

}  // namespace gs
