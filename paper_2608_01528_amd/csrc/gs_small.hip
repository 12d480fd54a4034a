// Streaming kernels for small codebooks (M <= 32, r <= 32): probability
// vectorisation, similarity (+ argmax) and attention score on Gram-loc.
//
// At these sizes every output row costs at most M*r multiply-adds against
// 4(M + r) bytes of traffic, so the kernels are bound by memory traffic and
// latency, not arithmetic.  Each work-group stages the codebook coordinates R
// (and their norms) in LDS once, streams a tile of ROWS batch rows through
// LDS with coalesced loads, computes one row per thread from LDS, and writes
// the output tile back through LDS with coalesced stores.
#include "gs_internal.h"

namespace gs {
namespace {

constexpr int ROWS = 128;   // batch rows per work-group = threads per work-group
constexpr int MAXK = SMALL_MAX;

enum Mode { MODE_P2V = 0, MODE_SIM = 1, MODE_ATT = 2 };

// Odd row stride of a staged tile of `w` columns: conflict-free when each
// thread walks its own row.
__device__ __forceinline__ int odd_stride(int64_t w) { return (int)(w | 1); }

template <typename TI, typename TO, int MODE>
__global__ void __launch_bounds__(ROWS) small_kernel(SmallArgs a) {
    __shared__ float Rs[MAXK * MAXK];               // R, M x r
    __shared__ float Rn[MAXK];                      // 1/||c_j|| (cosine) or 1
    __shared__ float tile_in[ROWS * (MAXK + 1)];
    __shared__ float tile_out[ROWS * (MAXK + 1)];
    // attention-weighted sum of a row: written over the thread's own input row
    // once that row is in registers (input and output rows share the stride)
    float *tile_o = tile_in;

    const int t = threadIdx.x;
    const int64_t b0 = (int64_t)blockIdx.x * ROWS;
    const int M = (int)a.M, r = (int)a.r;
    const TI *R = static_cast<const TI *>(a.R);
    const TI *In = static_cast<const TI *>(a.In);

    for (int e = t; e < M * r; e += ROWS) Rs[e] = ld_f32<TI>(R, (int64_t)(e / r) * a.ldr + e % r);
    // input tile: P rows (width M) or T rows (width r)
    const int win = (MODE == MODE_P2V) ? M : r;
    const int sin = odd_stride(win);
    const int64_t nrow = (a.B - b0 < ROWS) ? (a.B - b0) : ROWS;
    for (int e = t; e < nrow * win; e += ROWS) {
        const int row = e / win, col = e % win;
        tile_in[row * sin + col] = ld_f32<TI>(In, (b0 + row) * a.ldin + col);
    }
    __syncthreads();
    if (MODE != MODE_P2V && t < M) {
        float c = 1.f;
        if (a.cosine) {
            float n;
            if (a.cnorm) n = a.cnorm[t];
            else {
                float s = 0.f;
                for (int k = 0; k < r; ++k) s += Rs[t * r + k] * Rs[t * r + k];
                n = sqrtf(s);
            }
            c = (n > 0.f) ? 1.f / n : 0.f;
        }
        Rn[t] = c;
    }
    __syncthreads();

    const int64_t row = b0 + t;
    const float *x = tile_in + t * sin;
    if (MODE == MODE_P2V) {
        const int sout = odd_stride(r);
        if (t < nrow) {
            float acc[MAXK];
#pragma unroll
            for (int k = 0; k < MAXK; ++k) acc[k] = 0.f;
            for (int j = 0; j < M; ++j) {
                const float p = x[j];
#pragma unroll
                for (int k = 0; k < MAXK; ++k)
                    if (k < r) acc[k] += p * Rs[j * r + k];
            }
#pragma unroll
            for (int k = 0; k < MAXK; ++k)
                if (k < r) tile_out[t * sout + k] = acc[k];
        }
        __syncthreads();
        TO *T = static_cast<TO *>(a.Out);
        for (int e = t; e < nrow * r; e += ROWS) {
            const int rr = e / r, k = e % r;
            st_f32<TO>(T, (b0 + rr) * a.ldout + k, tile_out[rr * sout + k]);
        }
        return;
    }

    // similarity / attention: scores of this thread's row against all M codes
    const int ss = odd_stride(M);
    if (t < nrow) {
        float xr[MAXK];
        float n2 = 0.f;
#pragma unroll
        for (int k = 0; k < MAXK; ++k) {
            xr[k] = (k < r) ? x[k] : 0.f;
            n2 += xr[k] * xr[k];
        }
        float q = 1.f;
        if (a.cosine) {
            if (a.qnorm2) n2 = a.qnorm2[row];
            q = (n2 > 0.f) ? 1.f / sqrtf(n2) : 0.f;
        }
        const float mul = (MODE == MODE_ATT) ? a.scale * a.beta : a.scale;
        float best = -INFINITY;
        int bi = 0;
        for (int j = 0; j < M; ++j) {
            float d = 0.f;
#pragma unroll
            for (int k = 0; k < MAXK; ++k)
                if (k < r) d += xr[k] * Rs[j * r + k];
            const float s = mul * d * q * Rn[j];
            tile_out[t * ss + j] = s;
            if (s > best) { best = s; bi = j; }
        }
        if (MODE == MODE_SIM) {
            if (a.argmax) a.argmax[row] = bi;
        } else {
            float z = 0.f;
            for (int j = 0; j < M; ++j) {
                const float e = __expf(tile_out[t * ss + j] - best);
                tile_out[t * ss + j] = e;
                z += e;
            }
            const float iz = 1.f / z;
            for (int j = 0; j < M; ++j) tile_out[t * ss + j] *= iz;
            if (a.O) {
                const int so = odd_stride(r);
                float o[MAXK];
#pragma unroll
                for (int k = 0; k < MAXK; ++k) o[k] = 0.f;
                for (int j = 0; j < M; ++j) {
                    const float p = tile_out[t * ss + j];
#pragma unroll
                    for (int k = 0; k < MAXK; ++k)
                        if (k < r) o[k] += p * Rs[j * r + k];
                }
#pragma unroll
                for (int k = 0; k < MAXK; ++k)
                    if (k < r) tile_o[t * so + k] = o[k];
            }
        }
    }
    __syncthreads();
    float *S = static_cast<float *>(a.Out);
    if (S) {
        for (int e = t; e < nrow * M; e += ROWS) {
            const int rr = e / M, j = e % M;
            S[(b0 + rr) * a.ldout + j] = tile_out[rr * ss + j];
        }
    }
    if (MODE == MODE_ATT && a.O) {
        const int so = odd_stride(r);
        TO *O = static_cast<TO *>(a.O);
        for (int e = t; e < nrow * r; e += ROWS) {
            const int rr = e / r, k = e % r;
            st_f32<TO>(O, (b0 + rr) * a.ldo + k, tile_o[rr * so + k]);
        }
    }
}

template <typename TI, typename TO, int MODE>
hipError_t launch(const SmallArgs &a, hipStream_t s) {
    if (a.B == 0) return hipSuccess;
    const int64_t grid = (a.B + ROWS - 1) / ROWS;
    hipLaunchKernelGGL((small_kernel<TI, TO, MODE>), dim3(grid), dim3(ROWS), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_small_prob2vec(gs_dtype tin, gs_dtype tout, const SmallArgs &a, hipStream_t s) {
    if (tin == GS_F32 && tout == GS_F32) return launch<float, float, MODE_P2V>(a, s);
    if (tin == GS_F32 && tout == GS_BF16) return launch<float, bf16_t, MODE_P2V>(a, s);
    if (tin == GS_BF16 && tout == GS_F32) return launch<bf16_t, float, MODE_P2V>(a, s);
    if (tin == GS_BF16 && tout == GS_BF16) return launch<bf16_t, bf16_t, MODE_P2V>(a, s);
    return hipErrorInvalidValue;
}

hipError_t launch_small_similarity(gs_dtype tin, const SmallArgs &a, hipStream_t s) {
    if (tin == GS_F32) return launch<float, float, MODE_SIM>(a, s);
    if (tin == GS_BF16) return launch<bf16_t, float, MODE_SIM>(a, s);
    return hipErrorInvalidValue;
}

hipError_t launch_small_attention(gs_dtype tin, gs_dtype to, const SmallArgs &a, hipStream_t s) {
    if (tin == GS_F32 && to == GS_F32) return launch<float, float, MODE_ATT>(a, s);
    if (tin == GS_F32 && to == GS_BF16) return launch<float, bf16_t, MODE_ATT>(a, s);
    if (tin == GS_BF16 && to == GS_F32) return launch<bf16_t, float, MODE_ATT>(a, s);
    if (tin == GS_BF16 && to == GS_BF16) return launch<bf16_t, bf16_t, MODE_ATT>(a, s);
    return hipErrorInvalidValue;
}

}  // namespace gs
