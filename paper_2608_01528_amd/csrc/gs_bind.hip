// Component-wise binding of restored vectors (the operators that run in the
// original domain after a restore): element-wise product, exclusive or of
// binary vectors, and blockwise circular convolution / correlation.
//
// Circular convolution and correlation of a block of L values go through one
// complex fp32 FFT of z = x + i y (both spectra from one transform: for real
// x and y, X_k = (Z_k + conj Z_{L-k}) / 2 and Y_k = (Z_k - conj Z_{L-k}) / 2i),
// the product of the spectra (X_k Y_k, or X_k conj Y_k for the correlation),
// and one inverse FFT whose real part is the result.  A work-group holds one
// block (or several short blocks of one row) in LDS: the forward transform is
// a radix-2 decimation in time over the bit-reversed input, the inverse a
// decimation in frequency whose output comes out bit-reversed and is read
// back in that order; twiddles exp(-2 pi i m / L) are tabulated once per
// work-group.
#include "gs_internal.h"

namespace gs {
namespace {

constexpr int BT = 256;     // threads per work-group
constexpr int SEG = 4096;   // values per work-group when blocks are short

typedef float f2v __attribute__((ext_vector_type(2)));

__device__ __forceinline__ f2v cmul(f2v a, f2v b) { return f2v{a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x}; }
__device__ __forceinline__ f2v conjv(f2v a) { return f2v{a.x, -a.y}; }

// index i (lg bits) in reversed bit order
__device__ __forceinline__ int brev(int i, int lg) { return (int)(__builtin_bitreverse32((unsigned)i) >> (32 - lg)); }

template <typename TI, typename TO, bool CORR>
__global__ void __launch_bounds__(BT) circular_kernel(BindArgs a) {
    extern __shared__ f2v smem[];
    const int L = (int)a.L, lg = a.lg, nbmax = a.nb;
    const int64_t wpr = (a.nblocks + nbmax - 1) / nbmax;          // work-groups per row
    const int64_t row = (int64_t)blockIdx.x / wpr;
    const int64_t blk0 = ((int64_t)blockIdx.x - row * wpr) * nbmax;
    const int nb = (int)((a.nblocks - blk0 < nbmax) ? (a.nblocks - blk0) : nbmax);
    const int S = nb * L;
    const int t = threadIdx.x;
    f2v *z = smem;                   // nbmax * L values
    f2v *W = smem + nbmax * L;       // L / 2 twiddles
    const TI *x = static_cast<const TI *>(a.X) + row * a.ldx + blk0 * L;
    const TI *y = static_cast<const TI *>(a.Y) + row * a.ldy + blk0 * L;
    TO *out = static_cast<TO *>(a.Z) + row * a.ldz + blk0 * L;

    for (int m = t; m < L / 2; m += BT) {
        float s, c;
        sincospif(-2.0f * (float)m / (float)L, &s, &c);
        W[m] = f2v{c, s};
    }
    for (int e = t; e < S; e += BT) {
        const int j = e & (L - 1);
        z[(e - j) + brev(j, lg)] = f2v{ld_f32<TI>(x, e), ld_f32<TI>(y, e)};
    }
    __syncthreads();

    // forward transform of every block: butterflies of half-size h = 2^sh
    for (int sh = 0; sh < lg; ++sh) {
        const int h = 1 << sh;
        for (int q = t; q < S / 2; q += BT) {
            const int blk = q >> (lg - 1), qb = q & (L / 2 - 1);
            const int pos = qb & (h - 1);
            const int i0 = (blk << lg) + ((qb >> sh) << (sh + 1)) + pos, i1 = i0 + h;
            const f2v u = z[i0], v = cmul(z[i1], W[pos << (lg - 1 - sh)]);
            z[i0] = u + v;
            z[i1] = u - v;
        }
        __syncthreads();
    }

    // product of the two spectra; P_{L-k} = conj P_k (real signals)
    for (int q = t; q < nb * (L / 2 + 1); q += BT) {
        const int blk = q / (L / 2 + 1), k = q - blk * (L / 2 + 1);
        const int kk = (L - k) & (L - 1);
        f2v *zb = z + (blk << lg);
        const f2v zk = zb[k], zm = conjv(zb[kk]);
        const f2v X = (zk + zm) * 0.5f;
        const f2v iY = (zk - zm) * 0.5f;        // i Y_k
        const f2v Yk = f2v{iY.y, -iY.x};
        const f2v P = CORR ? cmul(X, conjv(Yk)) : cmul(X, Yk);
        zb[k] = P;
        if (kk != k) zb[kk] = conjv(P);
    }
    __syncthreads();

    // inverse transform (decimation in frequency, conjugate twiddles)
    for (int sh = lg - 1; sh >= 0; --sh) {
        const int h = 1 << sh;
        for (int q = t; q < S / 2; q += BT) {
            const int blk = q >> (lg - 1), qb = q & (L / 2 - 1);
            const int pos = qb & (h - 1);
            const int i0 = (blk << lg) + ((qb >> sh) << (sh + 1)) + pos, i1 = i0 + h;
            const f2v u = z[i0], v = z[i1];
            z[i0] = u + v;
            z[i1] = cmul(u - v, conjv(W[pos << (lg - 1 - sh)]));
        }
        __syncthreads();
    }

    const float inv = 1.0f / (float)L;
    for (int e = t; e < S; e += BT) {
        const int j = e & (L - 1);
        st_f32<TO>(out, e, z[(e - j) + brev(j, lg)].x * inv);
    }
}

// Element-wise product or exclusive or; one work-group per 2048 values of a row.
template <typename TI, typename TO, bool XOR>
__global__ void __launch_bounds__(BT) elementwise_kernel(BindArgs a) {
    constexpr int CH = 2048;
    const int64_t cpr = (a.D + CH - 1) / CH;
    const int64_t row = (int64_t)blockIdx.x / cpr;
    const int64_t c0 = ((int64_t)blockIdx.x - row * cpr) * CH;
    const TI *x = static_cast<const TI *>(a.X) + row * a.ldx;
    const TI *y = static_cast<const TI *>(a.Y) + row * a.ldy;
    TO *out = static_cast<TO *>(a.Z) + row * a.ldz;
    for (int64_t c = c0 + threadIdx.x; c < c0 + CH && c < a.D; c += BT) {
        const float u = ld_f32<TI>(x, c), v = ld_f32<TI>(y, c);
        st_f32<TO>(out, c, XOR ? (((u >= 0.5f) != (v >= 0.5f)) ? 1.f : 0.f) : u * v);
    }
}

template <typename TI, typename TO>
hipError_t launch_typed(int op, const BindArgs &a, hipStream_t s) {
    if (op == GS_BINDOP_MUL || op == GS_BINDOP_XOR) {
        const int64_t cpr = (a.D + 2047) / 2048;
        const dim3 grid((unsigned)(a.B * cpr));
        if (op == GS_BINDOP_XOR) hipLaunchKernelGGL((elementwise_kernel<TI, TO, true>), grid, dim3(BT), 0, s, a);
        else hipLaunchKernelGGL((elementwise_kernel<TI, TO, false>), grid, dim3(BT), 0, s, a);
        return hipGetLastError();
    }
    const int64_t wpr = (a.nblocks + a.nb - 1) / a.nb;
    const dim3 grid((unsigned)(a.B * wpr));
    const size_t lds = ((size_t)a.nb * a.L + a.L / 2) * sizeof(f2v);
    const void *k = (op == GS_BINDOP_CORR) ? reinterpret_cast<const void *>(circular_kernel<TI, TO, true>)
                                           : reinterpret_cast<const void *>(circular_kernel<TI, TO, false>);
    hipError_t e = raise_lds_limit(k, lds);
    if (e != hipSuccess) return e;
    if (op == GS_BINDOP_CORR) hipLaunchKernelGGL((circular_kernel<TI, TO, true>), grid, dim3(BT), lds, s, a);
    else hipLaunchKernelGGL((circular_kernel<TI, TO, false>), grid, dim3(BT), lds, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_bind(gs_dtype tin, gs_dtype tout, int op, const BindArgs &a_in, hipStream_t s) {
    if (a_in.B == 0) return hipSuccess;
    BindArgs a = a_in;
    if (op == GS_BINDOP_CONV || op == GS_BINDOP_CORR) {
        a.lg = 0;
        while ((int64_t)1 << a.lg < a.L) ++a.lg;
        a.nblocks = a.D / a.L;
        const int64_t per = (a.L >= SEG) ? 1 : SEG / a.L;
        a.nb = (int)(per < a.nblocks ? per : a.nblocks);
    }
    if (tin == GS_F32 && tout == GS_F32) return launch_typed<float, float>(op, a, s);
    if (tin == GS_F32 && tout == GS_BF16) return launch_typed<float, bf16_t>(op, a, s);
    if (tin == GS_BF16 && tout == GS_F32) return launch_typed<bf16_t, float>(op, a, s);
    if (tin == GS_BF16 && tout == GS_BF16) return launch_typed<bf16_t, bf16_t>(op, a, s);
    return hipErrorInvalidValue;
}

}  // namespace gs
