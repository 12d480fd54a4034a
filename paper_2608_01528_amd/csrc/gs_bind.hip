// Component-wise binding of restored vectors (the operators that run in the
// original domain after a restore): element-wise product, exclusive or of
// binary vectors, and blockwise circular convolution / correlation.
//
// Circular convolution and correlation of a block of L values go through one
// complex fp32 FFT of z = x + i y (both spectra from one transform: for real
// x and y, X_k = (Z_k + conj Z_{L-k}) / 2 and Y_k = (Z_k - conj Z_{L-k}) / 2i),
// the product of the spectra (X_k Y_k, or X_k conj Y_k for the correlation),
// and an inverse transform taken as the forward transform of the conjugate
// (ifft(P) = conj(fft(conj P)) / L; the result is real, so its real part
// divided by L).  A work-group holds one block (or several short blocks of one
// row, up to 4096 values) in LDS.  The transform is a Stockham autosort FFT
// (natural order in and out, no bit reversal) in passes of radix 16 (and one
// of radix 8, 4 or 2 when log2 L is not a multiple of 4): in each pass every
// thread gathers the R values of its butterflies from LDS into registers,
// applies the pass twiddles exp(-2 pi i (j mod Ns) r / (Ns R)), takes the
// R-point DFT in registers and scatters the results back, with a barrier
// between the gather and the scatter (so one buffer serves as input and
// output) and after the scatter.  The first pass gathers straight from the
// inputs and the last pass of the inverse scatters straight to the output.
#include "gs_internal.h"

namespace gs {
namespace {

constexpr int BT = 256;     // threads per work-group
constexpr int SEG = 4096;   // values per work-group when blocks are short

typedef float f2v __attribute__((ext_vector_type(2)));

__device__ __forceinline__ f2v cmul(f2v a, f2v b) { return f2v{a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x}; }
__device__ __forceinline__ f2v conjv(f2v a) { return f2v{a.x, -a.y}; }
__device__ __forceinline__ f2v mul_mi(f2v a) { return f2v{a.y, -a.x}; }     // -i a

// LDS slot of value i: one pad slot per 16 values, so the stride-16 scatter
// of a radix-16 pass spreads over the banks
__device__ __forceinline__ int pad(int i) { return i + (i >> 4); }

// exp(-2 pi i m / 16), m = 0 .. 15
__constant__ const float W16C[16] = {1.f, 0.92387953251128674f, 0.70710678118654752f, 0.38268343236508978f,
                                     0.f, -0.38268343236508978f, -0.70710678118654752f, -0.92387953251128674f,
                                     -1.f, -0.92387953251128674f, -0.70710678118654752f, -0.38268343236508978f,
                                     0.f, 0.38268343236508978f, 0.70710678118654752f, 0.92387953251128674f};
__device__ __forceinline__ f2v w16(int m) { return f2v{W16C[m & 15], -W16C[(m + 12) & 15]}; }

// R-point forward DFT in registers, natural order in and out:
// v[k] <- sum_n v[n] exp(-2 pi i n k / R)
template <int R> __device__ __forceinline__ void dft(f2v *v);
template <> __device__ __forceinline__ void dft<2>(f2v *v) {
    const f2v a = v[0], b = v[1];
    v[0] = a + b;
    v[1] = a - b;
}
template <> __device__ __forceinline__ void dft<4>(f2v *v) {
    const f2v t0 = v[0] + v[2], t1 = v[0] - v[2], t2 = v[1] + v[3], t3 = mul_mi(v[1] - v[3]);
    v[0] = t0 + t2;
    v[2] = t0 - t2;
    v[1] = t1 + t3;
    v[3] = t1 - t3;
}
// 8 = 4 x 2: the DFTs of the even and the odd values, combined with exp(-2 pi i k / 8)
template <> __device__ __forceinline__ void dft<8>(f2v *v) {
    f2v e[4] = {v[0], v[2], v[4], v[6]}, o[4] = {v[1], v[3], v[5], v[7]};
    dft<4>(e);
    dft<4>(o);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const f2v t = (k == 0) ? o[k] : cmul(o[k], w16(2 * k));
        v[k] = e[k] + t;
        v[k + 4] = e[k] - t;
    }
}
// 16 = 4 x 4 (n = 4 n1 + n2, k = k1 + 4 k2): 4-point DFTs over n1, twiddles
// exp(-2 pi i n2 k1 / 16), 4-point DFTs over n2
template <> __device__ __forceinline__ void dft<16>(f2v *v) {
    f2v y[4][4];
#pragma unroll
    for (int n2 = 0; n2 < 4; ++n2) {
#pragma unroll
        for (int n1 = 0; n1 < 4; ++n1) y[n2][n1] = v[4 * n1 + n2];
        dft<4>(y[n2]);
    }
#pragma unroll
    for (int n2 = 1; n2 < 4; ++n2)
#pragma unroll
        for (int k1 = 1; k1 < 4; ++k1) y[n2][k1] = cmul(y[n2][k1], w16(n2 * k1));
#pragma unroll
    for (int k1 = 0; k1 < 4; ++k1) {
        f2v c[4] = {y[0][k1], y[1][k1], y[2][k1], y[3][k1]};
        dft<4>(c);
#pragma unroll
        for (int k2 = 0; k2 < 4; ++k2) v[k1 + 4 * k2] = c[k2];
    }
}

// Where a transform starts and ends: the first pass of the forward transform
// gathers x + i y straight from the inputs, the last pass of the inverse
// scatters Re / L straight to the output (both in natural order, coalesced).
template <typename TI, typename TO> struct BlockIo {
    const TI *x, *y;
    TO *out;
    float inv;
    __device__ __forceinline__ f2v load(int e) const { return f2v{ld_f32<TI>(x, e), ld_f32<TI>(y, e)}; }
    __device__ __forceinline__ void store(int e, f2v v) const { st_f32<TO>(out, e, v.x * inv); }
};

// One Stockham pass of radix R over the S values in LDS (blocks of L = 2^lg
// values), the sub-transforms done so far having length Ns: butterfly q of
// block blk (j = q mod L/R) takes values j + r L/R and writes its outputs to
// (j / Ns) Ns R + (j mod Ns) + r Ns.  Each thread holds VPT values.  GIN:
// gather from io.load instead of LDS; GOUT: scatter to io.store instead.
template <int R, int VPT, bool GIN, bool GOUT, class Io>
__device__ __forceinline__ void stockham_pass(f2v *z, int S, int lg, int Ns, int t, const Io &io) {
    constexpr int G = VPT / R;
    constexpr int LOGR = R == 16 ? 4 : R == 8 ? 3 : R == 4 ? 2 : 1;
    const int lr = lg - LOGR, LR = 1 << lr, nq = S >> LOGR;
    f2v v[G][R];
#pragma unroll
    for (int g = 0; g < G; ++g) {
        const int q = t + g * BT;
        if (q < nq) {
            const int blk = q >> lr, j = q & (LR - 1);
            const int base = (blk << lg) + j;
#pragma unroll
            for (int r = 0; r < R; ++r) v[g][r] = GIN ? io.load(base + r * LR) : z[pad(base + r * LR)];
        }
    }
    if (!GIN && !GOUT) __syncthreads();   // every gather is done before LDS is overwritten
#pragma unroll
    for (int g = 0; g < G; ++g) {
        const int q = t + g * BT;
        if (q < nq) {
            const int blk = q >> lr, j = q & (LR - 1);
            const int jm = j & (Ns - 1);
            if (Ns > 1) {
                float sn, cs;
                sincospif(-2.0f * (float)jm / (float)(Ns * R), &sn, &cs);
                const f2v w = f2v{cs, sn};
                f2v wr = w;
#pragma unroll
                for (int r = 1; r < R; ++r) {
                    v[g][r] = cmul(v[g][r], wr);
                    wr = cmul(wr, w);
                }
            }
            dft<R>(v[g]);
            const int out = (blk << lg) + (j - jm) * R + jm;
#pragma unroll
            for (int r = 0; r < R; ++r) {
                if (GOUT) io.store(out + r * Ns, v[g][r]);
                else z[pad(out + r * Ns)] = v[g][r];
            }
        }
    }
    if (!GOUT) __syncthreads();
}

template <int R, int VPT, bool GIN, bool GOUT, class Io>
__device__ __forceinline__ void pass_io(f2v *z, int S, int lg, int Ns, int t, const Io &io, bool first, bool last) {
    if (GIN && first && GOUT && last) stockham_pass<R, VPT, true, true>(z, S, lg, Ns, t, io);
    else if (GIN && first) stockham_pass<R, VPT, true, false>(z, S, lg, Ns, t, io);
    else if (GOUT && last) stockham_pass<R, VPT, false, true>(z, S, lg, Ns, t, io);
    else stockham_pass<R, VPT, false, false>(z, S, lg, Ns, t, io);
}

// Forward transform of every block: radix-16 passes, then one pass of the
// remaining radix; GIN / GOUT as in stockham_pass, for the first / last pass.
template <int VPT, bool GIN, bool GOUT, class Io>
__device__ __forceinline__ void fft_blocks(f2v *z, int S, int lg, int t, const Io &io) {
    const int n16 = lg >> 2, rem = lg & 3, npass = n16 + (rem != 0);
    int Ns = 1;
    for (int p = 0; p < n16; ++p, Ns <<= 4)
        pass_io<16, VPT, GIN, GOUT>(z, S, lg, Ns, t, io, p == 0, p == npass - 1);
    const bool first = n16 == 0;
    if (rem == 3) pass_io<8, VPT, GIN, GOUT>(z, S, lg, Ns, t, io, first, true);
    else if (rem == 2) pass_io<4, VPT, GIN, GOUT>(z, S, lg, Ns, t, io, first, true);
    else if (rem == 1) pass_io<2, VPT, GIN, GOUT>(z, S, lg, Ns, t, io, first, true);
}

template <typename TI, typename TO, bool CORR, int VPT>
__global__ void __launch_bounds__(BT) circular_kernel(BindArgs a) {
    extern __shared__ f2v smem[];
    const int L = (int)a.L, lg = a.lg, nbmax = a.nb;
    const int64_t wpr = (a.nblocks + nbmax - 1) / nbmax;          // work-groups per row
    const int64_t row = (int64_t)blockIdx.x / wpr;
    const int64_t blk0 = ((int64_t)blockIdx.x - row * wpr) * nbmax;
    const int nb = (int)((a.nblocks - blk0 < nbmax) ? (a.nblocks - blk0) : nbmax);
    const int S = nb * L;                                        // <= VPT * BT
    const int t = threadIdx.x;
    f2v *z = smem;
    BlockIo<TI, TO> io;
    io.x = static_cast<const TI *>(a.X) + row * a.ldx + blk0 * L;
    io.y = static_cast<const TI *>(a.Y) + row * a.ldy + blk0 * L;
    io.out = static_cast<TO *>(a.Z) + row * a.ldz + blk0 * L;
    io.inv = 1.0f / (float)L;

    fft_blocks<VPT, true, false>(z, S, lg, t, io);

    // product of the two spectra, stored conjugated for the inverse;
    // P_{L-k} = conj P_k (real signals)
    for (int q = t; q < nb * (L / 2 + 1); q += BT) {
        const int blk = q / (L / 2 + 1), k = q - blk * (L / 2 + 1);
        const int kk = (L - k) & (L - 1);
        const int ik = pad((blk << lg) + k), ikk = pad((blk << lg) + kk);
        const f2v zk = z[ik], zm = conjv(z[ikk]);
        const f2v X = (zk + zm) * 0.5f;
        const f2v Yk = mul_mi((zk - zm) * 0.5f);
        const f2v P = CORR ? cmul(X, conjv(Yk)) : cmul(X, Yk);
        z[ik] = conjv(P);
        if (kk != k) z[ikk] = P;
    }
    __syncthreads();
    fft_blocks<VPT, false, true>(z, S, lg, t, io);
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

template <typename TI, typename TO, int VPT>
hipError_t launch_circular(int op, dim3 grid, size_t lds, const BindArgs &a, hipStream_t s) {
    const void *k = (op == GS_BINDOP_CORR) ? reinterpret_cast<const void *>(circular_kernel<TI, TO, true, VPT>)
                                           : reinterpret_cast<const void *>(circular_kernel<TI, TO, false, VPT>);
    hipError_t e = raise_lds_limit(k, lds);
    if (e != hipSuccess) return e;
    if (op == GS_BINDOP_CORR) hipLaunchKernelGGL((circular_kernel<TI, TO, true, VPT>), grid, dim3(BT), lds, s, a);
    else hipLaunchKernelGGL((circular_kernel<TI, TO, false, VPT>), grid, dim3(BT), lds, s, a);
    return hipGetLastError();
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
    const int64_t S = a.nb * a.L;                         // values per work-group
    const size_t lds = (size_t)(S + S / 16) * sizeof(f2v);
    if (S > 32 * BT) return hipErrorInvalidValue;
    if (S <= 16 * BT) return launch_circular<TI, TO, 16>(op, grid, lds, a, s);
    return launch_circular<TI, TO, 32>(op, grid, lds, a, s);
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
