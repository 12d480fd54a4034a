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

// Pass P of a transform of L = 2^LG values: radix-16 passes, then one pass of
// the remaining radix; the sub-transforms before it have length NS.
template <int LG, int P> struct PassShape {
    static constexpr int N16 = LG / 4, REM = LG % 4, NPASS = N16 + (REM != 0);
    static constexpr int R = P < N16 ? 16 : (REM == 3 ? 8 : REM == 2 ? 4 : 2);
    static constexpr int LOGR = R == 16 ? 4 : R == 8 ? 3 : R == 4 ? 2 : 1;
    static constexpr int NS = 1 << (4 * P);
    static constexpr int LR = 1 << (LG - LOGR);
};

// The pass twiddles exp(-2 pi i (j mod NS) r / (NS R)), r = 1 .. R - 1, of
// this thread's butterflies in passes P, P + 1, ... (pass 0 has none): the
// forward and the inverse transform take the same passes with the same
// butterflies, so each thread computes its own once and keeps them in
// registers (with 16 values per thread; with 32, L = 8192, they would not
// fit and each pass computes its own).  Powers by repeated products of
// exp(-2 pi i (j mod NS) / (NS R)).
template <int LG, int P> __device__ __forceinline__ void pass_twiddles(f2v *w, int q) {
    typedef PassShape<LG, P> Sh;
    const int jm = (q & (Sh::LR - 1)) & (Sh::NS - 1);
    float sn, cs;
    // -2 jm / (NS R) exactly: the divisor is a power of two
    sincospif((-2.0f / (float)(Sh::NS * Sh::R)) * (float)jm, &sn, &cs);
    const f2v w1 = f2v{cs, sn};
    f2v wr = w1;
#pragma unroll
    for (int r = 0; r < Sh::R - 1; ++r) {
        w[r] = wr;
        wr = cmul(wr, w1);
    }
}
template <int LG, int P, int VPT, bool END = (P >= PassShape<LG, P>::NPASS || VPT > 16)> struct Twiddles {
    static constexpr bool CACHED = true;
    typedef PassShape<LG, P> Sh;
    static constexpr int G = VPT / Sh::R;
    f2v w[G][Sh::R - 1];
    Twiddles<LG, P + 1, VPT> next;
    __device__ __forceinline__ void init(int S, int t) {
        const int nq = S >> Sh::LOGR;
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const int q = t + g * BT;
            if (q < nq) pass_twiddles<LG, P>(w[g], q);
        }
        next.init(S, t);
    }
};
template <int LG, int P, int VPT> struct Twiddles<LG, P, VPT, true> {
    static constexpr bool CACHED = false;
    __device__ __forceinline__ void init(int, int) {}
};
// The twiddles from pass 1 on (pass 0 has none).
template <int LG, int VPT> struct TwiddlesAll {
    static constexpr bool CACHED = true;
    Twiddles<LG, 1, VPT> next;
};
// The twiddles of the passes after the one tw serves.
template <class Tw> __device__ __forceinline__ const auto &next_twiddles(const Tw &tw) {
    if constexpr (Tw::CACHED) return tw.next;
    else return tw;
}

// One Stockham pass of radix R over the S values in LDS (blocks of L = 2^LG
// values), the sub-transforms done so far having length NS: butterfly q of
// block blk (j = q mod L/R) takes values j + r L/R, multiplies value r by the
// pass twiddle r, and writes its outputs to (j / NS) NS R + (j mod NS) + r NS.
// Each thread holds VPT values.  GIN: gather from io.load instead of LDS;
// GOUT: scatter to io.store instead.  With L, R and NS known at compile time
// the element offsets of a gather or scatter are constants added to one
// padded base slot wherever a whole number of 16-value groups separates
// consecutive elements.
template <int LG, int P, int VPT, bool GIN, bool GOUT, class Io, class Tw>
__device__ __forceinline__ void stockham_pass(f2v *z, int S, int t, const Io &io, const Tw &tw) {
    typedef PassShape<LG, P> Sh;
    constexpr int R = Sh::R, NS = Sh::NS, LR = Sh::LR, LOGR = Sh::LOGR;
    constexpr int G = VPT / R;
    // consecutive gather elements LR apart; scatter elements NS apart (or the
    // 16 outputs of a first radix-16 pass filling one group)
    constexpr bool GC = LR % 16 == 0, SC = NS % 16 == 0 || (NS == 1 && R == 16);
    const int nq = S >> LOGR;
    f2v v[G][R];
#pragma unroll
    for (int g = 0; g < G; ++g) {
        const int q = t + g * BT;
        if (q < nq) {
            const int blk = q >> (LG - LOGR), j = q & (LR - 1);
            const int base = (blk << LG) + j;
            const int pb = pad(base);
#pragma unroll
            for (int r = 0; r < R; ++r) {
                if (GIN) v[g][r] = io.load(base + r * LR);
                else v[g][r] = z[GC ? pb + r * (LR + LR / 16) : pad(base + r * LR)];
            }
        }
    }
    if (!GIN && !GOUT) __syncthreads();   // every gather is done before LDS is overwritten
#pragma unroll
    for (int g = 0; g < G; ++g) {
        const int q = t + g * BT;
        if (q < nq) {
            const int blk = q >> (LG - LOGR), j = q & (LR - 1);
            const int jm = j & (NS - 1);
            if constexpr (NS > 1) {
                if constexpr (Tw::CACHED) {
#pragma unroll
                    for (int r = 1; r < R; ++r) v[g][r] = cmul(v[g][r], tw.w[g][r - 1]);
                } else {
                    f2v w[R - 1];
                    pass_twiddles<LG, P>(w, q);
#pragma unroll
                    for (int r = 1; r < R; ++r) v[g][r] = cmul(v[g][r], w[r - 1]);
                }
            }
            dft<R>(v[g]);
            const int out = (blk << LG) + (j - jm) * R + jm;
            const int po = pad(out);
#pragma unroll
            for (int r = 0; r < R; ++r) {
                if (GOUT) io.store(out + r * NS, v[g][r]);
                else z[SC ? po + r * (NS + NS / 16) : pad(out + r * NS)] = v[g][r];
            }
        }
    }
    if (!GOUT) __syncthreads();
}

// Passes P .. of the forward transform of every block; GIN / GOUT as in
// stockham_pass, for the first / last pass.
template <int LG, int P, int VPT, bool GIN, bool GOUT, class Io, class Tw>
__device__ __forceinline__ void fft_passes(f2v *z, int S, int t, const Io &io, const Tw &tw) {
    typedef PassShape<LG, P> Sh;
    if constexpr (P < Sh::NPASS) {
        stockham_pass<LG, P, VPT, GIN && P == 0, GOUT && P == Sh::NPASS - 1>(z, S, t, io, tw);
        fft_passes<LG, P + 1, VPT, GIN, GOUT>(z, S, t, io, next_twiddles(tw));
    }
}

// Blocks of L = 2^LG values; a work-group holds nb of them (S = nb L <= VPT BT).
template <typename TI, typename TO, bool CORR, int LG>
__global__ void __launch_bounds__(BT) circular_kernel(BindArgs a) {
    constexpr int L = 1 << LG, VPT = L > 16 * BT ? L / BT : 16;
    extern __shared__ f2v smem[];
    const int nbmax = a.nb;
    const int64_t wpr = (a.nblocks + nbmax - 1) / nbmax;          // work-groups per row
    const int64_t row = (int64_t)blockIdx.x / wpr;
    const int64_t blk0 = ((int64_t)blockIdx.x - row * wpr) * nbmax;
    // blocks of 4096 values or more: one per work-group, known here
    const int nb = (L >= SEG) ? 1 : (int)((a.nblocks - blk0 < nbmax) ? (a.nblocks - blk0) : nbmax);
    const int S = nb * L;                                        // <= VPT * BT
    const int t = threadIdx.x;
    f2v *z = smem;
    BlockIo<TI, TO> io;
    io.x = static_cast<const TI *>(a.X) + row * a.ldx + blk0 * L;
    io.y = static_cast<const TI *>(a.Y) + row * a.ldy + blk0 * L;
    io.out = static_cast<TO *>(a.Z) + row * a.ldz + blk0 * L;
    io.inv = 1.0f / (float)L;

    TwiddlesAll<LG, VPT> tw;
    tw.next.init(S, t);
    fft_passes<LG, 0, VPT, true, false>(z, S, t, io, tw);

    // product of the two spectra, stored conjugated for the inverse;
    // P_{L-k} = conj P_k (real signals): k = 0 .. L/2 - 1 with its partner
    // L - k (k = 0 is its own), then k = L/2 (its own) of every block
    auto product = [&](int blk, int k) {
        const int kk = (L - k) & (L - 1);
        const int ik = pad((blk << LG) + k), ikk = pad((blk << LG) + kk);
        const f2v zk = z[ik], zm = conjv(z[ikk]);
        const f2v X = (zk + zm) * 0.5f;
        const f2v Yk = mul_mi((zk - zm) * 0.5f);
        const f2v P = CORR ? cmul(X, conjv(Yk)) : cmul(X, Yk);
        z[ik] = conjv(P);
        if (kk != k) z[ikk] = P;
    };
    for (int q = t; q < nb * (L / 2); q += BT) product(q >> (LG - 1), q & (L / 2 - 1));
    for (int blk = t; blk < nb; blk += BT) product(blk, L / 2);
    __syncthreads();
    fft_passes<LG, 0, VPT, false, true>(z, S, t, io, tw);
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

template <typename TI, typename TO, int LG>
hipError_t launch_circular(int op, dim3 grid, size_t lds, const BindArgs &a, hipStream_t s) {
    const void *k = (op == GS_BINDOP_CORR) ? reinterpret_cast<const void *>(circular_kernel<TI, TO, true, LG>)
                                           : reinterpret_cast<const void *>(circular_kernel<TI, TO, false, LG>);
    hipError_t e = raise_lds_limit(k, lds);
    if (e != hipSuccess) return e;
    if (op == GS_BINDOP_CORR) hipLaunchKernelGGL((circular_kernel<TI, TO, true, LG>), grid, dim3(BT), lds, s, a);
    else hipLaunchKernelGGL((circular_kernel<TI, TO, false, LG>), grid, dim3(BT), lds, s, a);
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
    if (S > (a.lg == 13 ? 32 : 16) * BT) return hipErrorInvalidValue;
    switch (a.lg) {
    case 1: return launch_circular<TI, TO, 1>(op, grid, lds, a, s);
    case 2: return launch_circular<TI, TO, 2>(op, grid, lds, a, s);
    case 3: return launch_circular<TI, TO, 3>(op, grid, lds, a, s);
    case 4: return launch_circular<TI, TO, 4>(op, grid, lds, a, s);
    case 5: return launch_circular<TI, TO, 5>(op, grid, lds, a, s);
    case 6: return launch_circular<TI, TO, 6>(op, grid, lds, a, s);
    case 7: return launch_circular<TI, TO, 7>(op, grid, lds, a, s);
    case 8: return launch_circular<TI, TO, 8>(op, grid, lds, a, s);
    case 9: return launch_circular<TI, TO, 9>(op, grid, lds, a, s);
    case 10: return launch_circular<TI, TO, 10>(op, grid, lds, a, s);
    case 11: return launch_circular<TI, TO, 11>(op, grid, lds, a, s);
    case 12: return launch_circular<TI, TO, 12>(op, grid, lds, a, s);
    case 13: return launch_circular<TI, TO, 13>(op, grid, lds, a, s);
    default: return hipErrorInvalidValue;
    }
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
