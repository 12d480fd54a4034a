// Dense contractions of the Gram-Space operators on CDNA4 matrix cores.
//
//   project      T = X Q^T          (A = X,  B = Q stored N x K)
//   reconstruct  X = T Q            (A = T,  B = Q stored K x N)
//   bind         X = (T Q) .* (T2 Q)
//   prob2vec     T = P R            (A = P,  B = R stored K x N)
//   similarity   S = scale * T R^T  (A = T,  B = R stored N x K), cosine
//                normalisation and row argmax fused in the epilogue
//   attention    A = softmax(beta * S) fused, two passes over the row block
//
// Work-group tile 128 x 128, K-step 32, 256 threads = 4 waves in a 2 x 2
// arrangement, each wave owning a 64 x 64 sub-tile as 2 x 2 blocks of the
// 32x32x2 fp32 MFMA.  Both operands are staged through LDS k-major
// ([k][m] / [k][n]), so every MFMA operand read is one conflict-free
// ds_read_b32 per lane; bf16 operands are widened to fp32 on the way in.
// The next K-step is fetched into registers while the current one is
// multiplied (double-buffered LDS, one barrier per K-step).
#include <mutex>
#include <unordered_set>

#include "gs_internal.h"

namespace gs {
namespace {

constexpr int BM = 128, BN = 128, BK = 32;
constexpr int NTHR = 256;
constexpr int LDS_STRIDE = BM + 4;            // floats per k-row of a staged tile
constexpr int TILE_FLOATS = BK * LDS_STRIDE;  // one staged operand tile

typedef float f16v __attribute__((ext_vector_type(16)));
typedef float f4v __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- loading
// Each thread moves 16 elements of a tile per K-step.

// Row-oriented operand (A, or B stored N x K): 128 rows x 32 k.  Lane l of
// wave w takes row (l % 32) + 32 w and the 16 contiguous k starting at
// 16 (l / 32).
template <typename T>
__device__ __forceinline__ void load_rows(const T *__restrict__ base, int64_t ld, int64_t row0,
                                          int64_t nrows, int64_t k0, int64_t K, bool vec,
                                          float v[16]) {
    const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int64_t row = row0 + (l & 31) + 32 * w;
    const int64_t kb = k0 + 16 * (l >> 5);
    if (row >= nrows) {
#pragma unroll
        for (int i = 0; i < 16; ++i) v[i] = 0.f;
        return;
    }
    const T *p = base + row * ld + kb;
    if constexpr (sizeof(T) == 4) {
        if (vec) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                if (kb + 4 * q < K) {
                    f4v t = *reinterpret_cast<const f4v *>(p + 4 * q);
                    v[4 * q] = t[0]; v[4 * q + 1] = t[1]; v[4 * q + 2] = t[2]; v[4 * q + 3] = t[3];
                } else {
                    v[4 * q] = v[4 * q + 1] = v[4 * q + 2] = v[4 * q + 3] = 0.f;
                }
            }
            return;
        }
    } else {
        if (vec) {
#pragma unroll
            for (int q = 0; q < 2; ++q) {
                if (kb + 8 * q < K) {
                    uint4 t = *reinterpret_cast<const uint4 *>(p + 8 * q);
                    uint32_t ww[4] = {t.x, t.y, t.z, t.w};
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        v[8 * q + 2 * e] = __uint_as_float(ww[e] << 16);
                        v[8 * q + 2 * e + 1] = __uint_as_float(ww[e] & 0xffff0000u);
                    }
                } else {
#pragma unroll
                    for (int e = 0; e < 8; ++e) v[8 * q + e] = 0.f;
                }
            }
            return;
        }
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) v[i] = (kb + i < K) ? ld_f32<T>(p, i) : 0.f;
}

__device__ __forceinline__ void store_rows(float *tile, const float v[16]) {
    const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int m = (l & 31) + 32 * w;
    const int kb = 16 * (l >> 5);
#pragma unroll
    for (int i = 0; i < 16; ++i) tile[(kb + i) * LDS_STRIDE + m] = v[i];
}

// K-major operand (B stored K x N): 32 k-rows x 128 columns.  Thread t takes
// k-row t / 8 and the 16 contiguous columns starting at 16 (t % 8).
template <typename T>
__device__ __forceinline__ void load_kmajor(const T *__restrict__ base, int64_t ld, int64_t k0,
                                            int64_t K, int64_t n0, int64_t N, bool vec,
                                            float v[16]) {
    const int t = threadIdx.x;
    const int64_t k = k0 + (t >> 3);
    const int64_t nb = n0 + 16 * (t & 7);
    if (k >= K) {
#pragma unroll
        for (int i = 0; i < 16; ++i) v[i] = 0.f;
        return;
    }
    const T *p = base + k * ld + nb;
    if constexpr (sizeof(T) == 4) {
        if (vec) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                if (nb + 4 * q < N) {
                    f4v x = *reinterpret_cast<const f4v *>(p + 4 * q);
                    v[4 * q] = x[0]; v[4 * q + 1] = x[1]; v[4 * q + 2] = x[2]; v[4 * q + 3] = x[3];
                } else {
                    v[4 * q] = v[4 * q + 1] = v[4 * q + 2] = v[4 * q + 3] = 0.f;
                }
            }
            return;
        }
    } else {
        if (vec) {
#pragma unroll
            for (int q = 0; q < 2; ++q) {
                if (nb + 8 * q < N) {
                    uint4 x = *reinterpret_cast<const uint4 *>(p + 8 * q);
                    uint32_t ww[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        v[8 * q + 2 * e] = __uint_as_float(ww[e] << 16);
                        v[8 * q + 2 * e + 1] = __uint_as_float(ww[e] & 0xffff0000u);
                    }
                } else {
#pragma unroll
                    for (int e = 0; e < 8; ++e) v[8 * q + e] = 0.f;
                }
            }
            return;
        }
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) v[i] = (nb + i < N) ? ld_f32<T>(p, i) : 0.f;
}

__device__ __forceinline__ void store_kmajor(float *tile, const float v[16]) {
    const int t = threadIdx.x;
    float *p = tile + (t >> 3) * LDS_STRIDE + 16 * (t & 7);
#pragma unroll
    for (int q = 0; q < 4; ++q)
        *reinterpret_cast<f4v *>(p + 4 * q) = f4v{v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]};
}

// Row of the output held by accumulator register g of a 32x32 block, for lane l.
__device__ __forceinline__ int acc_row(int g, int l) { return 8 * (g >> 2) + 4 * (l >> 5) + (g & 3); }

// ------------------------------------------------------------- main loop
//
// Computes the 128 x 128 block (m0, n0) of A * Bop into acc (and A2 * Bop into
// acc2 when TWO).  On return LDS is free for reuse by the caller (a barrier
// has been passed after the last MFMA read).
//
// When SQA, every thread t < 128 also accumulates sum_k A[m0 + t, k]^2 into
// *sqa; when SQB, every thread t < 128 accumulates sum_k Bop[k, n0 + t]^2.
template <typename TA, typename TB, bool BNN, bool TWO>
__device__ __forceinline__ void block_mma(const GemmArgs &g, int64_t m0, int64_t n0, bool veca,
                                          bool vecb, float *lds, f16v acc[2][2], f16v acc2[2][2],
                                          bool sqa, float *sqa_out, bool sqb, float *sqb_out) {
    const TA *A = static_cast<const TA *>(g.A);
    const TA *A2 = static_cast<const TA *>(g.A2);
    const TB *B = static_cast<const TB *>(g.B);
    const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int wm = (w >> 1) * 64, wn = (w & 1) * 64;
    // operand tiles per buffer; buffers are addressed as offsets from the
    // LDS base (a pointer select would make the compiler fall back to flat
    // addressing, whose waits also cover the in-flight global prefetch)
    constexpr int nstage = TWO ? 3 : 2;
    auto buf = [&](int64_t i) { return lds + (int)(i & 1) * (nstage * TILE_FLOATS); };

#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            acc[i][j] = f16v{};
            if (TWO) acc2[i][j] = f16v{};
        }
    float sa = 0.f, sb = 0.f;

    float va[16], vb[16], va2[16];
    const int64_t nk = (g.K + BK - 1) / BK;
    auto fetch = [&](int64_t kt) {
        load_rows<TA>(A, g.lda, m0, g.M, kt * BK, g.K, veca, va);
        if (TWO) load_rows<TA>(A2, g.lda2, m0, g.M, kt * BK, g.K, veca, va2);
        if (BNN) load_kmajor<TB>(B, g.ldb, kt * BK, g.K, n0, g.N, vecb, vb);
        else load_rows<TB>(B, g.ldb, n0, g.N, kt * BK, g.K, vecb, vb);
    };
    auto stash = [&](float *b) {
        store_rows(b, va);
        if (BNN) store_kmajor(b + TILE_FLOATS, vb);
        else store_rows(b + TILE_FLOATS, vb);
        if (TWO) store_rows(b + 2 * TILE_FLOATS, va2);
    };

    fetch(0);
    stash(buf(0));
    lds_barrier();
    for (int64_t kt = 0; kt < nk; ++kt) {
        float *cur = buf(kt);
        if (kt + 1 < nk) fetch(kt + 1);
        const float *As = cur, *Bs = cur + TILE_FLOATS, *As2 = cur + 2 * TILE_FLOATS;
#pragma unroll
        for (int kk = 0; kk < BK; kk += 2) {
            const int kr = (kk + (l >> 5)) * LDS_STRIDE;
            float a0 = As[kr + wm + (l & 31)], a1 = As[kr + wm + 32 + (l & 31)];
            float b0 = Bs[kr + wn + (l & 31)], b1 = Bs[kr + wn + 32 + (l & 31)];
            acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b0, acc[0][0], 0, 0, 0);
            acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b1, acc[0][1], 0, 0, 0);
            acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b0, acc[1][0], 0, 0, 0);
            acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b1, acc[1][1], 0, 0, 0);
            if (TWO) {
                float c0 = As2[kr + wm + (l & 31)], c1 = As2[kr + wm + 32 + (l & 31)];
                acc2[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(c0, b0, acc2[0][0], 0, 0, 0);
                acc2[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(c0, b1, acc2[0][1], 0, 0, 0);
                acc2[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(c1, b0, acc2[1][0], 0, 0, 0);
                acc2[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(c1, b1, acc2[1][1], 0, 0, 0);
            }
        }
        if (threadIdx.x < 128) {
            if (sqa) {
#pragma unroll 8
                for (int k = 0; k < BK; ++k) { float x = As[k * LDS_STRIDE + threadIdx.x]; sa += x * x; }
            }
            if (sqb) {
#pragma unroll 8
                for (int k = 0; k < BK; ++k) { float x = Bs[k * LDS_STRIDE + threadIdx.x]; sb += x * x; }
            }
        }
        if (kt + 1 < nk) stash(buf(kt + 1));
        lds_barrier();
    }
    if (threadIdx.x < 128) {
        if (sqa) *sqa_out = sa;
        if (sqb) *sqb_out = sb;
    }
}

// ------------------------------------------------------- bf16 main loop
//
// Both operands bf16: v_mfma_f32_32x32x16_bf16 on the same 128 x 128 block
// with K-steps of 64.  Operands stay bf16 in LDS, k-contiguous per row
// ([m][k] and [n][k], row stride BSTR), so every MFMA operand is one 16-byte
// LDS read (8 consecutive k) per lane.  A K x N operand (b_nn) is transposed
// while it is written to LDS.  Same accumulator layout as the fp32 loop.

constexpr int BK16 = 64;                       // K-step of the bf16 loop
constexpr int BSTR = BK16 + 8;                 // bf16 per staged row (16-byte pad)
constexpr int BTILE = 128 * BSTR;              // bf16 per staged operand tile

typedef __bf16 bf8v __attribute__((ext_vector_type(8)));

// LDS floats used by the staging buffers of either loop.
template <typename TA, typename TB, bool TWO>
constexpr size_t mma_lds_floats() {
    if constexpr (sizeof(TA) == 2 && sizeof(TB) == 2) return (size_t)2 * (TWO ? 3 : 2) * BTILE / 2;
    else return (size_t)2 * (TWO ? 3 : 2) * TILE_FLOATS;
}

// 8 consecutive bf16 (raw bits) starting at p, zeros at or beyond `lim`
// elements from p (lim <= 0: all zero); vector load when allowed.
__device__ __forceinline__ uint4 load8_bf16(const bf16_t *p, int64_t lim, bool vec) {
    if (lim >= 8 && vec) return *reinterpret_cast<const uint4 *>(p);
    uint16_t h[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) h[i] = (i < lim) ? p[i].bits : (uint16_t)0;
    return uint4{(uint32_t)h[0] | ((uint32_t)h[1] << 16), (uint32_t)h[2] | ((uint32_t)h[3] << 16),
                 (uint32_t)h[4] | ((uint32_t)h[5] << 16), (uint32_t)h[6] | ((uint32_t)h[7] << 16)};
}

// Row operand (128 rows x 64 k): thread t moves rows t / 8 + 32 i (i < 4),
// k-chunk 8 (t % 8).  The chunk's validity is all-or-nothing in vector mode
// (K a multiple of 8), element-wise otherwise.
__device__ __forceinline__ void fetch_rows_bf16(const bf16_t *base, int64_t ld, int64_t row0, int64_t nrows,
                                                int64_t k0, int64_t K, bool vec, uint4 v[4]) {
    const int t = threadIdx.x;
    const int64_t kc = k0 + 8 * (t & 7);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t row = row0 + (t >> 3) + 32 * i;
        v[i] = (row < nrows && kc < K) ? load8_bf16(base + row * ld + kc, K - kc, vec) : uint4{0, 0, 0, 0};
    }
}

__device__ __forceinline__ void stash_rows_bf16(uint16_t *tile, const uint4 v[4]) {
    const int t = threadIdx.x;
#pragma unroll
    for (int i = 0; i < 4; ++i)
        *reinterpret_cast<uint4 *>(tile + ((t >> 3) + 32 * i) * BSTR + 8 * (t & 7)) = v[i];
}

// K x N operand (64 k x 128 n), written transposed ([n][k]) into LDS.
// Thread t owns the 4 x 8 block k = 4 (t % 16) + 0..3, n = 8 (t / 16) + 0..7:
// four 16-byte loads (one per k), a register transpose with v_perm_b32, and
// eight 8-byte LDS writes (four k-values of one n each).  Lanes vary along k
// first, so every 16 lanes fill one contiguous 128-byte LDS row segment.
__device__ __forceinline__ void fetch_kmajor_bf16(const bf16_t *base, int64_t ld, int64_t k0, int64_t K,
                                                  int64_t n0, int64_t N, bool vec, uint4 v[4]) {
    const int t = threadIdx.x;
    const int64_t nc = n0 + 8 * (t >> 4);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t k = k0 + 4 * (t & 15) + i;
        v[i] = (k < K && nc < N) ? load8_bf16(base + k * ld + nc, N - nc, vec) : uint4{0, 0, 0, 0};
    }
}

__device__ __forceinline__ void stash_kmajor_bf16(uint16_t *tile, const uint4 v[4]) {
    const int t = threadIdx.x;
    const int kb = 4 * (t & 15), nb = 8 * (t >> 4);
    const uint32_t w0[4] = {v[0].x, v[0].y, v[0].z, v[0].w}, w1[4] = {v[1].x, v[1].y, v[1].z, v[1].w};
    const uint32_t w2[4] = {v[2].x, v[2].y, v[2].z, v[2].w}, w3[4] = {v[3].x, v[3].y, v[3].z, v[3].w};
#pragma unroll
    for (int m = 0; m < 4; ++m) {
        // low halves: column n = nb + 2m; high halves: n = nb + 2m + 1
        const uint2 lo = {__builtin_amdgcn_perm(w1[m], w0[m], 0x05040100u), __builtin_amdgcn_perm(w3[m], w2[m], 0x05040100u)};
        const uint2 hi = {__builtin_amdgcn_perm(w1[m], w0[m], 0x07060302u), __builtin_amdgcn_perm(w3[m], w2[m], 0x07060302u)};
        *reinterpret_cast<uint2 *>(tile + (nb + 2 * m) * BSTR + kb) = lo;
        *reinterpret_cast<uint2 *>(tile + (nb + 2 * m + 1) * BSTR + kb) = hi;
    }
}

__device__ __forceinline__ bf8v lds_frag(const uint16_t *tile, int row, int kofs) {
    return *reinterpret_cast<const bf8v *>(tile + row * BSTR + kofs);
}

// Sum of squares of the 64 staged k-values of row t (t < 128).
__device__ __forceinline__ float row_sq_bf16(const uint16_t *tile, int row) {
    float s = 0.f;
#pragma unroll
    for (int q = 0; q < BK16 / 8; ++q) {
        const uint4 u = *reinterpret_cast<const uint4 *>(tile + row * BSTR + 8 * q);
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float lo = __uint_as_float(w[e] << 16), hi = __uint_as_float(w[e] & 0xffff0000u);
            s += lo * lo + hi * hi;
        }
    }
    return s;
}

template <bool BNN, bool TWO>
__device__ __forceinline__ void block_mma_bf16(const GemmArgs &g, int64_t m0, int64_t n0, bool veca, bool vecb,
                                               float *lds_f, f16v acc[2][2], f16v acc2[2][2], bool sqa,
                                               float *sqa_out, bool sqb, float *sqb_out) {
    const bf16_t *A = static_cast<const bf16_t *>(g.A);
    const bf16_t *A2 = static_cast<const bf16_t *>(g.A2);
    const bf16_t *B = static_cast<const bf16_t *>(g.B);
    uint16_t *lds = reinterpret_cast<uint16_t *>(lds_f);
    const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int wm = (w >> 1) * 64, wn = (w & 1) * 64;
    constexpr int nstage = TWO ? 3 : 2;
    auto buf = [&](int64_t i) { return lds + (int)(i & 1) * (nstage * BTILE); };

#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            acc[i][j] = f16v{};
            if (TWO) acc2[i][j] = f16v{};
        }
    float sa = 0.f, sb = 0.f;
    uint4 va[4], vb[4], va2[4];
    const int64_t nk = (g.K + BK16 - 1) / BK16;
    auto fetch = [&](int64_t kt) {
        fetch_rows_bf16(A, g.lda, m0, g.M, kt * BK16, g.K, veca, va);
        if (TWO) fetch_rows_bf16(A2, g.lda2, m0, g.M, kt * BK16, g.K, veca, va2);
        if (BNN) fetch_kmajor_bf16(B, g.ldb, kt * BK16, g.K, n0, g.N, vecb, vb);
        else fetch_rows_bf16(B, g.ldb, n0, g.N, kt * BK16, g.K, vecb, vb);
    };
    auto stash = [&](uint16_t *b) {
        stash_rows_bf16(b, va);
        if (BNN) stash_kmajor_bf16(b + BTILE, vb);
        else stash_rows_bf16(b + BTILE, vb);
        if (TWO) stash_rows_bf16(b + 2 * BTILE, va2);
    };

    fetch(0);
    stash(buf(0));
    lds_barrier();
    for (int64_t kt = 0; kt < nk; ++kt) {
        uint16_t *cur = buf(kt);
        if (kt + 1 < nk) fetch(kt + 1);
        const uint16_t *As = cur, *Bs = cur + BTILE, *As2 = cur + 2 * BTILE;
#pragma unroll
        for (int kk = 0; kk < BK16; kk += 16) {
            const int ko = kk + 8 * (l >> 5);
            const bf8v a0 = lds_frag(As, wm + (l & 31), ko), a1 = lds_frag(As, wm + 32 + (l & 31), ko);
            const bf8v b0 = lds_frag(Bs, wn + (l & 31), ko), b1 = lds_frag(Bs, wn + 32 + (l & 31), ko);
            acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b0, acc[0][0], 0, 0, 0);
            acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b1, acc[0][1], 0, 0, 0);
            acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b0, acc[1][0], 0, 0, 0);
            acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b1, acc[1][1], 0, 0, 0);
            if (TWO) {
                const bf8v c0 = lds_frag(As2, wm + (l & 31), ko), c1 = lds_frag(As2, wm + 32 + (l & 31), ko);
                acc2[0][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(c0, b0, acc2[0][0], 0, 0, 0);
                acc2[0][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(c0, b1, acc2[0][1], 0, 0, 0);
                acc2[1][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(c1, b0, acc2[1][0], 0, 0, 0);
                acc2[1][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(c1, b1, acc2[1][1], 0, 0, 0);
            }
        }
        if (threadIdx.x < 128) {
            if (sqa) sa += row_sq_bf16(As, threadIdx.x);
            if (sqb) sb += row_sq_bf16(Bs, threadIdx.x);
        }
        if (kt + 1 < nk) stash(buf(kt + 1));
        lds_barrier();
    }
    if (threadIdx.x < 128) {
        if (sqa) *sqa_out = sa;
        if (sqb) *sqb_out = sb;
    }
}

// --------------------------------------------- bf16 pipelined main loop
//
// The same 128 x 128 block and K-steps of 64, with operand tiles brought
// into LDS by asynchronous global->LDS loads (global_load_lds_dwordx4), NS
// stages deep: the loads for K-step kt + NS - 1 are in flight while step kt
// is multiplied, with one barrier per step and no register staging.  Each
// load instruction fills 1 KB of LDS in lane order, so the layout is chosen
// through which 16-byte chunk each lane fetches:
//   row tile   [128][64]: chunk c of row r sits at position c ^ ((r >> 1) & 7);
//   k-row tile [64][128]: chunk c of k-row k sits at position c ^ (4 (k & 3)).
// A 128-byte row covers half of the 64 LDS banks, so 16 consecutive rows (one
// 256-byte read phase of ds_read_b128) reach all 16 bank groups only if the
// swizzle changes with r >> 1; a transpose read takes 4 chunks from each of 4
// consecutive k-rows per 32 lanes, which the k-row swizzle spreads over all 64
// banks.  Both make the fragment reads conflict-free without padding.  Fragments of a k-row tile (b_nn) come from transpose reads
// (ds_read_b64_tr_b16), which hand each lane 4 consecutive k of one column.
// Rows beyond the matrix reuse its last row (their results are discarded);
// k beyond K is zeroed in LDS in the last step.  Requires 16-byte aligned
// rows (ld a multiple of 8): rows are read in 16-byte units up to column
// ceil(cols / 8) * 8 <= ld.

constexpr int DTILE = 128 * 64;                 // bf16 per operand tile (16 KB)

#define GS_G1 __attribute__((address_space(1)))
#define GS_L3 __attribute__((address_space(3)))
typedef short s4v __attribute__((ext_vector_type(4)));

template <bool TWO, int NS>
constexpr size_t dma_lds_floats() { return (size_t)NS * (TWO ? 3 : 2) * DTILE / 2; }

// s_waitcnt with vmcnt <= n (expcnt and lgkmcnt unconstrained), gfx9 encoding.
template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Wait until at most `later` stages of OPS loads each (this wave's) are still
// in flight; later is clamped to MAXS.
template <int OPS, int MAXS>
__device__ __forceinline__ void wait_stages(int64_t later) {
    if constexpr (MAXS <= 0) {
        wait_vm<0>();
    } else {
        if (later >= MAXS) wait_vm<OPS * MAXS>();
        else wait_stages<OPS, MAXS - 1>(later);
    }
}

__device__ __forceinline__ void dma16(const void *g, uint16_t *lds_wave_base) {
    __builtin_amdgcn_global_load_lds((const GS_G1 void *)g, (GS_L3 void *)lds_wave_base, 16, 0, 0);
}

// 16 load instructions of 1 KB per row tile: wave w issues blocks 4w .. 4w+3
// (8 rows each).  Lane L of block b lands at row r = 8b + L/8, position L%8,
// so it fetches chunk (L%8) ^ ((r >> 1) & 7) = (L%8) ^ (4 (b & 1) + L/16).
__device__ __forceinline__ void dma_rows(const bf16_t *base, int64_t ld, int64_t row0, int64_t nrows,
                                         int64_t k0, int64_t K, uint16_t *tile) {
    const int L = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int rl = L >> 3;
    const int64_t klast = ((K - 1) >> 3) << 3;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int b = 4 * w + q;
        const int c = (L & 7) ^ (4 * (q & 1) + (rl >> 1));
        int64_t kc = k0 + 8 * c;
        if (kc > klast) kc = klast;
        int64_t row = row0 + 8 * b + rl;
        if (row > nrows - 1) row = nrows - 1;
        dma16(base + row * ld + kc, tile + b * 512);
    }
}

// 16 load instructions of 1 KB per k-row tile: wave w issues blocks 4w .. 4w+3
// (4 k-rows each).  Lane L of block b fetches k-row 4b + L/16, chunk
// (L%16) ^ (4 (k-row % 4)).
__device__ __forceinline__ void dma_krows(const bf16_t *base, int64_t ld, int64_t k0, int64_t K, int64_t n0,
                                          int64_t N, uint16_t *tile) {
    const int L = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t nlast = ((N - 1) >> 3) << 3;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int b = 4 * w + q;
        const int kl = 4 * b + (L >> 4);
        const int c = (L & 15) ^ (4 * (kl & 3));
        int64_t nc = n0 + 8 * c;
        if (nc > nlast) nc = nlast;
        int64_t k = k0 + kl;
        if (k > K - 1) k = K - 1;
        dma16(base + k * ld + nc, tile + b * 512);
    }
}

// Zero the k >= kvalid part of a staged row tile / k-row tile.
__device__ __forceinline__ void zero_rows_tail(uint16_t *tile, int kvalid) {
    for (int e = threadIdx.x; e < 128 * 64; e += NTHR) {
        const int r = e >> 6, kl = e & 63;
        if (kl >= kvalid) tile[r * 64 + ((((kl >> 3) ^ ((r >> 1) & 7))) << 3) + (kl & 7)] = 0;
    }
}
__device__ __forceinline__ void zero_krows_tail(uint16_t *tile, int kvalid) {
    for (int e = threadIdx.x; e < 64 * 128; e += NTHR)
        if ((e >> 7) >= kvalid) tile[e] = 0;
}

__device__ __forceinline__ bf8v frag_rows(const uint16_t *tile, int r, int c) {
    return *reinterpret_cast<const bf8v *>(tile + r * 64 + ((c ^ ((r >> 1) & 7)) << 3));
}

// B fragment (8 consecutive k at kk + 8 (lane / 32), column n0w + lane % 32)
// from a k-row tile, by two transpose reads of 4 k each.
__device__ __forceinline__ bf8v frag_krows(const uint16_t *tile, int kk, int n0w) {
    const int l = threadIdx.x & 63;
    const int g = l >> 4, a = l & 15;
    const int n = n0w + 16 * (g & 1) + 4 * (a & 3);
    const int k = kk + 8 * (g >> 1) + (a >> 2);
    const int c = n >> 3;
    const uint16_t *p0 = tile + k * 128 + ((c ^ (4 * (k & 3))) << 3) + (n & 7);
    const uint16_t *p1 = tile + (k + 4) * 128 + ((c ^ (4 * (k & 3))) << 3) + (n & 7);
    const s4v lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((GS_L3 s4v *)(p0));
    const s4v hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((GS_L3 s4v *)(p1));
    const s4v both[2] = {lo, hi};
    return *reinterpret_cast<const bf8v *>(both);
}

// Sum of squares of row r of a row tile (all 8 chunks, started at a position
// that differs between neighbouring row pairs so the 16-lane phases of the
// reads do not collide on banks).
__device__ __forceinline__ float row_sq_dma(const uint16_t *tile, int r) {
    float s = 0.f;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        const uint4 u = *reinterpret_cast<const uint4 *>(tile + r * 64 + 8 * ((q + (r >> 1)) & 7));
        const uint32_t wv[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float lo = __uint_as_float(wv[e] << 16), hi = __uint_as_float(wv[e] & 0xffff0000u);
            s += lo * lo + hi * hi;
        }
    }
    return s;
}

template <bool BNN, bool TWO, int DMA_STAGES>
__device__ __forceinline__ void block_mma_bf16_dma(const GemmArgs &g, int64_t m0, int64_t n0, float *lds_f,
                                                   f16v acc[2][2], f16v acc2[2][2], bool sqa, float *sqa_out,
                                                   bool sqb, float *sqb_out) {
    const bf16_t *A = static_cast<const bf16_t *>(g.A);
    const bf16_t *A2 = static_cast<const bf16_t *>(g.A2);
    const bf16_t *B = static_cast<const bf16_t *>(g.B);
    uint16_t *lds = reinterpret_cast<uint16_t *>(lds_f);
    constexpr int NT_ = TWO ? 3 : 2;                 // tiles per stage
    constexpr int OPS = 4 * NT_;                     // load instructions per stage per wave
    const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int wm = (w >> 1) * 64, wn = (w & 1) * 64;

#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            acc[i][j] = f16v{};
            if (TWO) acc2[i][j] = f16v{};
        }
    float sa = 0.f, sb = 0.f;
    const int64_t nk = (g.K + BK16 - 1) / BK16;
    auto stage = [&](int s) { return lds + s * NT_ * DTILE; };
    auto issue = [&](int64_t kt) {
        uint16_t *st = stage((int)(kt % DMA_STAGES));
        dma_rows(A, g.lda, m0, g.M, kt * BK16, g.K, st);
        if (BNN) dma_krows(B, g.ldb, kt * BK16, g.K, n0, g.N, st + DTILE);
        else dma_rows(B, g.ldb, n0, g.N, kt * BK16, g.K, st + DTILE);
        if (TWO) dma_rows(A2, g.lda2, m0, g.M, kt * BK16, g.K, st + 2 * DTILE);
    };

    for (int s = 0; s < DMA_STAGES - 1; ++s)
        if (s < nk) issue(s);
    for (int64_t kt = 0; kt < nk; ++kt) {
        // the loads of step kt are complete once at most those of the later
        // stages already issued (kt + 1 .. min(kt + NS - 2, nk - 1)) remain
        wait_stages<OPS, DMA_STAGES - 2>(nk - 1 - kt);
        __builtin_amdgcn_s_barrier();
        if (kt + DMA_STAGES - 1 < nk) issue(kt + DMA_STAGES - 1);
        uint16_t *cur = stage((int)(kt % DMA_STAGES));
        const uint16_t *As = cur, *Bs = cur + DTILE, *As2 = cur + 2 * DTILE;
        const int64_t kvalid = g.K - kt * BK16;
        if (kvalid < BK16) {
            zero_rows_tail(cur, (int)kvalid);
            if (BNN) zero_krows_tail(cur + DTILE, (int)kvalid);
            else zero_rows_tail(cur + DTILE, (int)kvalid);
            if (TWO) zero_rows_tail(cur + 2 * DTILE, (int)kvalid);
            __builtin_amdgcn_s_waitcnt(0xc07f);    // lgkmcnt(0): the zeros are in LDS
            __builtin_amdgcn_s_barrier();
        }
#pragma unroll
        for (int kk = 0; kk < BK16; kk += 16) {
            const int c = (kk >> 3) + (l >> 5);
            const bf8v a0 = frag_rows(As, wm + (l & 31), c), a1 = frag_rows(As, wm + 32 + (l & 31), c);
            bf8v b0, b1;
            if (BNN) {
                b0 = frag_krows(Bs, kk, wn);
                b1 = frag_krows(Bs, kk, wn + 32);
            } else {
                b0 = frag_rows(Bs, wn + (l & 31), c);
                b1 = frag_rows(Bs, wn + 32 + (l & 31), c);
            }
            acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b0, acc[0][0], 0, 0, 0);
            acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b1, acc[0][1], 0, 0, 0);
            acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b0, acc[1][0], 0, 0, 0);
            acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b1, acc[1][1], 0, 0, 0);
            if (TWO) {
                const bf8v c0 = frag_rows(As2, wm + (l & 31), c), c1 = frag_rows(As2, wm + 32 + (l & 31), c);
                acc2[0][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(c0, b0, acc2[0][0], 0, 0, 0);
                acc2[0][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(c0, b1, acc2[0][1], 0, 0, 0);
                acc2[1][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(c1, b0, acc2[1][0], 0, 0, 0);
                acc2[1][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(c1, b1, acc2[1][1], 0, 0, 0);
            }
        }
        if (threadIdx.x < 128) {
            if (sqa) sa += row_sq_dma(As, threadIdx.x);
            if (sqb && !BNN) sb += row_sq_dma(Bs, threadIdx.x);
        }
    }
    // every wave is done reading LDS before the caller reuses it
    lds_barrier();
    if (threadIdx.x < 128) {
        if (sqa) *sqa_out = sa;
        if (sqb) *sqb_out = sb;
    }
}

// Dispatch on the operand types: both bf16 -> bf16 matrix cores (pipelined
// asynchronous loads when every operand has 16-byte aligned rows, register
// staging otherwise), else fp32 matrix cores on widened operands.
template <typename TA, typename TB, bool BNN, bool TWO, int NS>
__device__ __forceinline__ void block_mma_any(const GemmArgs &g, int64_t m0, int64_t n0, bool veca, bool vecb,
                                              float *lds, f16v acc[2][2], f16v acc2[2][2], bool sqa,
                                              float *sqa_out, bool sqb, float *sqb_out) {
    if constexpr (sizeof(TA) == 2 && sizeof(TB) == 2) {
        if (g.dma)
            block_mma_bf16_dma<BNN, TWO, NS>(g, m0, n0, lds, acc, acc2, sqa, sqa_out, sqb, sqb_out);
        else
            block_mma_bf16<BNN, TWO>(g, m0, n0, veca, vecb, lds, acc, acc2, sqa, sqa_out, sqb, sqb_out);
    } else {
        block_mma<TA, TB, BNN, TWO>(g, m0, n0, veca, vecb, lds, acc, acc2, sqa, sqa_out, sqb, sqb_out);
    }
}

// LDS floats for the operand staging of a launch: the pipelined bf16 loop's
// stages when it runs (dma), the register-staged loop's buffers otherwise.
template <typename TA, typename TB, bool TWO, int NS>
__host__ __device__ size_t stage_lds_floats(bool dma) {
    if constexpr (sizeof(TA) == 2 && sizeof(TB) == 2)
        if (dma) return dma_lds_floats<TWO, NS>();
    return mma_lds_floats<TA, TB, TWO>();
}

// Pipeline depth of the asynchronous loop: 4 stages (128 KiB) for a single
// product, 3 (144 KiB) when a second A operand is staged.
template <bool TWO>
constexpr int store_stages() { return TWO ? 3 : 4; }
constexpr int SWEEP_STAGES = 2;

// XCD-aware tile order: work-group ids are dealt to the 8 XCDs round-robin,
// so logical tile L is given to ids that share an XCD for consecutive L.
// Consecutive logical tiles share their A row block (n varies fastest), which
// then stays in that XCD's L2.
__device__ __forceinline__ int64_t logical_tile(int64_t total) {
    const int64_t per = (total + 7) / 8;
    const int64_t w = blockIdx.x;
    return (w & 7) * per + (w >> 3);
}

// --------------------------------------------------------- epilogue: store

template <typename TA, typename TB, typename TO, bool BNN, bool BIND>
__global__ void __launch_bounds__(NTHR) gemm_store_kernel(GemmArgs g, int veca, int vecb) {
    extern __shared__ float lds[];
    const int64_t nM = (g.M + BM - 1) / BM, nN = (g.N + BN - 1) / BN;
    const int64_t L = logical_tile(nM * nN);
    if (L >= nM * nN) return;
    const int64_t m0 = (L / nN) * BM, n0 = (L % nN) * BN;
    f16v acc[2][2], acc2[2][2];
    const bool sqa = (g.rownorm2 != nullptr) && (n0 == 0);
    float sa = 0.f, sb = 0.f;
    block_mma_any<TA, TB, BNN, BIND, store_stages<BIND>()>(g, m0, n0, veca, vecb, lds, acc, acc2, sqa, &sa, false,
                                                          &sb);
    if (sqa && threadIdx.x < 128 && m0 + threadIdx.x < g.M) g.rownorm2[m0 + threadIdx.x] = sa;

    TO *C = static_cast<TO *>(g.C);
    const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int wm = (w >> 1) * 64, wn = (w & 1) * 64;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int64_t col = n0 + wn + 32 * j + (l & 31);
            if (col >= g.N) continue;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t row = m0 + wm + 32 * i + acc_row(r, l);
                if (row < g.M) {
                    float v = acc[i][j][r];
                    if (BIND) v *= acc2[i][j][r];
                    st_f32<TO>(C, row * g.ldc + col, v);
                }
            }
        }
}

// ------------------------------------------------- epilogue: scores
//
// Similarity / attention when the scores (or weights) are written anyway:
// out = scale * acc / (||x|| ||c||) for cosine, scale * acc for dot (scale
// includes beta for attention); the row pass (argmax, or softmax in place)
// follows as its own launch.  Row norms come from qnorm2 or from the A tile,
// column norms from cnorm or from the B tile, both accumulated by the main
// loop.

template <typename TA, typename TB>
__global__ void __launch_bounds__(NTHR) gemm_scores_kernel(GemmArgs g, int veca, int vecb) {
    extern __shared__ float lds[];
    const int64_t nM = (g.M + BM - 1) / BM, nN = (g.N + BN - 1) / BN;
    const int64_t L = logical_tile(nM * nN);
    if (L >= nM * nN) return;
    const int64_t m0 = (L / nN) * BM, n0 = (L % nN) * BN;
    f16v acc[2][2], acc2[2][2];
    const bool sqa = g.cosine && g.qnorm2 == nullptr, sqb = g.cosine && g.cnorm == nullptr;
    float sa = 0.f, sb = 0.f;
    block_mma_any<TA, TB, false, false, store_stages<false>()>(g, m0, n0, veca, vecb, lds, acc, acc2, sqa, &sa,
                                                               sqb, &sb);
    // the main loop has passed a barrier after its last LDS read
    float *rq = lds, *cn = lds + BM;
    const int t = threadIdx.x;
    if (t < 128) {
        float q = g.scale;
        if (g.cosine) {
            const float n2 = g.qnorm2 ? ((m0 + t < g.M) ? g.qnorm2[m0 + t] : 1.f) : sa;
            q = (n2 > 0.f) ? g.scale / sqrtf(n2) : 0.f;
        }
        rq[t] = q;
        float c = 1.f;
        if (g.cosine) {
            const float cc = g.cnorm ? ((n0 + t < g.N) ? g.cnorm[n0 + t] : 1.f) : sqrtf(sb);
            c = (cc > 0.f) ? 1.f / cc : 0.f;
        }
        cn[t] = c;
    }
    lds_barrier();
    float *C = static_cast<float *>(g.C);
    const int l = t & 63, w = t >> 6;
    const int wm = (w >> 1) * 64, wn = (w & 1) * 64;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int cl = wn + 32 * j + (l & 31);
            const int64_t col = n0 + cl;
            if (col >= g.N) continue;
            const float cf = cn[cl];
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int rl = wm + 32 * i + acc_row(r, l);
                const int64_t row = m0 + rl;
                if (row < g.M) C[row * g.ldc + col] = acc[i][j][r] * rq[rl] * cf;
            }
        }
}

// ---------------------------------------- epilogue: similarity / softmax
//
// One work-group owns a 128-row block and sweeps every 128-column block of
// the codebook.  Scores of a column block are parked in LDS, where one pair
// of threads per row folds them into the row's running state: (max, argmax)
// for similarity, (max, sum of exp) for softmax.  Softmax rows are finished
// by a second sweep over the row block's outputs, which that same work-group
// has just written (still in L2).

constexpr int SS_STRIDE = BN + 1;

template <typename TA, typename TB, bool SOFTMAX>
__global__ void __launch_bounds__(NTHR) gemm_rowsweep_kernel(GemmArgs g, int veca, int vecb) {
    extern __shared__ float lds[];
    float *ss = lds + stage_lds_floats<TA, TB, false, SWEEP_STAGES>(g.dma);   // scores [BM][SS_STRIDE]
    float *rq = ss + BM * SS_STRIDE;               // 1 / ||x|| per row (or 1)
    float *cn = rq + BM;                           // 1 / ||c|| per column (or 1)
    const int64_t nM = (g.M + BM - 1) / BM;
    const int64_t L = logical_tile(nM);
    if (L >= nM) return;
    const int64_t m0 = L * BM;
    const int64_t nN = (g.N + BN - 1) / BN;
    const int t = threadIdx.x;
    const int l = t & 63, w = t >> 6;
    const int wm = (w >> 1) * 64, wn = (w & 1) * 64;
    float *out = static_cast<float *>(g.C);
    const bool vec_out = (reinterpret_cast<uintptr_t>(out) & 15) == 0 && g.ldc % 4 == 0;

    // running row state, identical in both threads of a pair
    const int prow = t >> 1, half = t & 1;
    float run_max = -INFINITY, run_sum = 0.f;
    int run_idx = 0;

    for (int64_t nt = 0; nt < nN; ++nt) {
        const int64_t n0 = nt * BN;
        f16v acc[2][2], acc2[2][2];
        const bool sqa = g.cosine && g.qnorm2 == nullptr && nt == 0;
        const bool sqb = g.cosine && g.cnorm == nullptr;
        float sa = 0.f, sb = 0.f;
        block_mma_any<TA, TB, false, false, SWEEP_STAGES>(g, m0, n0, veca, vecb, lds, acc, acc2, sqa, &sa, sqb, &sb);
        if (t < 128) {
            if (nt == 0) {
                float q = 1.f;
                if (g.cosine) {
                    float n2 = g.qnorm2 ? ((m0 + t < g.M) ? g.qnorm2[m0 + t] : 1.f) : sa;
                    q = (n2 > 0.f) ? 1.f / sqrtf(n2) : 0.f;
                }
                rq[t] = q;
            }
            float c = 1.f;
            if (g.cosine) {
                float cc = g.cnorm ? ((n0 + t < g.N) ? g.cnorm[n0 + t] : 1.f) : sqrtf(sb);
                c = (cc > 0.f) ? 1.f / cc : 0.f;
            }
            cn[t] = c;
        }
        lds_barrier();
        // scores -> LDS and (optionally) global
        const float mul = SOFTMAX ? g.scale * g.beta : g.scale;
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int cl = wn + 32 * j + (l & 31);
                const int64_t col = n0 + cl;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int rl = wm + 32 * i + acc_row(r, l);
                    const float v = mul * acc[i][j][r] * rq[rl] * cn[cl];
                    ss[rl * SS_STRIDE + cl] = (col < g.N) ? v : -INFINITY;
                }
            }
        lds_barrier();
        if (SOFTMAX || g.write_out) {
            // the block's scores leave from the LDS tile, four columns per
            // thread: rows t / 32 + 8 q, columns 4 (t % 32) .. + 3
            const int c4 = 4 * (t & 31);
            const int64_t col = n0 + c4;
            for (int q = 0; q < 16; ++q) {
                const int rl = (t >> 5) + 8 * q;
                const int64_t row = m0 + rl;
                if (row >= g.M || col >= g.N) continue;
                const float *src = ss + rl * SS_STRIDE + c4;
                float *dst = out + row * g.ldc + col;
                if (vec_out && col + 4 <= g.N) {
                    *reinterpret_cast<f4v *>(dst) = f4v{src[0], src[1], src[2], src[3]};
                } else {
                    for (int e = 0; e < 4 && col + e < g.N; ++e) dst[e] = src[e];
                }
            }
        }
        // fold this column block into the running row state
        const int ncols = (int)((g.N - n0 < BN) ? (g.N - n0) : BN);
        float bm = -INFINITY, bs = 0.f;
        int bi = 0;
        for (int c = half; c < ncols; c += 2) {
            float v = ss[prow * SS_STRIDE + c];
            if (v > bm) { bm = v; bi = c; }
        }
        if (SOFTMAX) {
            for (int c = half; c < ncols; c += 2) bs += __expf(ss[prow * SS_STRIDE + c] - bm);
        }
        float om = __shfl_xor(bm, 1), os = __shfl_xor(bs, 1);
        int oi = __shfl_xor(bi, 1);
        if (SOFTMAX) {
            float nm = fmaxf(bm, om);
            float tsum = (bm == -INFINITY ? 0.f : bs * __expf(bm - nm)) +
                         (om == -INFINITY ? 0.f : os * __expf(om - nm));
            float m2 = fmaxf(run_max, nm);
            run_sum = (run_max == -INFINITY ? 0.f : run_sum * __expf(run_max - m2)) +
                      (nm == -INFINITY ? 0.f : tsum * __expf(nm - m2));
            run_max = m2;
        } else {
            // lowest column index wins a tie
            if (om > bm || (om == bm && oi < bi)) { bm = om; bi = oi; }
            if (bm > run_max) { run_max = bm; run_idx = (int)(n0 + bi); }
        }
        lds_barrier();   // ss and the staged tiles are reused by the next block
    }

    if (!SOFTMAX) {
        if (g.argmax && half == 0 && m0 + prow < g.M) g.argmax[m0 + prow] = run_idx;
        return;
    }
    // second sweep: normalise the row block
    float *rmax = rq, *rinv = cn;   // reuse
    if (half == 0) {
        rmax[prow] = run_max;
        rinv[prow] = 1.f / run_sum;
    }
    // the second sweep reads scores that other threads stored to global
    // memory: a full barrier (their stores complete and visible)
    __syncthreads();
    softmax_rows(out, g.ldc, m0, (g.M - m0 < BM) ? (g.M - m0) : BM, g.N, rmax, rinv, vec_out, NTHR);
}

template <typename K>
hipError_t launch_with_lds(K kernel, dim3 grid, size_t lds, hipStream_t s, const GemmArgs &a, int veca,
                           int vecb) {
    if (lds > 65536) {
        hipError_t e = raise_lds_limit(reinterpret_cast<const void *>(kernel), lds);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(kernel, grid, dim3(NTHR), lds, s, a, veca, vecb);
    return hipGetLastError();
}

template <typename TA, typename TB, typename TO>
hipError_t dispatch_store(bool b_nn, bool bind, const GemmArgs &a, bool veca, bool vecb,
                          hipStream_t s) {
    const int64_t nM = (a.M + BM - 1) / BM, nN = (a.N + BN - 1) / BN;
    const int64_t total = nM * nN;
    const dim3 grid((unsigned)(8 * ((total + 7) / 8)));
    const size_t lds = (bind ? stage_lds_floats<TA, TB, true, store_stages<true>()>(a.dma)
                             : stage_lds_floats<TA, TB, false, store_stages<false>()>(a.dma)) * sizeof(float);
    if (b_nn) {
        if (bind) return launch_with_lds(gemm_store_kernel<TA, TB, TO, true, true>, grid, lds, s, a, veca, vecb);
        return launch_with_lds(gemm_store_kernel<TA, TB, TO, true, false>, grid, lds, s, a, veca, vecb);
    }
    if (bind) return launch_with_lds(gemm_store_kernel<TA, TB, TO, false, true>, grid, lds, s, a, veca, vecb);
    return launch_with_lds(gemm_store_kernel<TA, TB, TO, false, false>, grid, lds, s, a, veca, vecb);
}

template <typename TA, typename TB>
hipError_t dispatch_scores(bool softmax, const GemmArgs &a_in, bool veca, bool vecb, hipStream_t s) {
    GemmArgs a = a_in;
    if (softmax) a.scale = a_in.scale * a_in.beta;   // the softmax acts on beta * score
    const int64_t nM = (a.M + BM - 1) / BM, nN = (a.N + BN - 1) / BN;
    const dim3 grid((unsigned)(8 * ((nM * nN + 7) / 8)));
    const size_t lds = stage_lds_floats<TA, TB, false, store_stages<false>()>(a.dma) * sizeof(float);
    hipError_t e = launch_with_lds(gemm_scores_kernel<TA, TB>, grid, lds, s, a, veca, vecb);
    if (e != hipSuccess) return e;
    return launch_rows_pass(softmax, static_cast<float *>(a.C), a.ldc, a.M, a.N, softmax ? nullptr : a.argmax, s);
}

template <typename TA, typename TB>
hipError_t dispatch_rowsweep(bool softmax, const GemmArgs &a, bool veca, bool vecb, hipStream_t s) {
    const int64_t nM = (a.M + BM - 1) / BM;
    const dim3 grid((unsigned)(8 * ((nM + 7) / 8)));
    const size_t lds = (stage_lds_floats<TA, TB, false, SWEEP_STAGES>(a.dma) + BM * SS_STRIDE + 2 * BM) * sizeof(float);
    if (softmax) return launch_with_lds(gemm_rowsweep_kernel<TA, TB, true>, grid, lds, s, a, veca, vecb);
    return launch_with_lds(gemm_rowsweep_kernel<TA, TB, false>, grid, lds, s, a, veca, vecb);
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Vector loads along the contiguous dimension need a 16-byte aligned base, a
// leading dimension that keeps every row 16-byte aligned, and a contiguous
// extent that is a whole number of vectors.
bool vec_ok(const void *p, gs_dtype t, int64_t ld, int64_t extent) {
    const int64_t per = (t == GS_BF16) ? 8 : 4;
    return aligned16(p) && (ld % per == 0) && (extent % per == 0);
}

}  // namespace

// Kernels whose dynamic LDS exceeds the default 64 KiB limit raise it once,
// before their first launch, to the whole 160 KiB of a CU: a kernel's
// launches differ in size (pipelined or register-staged operands), and the
// attribute only permits; occupancy follows each launch's own size.
hipError_t raise_lds_limit(const void *kernel, size_t lds) {
    constexpr size_t LDS_MAX = 160 * 1024;
    static std::mutex mu;
    static std::unordered_set<const void *> done;
    if (lds > LDS_MAX) return hipErrorInvalidValue;
    std::lock_guard<std::mutex> lock(mu);
    if (done.count(kernel)) return hipSuccess;
    hipError_t e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)LDS_MAX);
    if (e == hipSuccess) done.insert(kernel);
    return e;
}

hipError_t launch_gemm(gs_dtype ta, gs_dtype tb, gs_dtype tout, bool b_nn, Epi epi,
                       const GemmArgs &a_in, hipStream_t s) {
    if (a_in.M == 0 || a_in.N == 0) return hipSuccess;
    GemmArgs a = a_in;
    // asynchronous-load loops: operands of one type, every row 16-byte aligned
    const bool same = (ta == GS_BF16 && tb == GS_BF16) || (ta == GS_F32 && tb == GS_F32);
    const int64_t per = (ta == GS_BF16) ? 8 : 4;
    auto rows16 = [&](const void *p, int64_t ld) { return aligned16(p) && ld % per == 0; };
    const bool rows_ok = same && rows16(a.A, a.lda) && rows16(a.B, a.ldb) &&
                         (epi != EPI_BIND || rows16(a.A2, a.lda2));
    a.dma = rows_ok && ta == GS_BF16;   // the 128 x 128 pipelined loop is bf16 only
    if (epi == EPI_STORE && rows_ok && gemm256_fits(ta, a, b_nn)) return launch_gemm256(ta, tout, b_nn, a, s);
    if (epi == EPI_BIND && rows_ok && tout == GS_F32 && gemm256_fits(ta, a, b_nn)) {
        // bound product on the large tiles: X = T Q, then X = X .* (T2 Q) in
        // the second product's epilogue (fp32 X holds the first factor exactly)
        GemmArgs first = a, second = a;
        first.A2 = nullptr;
        second.A = a.A2;
        second.lda = a.lda2;
        second.A2 = nullptr;
        second.mul_out = 1;
        hipError_t e = launch_gemm256(ta, tout, b_nn, first, s);
        if (e != hipSuccess) return e;
        return launch_gemm256(ta, tout, b_nn, second, s);
    }
    bool veca = vec_ok(a.A, ta, a.lda, a.K);
    if (epi == EPI_BIND) veca = veca && vec_ok(a.A2, ta, a.lda2, a.K);
    const bool vecb = b_nn ? vec_ok(a.B, tb, a.ldb, a.N) : vec_ok(a.B, tb, a.ldb, a.K);
    const bool bf_a = ta == GS_BF16, bf_b = tb == GS_BF16, bf_o = tout == GS_BF16;
    if (epi == EPI_STORE || epi == EPI_BIND) {
        const bool bind = epi == EPI_BIND;
        if (!bf_a && !bf_b && !bf_o) return dispatch_store<float, float, float>(b_nn, bind, a, veca, vecb, s);
        if (!bf_a && !bf_b && bf_o) return dispatch_store<float, float, bf16_t>(b_nn, bind, a, veca, vecb, s);
        if (bf_a && bf_b && !bf_o) return dispatch_store<bf16_t, bf16_t, float>(b_nn, bind, a, veca, vecb, s);
        if (bf_a && bf_b && bf_o) return dispatch_store<bf16_t, bf16_t, bf16_t>(b_nn, bind, a, veca, vecb, s);
        if (!bf_a && bf_b && !bf_o) return dispatch_store<float, bf16_t, float>(b_nn, bind, a, veca, vecb, s);
        if (!bf_a && bf_b && bf_o) return dispatch_store<float, bf16_t, bf16_t>(b_nn, bind, a, veca, vecb, s);
        return hipErrorInvalidValue;
    }
    const bool sm = epi == EPI_SOFTMAX;
    // a few query rows: the K range is split over whole work-groups instead
    // of walked by one tile
    if (!b_nn && (sm || a.write_out) && a.M <= FEW_ROWS && ta == tb) return launch_few_rows(ta, a, sm, s);
    // scores written, or whole rows in one tile (the row results come from
    // the product's epilogue): the large tiles
    if (rows_ok && !b_nn && (sm || a.write_out || a.N <= 256) && gemm256_fits(ta, a, false))
        return launch_scores256(ta, a, sm, s);
    if (rows_ok && !b_nn && sweep256_fits(ta, a)) return launch_sweep256(ta, sm, a, s);
    // scores or weights written anyway: product with a scaled epilogue, then
    // the row pass; argmax alone: the row sweep (no score matrix in memory)
    if ((sm || a.write_out) && !b_nn) {
        if (!bf_a && !bf_b) return dispatch_scores<float, float>(sm, a, veca, vecb, s);
        if (bf_a && bf_b) return dispatch_scores<bf16_t, bf16_t>(sm, a, veca, vecb, s);
    }
    if (!bf_a && !bf_b) return dispatch_rowsweep<float, float>(sm, a, veca, vecb, s);
    if (bf_a && bf_b) return dispatch_rowsweep<bf16_t, bf16_t>(sm, a, veca, vecb, s);
    return hipErrorInvalidValue;
}

}  // namespace gs
