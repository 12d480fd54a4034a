// Streaming kernels for small codebooks (M <= 32, r <= 32): probability
// vectorisation, similarity (+ argmax), attention score, and the fused
// soft-selection pass over several codebooks in one launch.
//
// At these sizes an output row costs at most M*r multiply-adds against
// 4(M + r) bytes of traffic.  One thread owns one batch row.  Batch tiles move
// between HBM and LDS with coalesced (vector, when rows are contiguous)
// accesses; each thread reads its own row from the tile.
//
// The codebook coordinates R are widened once per work-group into a
// zero-padded fp32 MB x MB block in LDS and read as broadcast 16-byte
// vectors (measured faster here than scalar loads into SGPRs, whose address
// and latency overhead outweighed the saved LDS traffic).  Loops run to a
// compile-time bound MB >= M (8, 16, 24 or 32) with padded terms contributing
// exact zeros.
#include "gs_internal.h"

namespace gs {
namespace {


// Batch rows (and threads) per work-group of the separate calls: 256, or 128
// for the widest codebooks (keeps the row tile and codebook block within
// 64 KiB of LDS).
template <int MB> constexpr int rows_of() { return MB <= 48 ? 256 : 128; }
constexpr int MAXK = SOFT_MAX_M;          // widest row of the fused soft selection (32)

enum Mode { MODE_P2V = 0, MODE_SIM = 1, MODE_ATT = 2 };

typedef float f4v __attribute__((ext_vector_type(4)));
typedef float gs16v __attribute__((ext_vector_type(16)));

__device__ __forceinline__ bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

// Four consecutive elements as fp32 (16-byte aligned fp32, 8-byte aligned bf16).
__device__ __forceinline__ f4v ld4(const float *p) { return *reinterpret_cast<const f4v *>(p); }
__device__ __forceinline__ f4v ld4(const bf16_t *p) {
    const uint2 u = *reinterpret_cast<const uint2 *>(p);
    return f4v{__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
               __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u)};
}
__device__ __forceinline__ void st4(float *p, f4v v) { *reinterpret_cast<f4v *>(p) = v; }
__device__ __forceinline__ void st4(bf16_t *p, f4v v) {
    uint2 u;
    u.x = (uint32_t)f32_to_bf16(v[0]) | ((uint32_t)f32_to_bf16(v[1]) << 16);
    u.y = (uint32_t)f32_to_bf16(v[2]) | ((uint32_t)f32_to_bf16(v[3]) << 16);
    *reinterpret_cast<uint2 *>(p) = u;
}

// Output stores: fp32 outputs are written with streaming (non-temporal)
// stores, which leave the cache for data the kernel never reads back.
__device__ __forceinline__ void st4_out(float *p, f4v v) { __builtin_nontemporal_store(v, reinterpret_cast<f4v *>(p)); }
__device__ __forceinline__ void st4_out(bf16_t *p, f4v v) { st4(p, v); }
template <typename T> __device__ __forceinline__ void st1_out(T *p, int64_t i, float v) { st_f32<T>(p, i, v); }
template <> __device__ __forceinline__ void st1_out<float>(float *p, int64_t i, float v) {
    __builtin_nontemporal_store(v, p + i);
}

// Smallest supported padded size for a codebook of M entries.
__host__ __device__ __forceinline__ int pad_of(int64_t M) { return M <= 8 ? 8 : M <= 16 ? 16 : M <= 24 ? 24 : 32; }
// ... for the separate calls, up to 64 entries.
__host__ __device__ __forceinline__ int pad_small(int64_t M) { return M <= 32 ? pad_of(M) : M <= 48 ? 48 : 64; }

// ------------------------------------------------------------- tile moves
//
// A tile holds rows [b0, b0 + nrow) x [0, w) densely (row stride w): tile
// element e is matrix element (e / w, e % w).  With contiguous rows
// (ld == w) and an aligned base, tile and matrix are one linear range moved
// as 4-element vectors; otherwise element by element with the row and column
// advanced incrementally.  NT threads take part, thread t of them (by
// default the work-group's threads).

template <typename T, int NT, int WMAX = MAXK>
__device__ __forceinline__ void tile_load(const T *__restrict__ g, int64_t ld, int64_t b0, int nrow, int w,
                                          float *tile, int t = threadIdx.x) {
    const int n = nrow * w;
    const T *base = g + b0 * ld;
    if constexpr (sizeof(T) == 2) if (ld == w && aligned16(base)) {
        // bf16: 16-byte pieces of eight values
        typedef unsigned int u4v __attribute__((ext_vector_type(4)));
        const int n8 = n >> 3;
        constexpr int V = (NT * WMAX / 8 + NT - 1) / NT;
        u4v v[V];
#pragma unroll
        for (int i = 0; i < V; ++i) {
            const int e8 = t + i * NT;
            if (e8 < n8) v[i] = *reinterpret_cast<const u4v *>(base + 8 * e8);
        }
#pragma unroll
        for (int i = 0; i < V; ++i) {
            const int e8 = t + i * NT;
            if (e8 < n8) {
                const u4v u = v[i];
                st4(tile + 8 * e8, f4v{__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                                       __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u)});
                st4(tile + 8 * e8 + 4, f4v{__uint_as_float(u.z << 16), __uint_as_float(u.z & 0xffff0000u),
                                           __uint_as_float(u.w << 16), __uint_as_float(u.w & 0xffff0000u)});
            }
        }
        for (int e = 8 * n8 + t; e < n; e += NT) tile[e] = ld_f32<T>(base, e);
        return;
    }
    if (ld == w && aligned16(base)) {
        const int n4 = n >> 2;
        constexpr int V = (NT * WMAX / 4 + NT - 1) / NT;
        f4v v[V];
#pragma unroll
        for (int i = 0; i < V; ++i) {
            const int e4 = t + i * NT;
            if (e4 < n4) v[i] = ld4(base + 4 * e4);
        }
#pragma unroll
        for (int i = 0; i < V; ++i) {
            const int e4 = t + i * NT;
            if (e4 < n4) st4(tile + 4 * e4, v[i]);
        }
        const int e = 4 * n4 + t;
        if (e < n) tile[e] = ld_f32<T>(base, e);
        return;
    }
    int row = t / w, col = t - (t / w) * w;
    const int dq = NT / w, dc = NT - (NT / w) * w;
    for (int i0 = 0; i0 * NT < n; i0 += 8) {   // 8 loads in flight per chunk
        float v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int e = t + (i0 + i) * NT;
            v[i] = (e < n) ? ld_f32<T>(base, (int64_t)row * ld + col) : 0.f;
            row += dq;
            col += dc;
            if (col >= w) { col -= w; ++row; }
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int e = t + (i0 + i) * NT;
            if (e < n) tile[e] = v[i];
        }
    }
}

template <typename T, int NT>
__device__ __forceinline__ void tile_store(T *__restrict__ g, int64_t ld, int64_t b0, int nrow, int w,
                                           const float *tile, int t = threadIdx.x) {
    const int n = nrow * w;
    T *base = g + b0 * ld;
    if (ld == w && aligned16(base)) {
        const int n4 = n >> 2;
        for (int e4 = t; e4 < n4; e4 += NT) st4_out(base + 4 * e4, *reinterpret_cast<const f4v *>(tile + 4 * e4));
        const int e = 4 * n4 + t;
        if (e < n) st1_out<T>(base, e, tile[e]);
        return;
    }
    int row = t / w, col = t - (t / w) * w;
    const int dq = NT / w, dc = NT - (NT / w) * w;
    for (int e = t; e < n; e += NT) {
        st1_out<T>(base, (int64_t)row * ld + col, tile[e]);
        row += dq;
        col += dc;
        if (col >= w) { col -= w; ++row; }
    }
}

// --------------------------------------------------- codebook row sources

// Zero-padded MB x MB fp32 block in LDS.
template <int MB>
struct LdsRows {
    const float *Rs;
    __device__ __forceinline__ void row(int j, float rr[MB]) const {
        const f4v *p = reinterpret_cast<const f4v *>(Rs + j * MB);
#pragma unroll
        for (int q = 0; q < MB / 4; ++q) {
            const f4v v = p[q];
            rr[4 * q] = v[0]; rr[4 * q + 1] = v[1]; rr[4 * q + 2] = v[2]; rr[4 * q + 3] = v[3];
        }
    }
};

// Reciprocal codebook norms for cosine scores (ones for dot), zeros beyond M.
// Without given norms they are ||R_j||, summed in fp32 from the source rows.
template <typename T, int NT>
__device__ __forceinline__ void stage_norms(const T *R, int64_t ldr, int M, int r, const float *cnorm,
                                            bool cosine, int MB, float *Rn) {
    for (int j = threadIdx.x; j < MB; j += NT) {
        float c = 0.f;
        if (j < M) {
            c = 1.f;
            if (cosine) {
                float n;
                if (cnorm) {
                    n = cnorm[j];
                } else {
                    float s2 = 0.f;
                    for (int k = 0; k < r; ++k) {
                        const float v = ld_f32<T>(R, (int64_t)j * ldr + k);
                        s2 += v * v;
                    }
                    n = sqrtf(s2);
                }
                c = (n > 0.f) ? 1.f / n : 0.f;
            }
        }
        Rn[j] = c;
    }
}

// ---------------------------------------------------------------- row ops

// out[k] = sum_{j < M} p_j R[j, k], p_j read from the thread's own tile row.
template <int MB, class Rows>
__device__ __forceinline__ void row_prob2vec(const float *prow, int M, const Rows &R, float out[MB]) {
#pragma unroll
    for (int k = 0; k < MB; ++k) out[k] = 0.f;
#pragma unroll 2
    for (int j = 0; j < M; ++j) {
        float rr[MB];
        R.row(j, rr);
        const float pj = prow[j];
#pragma unroll
        for (int k = 0; k < MB; ++k) out[k] += pj * rr[k];
    }
}

// srow[j] = mul * <x, R_j> * q * Rn[j] for j < M, into the thread's own tile
// row; the row maximum and its lowest index.
template <int MB, class Rows>
__device__ __forceinline__ void row_scores(const float x[MB], int M, const Rows &R, const float *Rn, float mul,
                                           float q, float *srow, float &best, int &bi) {
    best = -INFINITY;
    bi = 0;
#pragma unroll 2
    for (int j = 0; j < M; ++j) {
        float rr[MB];
        R.row(j, rr);
        float d = 0.f;
#pragma unroll
        for (int k = 0; k < MB; ++k) d += x[k] * rr[k];
        const float sj = mul * d * q * Rn[j];
        srow[j] = sj;
        if (sj > best) { best = sj; bi = j; }
    }
}

// In-place softmax of f * srow[0..M), given max_j f * srow[j] = mx.
__device__ __forceinline__ void row_softmax(float *srow, int M, float f, float mx) {
    float z = 0.f;
    for (int j = 0; j < M; ++j) {
        const float e = __expf(f * srow[j] - mx);
        srow[j] = e;
        z += e;
    }
    const float iz = 1.f / z;
    for (int j = 0; j < M; ++j) srow[j] *= iz;
}

template <int MB>
__device__ __forceinline__ void regs_to_tile(const float v[MB], int w, float *tile) {
#pragma unroll
    for (int k = 0; k < MB; ++k)
        if (k < w) tile[threadIdx.x * w + k] = v[k];
}

template <int MB>
__device__ __forceinline__ void tile_to_regs(const float *tile, int w, float v[MB]) {
#pragma unroll
    for (int k = 0; k < MB; ++k) v[k] = (k < w) ? tile[threadIdx.x * w + k] : 0.f;
}

// ------------------------------------------------------- separate calls

// Matrix-core product of the wave's 64 tile rows (two blocks of 32, rows
// 64 (t / 64) + 32 b + i, row stride W) with a K x 32 operand:
// acc[b][g] = sum_k A[32 b + i][k] B[k][l % 32] for row i = 8 (g / 4) +
// 4 (l / 32) + g % 4 (v_mfma_f32_32x32x2f32).  Step kk pairs k = kk (lanes
// 0..31) and k = kk + KH (lanes 32..63); bk[kk] is this lane's B[k][l % 32]
// (zero for k >= K), and A elements at k >= K are zeroed.  Rows past the
// tile's valid rows give results that are never stored.
template <int KH>
__device__ __forceinline__ void wave_rows_mm(const float *tile, int W, int K, const float (&bk)[KH],
                                             gs16v acc[2]) {
    const int t = threadIdx.x, l = t & 63, c = l & 31, h = l >> 5;
#pragma unroll
    for (int b = 0; b < 2; ++b) {
        const float *arow = tile + ((t & ~63) + 32 * b + c) * W;
        acc[b] = gs16v{};
#pragma unroll
        for (int kk = 0; kk < KH; ++kk) {
            const int k = kk + KH * h;
            const float x = (k < K) ? arow[k] : 0.f;
            acc[b] = __builtin_amdgcn_mfma_f32_32x32x2f32(x, bk[kk], acc[b], 0, 0, 0);
        }
    }
}

// The results of wave_rows_mm to the tile at row stride W, columns < ncol.
__device__ __forceinline__ void wave_rows_out(const gs16v acc[2], int W, int ncol, float *tile) {
    const int t = threadIdx.x, l = t & 63, c = l & 31, h = l >> 5;
    if (c >= ncol) return;
#pragma unroll
    for (int b = 0; b < 2; ++b) {
        float *drow = tile + ((t & ~63) + 32 * b + 4 * h) * W + c;
#pragma unroll
        for (int g = 0; g < 16; ++g) drow[(8 * (g >> 2) + (g & 3)) * W] = acc[b][g];
    }
}

template <typename TI, typename TO, int MODE, int MB, class Rows>
__device__ __forceinline__ void small_body(const SmallArgs &a, const Rows &R, const float *Rn, float *tile) {
    constexpr int NR = rows_of<MB>();
    const int t = threadIdx.x;
    const int64_t b0 = (int64_t)blockIdx.x * NR;
    const int M = (int)a.M, r = (int)a.r;
    const int nrow = (int)((a.B - b0 < NR) ? (a.B - b0) : NR);
    // prob2vec with codebooks of 17..32 entries runs on the matrix cores
    constexpr bool MM = MB == 24 || MB == 32;
    constexpr int KH = MB / 2;
    [[maybe_unused]] const int c = t & 31, h = (t >> 5) & 1;
    float x[MB];
    if (MODE == MODE_P2V) {
        if constexpr (MM) {
            // T = P R: B[k][j] = R[k][j]
            float bk[KH];
#pragma unroll
            for (int kk = 0; kk < KH; ++kk) bk[kk] = (c < r) ? R.Rs[(kk + KH * h) * MB + c] : 0.f;
            gs16v acc[2];
            wave_rows_mm<KH>(tile, M, M, bk, acc);
            lds_barrier();   // the tile is reused for the outputs
            wave_rows_out(acc, r, r, tile);
        } else {
            row_prob2vec<MB>(tile + t * M, M, R, x);
            lds_barrier();   // the tile is reused for the outputs
            regs_to_tile<MB>(x, r, tile);
        }
        lds_barrier();
        tile_store<TO, NR>(static_cast<TO *>(a.Out), a.ldout, b0, nrow, r, tile);
        return;
    }
    // (scores stay on the vector units: there the matrix-core form, which
    // returns the products through the tile, measured slower)
    tile_to_regs<MB>(tile, r, x);
    lds_barrier();   // the tile is reused for the outputs
    float n2 = 0.f;
#pragma unroll
    for (int k = 0; k < MB; ++k) n2 += x[k] * x[k];
    float q = 1.f;
    if (a.cosine) {
        if (a.qnorm2 && t < nrow) n2 = a.qnorm2[b0 + t];
        q = (n2 > 0.f) ? 1.f / sqrtf(n2) : 0.f;
    }
    const float mul = (MODE == MODE_ATT) ? a.scale * a.beta : a.scale;
    float *srow = tile + t * M;
    float best;
    int bi;
    row_scores<MB>(x, M, R, Rn, mul, q, srow, best, bi);
    if (MODE == MODE_SIM) {
        if (a.argmax && t < nrow) __builtin_nontemporal_store(bi, a.argmax + b0 + t);
        if (!a.Out) return;
        lds_barrier();
        tile_store<float, NR>(static_cast<float *>(a.Out), a.ldout, b0, nrow, M, tile);
        return;
    }
    row_softmax(srow, M, 1.f, best);
    lds_barrier();
    tile_store<float, NR>(static_cast<float *>(a.Out), a.ldout, b0, nrow, M, tile);
    if (!a.O) return;
    float o[MB];
    row_prob2vec<MB>(srow, M, R, o);
    lds_barrier();
    regs_to_tile<MB>(o, r, tile);
    lds_barrier();
    tile_store<TO, NR>(static_cast<TO *>(a.O), a.ldo, b0, nrow, r, tile);
}

// The codebook block and the given norms are requested first, then the row
// tile, so their global round trips overlap (the loads are all in flight
// before the first wait); missing norms are then summed from the block in LDS.
template <typename TI, typename TO, int MODE, int MB>
__global__ void __launch_bounds__(rows_of<MB>()) small_kernel(SmallArgs a) {
    constexpr int NR = rows_of<MB>();
    constexpr int RE = (MB * MB + NR - 1) / NR;   // codebook block elements per thread
    __shared__ __attribute__((aligned(16))) float tile[NR * MB];
    __shared__ __attribute__((aligned(16))) float Rs[MB * MB];
    __shared__ float Rn[MB];
    const int t = threadIdx.x;
    const int64_t b0 = (int64_t)blockIdx.x * NR;
    const int M = (int)a.M, r = (int)a.r;
    const int nrow = (int)((a.B - b0 < NR) ? (a.B - b0) : NR);
    const TI *R = static_cast<const TI *>(a.R);
    const bool cosine = a.cosine != 0;
    float rv[RE];
#pragma unroll
    for (int i = 0; i < RE; ++i) {
        const int e = t + i * NR, j = e / MB, k = e - (e / MB) * MB;
        rv[i] = (e < MB * MB && j < M && k < r) ? ld_f32<TI>(R, (int64_t)j * a.ldr + k) : 0.f;
    }
    float cn = 0.f;
    if (MODE != MODE_P2V && cosine && a.cnorm && t < M) cn = a.cnorm[t];
    tile_load<TI, NR, MB>(static_cast<const TI *>(a.In), a.ldin, b0, nrow, (MODE == MODE_P2V) ? M : r, tile);
#pragma unroll
    for (int i = 0; i < RE; ++i)
        if (t + i * NR < MB * MB) Rs[t + i * NR] = rv[i];
    lds_barrier();
    if (MODE != MODE_P2V) {
        // reciprocal codebook norms for cosine scores (ones for dot), zeros
        // beyond M; without given norms ||R_j||, summed in fp32 over k < r
        if (t < MB) {
            float c = 0.f;
            if (t < M) {
                c = 1.f;
                if (cosine) {
                    float n = cn;
                    if (!a.cnorm) {
                        float s2 = 0.f;
                        for (int k = 0; k < r; ++k) s2 += Rs[t * MB + k] * Rs[t * MB + k];
                        n = sqrtf(s2);
                    }
                    c = (n > 0.f) ? 1.f / n : 0.f;
                }
            }
            Rn[t] = c;
        }
        lds_barrier();
    }
    small_body<TI, TO, MODE, MB>(a, LdsRows<MB>{Rs}, Rn, tile);
}

// ---------------------------------------------------------------------------
// Fused soft selection.  A work-group of SROWS threads owns SROWS * RPT
// consecutive rows of one codebook group; thread t owns rows t, t + SROWS, ...
// so that every codebook value it reads serves RPT rows.  The probability
// tile is requested first (vector loads into registers), the codebook block
// and norms are staged in LDS while those loads are in flight, then the tile
// goes through LDS to the threads' rows.  Outputs leave through the same LDS
// tile with coalesced stores.

constexpr int SROWS = 256;               // threads per work-group
constexpr int RPT = 1;                   // rows per thread (the Gram form below assumes one)
constexpr int SBLK = SROWS * RPT;        // rows per work-group

__device__ __forceinline__ int soft_group(const SoftArgs &a, int64_t blk) {
    int gi = 0;
    while (gi + 1 < a.ngroups && blk >= a.tile_start[gi + 1]) ++gi;
    return gi;
}

// --------------------------------------------- soft selection, Gram form
//
// Without a coordinate output the coordinates t = p R are never formed: with
// the Gram matrix G = R R^T of the codebook block (G[j][k] = <c_j, c_k>, Q
// having orthonormal rows), <t, R_j> = sum_k p_k G[k][j] and
// ||t||^2 = sum_j p_j <t, R_j>.  Per row this is M^2 multiply-adds in place
// of 2 M r, all in registers.

// Probability tile request: 16-byte pieces into registers.  fp32 rows use
// buffer loads whose range is the tile itself, so every thread issues the same
// number of loads whatever the row count (the pieces beyond the range read as
// zero and are not used) and the codebook loads issued before them can be
// waited for alone.
// Cache-policy operand of the fp32 tile loads: non-temporal (nt), since the
// tile is read once.  Measured on the vsa step: 9.5 -> 8.8 us with the batch
// coming from HBM, unchanged (8.1 -> 8.0 us) with it cache resident.  Plain
// loads marked non-temporal in the separate calls' tile moves were 10-25 %
// slower when their inputs were cache resident, so those stay plain.
constexpr int NT_LOAD = 2;
template <typename TI> struct TileReq;
template <> struct TileReq<float> {
    static constexpr int V = 64 * MAXK / 4 / 64;   // 16-byte pieces per lane of a wave's 64 rows
    f4v v[V];
    __device__ __forceinline__ void issue(const float *base, int n, int lane) {
        const __amdgpu_buffer_rsrc_t rs =
            __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(base), (short)0, n * 4, 0x00020000);
#pragma unroll
        for (int i = 0; i < V; ++i)
            v[i] = __builtin_bit_cast(f4v, __builtin_amdgcn_raw_buffer_load_b128(rs, (lane + i * 64) * 16, 0, NT_LOAD));
    }
    // the requested pieces, then the last n % 4 elements, to the wave's tile
    __device__ __forceinline__ void store(float *wtile, const float *base, int n, int lane) const {
        const int n4 = n >> 2;
#pragma unroll
        for (int i = 0; i < V; ++i) {
            const int e4 = lane + i * 64;
            if (e4 < n4) st4(wtile + 4 * e4, v[i]);
        }
        const int e = 4 * n4 + lane;
        if (e < n) wtile[e] = base[e];
    }
};
// bf16 rows: 16-byte pieces of 8 elements (the tile start is 16-byte aligned).
template <> struct TileReq<bf16_t> {
    typedef unsigned int u4v __attribute__((ext_vector_type(4)));
    static constexpr int V = 64 * MAXK / 8 / 64;   // 8-element pieces per lane
    u4v v[V];
    __device__ __forceinline__ void issue(const bf16_t *base, int n, int lane) {
        const int n8 = n >> 3;
#pragma unroll
        for (int i = 0; i < V; ++i) {
            const int e8 = lane + i * 64;
            if (e8 < n8) v[i] = *reinterpret_cast<const u4v *>(base + 8 * e8);
        }
    }
    __device__ __forceinline__ void store(float *wtile, const bf16_t *base, int n, int lane) const {
        const int n8 = n >> 3;
#pragma unroll
        for (int i = 0; i < V; ++i) {
            const int e8 = lane + i * 64;
            if (e8 < n8) {
                const u4v u = v[i];
                st4(wtile + 8 * e8, f4v{__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                                        __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u)});
                st4(wtile + 8 * e8 + 4, f4v{__uint_as_float(u.z << 16), __uint_as_float(u.z & 0xffff0000u),
                                            __uint_as_float(u.w << 16), __uint_as_float(u.w & 0xffff0000u)});
            }
        }
        for (int e = 8 * n8 + lane; e < n; e += 64) wtile[e] = ld_f32<bf16_t>(base, e);
    }
};

// Gram matrix of the codebook, formed by wave 0 on the matrix cores as one
// 32 x 32 block of v_mfma_f32_32x32x2f32 with A = R and B = R^T in the same
// register: lane l holds R[l % 32][2 kk + l / 32] in rk[kk] (zero past M
// rows and r columns).  G[j][i] goes to Gs[j * GS + i] for i, j < M, and the
// per-entry factors to Rn (1 / ||c_j|| for cosine, from the given norms or
// from the codebook rows; 1 for dot).
template <int M, int GS>
__device__ __forceinline__ void gram_stage(const float (&rk)[(M + 1) / 2], float *Gs, float *Rn, bool cosine,
                                           bool given, float cn) {
    const int l = threadIdx.x;
    const int row = l & 31, h = l >> 5;
    gs16v acc = {};
    float s2 = 0.f;
#pragma unroll
    for (int kk = 0; kk < (M + 1) / 2; ++kk) {
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(rk[kk], rk[kk], acc, 0, 0, 0);
        s2 += rk[kk] * rk[kk];
    }
    s2 += __shfl_xor(s2, 32);   // ||R_row||^2: even and odd columns
    if (row < M) {
#pragma unroll
        for (int g = 0; g < 16; ++g) {
            const int j = 8 * (g >> 2) + 4 * h + (g & 3);
            if (j < M) Gs[j * GS + row] = acc[g];
        }
    }
    if (l < M) {
        float c = 1.f;
        if (cosine) {
            const float n = given ? cn : sqrtf(s2);
            c = (n > 0.f) ? 1.f / n : 0.f;
        }
        Rn[l] = c;
    }
}

// Coordinate form: wave 0 publishes the codebook coordinates themselves,
// Rs[j * GS + k] = R[j][k] (zero for k >= r), from the same operand layout,
// their transpose Rs[MAXK * MAXK + k * GS + j] for codebooks of at most 8
// entries, and the per-entry factors as gram_stage does.
template <int M, int GS>
__device__ __forceinline__ void rows_stage(const float (&rk)[(M + 1) / 2], float *Rs, float *Rn, bool cosine,
                                           bool given, float cn) {
    const int l = threadIdx.x;
    const int row = l & 31, h = l >> 5;
    float s2 = 0.f;
#pragma unroll
    for (int kk = 0; kk < (M + 1) / 2; ++kk) {
        s2 += rk[kk] * rk[kk];
        if (row < M) {
            Rs[row * GS + 2 * kk + h] = rk[kk];
            if (M <= 8) Rs[MAXK * MAXK + (2 * kk + h) * GS + row] = rk[kk];
        }
    }
    s2 += __shfl_xor(s2, 32);   // ||R_row||^2: even and odd columns
    if (l < M) {
        float c = 1.f;
        if (cosine) {
            const float n = given ? cn : sqrtf(s2);
            c = (n > 0.f) ? 1.f / n : 0.f;
        }
        Rn[l] = c;
    }
}

// LDS accesses of one wave complete in order: fences that keep the compiler
// from moving this wave's LDS reads and writes across each other.
__device__ __forceinline__ void wave_lds_fence() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
}

// One row block of one group, for a codebook of exactly M entries.  Each
// wave loads, scores and stores its own 64 rows (rows 64 w .. 64 w + 63 of
// the block, their own part of the tile), so after the one work-group
// barrier that publishes the Gram matrix the waves go on independently: one
// wave's arithmetic overlaps another's loads and stores.
// Coordinate form of step 5 for the wave's 64 rows (rows wrow0 .. + 63 of
// the block, in wtile): t = p R for each row, stored (bf16 or fp32) when the group
// asks for T, then the raw scores d_j = <t, R_j> of this thread's row and
// ||t||^2 in n2.  Rs holds R (row stride GS, zero past r columns).
//   M <= 8: vector units, each thread its own row (2 M^2 multiply-adds).
//   9 <= M <= 16: matrix cores, 16 x 16 blocks (below).
//   M > 16: matrix cores, the wave's rows as two 32-row blocks.  First
//     T^T = R^T P^T (v_mfma_f32_32x32x2f32, step kk pairing m = kk and
//     kk + KH over the half-waves): lane l supplies R[m][l % 32] and
//     P[row l % 32][m], and its register g then holds T[row l % 32][k] for
//     k = 8 (g / 4) + 4 (l / 32) + g % 4.  Those registers are directly the
//     A operand of S = T R^T (step s pairing the same k with B = R[l % 32][k]
//     from registers), whose result block (lane l, register g: row
//     8 (g / 4) + 4 (l / 32) + g % 4, entry l % 32) goes through the tile to
//     the threads' rows.
// The wave's rows of T (row stride r in wtile) to the output, in bf16 or fp32.
__device__ __forceinline__ void store_coords(const SoftGroup &G, bool t_bf16, int64_t b0, int wrow0, int nroww,
                                             const float *wtile, int lane) {
    if (t_bf16) tile_store<bf16_t, 64>(static_cast<bf16_t *>(G.T), G.ldt, b0 + wrow0, nroww, (int)G.r, wtile, lane);
    else tile_store<float, 64>(static_cast<float *>(G.T), G.ldt, b0 + wrow0, nroww, (int)G.r, wtile, lane);
}

template <int M, int GS>
__device__ __forceinline__ void soft_coords(const SoftGroup &G, bool t_bf16, int64_t b0, int wrow0, int nroww,
                                            float *tile, float *wtile, const float *Rs, float (&d)[M], float &n2) {
    const int t = threadIdx.x;
    const int lane = t & 63;
    const int r = (int)G.r;
    float *srow = tile + t * M;
    if constexpr (M <= 8) {
        float p[M], tk[M];
#pragma unroll
        for (int k = 0; k < M; ++k) p[k] = srow[k];
#pragma unroll
        for (int k = 0; k < M; ++k) tk[k] = 0.f;
#pragma unroll
        for (int j = 0; j < M; ++j) {
            const f4v *rq = reinterpret_cast<const f4v *>(Rs + j * GS);
#pragma unroll
            for (int qq = 0; qq < GS / 4; ++qq) {
                const f4v v = rq[qq];
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (4 * qq + i < M) tk[4 * qq + i] += p[j] * v[i];
            }
        }
        // d_j = sum_k t_k R[j][k], one row of R^T at a time into M
        // independent sums
        const float *Rt = Rs + MAXK * MAXK;
#pragma unroll
        for (int j = 0; j < M; ++j) d[j] = 0.f;
#pragma unroll
        for (int k = 0; k < M; ++k) {
            const f4v *rq = reinterpret_cast<const f4v *>(Rt + k * GS);
#pragma unroll
            for (int qq = 0; qq < GS / 4; ++qq) {
                const f4v v = rq[qq];
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (4 * qq + i < M) d[4 * qq + i] += tk[k] * v[i];
            }
        }
        n2 = 0.f;
#pragma unroll
        for (int k = 0; k < M; ++k) n2 += tk[k] * tk[k];
        if (G.T) {
            // rows of r values in the wave's tile, after every lane's row reads
            wave_lds_fence();
            float *trow = wtile + lane * r;
#pragma unroll
            for (int k = 0; k < M; ++k)
                if (k < r) trow[k] = tk[k];
            wave_lds_fence();
            store_coords(G, t_bf16, b0, wrow0, nroww, wtile, lane);
            wave_lds_fence();
        }
    } else if constexpr (M <= 16) {
        // 16 x 16 blocks (v_mfma_f32_16x16x4f32), the wave's rows as four
        // 16-row blocks.  T^T = R^T P^T in steps of four entries m = 4 s + q
        // (q = lane / 16): lane l supplies R[m][l % 16] and P[row l % 16][m],
        // and its register g then holds T[row l % 16][4 q + g], directly the
        // A operand of S = T R^T at step g (B = R[l % 16][4 q + g]); the
        // result (lane l, register g: row 4 q + g, entry l % 16) goes through
        // the tile to the threads' rows.
        constexpr int KS = (M + 3) / 4;
        const int c = lane & 15, qd = lane >> 4;
        f4v tq[4];
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const float *prow = tile + (wrow0 + 16 * b + c) * M;
            tq[b] = f4v{};
#pragma unroll
            for (int st = 0; st < KS; ++st) {
                const int m = 4 * st + qd;
                const float ra = (m < M && c < M) ? Rs[m * GS + c] : 0.f;
                const float x = (m < M) ? prow[m] : 0.f;
                tq[b] = __builtin_amdgcn_mfma_f32_16x16x4f32(ra, x, tq[b], 0, 0, 0);
            }
        }
        // ||t||^2 of row l % 16 of each block (coordinates past r are zero)
        float nb[4];
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            float s2 = tq[b][0] * tq[b][0] + tq[b][1] * tq[b][1] + tq[b][2] * tq[b][2] + tq[b][3] * tq[b][3];
            s2 += __shfl_xor(s2, 16);
            nb[b] = s2 + __shfl_xor(s2, 32);
        }
        n2 = (qd == 0) ? nb[0] : (qd == 1) ? nb[1] : (qd == 2) ? nb[2] : nb[3];   // block l / 16, row l % 16
        if (G.T) {
            // the products consumed every probability read of the wave
            wave_lds_fence();
#pragma unroll
            for (int b = 0; b < 4; ++b)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int k = 4 * qd + g;
                    if (k < r) wtile[(16 * b + c) * r + k] = tq[b][g];
                }
            wave_lds_fence();
            store_coords(G, t_bf16, b0, wrow0, nroww, wtile, lane);
        }
        float rb[4];
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int k = 4 * qd + g;
            rb[g] = (c < M && k < M) ? Rs[c * GS + k] : 0.f;
        }
        wave_lds_fence();   // T (or the probabilities) have left the tile
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            f4v acc = {};
#pragma unroll
            for (int g = 0; g < 4; ++g) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(tq[b][g], rb[g], acc, 0, 0, 0);
            if (c < M) {
                float *drow = tile + (wrow0 + 16 * b + 4 * qd) * M + c;
#pragma unroll
                for (int g = 0; g < 4; ++g) drow[g * M] = acc[g];
            }
        }
        wave_lds_fence();
#pragma unroll
        for (int j = 0; j < M; ++j) d[j] = srow[j];
    } else {
        constexpr int KH = (M + 1) / 2;
        // steps of the second product: s with 8 (s / 4) + s % 4 < M
        constexpr int NS = 4 * (M / 8) + (M % 8 < 4 ? M % 8 : 4);
        const int l = lane, c = l & 31, h = l >> 5;
        gs16v tq[2];
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            const float *arow = tile + (wrow0 + 32 * b + c) * M + KH * h;
            tq[b] = gs16v{};
#pragma unroll
            for (int kk = 0; kk < KH; ++kk) {
                const int m = kk + KH * h;
                const float ra = (m < M && c < M) ? Rs[m * GS + c] : 0.f;
                float x = arow[kk];
                if (M % 2 == 1 && kk == KH - 1) x = (h == 0) ? x : 0.f;
                tq[b] = __builtin_amdgcn_mfma_f32_32x32x2f32(ra, x, tq[b], 0, 0, 0);
            }
        }
        // ||t||^2 of row l % 32 of each block (coordinates past r are zero)
        float nb[2];
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            float s2 = 0.f;
#pragma unroll
            for (int g = 0; g < 16; ++g) s2 += tq[b][g] * tq[b][g];
            nb[b] = s2 + __shfl_xor(s2, 32);
        }
        n2 = h ? nb[1] : nb[0];   // this thread's row: block l / 32, row l % 32
        if (G.T) {
            // the products consumed every probability read of the wave
            wave_lds_fence();
#pragma unroll
            for (int b = 0; b < 2; ++b)
#pragma unroll
                for (int g = 0; g < 16; ++g) {
                    const int k = 8 * (g >> 2) + 4 * h + (g & 3);
                    if (k < r) wtile[(32 * b + c) * r + k] = tq[b][g];
                }
            wave_lds_fence();
            store_coords(G, t_bf16, b0, wrow0, nroww, wtile, lane);
        }
        float rb[NS];
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            const int k = 8 * (s >> 2) + 4 * h + (s & 3);
            rb[s] = (c < M && k < M) ? Rs[c * GS + k] : 0.f;
        }
        wave_lds_fence();   // T (or the probabilities) have left the tile
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            gs16v acc = {};
#pragma unroll
            for (int s = 0; s < NS; ++s) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(tq[b][s], rb[s], acc, 0, 0, 0);
            if (c < M) {
                float *drow = tile + (wrow0 + 32 * b + 4 * h) * M + c;
#pragma unroll
                for (int g = 0; g < 16; ++g) drow[(8 * (g >> 2) + (g & 3)) * M] = acc[g];
            }
        }
        wave_lds_fence();
#pragma unroll
        for (int j = 0; j < M; ++j) d[j] = srow[j];
    }
}

// CO (coordinate form): the codebook coordinates go to Gs in place of the
// Gram matrix, and each row's coordinates t = p R are formed (stored
// when the group asks for T) and scored against R, 2 M^2 multiply-adds per
// row (R zero past r columns).
template <typename TI, int M, bool CO>
__device__ __forceinline__ void soft_gram(const SoftGroup &G, bool cosine, float scale, float beta, bool t_bf16,
                                          int64_t b0, int nrow, float *tile, float *Gs, float *Rn) {
    constexpr int GS = (M + 3) & ~3;   // row stride of G in LDS (16-byte rows)
    constexpr int KG = (M + 1) / 2;    // steps of the Gram product
    const int t = threadIdx.x;
    const int lane = t & 63, wrow0 = t & ~63;
    const int nroww = (nrow - wrow0 < 0) ? 0 : (nrow - wrow0 < 64) ? nrow - wrow0 : 64;   // this wave's rows
    float *wtile = tile + wrow0 * M;
    const int r = (int)G.r;

    // 1. wave 0: the codebook rows in the Gram product's operand layout and
    // the given norms, requested before the tile so that they return first
    float rk[KG];
    float cn = 0.f;
    if (t < 64) {
        const int row = t & 31, h = t >> 5;
        const TI *Rrow = static_cast<const TI *>(G.R) + (int64_t)((row < M) ? row : 0) * G.ldr;
#pragma unroll
        for (int kk = 0; kk < KG; ++kk) {
            const int k = 2 * kk + h;
            rk[kk] = (row < M && k < r) ? ld_f32<TI>(Rrow, k) : 0.f;
        }
        if (cosine && G.cnorm && t < M) cn = G.cnorm[t];
    }

    // 2. this wave's probability rows (contiguous rows: one linear range; the
    // wave's start stays 16-byte aligned when the block's does)
    const TI *bbase = static_cast<const TI *>(G.P) + b0 * G.ldp;
    const bool contig = G.ldp == M && aligned16(bbase);
    const TI *base = bbase + (int64_t)wrow0 * M;
    const int n = nroww * M;
    TileReq<TI> req;
    req.issue(base, contig ? n : 0, lane);   // an empty range issues nothing useful

    // 3. Gram matrix (coordinate form: the coordinates) and factors while the
    // tiles are in flight, published to every wave
    if (t < 64) {
        if constexpr (CO) rows_stage<M, GS>(rk, Gs, Rn, cosine, G.cnorm != nullptr, cn);
        else gram_stage<M, GS>(rk, Gs, Rn, cosine, G.cnorm != nullptr, cn);
    }
    lds_barrier();

    // 4. this wave's rows to its part of the tile
    if (contig) {
        req.store(wtile, base, n, lane);
    } else {
        tile_load<TI, 64>(static_cast<const TI *>(G.P), G.ldp, b0 + wrow0, nroww, M, wtile, lane);
    }
    wave_lds_fence();

    // 5. scores of the thread's row, in registers
    float *srow = tile + t * M;
    float d[M];
    float q;
    if constexpr (CO) {
        soft_coords<M, GS>(G, t_bf16, b0, wrow0, nroww, tile, wtile, Gs, d, q);
        q = cosine ? ((q > 0.f) ? 1.f / sqrtf(q) : 0.f) : 1.f;   // in span: ||v|| = ||t||
    } else {
    float p[M];
#pragma unroll
    for (int k = 0; k < M; ++k) p[k] = srow[k];
    if constexpr (M > 16) {
        // Matrix cores: the wave's 64 rows as two 32 x M blocks times G
        // (v_mfma_f32_32x32x2f32; step kk pairs k = kk and kk + KH over the
        // two half-waves).  Lane l supplies A = P[row l % 32][k] from the
        // tile and B = G[k][l % 32] from registers; the result block (lane l,
        // register g: row 8(g/4) + 4(l/32) + g % 4, column l % 32) replaces the
        // block's probabilities in the tile, from where each thread takes its
        // own row.  Columns past M are never stored; a k past M (odd M) is
        // zero on both sides.
        constexpr int KH = (M + 1) / 2;
        const int l = t & 63, c = l & 31, h = l >> 5;
        float bf[KH];
#pragma unroll
        for (int kk = 0; kk < KH; ++kk) {
            if (M % 2 == 1 && kk == KH - 1) {
                const float x = Gs[kk * GS + c];
                bf[kk] = (h == 0) ? x : 0.f;
            } else {
                bf[kk] = Gs[(kk + KH * h) * GS + c];
            }
        }
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            const int r0 = (t & ~63) + 32 * b;
            const float *arow = tile + (r0 + c) * M + KH * h;
            gs16v acc = {};
#pragma unroll
            for (int kk = 0; kk < KH; ++kk) {
                float x = arow[kk];
                if (M % 2 == 1 && kk == KH - 1) x = (h == 0) ? x : 0.f;
                acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x, bf[kk], acc, 0, 0, 0);
            }
            // the block's reads have returned (the products consumed them) and
            // only this wave touches its rows
            if (c < M) {
                float *drow = tile + (r0 + 4 * h) * M + c;
#pragma unroll
                for (int g = 0; g < 16; ++g) drow[(8 * (g >> 2) + (g & 3)) * M] = acc[g];
            }
        }
        // the row written by the other lanes is read back after these fences
        wave_lds_fence();
#pragma unroll
        for (int j = 0; j < M; ++j) d[j] = srow[j];
    } else {
        // d_j = sum_k p_k G[k][j], one G row at a time into M independent sums
#pragma unroll
        for (int j = 0; j < M; ++j) d[j] = 0.f;
#pragma unroll
        for (int k = 0; k < M; ++k) {
            const f4v *gq = reinterpret_cast<const f4v *>(Gs + k * GS);
#pragma unroll
            for (int q = 0; q < GS / 4; ++q) {
                const f4v g = gq[q];
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (4 * q + i < M) d[4 * q + i] += p[k] * g[i];
            }
        }
    }
    float n2 = 0.f;
#pragma unroll
    for (int j = 0; j < M; ++j) n2 += p[j] * d[j];
    q = cosine ? ((n2 > 0.f) ? 1.f / sqrtf(n2) : 0.f) : 1.f;   // in span: ||v|| = ||t||
    }
    const float mq = scale * q;
    float best = -INFINITY, worst = INFINITY;
    int bi = 0;
#pragma unroll
    for (int j = 0; j < M; ++j) {
        d[j] = mq * d[j] * Rn[j];
        if (d[j] > best) { best = d[j]; bi = j; }
        worst = fminf(worst, d[j]);
    }
    if (G.argmax && t < nrow) __builtin_nontemporal_store(bi, G.argmax + b0 + t);

    // 6. outputs through the wave's part of the tile (each thread overwrites
    // only its own row)
    if (G.S) {
#pragma unroll
        for (int j = 0; j < M; ++j) srow[j] = d[j];
        wave_lds_fence();
        tile_store<float, 64>(G.S, G.lds, b0 + wrow0, nroww, M, wtile, lane);
    }
    if (G.A) {
        // softmax of beta times the scores in base 2: exp(beta s) =
        // 2^(beta log2(e) s); the largest exponent is beta log2(e) times the
        // largest score, or the smallest one when beta is negative
        const float bl = beta * 1.44269504088896341f;
        const float m2 = (bl >= 0.f) ? bl * best : bl * worst;
        float z = 0.f;
#pragma unroll
        for (int j = 0; j < M; ++j) {
            d[j] = __builtin_amdgcn_exp2f(fmaf(bl, d[j], -m2));
            z += d[j];
        }
        const float iz = 1.f / z;
        if (G.S) wave_lds_fence();   // S has left the tile before it is overwritten
#pragma unroll
        for (int j = 0; j < M; ++j) srow[j] = d[j] * iz;
        wave_lds_fence();
        tile_store<float, 64>(G.A, G.lda, b0 + wrow0, nroww, M, wtile, lane);
    }
}

template <typename TI, int M, bool CO>
__device__ __forceinline__ void soft_gram_m(int m, const SoftGroup &G, bool cosine, float scale, float beta,
                                            bool t_bf16, int64_t b0, int nrow, float *tile, float *Gs, float *Rn) {
    if constexpr (M <= MAXK) {
        if (m == M) soft_gram<TI, M, CO>(G, cosine, scale, beta, t_bf16, b0, nrow, tile, Gs, Rn);
        else soft_gram_m<TI, M + 1, CO>(m, G, cosine, scale, beta, t_bf16, b0, nrow, tile, Gs, Rn);
    }
}

// Fused soft selection without a coordinate output: scores through the
// codebook's Gram matrix (G = R R^T = C C^T, Sec. 3.2): with t = p R,
// <t, R_j> = sum_k p_k G[k][j] and ||t||^2 = sum_j p_j <t, R_j>, so the
// coordinates are never formed; per row this is M^2 multiply-adds in place
// of 2 M r.  One work-group per 256-row block of a group; at least four
// work-groups per CU (at most 128 registers per lane).
template <typename TI>
__global__ void __launch_bounds__(SROWS, 4) soft_gram_kernel(SoftArgs a) {
    __shared__ __attribute__((aligned(16))) float tile[SBLK * MAXK];
    __shared__ __attribute__((aligned(16))) float Gs[MAXK * MAXK];
    __shared__ float Rn[MAXK];
    const int64_t blk = blockIdx.x;
    const int gi = soft_group(a, blk);
    const SoftGroup G = a.g[gi];   // by value: the group's descriptor in scalar registers
    const int64_t b0 = (blk - a.tile_start[gi]) * SBLK;
    const int nrow = (int)((G.B - b0 < SBLK) ? (G.B - b0) : SBLK);
    soft_gram_m<TI, 1, false>((int)G.M, G, a.cosine != 0, a.scale, a.beta, false, b0, nrow, tile, Gs, Rn);
}

// Fused soft selection in the coordinate form: t = p R is formed for every
// row (and stored when the group asks for T), then scored against R, on the
// same frame as the Gram form (specialised on M, waves independent after the
// barrier that publishes the codebook block).
template <typename TI>
__global__ void __launch_bounds__(SROWS, 4) soft_select_kernel(SoftArgs a) {
    __shared__ __attribute__((aligned(16))) float tile[SBLK * MAXK];
    __shared__ __attribute__((aligned(16))) float Rs[MAXK * MAXK + 8 * 8];   // R, then R^T for M <= 8
    __shared__ float Rn[MAXK];
    const int64_t blk = blockIdx.x;
    const int gi = soft_group(a, blk);
    const SoftGroup G = a.g[gi];   // by value: the group's descriptor in scalar registers
    const int64_t b0 = (blk - a.tile_start[gi]) * SBLK;
    const int nrow = (int)((G.B - b0 < SBLK) ? (G.B - b0) : SBLK);
    soft_gram_m<TI, 1, true>((int)G.M, G, a.cosine != 0, a.scale, a.beta, a.t_bf16 != 0, b0, nrow, tile, Rs, Rn);
}

template <typename TI, typename TO, int MODE>
hipError_t launch(const SmallArgs &a, hipStream_t s) {
    if (a.B == 0) return hipSuccess;
    const int nr = pad_small(a.M) <= 48 ? 256 : 128;   // rows_of
    const dim3 grid((unsigned)((a.B + nr - 1) / nr)), block(nr);
    switch (pad_small(a.M)) {
        case 8: hipLaunchKernelGGL((small_kernel<TI, TO, MODE, 8>), grid, block, 0, s, a); break;
        case 16: hipLaunchKernelGGL((small_kernel<TI, TO, MODE, 16>), grid, block, 0, s, a); break;
        case 24: hipLaunchKernelGGL((small_kernel<TI, TO, MODE, 24>), grid, block, 0, s, a); break;
        case 32: hipLaunchKernelGGL((small_kernel<TI, TO, MODE, 32>), grid, block, 0, s, a); break;
        case 48: hipLaunchKernelGGL((small_kernel<TI, TO, MODE, 48>), grid, block, 0, s, a); break;
        default: hipLaunchKernelGGL((small_kernel<TI, TO, MODE, 64>), grid, block, 0, s, a); break;
    }
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

hipError_t launch_soft_select(gs_dtype tin, gs_dtype tt, const SoftArgs &a, hipStream_t s) {
    if (a.ntiles == 0) return hipSuccess;
    const dim3 grid((unsigned)a.ntiles), block(SROWS);
    if (!a.coords) {
        if (tin == GS_F32) hipLaunchKernelGGL((soft_gram_kernel<float>), grid, block, 0, s, a);
        else if (tin == GS_BF16) hipLaunchKernelGGL((soft_gram_kernel<bf16_t>), grid, block, 0, s, a);
        else return hipErrorInvalidValue;
        return hipGetLastError();
    }
    if (tt != GS_F32 && tt != GS_BF16) return hipErrorInvalidValue;
    SoftArgs b = a;
    b.t_bf16 = tt == GS_BF16;
    if (tin == GS_F32) hipLaunchKernelGGL((soft_select_kernel<float>), grid, block, 0, s, b);
    else if (tin == GS_BF16) hipLaunchKernelGGL((soft_select_kernel<bf16_t>), grid, block, 0, s, b);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

int64_t soft_select_tiles(int64_t B) { return (B + SBLK - 1) / SBLK; }


}  // namespace gs
