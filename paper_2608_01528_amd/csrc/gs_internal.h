// Internal declarations shared by the HIP translation units of the Gram-Space
// library.  Not part of the public ABI (that is include/gramspace.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gramspace.h"

namespace gs {

// ------------------------------------------------------------ element types

// bfloat16 is carried as its 16-bit pattern; arithmetic is always fp32.
struct bf16_t { uint16_t bits; };

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(((uint32_t)b) << 16);
}

// fp32 -> bf16, round to nearest even (finite inputs; NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u) return (uint16_t)((u >> 16) | ((u & 0xffffu) ? 0x40u : 0u));
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// fp64 -> bf16, round to nearest even in one rounding: narrow to fp32 toward
// zero, fold the discarded bits into the last fp32 bit (round to odd), then
// round that to bf16.  fp32 keeps 16 more bits than bf16, so the result equals
// the correctly rounded fp64 -> bf16 conversion.
__device__ __forceinline__ uint16_t f64_to_bf16(double d) {
    float f = __double2float_rz(d);
    if ((double)f != d) f = __uint_as_float(__float_as_uint(f) | 1u);
    return f32_to_bf16(f);
}

// Work-group barrier for hand-offs through LDS: every thread's LDS accesses
// before it are complete and visible after it.  Global stores still in flight
// are not waited for (__syncthreads would wait for them to complete, which
// serialises the store phases of a work-group on memory latency).
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Second pass of the attention sweeps: row r of the block (rows m0 ..
// m0 + rows - 1 of out, leading dimension ldc, N columns) becomes
// exp(s - rmax[r]) * rinv[r].  Eight rows are in flight per thread (their
// loads are issued before any is used), in 16-byte chunks when vec (out
// 16-byte aligned, ldc a multiple of 4).  nthr threads take part.
__device__ __forceinline__ void softmax_rows(float *out, int64_t ldc, int64_t m0, int64_t rows, int64_t N,
                                             const float *rmax, const float *rinv, bool vec, int nthr) {
    typedef float f4 __attribute__((ext_vector_type(4)));
    const int t = threadIdx.x;
    const int64_t n4 = vec ? N / 4 : 0;
    for (int64_t r0 = 0; r0 < rows; r0 += 8) {
        const int nr = (int)((rows - r0 < 8) ? (rows - r0) : 8);
        for (int64_t c = t; c < n4; c += nthr) {
            f4 v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (u < nr) v[u] = *reinterpret_cast<const f4 *>(out + (m0 + r0 + u) * ldc + 4 * c);
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (u < nr) {
                    const float mx = rmax[r0 + u], iv = rinv[r0 + u];
                    f4 e;
#pragma unroll
                    for (int q = 0; q < 4; ++q) e[q] = __expf(v[u][q] - mx) * iv;
                    *reinterpret_cast<f4 *>(out + (m0 + r0 + u) * ldc + 4 * c) = e;
                }
        }
        for (int64_t c = 4 * n4 + t; c < N; c += nthr) {
            float v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (u < nr) v[u] = out[(m0 + r0 + u) * ldc + c];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (u < nr) out[(m0 + r0 + u) * ldc + c] = __expf(v[u] - rmax[r0 + u]) * rinv[r0 + u];
        }
    }
}

template <typename T> __device__ __forceinline__ float ld_f32(const T *p, int64_t i);
template <> __device__ __forceinline__ float ld_f32<float>(const float *p, int64_t i) { return p[i]; }
template <> __device__ __forceinline__ float ld_f32<bf16_t>(const bf16_t *p, int64_t i) {
    return bf16_to_f32(p[i].bits);
}

template <typename T> __device__ __forceinline__ void st_f32(T *p, int64_t i, float v);
template <> __device__ __forceinline__ void st_f32<float>(float *p, int64_t i, float v) { p[i] = v; }
template <> __device__ __forceinline__ void st_f32<bf16_t>(bf16_t *p, int64_t i, float v) {
    p[i].bits = f32_to_bf16(v);
}

// --------------------------------------------------------- launch plumbing

enum Epi { EPI_STORE = 0, EPI_BIND = 1, EPI_SIM = 2, EPI_SOFTMAX = 3 };

// One dense contraction  out[m, n] = sum_k A[m, k] * Bop[k, n]  with fp32
// accumulation on MFMA.  B is stored either N x K (b_nn = false: Bop = B^T)
// or K x N (b_nn = true).  The epilogue decides what is written.
struct GemmArgs {
    const void *A; int64_t lda;
    const void *A2; int64_t lda2;      // second left operand (EPI_BIND)
    const void *B; int64_t ldb;
    void *C; int64_t ldc;              // output (float for SIM / SOFTMAX)
    int64_t M, N, K;
    float *rownorm2;                   // EPI_STORE: sum_k A[m,k]^2, nullable
    const float *qnorm2;               // SIM / SOFTMAX, nullable
    const float *cnorm;                // SIM / SOFTMAX, nullable
    int cosine;
    float scale;
    float beta;
    int32_t *argmax;                   // EPI_SIM, nullable
    int write_out;                     // EPI_SIM: write scores to C
    int dma;                           // set by launch_gemm: bf16 pipelined loop
    int mul_out;                       // 256 x 256 store: C = C .* product (fp32 C)
    int echelon;                       // B is a lower-echelon R (R[j][k] == 0 for k > j)
};

hipError_t launch_gemm(gs_dtype ta, gs_dtype tb, gs_dtype tout, bool b_nn, Epi epi,
                       const GemmArgs &a, hipStream_t s);

// 256 x 256-tile product with a plain store (and optional row norms of A),
// both operands of type t (bf16 or fp32) with 16-byte aligned rows.
// gemm256_fits tells whether the product is large enough to fill the chip
// with such tiles.
bool gemm256_fits(gs_dtype t, const GemmArgs &a, bool b_nn);
hipError_t launch_gemm256(gs_dtype t, gs_dtype tout, bool b_nn, const GemmArgs &a, hipStream_t s);
// Row sweep of similarity (softmax = false) or attention scores over 256 x
// 256 blocks, same operand conditions (B stored N x K).
bool sweep256_fits(gs_dtype t, const GemmArgs &a);
hipError_t launch_sweep256(gs_dtype t, bool softmax, const GemmArgs &a, hipStream_t s);
// Scores written to memory (similarity with S, or attention): the 256 x 256
// product kernel with a scaled-score epilogue, then a row pass (argmax, or
// softmax in place).  Same operand conditions as launch_gemm256 (B N x K).
hipError_t launch_scores256(gs_dtype t, const GemmArgs &a, bool softmax, hipStream_t s);
// Scores of a few query rows (a.M <= FEW_ROWS) written to a.C, then the row
// pass (argmax, or softmax in place); any K, B stored N x K.
constexpr int64_t FEW_ROWS = 32;
hipError_t launch_few_rows(gs_dtype t, const GemmArgs &a, bool softmax, hipStream_t s);
// Row pass over a B x M fp32 score matrix (leading dimension ld): softmax in
// place, or the row argmax (lowest index on ties) into argmax when non-null.
hipError_t launch_rows_pass(bool softmax, float *out, int64_t ld, int64_t B, int64_t M, int32_t *argmax,
                            hipStream_t s);
// One pass over a B x M fp32 score matrix W: the row argmax (lowest index on
// ties) into argmax when non-null, and A = softmax(beta * W) row by row when
// A is non-null (A may be W itself).
hipError_t launch_sim_attn_pass(const float *W, int64_t ldw, int64_t B, int64_t M, int32_t *argmax, float beta,
                                float *A, int64_t lda, hipStream_t s);

// Raise a kernel's dynamic LDS limit (once per kernel, to a whole CU's LDS);
// fails for requests beyond that.
hipError_t raise_lds_limit(const void *kernel, size_t lds);

// Component-wise binding of restored vectors (gs_bind).
struct BindArgs {
    const void *X; int64_t ldx;
    const void *Y; int64_t ldy;
    void *Z; int64_t ldz;
    int64_t B, D;
    int64_t L;          // block length of the circular operators
    int lg;             // log2 L (set by launch_bind)
    int nb;             // blocks per work-group (set by launch_bind)
    int64_t nblocks;    // D / L (set by launch_bind)
};
hipError_t launch_bind(gs_dtype tin, gs_dtype tout, int op, const BindArgs &a, hipStream_t s);

// Z = ((T Q) .* (T2 Q)) Q^T, fp32, r <= BIND_COORDS_MAX_R
constexpr int64_t BIND_COORDS_MAX_R = 256;
struct BindCoordsArgs {
    const float *T; int64_t ldt;
    const float *T2; int64_t ldt2;
    const float *Q; int64_t ldq;
    float *Z; int64_t ldz;
    int64_t B, r, D;
    int vec, qvec;      // 16-byte aligned rows of T and T2 / of Q (set by launch_bind_coords)
};
hipError_t launch_bind_coords(const BindCoordsArgs &a, hipStream_t s);

// Small-codebook streaming kernels of the separate calls (r <= M <= SMALL_MAX)
// and of the fused soft selection (r <= M <= SOFT_MAX_M).
constexpr int SMALL_MAX = 64;
constexpr int SOFT_MAX_M = 32;

struct SmallArgs {
    const void *In; int64_t ldin;      // P (prob2vec) or T (similarity / attention)
    const void *R; int64_t ldr;        // M x r
    int64_t B, M, r;
    void *Out; int64_t ldout;          // T (prob2vec); S (similarity); A (attention)
    void *O; int64_t ldo;              // attention weighted sum, nullable
    const float *qnorm2, *cnorm;
    int cosine;
    float scale, beta;
    int32_t *argmax;
};

hipError_t launch_small_prob2vec(gs_dtype tin, gs_dtype tout, const SmallArgs &a, hipStream_t s);
hipError_t launch_small_similarity(gs_dtype tin, const SmallArgs &a, hipStream_t s);
hipError_t launch_small_attention(gs_dtype tin, gs_dtype to, const SmallArgs &a, hipStream_t s);

// Fused soft selection over up to SOFT_MAX_GROUPS small codebooks.
constexpr int SOFT_MAX_GROUPS = 8;

struct SoftGroup {
    const void *P; int64_t ldp;
    const void *R; int64_t ldr;
    const float *cnorm;
    int64_t B, M, r;
    void *T; int64_t ldt;
    float *S; int64_t lds;
    int32_t *argmax;
    float *A; int64_t lda;
};

struct SoftArgs {
    SoftGroup g[SOFT_MAX_GROUPS];
    int64_t tile_start[SOFT_MAX_GROUPS + 1];    // first work-group (row block) of each group
    int64_t ntiles;                             // work-groups in total
    int ngroups;
    int cosine;
    float scale, beta;
    int coords;                                 // form t = p R per row (else scores through R R^T)
    int t_bf16;                                 // coordinate outputs T in bf16 (else fp32)
};

int64_t soft_select_tiles(int64_t B);
hipError_t launch_soft_select(gs_dtype tin, gs_dtype tt, const SoftArgs &a, hipStream_t s);

// Probability vectorisation of sparse (CSR) probability rows.
struct SparseArgs {
    const int64_t *rowptr;             // B + 1 entries
    const int32_t *cols;               // nnz column indices
    const void *vals;                  // nnz values (type of R)
    int64_t B, M, nnz;
    const void *R; int64_t ldr;        // M x r
    int64_t r;
    void *T; int64_t ldt;              // B x r
};
hipError_t launch_sparse_prob2vec(gs_dtype tv, gs_dtype tt, const SparseArgs &a, hipStream_t s);

// Compression.
size_t compress_workspace(int64_t M, int64_t D);
// A second stream (non-blocking, default priority) on which compression runs
// the next panel's rows and the first part of its first pass while the
// current panel is factored, and two events (timing disabled) that fork it
// from and join it back into the caller's stream.  Without one (null), the
// same launches run in the same order on the caller's stream alone, with the
// same results bit for bit.
struct CompressOverlap {
    hipStream_t aux;
    hipEvent_t fork, join;
};
// row_base is added to the kept row indices (a subset's first codebook row).
hipError_t run_compress(const void *C, gs_dtype ct, int64_t M, int64_t D, int64_t ldc, double tol,
                        void *Q, gs_dtype qt, int64_t ldq, void *R, gs_dtype rt, int64_t ldr,
                        int32_t *kept, float *cnorm, int32_t *rank, int *nonfinite,
                        void *ws, hipStream_t s, int64_t row_base = 0, const CompressOverlap *ov = nullptr);
// Basis completed to k vectors by unit vectors (coordinates zero-padded),
// optionally transformed by an orthogonal k x k matrix H.
size_t compress_padded_workspace(int64_t M, int64_t D, int64_t k);
hipError_t run_compress_padded(const void *C, gs_dtype ct, int64_t M, int64_t D, int64_t ldc, double tol,
                               int64_t k, const double *H, int64_t ldh, void *Q, gs_dtype qt, int64_t ldq,
                               void *R, gs_dtype rt, int64_t ldr, int32_t *kept, float *cnorm, int32_t *rank,
                               int *nonfinite, void *ws, hipStream_t s, const CompressOverlap *ov = nullptr);
// Consecutive subsets of `subset` codebook rows, each compressed on its own;
// bases stacked in Q, coordinate blocks on R's block diagonal.
hipError_t run_compress_partitioned(const void *C, gs_dtype ct, int64_t M, int64_t D, int64_t ldc, double tol,
                                    int64_t subset, void *Q, gs_dtype qt, int64_t ldq, void *R, gs_dtype rt,
                                    int64_t ldr, int32_t *kept, float *cnorm, int32_t *ranks, int32_t *total,
                                    int *nonfinite, void *ws, hipStream_t s,
                                    const CompressOverlap *ov = nullptr);

}  // namespace gs
