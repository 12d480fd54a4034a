// Large-tile bf16 contraction for the long products of the Gram-Space path at
// batch sizes that fill the chip: project T = X Q^T (B stored N x K),
// reconstruct X = T Q and prob2vec T = P R (B stored K x N).
//
// Work-group tile 256 x 256, K-step 32, 256 threads = 4 waves in a 2 x 2
// arrangement; each wave owns a 128 x 128 sub-tile as 4 x 4 blocks of the
// 32x32x16 bf16 MFMA, whose 256 accumulators sit in the accumulation
// registers (one wave per SIMD).  Per flop this moves half the bytes of a
// 128 x 128 tile through L2 and LDS, and each wave issues 16 MFMAs per 8
// fragment reads, so the LDS reads of one k-substep hide behind the MFMAs of
// the previous one.
//
// Operand tiles come into LDS by asynchronous global->LDS loads
// (global_load_lds_dwordx4), 4 stages deep (4 x 32 KiB), one barrier per
// K-step.  Each load instruction fills 1 KiB of LDS in lane order, so the
// layout is chosen through the 16-byte chunk each lane fetches:
//   row tile   [256][32]: chunk c of row r sits at position c ^ ((r >> 2) & 3)
//   k-row tile [32][256]: chunk c of k-row k sits at position c ^ (4 (k & 3))
// A 64-byte row covers a quarter of the 64 banks, so the 16 rows of one read
// phase of ds_read_b128 reach all 16 bank groups only if the swizzle changes
// with r >> 2.  A transpose read (ds_read_b64_tr_b16) takes 4 chunks from each
// of 4 consecutive k-rows per 32 lanes, which the k-row swizzle spreads over
// all 64 banks.  Rows beyond the matrix reuse its last row (their results are
// discarded); k beyond K is zeroed in LDS in the last step.  Operands must have
// 16-byte aligned rows (ld a multiple of 8): rows are read in 16-byte units up
// to column ceil(cols / 8) * 8 <= ld.
#include "gs_internal.h"

namespace gs {
namespace {

constexpr int TM = 256, TN = 256, TK = 32;
constexpr int NTH = 256;
constexpr int NSTAGE = 4;
constexpr int OPT = TM * TK;        // bf16 per staged operand tile (16 KiB)
constexpr int OPS = 8;              // load instructions per stage and wave
constexpr int GROUP_M = 4;          // m-tiles that take each n-tile in turn
constexpr size_t LDS_BYTES = (size_t)NSTAGE * 2 * OPT * sizeof(uint16_t);

typedef float f16v __attribute__((ext_vector_type(16)));
typedef __bf16 bf8v __attribute__((ext_vector_type(8)));
typedef short s4v __attribute__((ext_vector_type(4)));
#define AS_G __attribute__((address_space(1)))
#define AS_L __attribute__((address_space(3)))

// s_waitcnt with vmcnt <= n (expcnt and lgkmcnt unconstrained), gfx9 encoding.
template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Wait until at most `later` stages of this wave's loads (clamped to MAXS)
// are still in flight.
template <int MAXS>
__device__ __forceinline__ void wait_stages(int64_t later) {
    if constexpr (MAXS <= 0) {
        wait_vm<0>();
    } else {
        if (later >= MAXS) wait_vm<OPS * MAXS>();
        else wait_stages<MAXS - 1>(later);
    }
}

__device__ __forceinline__ void dma16(const void *g, uint16_t *lds) {
    __builtin_amdgcn_global_load_lds((const AS_G void *)g, (AS_L void *)lds, 16, 0, 0);
}

// Row tile: 16 load instructions of 16 rows x 64 bytes; wave w issues blocks
// 4w .. 4w+3.  Lane L lands at row 16b + L/4, position L%4, so it fetches
// chunk (L%4) ^ ((L/16)%4).
__device__ __forceinline__ void dma_rows(const bf16_t *base, int64_t ld, int64_t row0, int64_t nrows,
                                         int64_t k0, int64_t K, uint16_t *tile) {
    const int L = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int c = (L & 3) ^ ((L >> 4) & 3);
    int64_t kc = k0 + 8 * c;
    const int64_t klast = ((K - 1) >> 3) << 3;
    if (kc > klast) kc = klast;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int b = 4 * w + q;
        int64_t row = row0 + 16 * b + (L >> 2);
        if (row > nrows - 1) row = nrows - 1;
        dma16(base + row * ld + kc, tile + b * 512);
    }
}

// k-row tile: 16 load instructions of 2 k-rows x 512 bytes; wave w issues
// blocks 4w .. 4w+3.  Lane L lands at k-row 2b + L/32, position L%32, so it
// fetches chunk (L%32) ^ (4 (k-row % 4)).
__device__ __forceinline__ void dma_krows(const bf16_t *base, int64_t ld, int64_t k0, int64_t K, int64_t n0,
                                          int64_t N, uint16_t *tile) {
    const int L = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t nlast = ((N - 1) >> 3) << 3;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int b = 4 * w + q;
        const int kl = 2 * b + (L >> 5);
        const int c = (L & 31) ^ (4 * (kl & 3));
        int64_t nc = n0 + 8 * c;
        if (nc > nlast) nc = nlast;
        int64_t k = k0 + kl;
        if (k > K - 1) k = K - 1;
        dma16(base + k * ld + nc, tile + b * 512);
    }
}

// Zero the k >= kvalid part of a staged row tile / k-row tile.
__device__ __forceinline__ void zero_rows_tail(uint16_t *tile, int kvalid) {
    for (int e = threadIdx.x; e < TM * TK; e += NTH) {
        const int r = e >> 5, kl = e & 31;
        if (kl >= kvalid) tile[r * TK + ((((kl >> 3) ^ ((r >> 2) & 3))) << 3) + (kl & 7)] = 0;
    }
}
__device__ __forceinline__ void zero_krows_tail(uint16_t *tile, int kvalid) {
    for (int e = threadIdx.x; e < TK * TN; e += NTH)
        if ((e >> 8) >= kvalid) tile[e] = 0;
}

// A (or N x K B) fragment: 8 consecutive k of chunk c of row r.
__device__ __forceinline__ bf8v frag_rows(const uint16_t *tile, int r, int c) {
    return *reinterpret_cast<const bf8v *>(tile + r * TK + ((c ^ ((r >> 2) & 3)) << 3));
}

// K x N B fragment (8 consecutive k at kk + 8 (lane / 32), column
// n0w + lane % 32) by two transpose reads of 4 k each.
__device__ __forceinline__ bf8v frag_krows(const uint16_t *tile, int kk, int n0w) {
    const int l = threadIdx.x & 63;
    const int g = l >> 4, a = l & 15;
    const int n = n0w + 16 * (g & 1) + 4 * (a & 3);
    const int k = kk + 8 * (g >> 1) + (a >> 2);
    const int off = (((n >> 3) ^ (4 * (k & 3))) << 3) + (n & 7);     // (k + 4) & 3 == k & 3
    const s4v lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((AS_L s4v *)(tile + k * TN + off));
    const s4v hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((AS_L s4v *)(tile + (k + 4) * TN + off));
    const s4v both[2] = {lo, hi};
    return *reinterpret_cast<const bf8v *>(both);
}

__device__ __forceinline__ float sum_sq(const bf8v v) {
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const float x = (float)v[e];
        s += x * x;
    }
    return s;
}

// Row of the output held by accumulator register g of a 32x32 block, for lane l.
__device__ __forceinline__ int acc_row(int g, int l) { return 8 * (g >> 2) + 4 * (l >> 5) + (g & 3); }

template <typename TO, bool BNN>
__global__ void __launch_bounds__(NTH) __attribute__((amdgpu_waves_per_eu(1, 1)))
gemm256_kernel(GemmArgs g) {
    extern __shared__ float lds_f[];
    uint16_t *lds = reinterpret_cast<uint16_t *>(lds_f);
    const int64_t nM = (g.M + TM - 1) / TM, nN = (g.N + TN - 1) / TN;
    const int64_t total = nM * nN;
    // Work-group ids are dealt to the 8 XCDs round robin: XCD x runs the
    // logical tiles [x per, (x + 1) per) in order.
    const int64_t per = (total + 7) / 8;
    const int64_t lt = (int64_t)(blockIdx.x & 7) * per + (blockIdx.x >> 3);
    if (lt >= total) return;
    // Logical order: groups of GROUP_M m-tiles take each n-tile in turn, so the
    // tiles one XCD runs together share A row blocks and B column blocks in L2.
    const int64_t grp = lt / (GROUP_M * nN);
    const int64_t first_m = grp * GROUP_M;
    const int64_t gm = (nM - first_m < GROUP_M) ? (nM - first_m) : GROUP_M;
    const int64_t within = lt - grp * GROUP_M * nN;
    const int64_t m0 = (first_m + within % gm) * TM;
    const int64_t n0 = (within / gm) * TN;

    const bf16_t *A = static_cast<const bf16_t *>(g.A);
    const bf16_t *B = static_cast<const bf16_t *>(g.B);
    const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int wm = (w >> 1) * 128, wn = (w & 1) * 128;

    f16v acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f16v{};
    // row norms of A from the fragments already in registers: the waves of
    // the left column (wn == 0) of the tiles with n0 == 0
    const bool sqa = g.rownorm2 != nullptr && n0 == 0 && (w & 1) == 0;
    float sq[4] = {0.f, 0.f, 0.f, 0.f};

    const int64_t nk = (g.K + TK - 1) / TK;
    auto stage = [&](int64_t kt) { return lds + (int)(kt % NSTAGE) * (2 * OPT); };
    auto issue = [&](int64_t kt) {
        uint16_t *st = stage(kt);
        dma_rows(A, g.lda, m0, g.M, kt * TK, g.K, st);
        if (BNN) dma_krows(B, g.ldb, kt * TK, g.K, n0, g.N, st + OPT);
        else dma_rows(B, g.ldb, n0, g.N, kt * TK, g.K, st + OPT);
    };

    for (int s = 0; s < NSTAGE - 1; ++s)
        if (s < nk) issue(s);
    for (int64_t kt = 0; kt < nk; ++kt) {
        // step kt has landed once at most the loads of the later stages
        // already issued (kt + 1 .. min(kt + NSTAGE - 2, nk - 1)) remain
        wait_stages<NSTAGE - 2>(nk - 1 - kt);
        __builtin_amdgcn_s_barrier();
        // refill the slot every wave finished reading in step kt - 1
        if (kt + NSTAGE - 1 < nk) issue(kt + NSTAGE - 1);
        uint16_t *cur = stage(kt);
        const uint16_t *As = cur, *Bs = cur + OPT;
        const int64_t kvalid = g.K - kt * TK;
        if (kvalid < TK) {
            zero_rows_tail(cur, (int)kvalid);
            if (BNN) zero_krows_tail(cur + OPT, (int)kvalid);
            else zero_rows_tail(cur + OPT, (int)kvalid);
            __builtin_amdgcn_s_waitcnt(0xc07f);    // lgkmcnt(0): the zeros are in LDS
            __builtin_amdgcn_s_barrier();
        }
#pragma unroll
        for (int kk = 0; kk < TK; kk += 16) {
            const int c = (kk >> 3) + (l >> 5);
            bf8v a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = frag_rows(As, wm + 32 * i + (l & 31), c);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                b[j] = BNN ? frag_krows(Bs, kk, wn + 32 * j) : frag_rows(Bs, wn + 32 * j + (l & 31), c);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
            if (sqa) {
#pragma unroll
                for (int i = 0; i < 4; ++i) sq[i] += sum_sq(a[i]);
            }
        }
    }

    if (sqa) {
        // lanes l and l + 32 hold the two k-halves of row wm + 32 i + l % 32
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float t = sq[i] + __shfl_xor(sq[i], 32);
            const int64_t row = m0 + wm + 32 * i + l;
            if (l < 32 && row < g.M) g.rownorm2[row] = t;
        }
    }

    TO *C = static_cast<TO *>(g.C);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t col = n0 + wn + 32 * j + (l & 31);
            if (col >= g.N) continue;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t row = m0 + wm + 32 * i + acc_row(r, l);
                if (row < g.M) st_f32<TO>(C, row * g.ldc + col, acc[i][j][r]);
            }
        }
}

template <typename TO>
hipError_t launch_to(bool b_nn, const GemmArgs &a, hipStream_t s) {
    const int64_t total = ((a.M + TM - 1) / TM) * ((a.N + TN - 1) / TN);
    const dim3 grid((unsigned)(8 * ((total + 7) / 8)));
    const void *k = b_nn ? reinterpret_cast<const void *>(gemm256_kernel<TO, true>)
                         : reinterpret_cast<const void *>(gemm256_kernel<TO, false>);
    hipError_t e = raise_lds_limit(k, LDS_BYTES);
    if (e != hipSuccess) return e;
    if (b_nn) hipLaunchKernelGGL((gemm256_kernel<TO, true>), grid, dim3(NTH), LDS_BYTES, s, a);
    else hipLaunchKernelGGL((gemm256_kernel<TO, false>), grid, dim3(NTH), LDS_BYTES, s, a);
    return hipGetLastError();
}

}  // namespace

bool gemm256_fits(const GemmArgs &a) {
    // at least one full round of 256 x 256 tiles over the 256 CUs; smaller
    // products keep the 128 x 128 tiles, which spread over more CUs
    const int64_t total = ((a.M + TM - 1) / TM) * ((a.N + TN - 1) / TN);
    return total >= 256;
}

hipError_t launch_gemm256(gs_dtype tout, bool b_nn, const GemmArgs &a, hipStream_t s) {
    if (a.M == 0 || a.N == 0) return hipSuccess;
    if (tout == GS_BF16) return launch_to<bf16_t>(b_nn, a, s);
    return launch_to<float>(b_nn, a, s);
}

}  // namespace gs
