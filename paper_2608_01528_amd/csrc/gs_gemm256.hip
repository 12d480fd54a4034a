// Large-tile bf16 contraction for the long products of the Gram-Space path at
// batch sizes that fill the chip: project T = X Q^T (B stored N x K),
// reconstruct X = T Q and prob2vec T = P R (B stored K x N).
//
// Work-group tile 256 x 256, K-step 64, 256 threads = 4 waves in a 2 x 2
// arrangement; each wave owns a 128 x 128 sub-tile as 4 x 4 blocks of the
// 32x32x16 bf16 MFMA, whose 256 accumulators sit in the accumulation
// registers (one wave per SIMD).  Per flop this moves half the bytes of a
// 128 x 128 tile through L2 and LDS, and each wave issues 16 MFMAs per 8
// fragment reads.  A K-step of 64 bf16 makes every row slice a whole
// 128-byte line, so L2 serves the operands in full-line requests.
//
// Operand tiles come into LDS by asynchronous buffer->LDS loads
// (buffer_load_dwordx4 ... lds) into two stages of 64 KiB, ordered by
// explicit vmcnt waits.  Each operand of a tile has its own buffer resource
// based at the tile's first row (or column) and sized to what the tile
// reads, so 32-bit offsets reach it and the hardware range check backs up
// the index clamping.  Each load instruction fills 1 KiB of LDS in lane
// order, so the layout is chosen through the 16-byte chunk each lane fetches:
//   row tile   [256][64]: chunk c of row r sits at position c ^ ((r >> 1) & 7)
//   k-row tile [64][256]: chunk c of k-row k sits at position c ^ (4 (k & 3))
// A 128-byte row covers half of the 64 banks, so the 16 rows of one read
// phase of ds_read_b128 reach all 16 bank groups only if the swizzle changes
// with r >> 1.  A transpose read (ds_read_b64_tr_b16) takes 4 chunks from each
// of 4 consecutive k-rows per 32 lanes, which the k-row swizzle spreads over
// all 64 banks.  Rows beyond the matrix reuse its last row (their results are
// discarded); fragment elements at k >= K are zeroed in registers in the last
// K-step.  Operands must have 16-byte aligned rows (ld a multiple of 8): rows
// are read in 16-byte units up to column ceil(cols / 8) * 8 <= ld.
#include "gs_internal.h"

namespace gs {
namespace {

constexpr int TM = 256, TN = 256, TK = 64;
constexpr int NTH = 256;
constexpr int NSTAGE = 2;
constexpr int OPT = TM * TK;        // bf16 per staged operand tile (32 KiB)
constexpr int OPS = 16;             // load instructions per stage and wave
constexpr int GROUP_M = 4;          // m-tiles that take each n-tile in turn
constexpr int EP_STRIDE_MAX = 128 * 4 + 32;   // staged fp32 output row: 128 values + 32-byte pad
constexpr size_t STAGE_BYTES = (size_t)NSTAGE * 2 * OPT * sizeof(uint16_t);
constexpr size_t EPI_BYTES = (size_t)4 * 64 * EP_STRIDE_MAX;
constexpr size_t LDS_BYTES = STAGE_BYTES > EPI_BYTES ? STAGE_BYTES : EPI_BYTES;

typedef float f16v __attribute__((ext_vector_type(16)));
typedef __bf16 bf8v __attribute__((ext_vector_type(8)));
typedef short s4v __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
#define AS_L __attribute__((address_space(3)))

// s_waitcnt with vmcnt <= n (expcnt and lgkmcnt unconstrained), gfx9 encoding.
template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Buffer resource: base address, stride 0, byte extent, raw 32-bit format.
typedef int rsrc_t __attribute__((ext_vector_type(4)));
constexpr int RSRC_WORD3 = 0x00020000;

// Resource over `bytes` bytes from base (at most 2^31 - 1); wave-uniform.
__device__ __forceinline__ rsrc_t make_rsrc(const void *base, int64_t bytes) {
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    const int n = bytes > 0x7fffffff ? 0x7fffffff : (int)bytes;
    rsrc_t r;
    r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
    r[1] = __builtin_amdgcn_readfirstlane((int)((uint32_t)(a >> 32) & 0xffffu));
    r[2] = __builtin_amdgcn_readfirstlane(n);
    r[3] = RSRC_WORD3;
    return r;
}

// One buffer->LDS load of 16 bytes per lane: lane l's bytes land at
// lds + 16 l.  Written as assembly so that the compiler neither waits for
// these loads before unrelated LDS reads (it cannot tell the stages apart)
// nor keeps the resource in vector registers; the loop's own vmcnt waits
// order them.  M0 holds the LDS base; one wait state separates its write
// from the load.
__device__ __forceinline__ void dma16(const rsrc_t &r, int64_t byte_off, const uint16_t *lds) {
    const int m0v = __builtin_amdgcn_readfirstlane((int)(size_t)(const AS_L void *)lds);
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
                 :
                 : "v"((int)byte_off), "s"(r), "s"(m0v)
                 : "memory", "m0");
}

// Row tile: 32 load instructions of 8 rows x 128 bytes; wave w issues blocks
// 8w .. 8w+7.  Lane L lands at row 8b + L/8, position L%8, so it fetches
// chunk (L%8) ^ (((8b + L/8) >> 1) % 8) = (L%8) ^ (4 (b % 2) + L/16).  `r`
// starts at the tile's first row; rows past the last one (nrows rows from
// there) reuse it.
__device__ __forceinline__ void dma_rows(const rsrc_t &r, int64_t ld, int64_t nrows, int64_t k0, int64_t K,
                                         uint16_t *tile) {
    const int L = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t klast = ((K - 1) >> 3) << 3;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        const int b = 8 * w + q;
        const int c = (L & 7) ^ (4 * (q & 1) + (L >> 4));
        int64_t kc = k0 + 8 * c;
        if (kc > klast) kc = klast;
        int64_t row = 8 * b + (L >> 3);
        if (row > nrows - 1) row = nrows - 1;
        dma16(r, 2 * (row * ld + kc), tile + b * 512);
    }
}

// k-row tile: 32 load instructions of 2 k-rows x 512 bytes; wave w issues
// blocks 8w .. 8w+7.  Lane L lands at k-row 2b + L/32, position L%32, so it
// fetches chunk (L%32) ^ (4 (k-row % 4)).  `r` starts at the tile's first
// column; ncols columns exist from there.
__device__ __forceinline__ void dma_krows(const rsrc_t &r, int64_t ld, int64_t k0, int64_t K, int64_t ncols,
                                          uint16_t *tile) {
    const int L = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t nlast = ((ncols - 1) >> 3) << 3;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        const int b = 8 * w + q;
        const int kl = 2 * b + (L >> 5);
        const int c = (L & 31) ^ (4 * (kl & 3));
        int64_t nc = 8 * c;
        if (nc > nlast) nc = nlast;
        int64_t k = k0 + kl;
        if (k > K - 1) k = K - 1;
        dma16(r, 2 * (k * ld + nc), tile + b * 512);
    }
}

// A (or N x K B) fragment: 8 consecutive k of chunk c of row r.
__device__ __forceinline__ bf8v frag_rows(const uint16_t *tile, int r, int c) {
    return *reinterpret_cast<const bf8v *>(tile + r * TK + ((c ^ ((r >> 1) & 7)) << 3));
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

template <typename TO> __device__ __forceinline__ TO to_out(float v);
template <> __device__ __forceinline__ float to_out<float>(float v) { return v; }
// hardware conversion, round to nearest even
template <> __device__ __forceinline__ bf16_t to_out<bf16_t>(float v) {
    return bf16_t{__builtin_bit_cast(uint16_t, (__bf16)v)};
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
    // buffer resources over exactly what this tile reads (row slices end at
    // column ceil(K / 8) * 8, k-row slices at column ceil(N / 8) * 8)
    const int64_t k8 = (g.K + 7) / 8 * 8, n8 = (g.N + 7) / 8 * 8;
    const int64_t rows_a = (g.M - m0 < TM) ? (g.M - m0) : TM;
    const rsrc_t ra = make_rsrc(A + m0 * g.lda, 2 * ((rows_a - 1) * g.lda + k8));
    int64_t rows_b, cols_b;
    rsrc_t rb;
    if (BNN) {
        cols_b = (g.N - n0 < TN) ? (g.N - n0) : TN;
        const int64_t span = (n8 - n0 < TN) ? (n8 - n0) : TN;
        rb = make_rsrc(B + n0, 2 * ((g.K - 1) * g.ldb + span));
        rows_b = 0;
    } else {
        rows_b = (g.N - n0 < TN) ? (g.N - n0) : TN;
        rb = make_rsrc(B + n0 * g.ldb, 2 * ((rows_b - 1) * g.ldb + k8));
        cols_b = 0;
    }

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
        dma_rows(ra, g.lda, rows_a, kt * TK, g.K, st);
        if (BNN) dma_krows(rb, g.ldb, kt * TK, g.K, cols_b, st + OPT);
        else dma_rows(rb, g.ldb, rows_b, kt * TK, g.K, st + OPT);
    };
    struct Frags { bf8v a[4], b[4]; };
    auto load_frags = [&](const uint16_t *st, int kk, Frags &f) {
        const int c = (kk >> 3) + (l >> 5);
#pragma unroll
        for (int i = 0; i < 4; ++i) f.a[i] = frag_rows(st, wm + 32 * i + (l & 31), c);
#pragma unroll
        for (int j = 0; j < 4; ++j)
            f.b[j] = BNN ? frag_krows(st + OPT, kk, wn + 32 * j) : frag_rows(st + OPT, wn + 32 * j + (l & 31), c);
    };
    // In the last K-step, zero the fragment elements at k >= K (both operands:
    // what lies there in LDS is row padding or a re-read chunk, possibly NaN).
    Frags f0, f1;
    auto mask_tail = [&](Frags &f, int64_t kt, int kk) {
        if (kt * TK + TK <= g.K) return;                 // a full step
        const int64_t kb = kt * TK + kk + 8 * (l >> 5);  // first k of this lane's fragments
#pragma unroll
        for (int e = 0; e < 8; ++e)
            if (kb + e >= g.K) {
#pragma unroll
                for (int i = 0; i < 4; ++i) f.a[i][e] = (__bf16)0.f;
#pragma unroll
                for (int j = 0; j < 4; ++j) f.b[j][e] = (__bf16)0.f;
            }
    };
    auto mma = [&](const Frags &f) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[i], f.b[j], acc[i][j], 0, 0, 0);
        if (sqa) {
#pragma unroll
            for (int i = 0; i < 4; ++i) sq[i] += sum_sq(f.a[i]);
        }
    };

    // Software pipeline over the four k-substeps of 16 of a step: the
    // fragments of the next substep are read while the MFMAs of the current
    // one run.  Before the last substep's MFMAs each wave has its reads of
    // the current slot back and the next stage landed; one barrier then
    // hands the current slot to the load of step kt + 2.
    auto step = [&](int64_t kt, bool next_is_last) {
        const uint16_t *cur = stage(kt);
        load_frags(cur, 16, f1);
        __builtin_amdgcn_sched_barrier(0);
        mma(f0);
        __builtin_amdgcn_sched_barrier(0);
        load_frags(cur, 32, f0);
        __builtin_amdgcn_sched_barrier(0);
        mma(f1);
        __builtin_amdgcn_sched_barrier(0);
        load_frags(cur, 48, f1);
        __builtin_amdgcn_sched_barrier(0);
        mma(f0);
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_waitcnt(0);       // this wave's reads and loads have returned
        __builtin_amdgcn_s_barrier();        // ... and every other wave's
        if (kt + 2 < nk) issue(kt + 2);      // into the slot just read
        load_frags(stage(kt + 1), 0, f0);
        if (next_is_last) mask_tail(f0, kt + 1, 0);
        __builtin_amdgcn_sched_barrier(0);
        mma(f1);
    };

    issue(0);
    if (nk > 1) {
        issue(1);
        wait_vm<OPS>();                      // stage 0 has landed (stage 1 may be in flight)
    } else {
        wait_vm<0>();
    }
    __builtin_amdgcn_s_barrier();
    load_frags(stage(0), 0, f0);
    if (nk == 1) mask_tail(f0, 0, 0);
    // the steady state has no tail handling: the last two steps are peeled
    for (int64_t kt = 0; kt + 2 < nk; ++kt) step(kt, false);
    if (nk >= 2) step(nk - 2, true);
    {
        const int64_t kt = nk - 1;
        const uint16_t *cur = stage(kt);
        load_frags(cur, 16, f1);
        mask_tail(f1, kt, 16);
        mma(f0);
        load_frags(cur, 32, f0);
        mask_tail(f0, kt, 32);
        mma(f1);
        load_frags(cur, 48, f1);
        mask_tail(f1, kt, 48);
        mma(f0);
        mma(f1);
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

    // Epilogue: each wave stages its 128 x 128 sub-tile through its own LDS
    // region in two halves of 64 rows (rows padded so the column-wise writes
    // of the accumulator layout do not collide on banks), then writes whole
    // 16-byte row chunks with streaming stores.
    __syncthreads();                      // every wave is done with the operand stages
    TO *C = static_cast<TO *>(g.C);
    constexpr int EPC = 16 / (int)sizeof(TO);                 // elements per 16-byte chunk
    constexpr int CPR = 128 / EPC;                            // chunks per sub-tile row
    constexpr int STRIDE = 128 * (int)sizeof(TO) + 16 * (int)sizeof(TO) / 2;   // bytes per staged row
    unsigned char *region = reinterpret_cast<unsigned char *>(lds) + w * (64 * EP_STRIDE_MAX);
    // whole tile inside the output, rows 16-byte aligned: plain 16-byte stores
    const bool interior = ((reinterpret_cast<uintptr_t>(C) & 15) == 0) && (g.ldc % EPC == 0) &&
                          m0 + TM <= g.M && n0 + TN <= g.N;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int ii = 0; ii < 2; ++ii)
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int row = 32 * ii + acc_row(r, l), col = 32 * j + (l & 31);
                    *reinterpret_cast<TO *>(region + row * STRIDE + col * (int)sizeof(TO)) =
                        to_out<TO>(acc[2 * h + ii][j][r]);
                }
        if (interior) {
#pragma unroll 4
            for (int id = l; id < 64 * CPR; id += 64) {
                const int rr = id / CPR, cc = id % CPR;
                const u32x4 v = *reinterpret_cast<const u32x4 *>(region + rr * STRIDE + cc * 16);
                TO *dst = C + (m0 + wm + 64 * h + rr) * g.ldc + (n0 + wn + cc * EPC);
                // streaming store: the output is not re-read by this kernel and
                // should not displace the operand slices other tiles share in L2
                __builtin_nontemporal_store(v, reinterpret_cast<u32x4 *>(dst));
            }
        } else {
            // edge tiles and unaligned outputs: element stores within bounds
            for (int id = l; id < 64 * 128; id += 64) {
                const int rr = id >> 7, cc = id & 127;
                const int64_t grow = m0 + wm + 64 * h + rr, gcol = n0 + wn + cc;
                if (grow < g.M && gcol < g.N)
                    C[grow * g.ldc + gcol] = *reinterpret_cast<const TO *>(region + rr * STRIDE + cc * (int)sizeof(TO));
            }
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

bool gemm256_fits(const GemmArgs &a, bool b_nn) {
    // at least one full round of 256 x 256 tiles over the 256 CUs; smaller
    // products keep the 128 x 128 tiles, which spread over more CUs
    const int64_t total = ((a.M + TM - 1) / TM) * ((a.N + TN - 1) / TN);
    if (total < 256) return false;
    // byte offsets within a tile's buffer resources stay below 2^31
    const int64_t lim = (int64_t)1 << 31;
    if (2 * (TM * a.lda + a.K + 8) >= lim) return false;
    if (b_nn) return 2 * (a.K * a.ldb + TN) < lim;
    return 2 * (TN * a.ldb + a.K + 8) < lim;
}

hipError_t launch_gemm256(gs_dtype tout, bool b_nn, const GemmArgs &a, hipStream_t s) {
    if (a.M == 0 || a.N == 0) return hipSuccess;
    if (tout == GS_BF16) return launch_to<bf16_t>(b_nn, a, s);
    return launch_to<float>(b_nn, a, s);
}

}  // namespace gs
