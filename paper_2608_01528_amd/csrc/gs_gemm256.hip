// Large-tile bf16 and fp32 contractions for the long products of the
// Gram-Space path at batch sizes that fill the chip: project T = X Q^T (B
// stored N x K), reconstruct X = T Q and prob2vec T = P R (B stored K x N),
// the bound product, and the similarity scores (with the row argmax or
// softmax folded in when a tile holds whole rows).
//
// Work-group tile 256 x 256, 512 threads = 8 waves in a 2 x 4 arrangement;
// each wave owns a 128 x 64 sub-tile as 4 x 2 blocks of the 32 x 32 MFMA
// (32x32x16 bf16 or 32x32x2 fp32), 128 accumulators, two waves per SIMD so
// that one wave's waits overlap the other's matrix work.  A K-step of 64
// bf16 or 32 fp32 makes every row slice a whole 128-byte line, so L2 serves
// the operands in full-line requests.
//
// Operand tiles come into LDS by asynchronous buffer->LDS loads
// (buffer_load_dwordx4 ... lds) into two stages of 64 KiB, ordered by
// explicit vmcnt waits.  Each operand of a tile has its own buffer resource
// based at the tile's first row (or column) and sized to what the tile
// reads, so 32-bit offsets reach it and the hardware range check backs up
// the index clamping.  Each load instruction fills 1 KiB of LDS in lane
// order, so the layout is chosen through the 16-byte chunk each lane fetches:
//   row tile   (256 rows x 128 bytes): chunk c of row r at c ^ ((r >> 1) & 7)
//   k-row tile bf16 (64 x 256): chunk c of k-row k at c ^ (4 (k & 3))
//   k-row tile fp32 (32 x 256): chunk c of k-row k at c ^ (8 ((k >> 4) & 1))
// A 128-byte row covers half of the 64 banks, so the 16 rows of one read
// phase of ds_read_b128 reach all 16 bank groups only if the swizzle changes
// with r >> 1.  A transpose read (ds_read_b64_tr_b16) takes 4 chunks from each
// of 4 consecutive k-rows per 32 lanes, which the k-row swizzle spreads over
// all 64 banks.  Rows beyond the matrix reuse its last row (their results are
// discarded); fragment elements at k >= K are zeroed in registers in the last
// K-step.  Operands must have 16-byte aligned rows (ld a multiple of 8 bf16
// or 4 fp32): rows are read in 16-byte units up to the end of the row's last
// 16-byte chunk, which lies within ld.
#include "gs_internal.h"

namespace gs {
namespace {

constexpr int TM = 256, TN = 256;
constexpr int NTH = 256;                // threads of the sweep (4 waves)
// Waves of the product kernel: 8 (two per SIMD, 128 x 64 each, so one wave's
// waits overlap the other's matrix work) or 4 (one per SIMD, 128 x 128).
constexpr int GEMM_NW = 8;
template <int NW> struct Waves {
    static constexpr int WTN = NW == 4 ? 128 : 64;   // columns of a wave's sub-tile
    static constexpr int NJ = WTN / 32;             // 32-column MFMA blocks per wave
    static constexpr int IPW = 32 / NW;             // 1 KiB load instructions per wave per operand tile
    static constexpr int NTHR = 64 * NW;
    // rows wm = 128 (w / (NW / 2)) .. + 127, columns wn = WTN (w % (NW / 2)) .. + WTN - 1
    static __device__ __forceinline__ int wm(int w) { return (w / (NW / 2)) * 128; }
    static __device__ __forceinline__ int wn(int w) { return (w % (NW / 2)) * WTN; }
};
constexpr int NSTAGE = 2;
constexpr int OPT = TM * 64;        // 16-bit units per staged operand tile (32 KiB)
constexpr int GROUP_M = 4;          // m-tiles that take each n-tile in turn
// bytes per staged output row of a wave's sub-tile (WTN values + 8 values of pad)
template <typename TO, int NW>
constexpr int ep_stride() { return Waves<NW>::WTN * (int)sizeof(TO) + 16 * (int)sizeof(TO) / 2; }
constexpr size_t STAGE_BYTES = (size_t)NSTAGE * 2 * OPT * sizeof(uint16_t);
constexpr size_t EPI_BYTES = (size_t)GEMM_NW * 64 * (Waves<GEMM_NW>::WTN * 4 + 32);   // fp32 staging of the product kernel
constexpr size_t LDS_BYTES = STAGE_BYTES > EPI_BYTES ? STAGE_BYTES : EPI_BYTES;

typedef float f16v __attribute__((ext_vector_type(16)));
typedef __bf16 bf8v __attribute__((ext_vector_type(8)));
typedef short s4v __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f4v __attribute__((ext_vector_type(4)));
#define AS_L __attribute__((address_space(3)))

// Operand element type: a staged row slice is always 128 bytes (TK elements)
// and a fragment one 16-byte chunk (PER elements) per lane.
template <typename T> struct Op;
template <> struct Op<bf16_t> {
    typedef bf8v V;
    typedef __bf16 E;
    static constexpr int TK = 64, PER = 8;
};
template <> struct Op<float> {
    typedef f4v V;
    typedef float E;
    static constexpr int TK = 32, PER = 4;
};

// s_waitcnt with vmcnt <= n (expcnt and lgkmcnt unconstrained), gfx9 encoding.
template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Buffer resource: base address, stride 0, byte extent, raw 32-bit format.
typedef int rsrc_t __attribute__((ext_vector_type(4)));
constexpr int RSRC_WORD3 = 0x00020000;

// Resource over the `bytes` bytes from base, starting DMA_BIAS bytes before
// it (only offsets of at least DMA_BIAS are used); wave-uniform.
constexpr int DMA_BIAS = 4096;
__device__ __forceinline__ rsrc_t make_rsrc(const void *base, int64_t bytes) {
    const uint64_t a = reinterpret_cast<uint64_t>(base) - DMA_BIAS;
    bytes += DMA_BIAS;
    const int n = bytes > 0x7fffffff ? 0x7fffffff : (int)bytes;
    rsrc_t r;
    r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
    r[1] = __builtin_amdgcn_readfirstlane((int)((uint32_t)(a >> 32) & 0xffffu));
    r[2] = __builtin_amdgcn_readfirstlane(n);
    r[3] = RSRC_WORD3;
    return r;
}

// Four buffer->LDS loads of 16 bytes per lane into four consecutive 1 KiB
// LDS blocks (lane l's bytes of load j land at lds + j KiB + 16 l), from one
// M0 value: the instruction offset (j KiB) moves both the LDS destination and
// the memory address, so the lane offset of load j is off[j] + DMA_BIAS -
// j KiB, which stays positive because the resource starts DMA_BIAS bytes
// before the operand.  Written as assembly so that the compiler neither
// waits for these loads before unrelated LDS reads (it cannot tell the
// stages apart) nor keeps the resource in vector registers; the loop's own
// vmcnt waits order them.  One wait state separates the M0 write from the
// first load.
__device__ __forceinline__ void dma16x4(const rsrc_t &r, const int off[4], const uint16_t *lds) {
    const int m0v = __builtin_amdgcn_readfirstlane((int)(size_t)(const AS_L void *)lds);
    asm volatile(
        "s_mov_b32 m0, %4\n\ts_nop 0\n\t"
        "buffer_load_dwordx4 %0, %5, 0 offen lds\n\t"
        "buffer_load_dwordx4 %1, %5, 0 offen offset:1024 lds\n\t"
        "buffer_load_dwordx4 %2, %5, 0 offen offset:2048 lds\n\t"
        "buffer_load_dwordx4 %3, %5, 0 offen offset:3072 lds"
        :
        : "v"(off[0] + DMA_BIAS), "v"(off[1] + DMA_BIAS - 1024), "v"(off[2] + DMA_BIAS - 2048),
          "v"(off[3] + DMA_BIAS - 3072), "s"(m0v), "s"(r)
        : "memory", "m0");
}

// Lane byte offset of instruction q (0..7) of this wave's share of a row tile.
template <typename T, int IPW>
__device__ __forceinline__ int rows_off(int64_t ld, int64_t nrows, int64_t k0, int64_t K, int tid, int q) {
    constexpr int P = Op<T>::PER;
    const int L = tid & 63;
    const int w = tid >> 6;
    const int64_t klast = ((K - 1) / P) * P;
    const int b = IPW * w + q;
    const int c = (L & 7) ^ (4 * (q & 1) + (L >> 4));
    int64_t kc = k0 + P * c;
    if (kc > klast) kc = klast;
    int64_t row = 8 * b + (L >> 3);
    if (row > nrows - 1) row = nrows - 1;
    return (int)((int64_t)sizeof(T) * (row * ld + kc));
}

// Instructions 4 h .. 4 h + 3 of this wave's share of a row tile.
template <typename T, int IPW>
__device__ __forceinline__ void dma_rows4(const rsrc_t &r, int64_t ld, int64_t nrows, int64_t k0, int64_t K,
                                          uint16_t *tile, int tid, int h) {
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    int off[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) off[j] = rows_off<T, IPW>(ld, nrows, k0, K, tid, 4 * h + j);
    dma16x4(r, off, tile + (IPW * w + 4 * h) * 512);
}

// k-row tile (bf16): 32 load instructions of 2 k-rows x 512 bytes; wave w
// issues blocks IPW w .. IPW w + IPW - 1 (IPW instructions per wave).  Lane L lands at k-row 2b + L/32, position L%32,
// so it fetches chunk (L%32) ^ (4 (k-row % 4)).  `r` starts at the tile's
// first column; ncols columns exist from there.
// k-row tile (fp32): 32 load instructions of one k-row x 1 KiB; lane L lands
// at position L of k-row b and fetches chunk L ^ (8 ((b / 16) % 2)), so the
// two half-waves of a column read (k-rows k and k + 16) use opposite halves
// of the banks.
template <typename T, int IPW>
__device__ __forceinline__ int krows_off(int64_t ld, int64_t k0, int64_t K, int64_t ncols, int tid, int q) {
    const int L = tid & 63;
    const int w = tid >> 6;
    constexpr int P = Op<T>::PER;
    const int64_t nlast = ((ncols - 1) / P) * P;
    const int b = IPW * w + q;
    int kl, c;
    if constexpr (sizeof(T) == 2) {
        kl = 2 * b + (L >> 5);
        c = (L & 31) ^ (4 * (kl & 3));
    } else {
        kl = b;
        c = L ^ (8 * ((b >> 4) & 1));
    }
    int64_t nc = P * c;
    if (nc > nlast) nc = nlast;
    int64_t k = k0 + kl;
    if (k > K - 1) k = K - 1;
    return (int)((int64_t)sizeof(T) * (k * ld + nc));
}

template <typename T, int IPW>
__device__ __forceinline__ void dma_krows4(const rsrc_t &r, int64_t ld, int64_t k0, int64_t K, int64_t ncols,
                                           uint16_t *tile, int tid, int h) {
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    int off[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) off[j] = krows_off<T, IPW>(ld, k0, K, ncols, tid, 4 * h + j);
    dma16x4(r, off, tile + (IPW * w + 4 * h) * 512);
}

// A (or N x K B) fragment: the 16-byte chunk c of row r (8 bf16 or 4 fp32
// consecutive k).
template <typename T>
__device__ __forceinline__ typename Op<T>::V frag_rows(const uint16_t *tile, int r, int c) {
    return *reinterpret_cast<const typename Op<T>::V *>(tile + r * 64 + ((c ^ ((r >> 1) & 7)) << 3));
}

// K x N fp32 fragment: the 4 consecutive k from 16 (lane / 32) + 4 q of
// column n0w + lane % 32, one read per k-row.
__device__ __forceinline__ f4v frag_krows_f32(const uint16_t *tile, int q, int n0w, int tid) {
    const int l = tid & 63, h = l >> 5;
    const int n = n0w + (l & 31);
    const float *base = reinterpret_cast<const float *>(tile) + (16 * h + 4 * q) * 256 +
                        ((((n >> 2) ^ (8 * h)) << 2) | (n & 3));
    return f4v{base[0], base[256], base[512], base[768]};
}

// K x N B fragment (8 consecutive k at kk + 8 (lane / 32), column
// n0w + lane % 32) by two transpose reads of 4 k each.
__device__ __forceinline__ bf8v frag_krows(const uint16_t *tile, int kk, int n0w, int tid) {
    const int l = tid & 63;
    const int g = l >> 4, a = l & 15;
    const int n = n0w + 16 * (g & 1) + 4 * (a & 3);
    const int k = kk + 8 * (g >> 1) + (a >> 2);
    const int off = (((n >> 3) ^ (4 * (k & 3))) << 3) + (n & 7);     // (k + 4) & 3 == k & 3
    const s4v lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((AS_L s4v *)(tile + k * TN + off));
    const s4v hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((AS_L s4v *)(tile + (k + 4) * TN + off));
    const s4v both[2] = {lo, hi};
    return *reinterpret_cast<const bf8v *>(both);
}

template <typename V>
__device__ __forceinline__ float sum_sq(const V v) {
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < (int)(sizeof(V) / sizeof(v[0])); ++e) {
        const float x = (float)v[e];
        s += x * x;
    }
    return s;
}

inline int64_t elt_bytes(gs_dtype t) { return t == GS_BF16 ? 2 : 4; }

template <typename TO> __device__ __forceinline__ TO to_out(float v);
template <> __device__ __forceinline__ float to_out<float>(float v) { return v; }
// hardware conversion, round to nearest even
template <> __device__ __forceinline__ bf16_t to_out<bf16_t>(float v) {
    return bf16_t{__builtin_bit_cast(uint16_t, (__bf16)v)};
}

// Two fp32 values as adjacent bf16 (round to nearest even), the first in the low half.
__device__ __forceinline__ uint32_t pack_bf16(float x, float y) {
    return (uint32_t)to_out<bf16_t>(x).bits | ((uint32_t)to_out<bf16_t>(y).bits << 16);
}

// Row of the output held by accumulator register g of a 32x32 block, for lane l.
__device__ __forceinline__ int acc_row(int g, int l) { return 8 * (g >> 2) + 4 * (l >> 5) + (g & 3); }

// The loads of one 256 x 256 tile (m0, n0): buffer resources over exactly
// what the tile reads (row slices end at column ceil(K / P) * P, k-row slices
// at column ceil(N / P) * P) and the issue of part p (0..1) of this wave's
// share of the operand tiles of K-step kt into a stage: with four waves,
// instructions 4p .. 4p + 3 (of 8) of each operand; with eight, the four of
// operand A (p = 0) or of operand B (p = 1).
template <typename T, bool BNN, int NW>
struct TileLoads {
    rsrc_t ra, rb;
    int64_t rows_a, rows_b, cols_b;
    __device__ __forceinline__ void init(const GemmArgs &g, int64_t m0, int64_t n0) {
        constexpr int P = Op<T>::PER;
        constexpr int64_t ES = sizeof(T);
        const T *A = static_cast<const T *>(g.A);
        const T *B = static_cast<const T *>(g.B);
        const int64_t kp = (g.K + P - 1) / P * P, np = (g.N + P - 1) / P * P;
        rows_a = (g.M - m0 < TM) ? (g.M - m0) : TM;
        ra = make_rsrc(A + m0 * g.lda, ES * ((rows_a - 1) * g.lda + kp));
        if (BNN) {
            cols_b = (g.N - n0 < TN) ? (g.N - n0) : TN;
            const int64_t span = (np - n0 < TN) ? (np - n0) : TN;
            rb = make_rsrc(B + n0, ES * ((g.K - 1) * g.ldb + span));
            rows_b = 0;
        } else {
            rows_b = (g.N - n0 < TN) ? (g.N - n0) : TN;
            rb = make_rsrc(B + n0 * g.ldb, ES * ((rows_b - 1) * g.ldb + kp));
            cols_b = 0;
        }
    }
    __device__ __forceinline__ void issue(const GemmArgs &g, int64_t kt, int p, uint16_t *st, int tid) const {
        constexpr int TK = Op<T>::TK, IPW = Waves<NW>::IPW;
        const int hp = (IPW == 8) ? p : 0;
        if (IPW == 8 || p == 0) dma_rows4<T, IPW>(ra, g.lda, rows_a, kt * TK, g.K, st, tid, hp);
        if (IPW == 8 || p == 1) {
            if (BNN) dma_krows4<T, IPW>(rb, g.ldb, kt * TK, g.K, cols_b, st + OPT, tid, hp);
            else dma_rows4<T, IPW>(rb, g.ldb, rows_b, kt * TK, g.K, st + OPT, tid, hp);
        }
    }
};

// LDS stage slot s (0 or 1): both operand tiles of one K-step.
__device__ __forceinline__ uint16_t *stage_slot(uint16_t *lds, int s) { return lds + s * (2 * OPT); }

// The 256 x 256 block (m0, n0) of A * Bop, accumulated into acc (zeroed
// here), by NW waves: wave w owns the rows and columns Waves<NW>::wm / wn
// give (128 x 128 with four waves, 128 x 64 with eight).  When SQA && sqa, sq[i] gathers this
// lane's share of sum_k A[row, k]^2 for row wm + 32 i + lane % 32 (lanes l
// and l + 32 hold the two k-halves of a row); when SQB && sqb, sb[j] does the same
// for row wn + 32 j + lane % 32 of an N x K operand.  Only k in [k_lo, k_hi)
// is accumulated (k_lo a multiple of the K-step).  K-step k_lo / TK + i uses
// stage slot (slot0 + i) mod 2.  With preissued the first stage's loads were
// issued by the caller, followed by `pending` (0, 16 or 32) other vector
// memory instructions of this wave that need not be waited for.  Returns once
// the last MFMA is issued; the stages stay in use until the caller's next
// barrier.
template <typename T, bool BNN, bool SQA, bool SQB, int NW, bool SWP = false>
__device__ __forceinline__ void mma_256(const GemmArgs &g, const TileLoads<T, BNN, NW> &tl, uint16_t *lds,
                                        int slot0, bool preissued, int pending,
                                        f16v acc[4][Waves<NW>::NJ], bool sqa, float sq[4], bool sqb,
                                        float sb[Waves<NW>::NJ], int64_t k_lo, int64_t k_hi, int tid) {
    constexpr int TK = Op<T>::TK, P = Op<T>::PER;
    constexpr int NJ = Waves<NW>::NJ;
    typedef typename Op<T>::V V;
    const int l = tid & 63, w = tid >> 6, h = l >> 5;
    const int wm = Waves<NW>::wm(w), wn = Waves<NW>::wn(w);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j) acc[i][j] = f16v{};
    const int64_t kt0 = k_lo / TK, kt1 = (k_hi + TK - 1) / TK;
    auto stage = [&](int64_t kt) { return stage_slot(lds, (int)((kt - kt0 + slot0) & 1)); };
    auto issue_part = [&](int64_t kt, int p) { tl.issue(g, kt, p, stage(kt), tid); };
    // Substep q (0..3) of a K-step: bf16 lanes take chunk 2q + lane / 32 (k
    // from 16 q + 8 (lane / 32)); fp32 lanes take chunk 4 (lane / 32) + q (k
    // from 16 (lane / 32) + 4 q), A and B alike, so each MFMA pairs the same k.
    struct Frags { V a[4], b[NJ]; };
    auto load_frags = [&](const uint16_t *st, int q, Frags &f) {
        const int c = (sizeof(T) == 2) ? 2 * q + h : 4 * h + q;
#pragma unroll
        for (int i = 0; i < 4; ++i) f.a[i] = frag_rows<T>(st, wm + 32 * i + (l & 31), c);
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            if constexpr (!BNN) f.b[j] = frag_rows<T>(st + OPT, wn + 32 * j + (l & 31), c);
            else if constexpr (sizeof(T) == 2) f.b[j] = frag_krows(st + OPT, 16 * q, wn + 32 * j, tid);
            else f.b[j] = frag_krows_f32(st + OPT, q, wn + 32 * j, tid);
        }
    };
    // In the last K-step, zero the fragment elements at k >= k_hi (both
    // operands: what lies there in LDS is row padding, a re-read chunk or
    // data past the range, possibly NaN).
    Frags f0, f1;
    auto mask_tail = [&](Frags &f, int64_t kt, int q) {
        if (kt * TK + TK <= k_hi) return;                // a full step
        const int64_t kb = kt * TK + ((sizeof(T) == 2) ? 16 * q + 8 * h : 16 * h + 4 * q);
#pragma unroll
        for (int e = 0; e < P; ++e)
            if (kb + e >= k_hi) {
#pragma unroll
                for (int i = 0; i < 4; ++i) f.a[i][e] = (typename Op<T>::E)0.f;
#pragma unroll
                for (int j = 0; j < NJ; ++j) f.b[j][e] = (typename Op<T>::E)0.f;
            }
    };
    auto mma = [&](const Frags &f) {
        // SWP: B's fragment is the first operand, so the block comes out
        // transposed (register g of lane l holds row l % 32, column
        // 8 (g / 4) + 4 (l / 32) + g % 4 of the block)
        if constexpr (sizeof(T) == 2) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < NJ; ++j)
                    acc[i][j] = SWP ? __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.b[j], f.a[i], acc[i][j], 0, 0, 0)
                                    : __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[i], f.b[j], acc[i][j], 0, 0, 0);
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < NJ; ++j)
                        acc[i][j] = SWP ? __builtin_amdgcn_mfma_f32_32x32x2f32(f.b[j][e], f.a[i][e], acc[i][j], 0, 0, 0)
                                        : __builtin_amdgcn_mfma_f32_32x32x2f32(f.a[i][e], f.b[j][e], acc[i][j], 0, 0, 0);
        }
        if (SQA && sqa) {
#pragma unroll
            for (int i = 0; i < 4; ++i) sq[i] += sum_sq(f.a[i]);
        }
        if (SQB && sqb) {
#pragma unroll
            for (int j = 0; j < NJ; ++j) sb[j] += sum_sq(f.b[j]);
        }
    };

    // Software pipeline over the four substeps of a step: the fragments of
    // the next substep are read while the MFMAs of the current one run, and
    // the loads of the next stage (into the slot the previous step read) go
    // out in two parts before the first two substeps, so they never queue
    // up in front of the MFMAs.  Before the last substep's MFMAs each
    // wave has its loads landed and its reads of the current slot back; one
    // barrier then makes the next stage visible and frees the current slot.
    auto step = [&](int64_t kt, bool next_is_last) {
        const uint16_t *cur = stage(kt);
        issue_part(kt + 1, 0);
        load_frags(cur, 1, f1);
        __builtin_amdgcn_sched_barrier(0);
        mma(f0);
        __builtin_amdgcn_sched_barrier(0);
        issue_part(kt + 1, 1);
        load_frags(cur, 2, f0);
        __builtin_amdgcn_sched_barrier(0);
        mma(f1);
        __builtin_amdgcn_sched_barrier(0);
        load_frags(cur, 3, f1);
        __builtin_amdgcn_sched_barrier(0);
        mma(f0);
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_waitcnt(0);       // this wave's loads and reads have returned
        __builtin_amdgcn_s_barrier();        // ... and every other wave's
        load_frags(stage(kt + 1), 0, f0);
        if (next_is_last) mask_tail(f0, kt + 1, 0);
        __builtin_amdgcn_sched_barrier(0);
        mma(f1);
    };

    if (!preissued) {
        issue_part(kt0, 0);
        issue_part(kt0, 1);
    }
    if (preissued && pending == 32) wait_vm<32>();
    else if (preissued && pending == 16) wait_vm<16>();
    else wait_vm<0>();
    __builtin_amdgcn_s_barrier();
    load_frags(stage(kt0), 0, f0);
    if (kt1 - kt0 == 1) mask_tail(f0, kt0, 0);
    // the steady state has no tail handling: the last two steps are peeled
    for (int64_t kt = kt0; kt + 2 < kt1; ++kt) step(kt, false);
    if (kt1 - kt0 >= 2) step(kt1 - 2, true);
    {
        const int64_t kt = kt1 - 1;
        const uint16_t *cur = stage(kt);
        load_frags(cur, 1, f1);
        mask_tail(f1, kt, 1);
        mma(f0);
        load_frags(cur, 2, f0);
        mask_tail(f0, kt, 2);
        mma(f1);
        load_frags(cur, 3, f1);
        mask_tail(f1, kt, 3);
        mma(f0);
        mma(f1);
    }
}

// Tile order shared by the 256 x 256 kernels.  Work-group ids are dealt to
// the 8 XCDs round robin, so XCD x runs logical tiles [x per, (x + 1) per);
// in logical order, groups of GROUP_M m-tiles take each n-tile in turn, so
// the tiles one XCD runs together share A row blocks and B column blocks in
// L2.
__device__ __forceinline__ void tile_of(int64_t lt, int64_t nM, int64_t nN, int64_t &m0, int64_t &n0) {
    const int64_t grp = lt / (GROUP_M * nN);
    const int64_t first_m = grp * GROUP_M;
    const int64_t gm = (nM - first_m < GROUP_M) ? (nM - first_m) : GROUP_M;
    const int64_t within = lt - grp * GROUP_M * nN;
    m0 = (first_m + within % gm) * TM;
    n0 = (within / gm) * TN;
}

// K range of tile column n0 when B is a lower-echelon R (R[j][k] == 0 for
// k > j): as the K x N operand (P R, A R) its rows j < n0 are zero in this
// tile's columns; as the N x K operand (T R^T) its columns k >= n0 + TN are
// zero in this tile's rows.  Row norms of A summed from the fragments need
// the whole K range.
template <typename T, bool BNN>
__device__ __forceinline__ void k_range(const GemmArgs &g, int64_t n0, bool a_norms, int64_t &k_lo, int64_t &k_hi) {
    k_lo = 0;
    k_hi = g.K;
    if (!g.echelon || a_norms) return;
    if (BNN) {
        if (n0 < g.K) k_lo = (n0 / Op<T>::TK) * Op<T>::TK;   // (else R is zero there: keep one range)
    } else {
        k_hi = (n0 + TN < g.K) ? n0 + TN : g.K;
    }
}

// Plain products on 256 x 256 tiles (project, prob2vec, reconstruct, the
// second factor of a bound product).  Work-group b takes tile lt = x per + b / 8
// of its XCD x's range, then every (grid / 8)-th after it in that range: with
// one work-group per tile that is the tile alone; with a persistent grid (one
// work-group per CU) it walks its share of the range.
// When a tile's last MFMAs are issued, the next tile's first stage is loaded
// into the stage slot the last K-step did not read, and the output is staged
// through the other slot, 32 rows of every wave at a time (16 for fp32 output;
// 36 KiB in all), then written as whole 16-byte row chunks with streaming
// stores that are not waited for: the next tile waits only for its own first
// stage (issued before those stores), so the stores drain while it computes.
// With bf16 output the MFMAs take the B fragment as their first operand, so
// each lane holds runs of four consecutive columns of one row and stages them
// with one 8-byte LDS write per run (two-byte writes otherwise).
template <typename T, typename TO, bool BNN>
__global__ void __launch_bounds__(Waves<GEMM_NW>::NTHR) __attribute__((amdgpu_waves_per_eu(GEMM_NW / 4, GEMM_NW / 4)))
gemm256_store_kernel(GemmArgs g) {
    typedef Waves<GEMM_NW> W;
    constexpr int NJ = W::NJ, WTN = W::WTN, TK = Op<T>::TK;
    constexpr bool SWP = sizeof(TO) == 2;                    // transposed accumulator blocks
    constexpr int PR = sizeof(TO) == 2 ? 32 : 16;            // rows per staging pass
    constexpr int RP = PR / 2;                               // accumulator registers per pass (fp32)
    constexpr int EPC = 16 / (int)sizeof(TO);                // elements per 16-byte chunk
    constexpr int CPR = WTN / EPC;                           // chunks per sub-tile row
    constexpr int STRIDE = ep_stride<TO, GEMM_NW>();         // bytes per staged row
    constexpr int NSTORES = 4 * (32 / PR) * (PR * CPR / 64); // streaming stores per wave per interior tile
    static_assert(NSTORES == 16 || NSTORES == 32, "waits of mma_256");
    static_assert(GEMM_NW * PR * STRIDE <= 2 * OPT * 2, "staging fits one stage slot");
    static_assert(STRIDE % 16 == 0, "16-byte reads of staged rows");
    extern __shared__ float lds_f[];
    uint16_t *lds = reinterpret_cast<uint16_t *>(lds_f);
    const int64_t nM = (g.M + TM - 1) / TM, nN = (g.N + TN - 1) / TN;
    const int64_t total = nM * nN;
    const int64_t per = (total + 7) / 8;
    const int64_t xcd = blockIdx.x & 7, nq = gridDim.x >> 3;
    const int64_t lt_end = ((xcd + 1) * per < total) ? (xcd + 1) * per : total;
    int64_t lt = xcd * per + (blockIdx.x >> 3);
    if (lt >= lt_end) return;
    TO *C = static_cast<TO *>(g.C);
    const bool a_norms = g.rownorm2 != nullptr;

    int64_t m0, n0, k_lo, k_hi;
    tile_of(lt, nM, nN, m0, n0);
    k_range<T, BNN>(g, n0, a_norms, k_lo, k_hi);
    TileLoads<T, BNN, GEMM_NW> tl;
    tl.init(g, m0, n0);
    int slot0 = 0, pending = 0;
    tl.issue(g, k_lo / TK, 0, stage_slot(lds, slot0), threadIdx.x);
    tl.issue(g, k_lo / TK, 1, stage_slot(lds, slot0), threadIdx.x);
    for (;;) {
        // the thread id passes through an empty asm per tile, so the
        // lane-dependent addresses are recomputed here rather than kept live
        // (and spilled) across the product loop
        int tid = threadIdx.x;
        asm volatile("" : "+v"(tid));
        const int l = tid & 63, w = tid >> 6, h = l >> 5;
        const int wm = W::wm(w), wn = W::wn(w);
        f16v acc[4][NJ];
        // row norms of A from the fragments (the waves of the left column):
        // the rownorm2 side output of the tiles with n0 == 0
        const bool sqa = a_norms && n0 == 0 && wn == 0;
        float sq[4] = {0.f, 0.f, 0.f, 0.f}, sb[NJ];
        mma_256<T, BNN, true, false, GEMM_NW, SWP>(g, tl, lds, slot0, true, pending, acc, sqa, sq, false, sb,
                                                   k_lo, k_hi, tid);
        if (sqa) {
            // lanes l and l + 32 hold the two k-halves of row wm + 32 i + l % 32
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float t = sq[i] + __shfl_xor(sq[i], 32);
                const int64_t row = m0 + wm + 32 * i + l;
                if (l < 32 && row < g.M) g.rownorm2[row] = t;
            }
        }
        // the next tile's first stage, into the slot the last K-step did not read
        const int next_slot = (int)((slot0 + (k_hi + TK - 1) / TK - k_lo / TK) & 1);
        const int64_t nlt = lt + nq;
        const bool has_next = nlt < lt_end;
        int64_t m1 = 0, n1 = 0, k_lo1 = 0, k_hi1 = 0;
        TileLoads<T, BNN, GEMM_NW> tl1;
        if (has_next) {
            tile_of(nlt, nM, nN, m1, n1);
            k_range<T, BNN>(g, n1, a_norms, k_lo1, k_hi1);
            tl1.init(g, m1, n1);
            tl1.issue(g, k_lo1 / TK, 0, stage_slot(lds, next_slot), tid);
            tl1.issue(g, k_lo1 / TK, 1, stage_slot(lds, next_slot), tid);
        }

        // whole tile inside the output, rows 16-byte aligned: staged 16-byte stores
        const bool interior = ((reinterpret_cast<uintptr_t>(C) & 15) == 0) && (g.ldc % EPC == 0) &&
                              m0 + TM <= g.M && n0 + TN <= g.N;
        if (interior) {
            __syncthreads();              // every wave is done reading this tile's stages
            // Each wave stages PR rows of its 128 x WTN sub-tile at a time in
            // its own part of the other slot (rows padded against bank
            // collisions), then writes whole 16-byte row chunks.
            unsigned char *region =
                reinterpret_cast<unsigned char *>(stage_slot(lds, next_slot ^ 1)) + w * (PR * STRIDE);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int hh = 0; hh < 32 / PR; ++hh) {
                    if constexpr (SWP) {
                        // register 4 m + e of block (i, j): row 32 i + l % 32,
                        // column 32 j + 8 m + 4 h + e of the wave's sub-tile
#pragma unroll
                        for (int j = 0; j < NJ; ++j)
#pragma unroll
                            for (int m = 0; m < 4; ++m) {
                                const f16v &a = acc[i][j];
                                const uint2 v = {pack_bf16(a[4 * m], a[4 * m + 1]),
                                                 pack_bf16(a[4 * m + 2], a[4 * m + 3])};
                                *reinterpret_cast<uint2 *>(region + (l & 31) * STRIDE +
                                                           (32 * j + 8 * m + 4 * h) * (int)sizeof(TO)) = v;
                            }
                    } else {
#pragma unroll
                        for (int j = 0; j < NJ; ++j)
#pragma unroll
                            for (int gg = 0; gg < RP; ++gg) {
                                const int row = acc_row(RP * hh + gg, l) - PR * hh, col = 32 * j + (l & 31);
                                *reinterpret_cast<TO *>(region + row * STRIDE + col * (int)sizeof(TO)) =
                                    to_out<TO>(acc[i][j][RP * hh + gg]);
                            }
                    }
                    const int64_t rb = m0 + wm + 32 * i + PR * hh;   // first output row of this pass
#pragma unroll
                    for (int id = l; id < PR * CPR; id += 64) {
                        const int rr = id / CPR, cc = id % CPR;
                        u32x4 v = *reinterpret_cast<const u32x4 *>(region + rr * STRIDE + cc * 16);
                        TO *dst = C + (rb + rr) * g.ldc + (n0 + wn + cc * EPC);
                        if constexpr (sizeof(TO) == 4) {
                            if (g.mul_out) {   // second factor of a bound product
                                const f4v x = __builtin_bit_cast(f4v, v) *
                                              __builtin_nontemporal_load(reinterpret_cast<const f4v *>(dst));
                                v = __builtin_bit_cast(u32x4, x);
                            }
                        }
                        // streaming store: the output is not re-read by this kernel and
                        // should not displace the operand slices other tiles share in L2
                        __builtin_nontemporal_store(v, reinterpret_cast<u32x4 *>(dst));
                    }
                }
        } else {
            // edge tiles and unaligned outputs: element stores within bounds,
            // straight from the accumulators
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < NJ; ++j)
#pragma unroll
                    for (int e = 0; e < 16; ++e) {
                        const int64_t row = m0 + wm + 32 * i + (SWP ? (l & 31) : acc_row(e, l));
                        const int64_t col = n0 + wn + 32 * j + (SWP ? 8 * (e >> 2) + 4 * h + (e & 3) : (l & 31));
                        if (row < g.M && col < g.N) {
                            TO x = to_out<TO>(acc[i][j][e]);
                            if constexpr (sizeof(TO) == 4) {
                                if (g.mul_out) x = x * C[row * g.ldc + col];
                            }
                            C[row * g.ldc + col] = x;
                        }
                    }
        }
        if (!has_next) break;
        // the stores just issued (a fixed count on interior tiles without
        // loads in the epilogue) need not land before the next tile starts
        pending = (interior && !g.mul_out) ? NSTORES : 0;
        lt = nlt;
        m0 = m1;
        n0 = n1;
        k_lo = k_lo1;
        k_hi = k_hi1;
        tl = tl1;
        slot0 = next_slot;
    }
}

// a, b: (value, index) pairs; the larger value wins, the lower index on ties
__device__ __forceinline__ void fold_max(float &v, int &i, float v2, int i2) {
    if (v2 > v || (v2 == v && i2 < i)) { v = v2; i = i2; }
}

// Row results folded into the scores epilogue when a tile holds whole rows.
constexpr int FUSE_NONE = 0, FUSE_ARGMAX = 1, FUSE_SOFTMAX = 2;

// Similarity scores on 256 x 256 tiles (fp32 output, B = R stored N x K):
// out = scale * acc / (||x_row|| ||c_col||) for cosine (row norms from qnorm2
// or from the A fragments, column norms from cnorm or from the B fragments),
// scale * acc for dot; one tile per work-group.  FUSE (only with N <= 256)
// also writes the row argmax, or replaces the scores by the row softmax.
template <typename T, int FUSE>
__global__ void __launch_bounds__(Waves<GEMM_NW>::NTHR) __attribute__((amdgpu_waves_per_eu(GEMM_NW / 4, GEMM_NW / 4)))
scores256_kernel(GemmArgs g) {
    typedef Waves<GEMM_NW> W;
    typedef float TO;
    constexpr bool BNN = false, SCALED = true;
    constexpr int NJ = W::NJ, WTN = W::WTN;
    extern __shared__ float lds_f[];
    uint16_t *lds = reinterpret_cast<uint16_t *>(lds_f);
    const int64_t nM = (g.M + TM - 1) / TM, nN = (g.N + TN - 1) / TN;
    const int64_t total = nM * nN;
    // Work-group ids are dealt to the 8 XCDs round robin: XCD x runs the
    // logical tiles [x per, (x + 1) per) in order.
    const int64_t per = (total + 7) / 8;
    const int64_t lt = (int64_t)(blockIdx.x & 7) * per + (blockIdx.x >> 3);
    if (lt >= total) return;
    int64_t m0, n0;
    tile_of(lt, nM, nN, m0, n0);

    const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int wm = W::wm(w), wn = W::wn(w);
    f16v acc[4][NJ];
    // row norms of A from the fragments already in registers (the waves of
    // the left column, wn == 0) for cosine scores without qnorm2; column
    // norms of B likewise (the waves of the top row, wm == 0) without cnorm
    const bool sqa = g.cosine && g.qnorm2 == nullptr && wn == 0;
    const bool sqb = g.cosine && g.cnorm == nullptr && wm == 0;
    float sq[4] = {0.f, 0.f, 0.f, 0.f}, sb[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j) sb[j] = 0.f;
    int64_t k_lo, k_hi;
    k_range<T, BNN>(g, n0, g.cosine && g.qnorm2 == nullptr, k_lo, k_hi);
    TileLoads<T, BNN, GEMM_NW> tl;
    tl.init(g, m0, n0);
    mma_256<T, BNN, true, SCALED, GEMM_NW>(g, tl, lds, 0, false, 0, acc, sqa, sq, sqb, sb, k_lo, k_hi, threadIdx.x);

    float *rq = lds_f + LDS_BYTES / sizeof(float);   // SCALED: scale / ||x|| per row of the tile
    float *cn = rq + TM;                             // SCALED: 1 / ||c|| per column of the tile
    if (SCALED) {
        const int t = threadIdx.x;
        if (!g.cosine) {
            if (t < TM) {
                rq[t] = g.scale;
                cn[t] = 1.f;
            }
        } else {
            if (g.qnorm2) {
                const float n2 = (t < TM && m0 + t < g.M) ? g.qnorm2[m0 + t] : 1.f;
                if (t < TM) rq[t] = (n2 > 0.f) ? g.scale / sqrtf(n2) : 0.f;
            } else if (sqa) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float n2 = sq[i] + __shfl_xor(sq[i], 32);
                    if (l < 32) rq[wm + 32 * i + l] = (n2 > 0.f) ? g.scale / sqrtf(n2) : 0.f;
                }
            }
            if (g.cnorm) {
                const float c = (t < TN && n0 + t < g.N) ? g.cnorm[n0 + t] : 1.f;
                if (t < TN) cn[t] = (c > 0.f) ? 1.f / c : 0.f;
            } else if (sqb) {
#pragma unroll
                for (int j = 0; j < NJ; ++j) {
                    const float n2 = sb[j] + __shfl_xor(sb[j], 32);
                    if (l < 32) cn[wn + 32 * j + l] = (n2 > 0.f) ? 1.f / sqrtf(n2) : 0.f;
                }
            }
        }
    }

    // Epilogue: each wave stages its 128 x 64 sub-tile through its own LDS
    // region in two halves of 64 rows (rows padded so the column-wise writes
    // of the accumulator layout do not collide on banks), then writes whole
    // 16-byte row chunks with streaming stores.  With FUSE the tile holds
    // whole rows (N <= 256): lane l of each wave first scales row l of its
    // region in place and folds it into a partial (maximum, lowest index of
    // the maximum) or (maximum, sum of exponentials) for its 64 columns; the
    // four waves that share the rows combine their partials through LDS in a
    // fixed order, so the argmax is written here and the weights leave
    // normalised, with no second pass over the stored matrix.
    __syncthreads();                      // every wave is done with the operand stages
    TO *C = static_cast<TO *>(g.C);
    constexpr int EPC = 16 / (int)sizeof(TO);                 // elements per 16-byte chunk
    constexpr int CPR = WTN / EPC;                            // chunks per sub-tile row
    constexpr int STRIDE = ep_stride<TO, GEMM_NW>();          // bytes per staged row
    unsigned char *region = reinterpret_cast<unsigned char *>(lds) + w * (64 * ep_stride<float, GEMM_NW>());
    // whole tile inside the output, rows 16-byte aligned: plain 16-byte stores
    const bool interior = ((reinterpret_cast<uintptr_t>(C) & 15) == 0) && (g.ldc % EPC == 0) &&
                          m0 + TM <= g.M && n0 + TN <= g.N;
    float *pm = cn + TN;                  // FUSE: [column quarter][row] partial maxima
    float *px = pm + (TN / WTN) * TM;     // FUSE: partial indices (int) or sums of exponentials
    const int cq = wn / WTN;              // this wave's column quarter
    const int64_t nv = g.N - n0 - wn;     // this wave's columns inside the output
    const int ncol = nv < 0 ? 0 : (nv < WTN ? (int)nv : WTN);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int ii = 0; ii < 2; ++ii)
#pragma unroll
            for (int j = 0; j < NJ; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int row = 32 * ii + acc_row(r, l), col = 32 * j + (l & 31);
                    *reinterpret_cast<TO *>(region + row * STRIDE + col * (int)sizeof(TO)) =
                        to_out<TO>(acc[2 * h + ii][j][r]);
                }
        if constexpr (FUSE != FUSE_NONE) {
            const int trow = wm + 64 * h + l;                 // tile row folded by this lane
            float *mrow = reinterpret_cast<float *>(region + l * STRIDE);
            const float rql = rq[trow];
            float m = -INFINITY;
            int mi = 0;
#pragma unroll 4
            for (int q = 0; q < CPR; ++q) {
                const int qq = (q + l) & (CPR - 1);           // rotated: lanes spread over the banks
                f4v v = *reinterpret_cast<const f4v *>(mrow + 4 * qq);
                v = v * rql * *reinterpret_cast<const f4v *>(cn + wn + 4 * qq);
                *reinterpret_cast<f4v *>(mrow + 4 * qq) = v;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int c = 4 * qq + e;
                    if (c < ncol) {
                        if constexpr (FUSE == FUSE_ARGMAX) fold_max(m, mi, v[e], wn + c);
                        else m = fmaxf(m, v[e]);
                    }
                }
            }
            pm[cq * TM + trow] = m;
            if constexpr (FUSE == FUSE_ARGMAX) reinterpret_cast<int *>(px)[cq * TM + trow] = mi;
            __syncthreads();
            float rm = pm[trow];
            int ri = 0;
            if constexpr (FUSE == FUSE_ARGMAX) {
                ri = reinterpret_cast<const int *>(px)[trow];
#pragma unroll
                for (int c = 1; c < TN / WTN; ++c)
                    fold_max(rm, ri, pm[c * TM + trow], reinterpret_cast<const int *>(px)[c * TM + trow]);
                if (cq == 0 && m0 + trow < g.M) g.argmax[m0 + trow] = ri;
                if (!g.write_out) continue;                   // argmax only: no scores leave
            } else {
#pragma unroll
                for (int c = 1; c < TN / WTN; ++c) rm = fmaxf(rm, pm[c * TM + trow]);
                float z = 0.f;
#pragma unroll 4
                for (int q = 0; q < CPR; ++q) {
                    const int qq = (q + l) & (CPR - 1);
                    f4v v = *reinterpret_cast<const f4v *>(mrow + 4 * qq);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        v[e] = __expf(v[e] - rm);
                        if (4 * qq + e < ncol) z += v[e];
                    }
                    *reinterpret_cast<f4v *>(mrow + 4 * qq) = v;
                }
                px[cq * TM + trow] = z;
                __syncthreads();
                float rz = px[trow];
#pragma unroll
                for (int c = 1; c < TN / WTN; ++c) rz += px[c * TM + trow];
                // the partial maxima of these rows have all been read: the
                // slot of this wave's own rows now holds their factor
                pm[cq * TM + trow] = 1.f / rz;
            }
        }
        if (interior) {
#pragma unroll 4
            for (int id = l; id < 64 * CPR; id += 64) {
                const int rr = id / CPR, cc = id % CPR;
                u32x4 v = *reinterpret_cast<const u32x4 *>(region + rr * STRIDE + cc * 16);
                if constexpr (FUSE == FUSE_NONE) {
                    const f4v x = __builtin_bit_cast(f4v, v) * rq[wm + 64 * h + rr] *
                                  *reinterpret_cast<const f4v *>(cn + wn + cc * EPC);
                    v = __builtin_bit_cast(u32x4, x);
                } else if constexpr (FUSE == FUSE_SOFTMAX) {
                    v = __builtin_bit_cast(u32x4, __builtin_bit_cast(f4v, v) * pm[cq * TM + wm + 64 * h + rr]);
                }
                TO *dst = C + (m0 + wm + 64 * h + rr) * g.ldc + (n0 + wn + cc * EPC);
                // streaming store: the output is not re-read by this kernel and
                // should not displace the operand slices other tiles share in L2
                __builtin_nontemporal_store(v, reinterpret_cast<u32x4 *>(dst));
            }
        } else {
            // edge tiles and unaligned outputs: element stores within bounds
            for (int id = l; id < 64 * WTN; id += 64) {
                const int rr = id / WTN, cc = id % WTN;
                const int64_t grow = m0 + wm + 64 * h + rr, gcol = n0 + wn + cc;
                if (grow < g.M && gcol < g.N) {
                    TO x = *reinterpret_cast<const TO *>(region + rr * STRIDE + cc * (int)sizeof(TO));
                    if constexpr (FUSE == FUSE_NONE) x = x * rq[wm + 64 * h + rr] * cn[wn + cc];
                    else if constexpr (FUSE == FUSE_SOFTMAX) x = x * pm[cq * TM + wm + 64 * h + rr];
                    C[grow * g.ldc + gcol] = x;
                }
            }
        }
    }
}

// ------------------------------------------------ similarity / softmax sweep
//
// One work-group owns 256 query rows and sweeps the codebook in column blocks
// of 256 with the same product loop (B = R stored N x K).  After each block,
// the scaled scores of one half of the rows at a time (rows wm + 64 h ..
// + 63 of each wave) are staged in LDS: from there they are stored (scores
// requested, or raw softmax scores for the second pass) with 16-byte row
// chunks, and two threads per row fold them into the row's running state:
// (max, lowest index of the max) for similarity, (max, sum of exp) for
// softmax.  Softmax rows are finished by a second pass over the row block's
// stored scores.

// (max, sum of exp(x - max)) pairs
__device__ __forceinline__ void fold_sum(float &m, float &z, float m2, float z2) {
    const float mx = fmaxf(m, m2);
    const float a = (m == -INFINITY) ? 0.f : z * __expf(m - mx);
    const float b = (m2 == -INFINITY) ? 0.f : z2 * __expf(m2 - mx);
    m = mx;
    z = a + b;
}

constexpr size_t SWEEP_LDS_BYTES = LDS_BYTES + 4 * TM * sizeof(float);   // + rq, cn, rmax, rinv

// ROWN: row norms of T from its fragments (cosine without qnorm2); COLN:
// column norms of R from its fragments (cosine without cnorm).
template <typename T, bool SOFTMAX, bool ROWN, bool COLN>
__global__ void __launch_bounds__(NTH) __attribute__((amdgpu_waves_per_eu(1, 1)))
sweep256_kernel(GemmArgs g) {
    extern __shared__ float lds_f[];
    uint16_t *lds = reinterpret_cast<uint16_t *>(lds_f);
    float *rq = lds_f + LDS_BYTES / sizeof(float);   // 1 / ||x|| per row (or 1)
    float *cn = rq + TM;                             // 1 / ||c|| per column of the block (or 1)
    float *rmax = cn + TN, *rinv = rmax + TM;        // softmax row results
    const int64_t nM = (g.M + TM - 1) / TM, nN = (g.N + TN - 1) / TN;
    // row blocks dealt to the XCDs in contiguous ranges: the blocks one XCD
    // runs together sweep the same codebook block at about the same time
    const int64_t per = (nM + 7) / 8;
    const int64_t lt = (int64_t)(blockIdx.x & 7) * per + (blockIdx.x >> 3);
    if (lt >= nM) return;
    const int64_t m0 = lt * TM;
    const int t = threadIdx.x, l = t & 63, w = t >> 6;
    const int wm = (w >> 1) * 128, wn = (w & 1) * 128;
    float *out = static_cast<float *>(g.C);
    const bool write = SOFTMAX || g.write_out;
    const bool interior_rows = m0 + TM <= g.M;
    const bool vec_out = (reinterpret_cast<uintptr_t>(out) & 15) == 0 && g.ldc % 4 == 0;
    const float mul = SOFTMAX ? g.scale * g.beta : g.scale;
    // the staged half h holds rows wm + 64 h + (0 .. 63) of every wave; thread
    // pair (t, t ^ 1) folds staged row t / 2 of that half: wave region
    // 2 (t / 128) + (t & 1), local row (t / 2) % 64
    const int srow = (t >> 1) & 63, sreg = 2 * (t >> 7) + (t & 1);
    float run_m[2] = {-INFINITY, -INFINITY}, run_z[2] = {0.f, 0.f};
    int run_i[2] = {0, 0};

    constexpr int STRIDE = 128 * 4 + 32;             // staged fp32 row: 128 values + pad
    for (int64_t nt = 0; nt < nN; ++nt) {
        const int64_t n0 = nt * TN;
        f16v acc[4][4];
        const bool sqa = ROWN && (w & 1) == 0;
        const bool sqb = COLN && (w >> 1) == 0;
        float sa[4] = {0.f, 0.f, 0.f, 0.f}, sb[4] = {0.f, 0.f, 0.f, 0.f};
        // the thread id passes through an empty asm per block, so the
        // product loop's lane-dependent addresses are recomputed here rather
        // than kept live (and spilled) across the whole sweep
        int tid = threadIdx.x;
        asm volatile("" : "+v"(tid));
        TileLoads<T, false, 4> tl;
        tl.init(g, m0, n0);
        if (ROWN && nt == 0)
            mma_256<T, false, ROWN, COLN, 4>(g, tl, lds, 0, false, 0, acc, sqa, sa, sqb, sb, 0, g.K, tid);
        else
            mma_256<T, false, false, COLN, 4>(g, tl, lds, 0, false, 0, acc, false, sa, sqb, sb, 0, g.K, tid);

        // cosine factors of the rows (first block) and of this block's columns
        if (nt == 0) {
            if (!g.cosine) {
                rq[t] = 1.f;
            } else if (!ROWN) {
                const float n2 = (m0 + t < g.M) ? g.qnorm2[m0 + t] : 1.f;
                rq[t] = (n2 > 0.f) ? 1.f / sqrtf(n2) : 0.f;
            } else if (sqa) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float n2 = sa[i] + __shfl_xor(sa[i], 32);
                    if (l < 32) rq[wm + 32 * i + l] = (n2 > 0.f) ? 1.f / sqrtf(n2) : 0.f;
                }
            }
        }
        if (!g.cosine) {
            cn[t] = 1.f;
        } else if (!COLN) {
            const float c = (n0 + t < g.N) ? g.cnorm[n0 + t] : 1.f;
            cn[t] = (c > 0.f) ? 1.f / c : 0.f;
        } else if (sqb) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const float n2 = sb[j] + __shfl_xor(sb[j], 32);
                if (l < 32) cn[wn + 32 * j + l] = (n2 > 0.f) ? 1.f / sqrtf(n2) : 0.f;
            }
        }
        // every wave is done with the stages (reused for staging) and the
        // factors are in place
        lds_barrier();

        const int64_t ncols = (g.N - n0 < TN) ? (g.N - n0) : TN;
        unsigned char *region = reinterpret_cast<unsigned char *>(lds) + w * (64 * STRIDE);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            // stage the raw accumulators of rows wm + 64 h .. + 63 of this wave
#pragma unroll
            for (int ii = 0; ii < 2; ++ii)
#pragma unroll
                for (int j = 0; j < 4; ++j)
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int row = 32 * ii + acc_row(r, l), col = 32 * j + (l & 31);
                        *reinterpret_cast<float *>(region + row * STRIDE + col * 4) = acc[2 * h + ii][j][r];
                    }
            lds_barrier();
            // score of staged (row, 4 columns): raw * (mul / (||x|| ||c||)), one
            // expression for the stored scores and the fold
            if (write) {
                const bool full = vec_out && interior_rows && n0 + wn + 128 <= g.N;
#pragma unroll 4
                for (int id = l; id < 64 * 32; id += 64) {
                    const int rr = id >> 5, cc = id & 31;
                    const int64_t grow = m0 + wm + 64 * h + rr, gcol = n0 + wn + 4 * cc;
                    const f4v raw = *reinterpret_cast<const f4v *>(region + rr * STRIDE + cc * 16);
                    const f4v cf = *reinterpret_cast<const f4v *>(cn + wn + 4 * cc);
                    const f4v v = raw * (mul * rq[wm + 64 * h + rr]) * cf;
                    float *dst = out + grow * g.ldc + gcol;
                    if (full) {
                        *reinterpret_cast<f4v *>(dst) = v;
                    } else if (grow < g.M) {
                        for (int e = 0; e < 4; ++e)
                            if (gcol + e < g.N) dst[e] = v[e];
                    }
                }
            }
            // fold: thread t scans the 128 staged columns of its row, then pairs up
            {
                const float *src = reinterpret_cast<const float *>(
                    reinterpret_cast<const unsigned char *>(lds) + sreg * (64 * STRIDE) + srow * STRIDE);
                const int half = 128 * (t & 1);
                const float f = mul * rq[128 * (t >> 7) + 64 * h + srow];
                float m = -INFINITY, z = 0.f;
                int mi = 0;
#pragma unroll 2
                for (int c4 = 0; c4 < 32; ++c4) {
                    const f4v v = *reinterpret_cast<const f4v *>(src + 4 * c4) * f *
                                  *reinterpret_cast<const f4v *>(cn + half + 4 * c4);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int c = half + 4 * c4 + e;
                        if (c < ncols && v[e] > m) { m = v[e]; mi = (int)n0 + c; }
                    }
                }
                if (SOFTMAX && m != -INFINITY) {
#pragma unroll 2
                    for (int c4 = 0; c4 < 32; ++c4) {
                        const f4v v = *reinterpret_cast<const f4v *>(src + 4 * c4) * f *
                                      *reinterpret_cast<const f4v *>(cn + half + 4 * c4);
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (half + 4 * c4 + e < ncols) z += __expf(v[e] - m);
                    }
                }
                // the partner thread holds the other 128 columns of the row
                const float m2 = __shfl_xor(m, 1), z2 = __shfl_xor(z, 1);
                const int i2 = __shfl_xor(mi, 1);
                if (SOFTMAX) {
                    fold_sum(m, z, m2, z2);
                    fold_sum(run_m[h], run_z[h], m, z);
                } else {
                    fold_max(m, mi, m2, i2);
                    fold_max(run_m[h], run_i[h], m, mi);
                }
            }
            lds_barrier();    // the staging region is rewritten next
        }
    }

    // rows owned by thread pair (t, t ^ 1) in half h: wm + 64 h + srow of wave
    // region sreg, i.e. 128 (t / 128) + 64 h + srow
    if (!SOFTMAX) {
        if (g.argmax && (t & 1) == 0) {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int64_t row = m0 + 128 * (t >> 7) + 64 * h + srow;
                if (row < g.M) g.argmax[row] = run_i[h];
            }
        }
        return;
    }
    if ((t & 1) == 0) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int rl = 128 * (t >> 7) + 64 * h + srow;
            rmax[rl] = run_m[h];
            rinv[rl] = 1.f / run_z[h];
        }
    }
    // the second pass reads scores other threads stored to global memory
    __syncthreads();
    softmax_rows(out, g.ldc, m0, (g.M - m0 < TM) ? (g.M - m0) : TM, g.N, rmax, rinv, vec_out, NTH);
}

template <typename T, typename TO>
hipError_t launch_to(bool b_nn, const GemmArgs &a, hipStream_t s) {
    // Tiles of equal work (all interior, the whole K range): one persistent
    // work-group per CU (256 CUs, 32 per XCD; the tile count is at least 256,
    // gemm256_fits).  Otherwise one work-group per tile, so the dispatcher
    // balances tiles of unequal work (edge tiles, echelon K ranges), which a
    // fixed stride would let drift apart and lose their shared L2 slices.
    const int64_t total = ((a.M + TM - 1) / TM) * ((a.N + TN - 1) / TN);
    const bool uniform = !a.echelon && a.M % TM == 0 && a.N % TN == 0;
    const dim3 grid(uniform ? 256u : (unsigned)(8 * ((total + 7) / 8)));
    const size_t lds = 2 * 2 * OPT * sizeof(uint16_t);      // the two stage slots
    const void *k = b_nn ? reinterpret_cast<const void *>(gemm256_store_kernel<T, TO, true>)
                         : reinterpret_cast<const void *>(gemm256_store_kernel<T, TO, false>);
    hipError_t e = raise_lds_limit(k, lds);
    if (e != hipSuccess) return e;
    const dim3 block(Waves<GEMM_NW>::NTHR);
    if (b_nn) hipLaunchKernelGGL((gemm256_store_kernel<T, TO, true>), grid, block, lds, s, a);
    else hipLaunchKernelGGL((gemm256_store_kernel<T, TO, false>), grid, block, lds, s, a);
    return hipGetLastError();
}

constexpr size_t SCORES_LDS_BYTES = LDS_BYTES + 2 * TM * sizeof(float);   // + row and column factors
// + partial row results of the four column quarters (FUSE)
constexpr size_t SCORES_FUSED_LDS_BYTES = SCORES_LDS_BYTES + 2 * (TN / Waves<GEMM_NW>::WTN) * TM * sizeof(float);

// One wave per row: the maximum of the row and its lowest column index.
__global__ void __launch_bounds__(256) rows_argmax_kernel(const float *S, int64_t lds, int64_t B, int64_t M,
                                                          int32_t *idx) {
    const int l = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= B) return;
    const float *s = S + row * lds;
    float m = -INFINITY;
    int mi = 0;
#pragma unroll 8
    for (int64_t c = l; c < M; c += 64) {
        const float v = s[c];
        if (v > m) { m = v; mi = (int)c; }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const float m2 = __shfl_xor(m, o);
        const int i2 = __shfl_xor(mi, o);
        fold_max(m, mi, m2, i2);
    }
    if (l == 0) idx[row] = mi;
}

// One wave per row, in place: softmax of the row (max-subtracted), the row
// held in registers (16-byte pieces; M <= 4 * 64 * V4, rows 16-byte aligned),
// so it is read once and written once.
template <int V4>
__global__ void __launch_bounds__(256) rows_softmax_reg_kernel(float *A, int64_t lda, int64_t B, int64_t M) {
    const int l = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= B) return;
    float *a = A + row * lda;
    f4v v[V4];
    float m = -INFINITY;
#pragma unroll
    for (int i = 0; i < V4; ++i) {
        const int64_t c = 4 * (l + 64 * i);
        if (c + 4 <= M) {
            v[i] = __builtin_nontemporal_load(reinterpret_cast<const f4v *>(a + c));
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) v[i][e] = (c + e < M) ? a[c + e] : -INFINITY;
        }
        m = fmaxf(m, fmaxf(fmaxf(v[i][0], v[i][1]), fmaxf(v[i][2], v[i][3])));
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
    float z = 0.f;
#pragma unroll
    for (int i = 0; i < V4; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            v[i][e] = __expf(v[i][e] - m);          // exp(-inf) = 0 past the row's end
            z += v[i][e];
        }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) z += __shfl_xor(z, o);
    const float iz = 1.f / z;
#pragma unroll
    for (int i = 0; i < V4; ++i) {
        const int64_t c = 4 * (l + 64 * i);
        const f4v w = v[i] * iz;
        if (c + 4 <= M) {
            __builtin_nontemporal_store(w, reinterpret_cast<f4v *>(a + c));
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (c + e < M) a[c + e] = w[e];
        }
    }
}

// One wave per row, in place: softmax of the row (max-subtracted).
__global__ void __launch_bounds__(256) rows_softmax_kernel(float *A, int64_t lda, int64_t B, int64_t M) {
    const int l = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= B) return;
    float *a = A + row * lda;
    float m = -INFINITY;
#pragma unroll 8
    for (int64_t c = l; c < M; c += 64) m = fmaxf(m, a[c]);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
    float z = 0.f;
#pragma unroll 8
    for (int64_t c = l; c < M; c += 64) z += __expf(a[c] - m);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) z += __shfl_xor(z, o);
    const float iz = 1.f / z;
#pragma unroll 8
    for (int64_t c = l; c < M; c += 64) a[c] = __expf(a[c] - m) * iz;
}

// One wave per row of the scores W: the lowest index of the row maximum into
// argmax (when non-null), then A = softmax(beta * W) (when non-null; A may be
// W itself: the row is in registers before anything is written).  Rows in
// registers as 16-byte pieces (M <= 4 * 64 * V4, rows of W and A 16-byte
// aligned), so W is read once and A written once.
template <int V4>
__global__ void __launch_bounds__(256) rows_sim_attn_reg_kernel(const float *W, int64_t ldw, int64_t B, int64_t M,
                                                               int32_t *argmax, float beta, float *A, int64_t lda) {
    const int l = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= B) return;
    const float *w = W + row * ldw;
    f4v v[V4];
#pragma unroll
    for (int i = 0; i < V4; ++i) {
        const int64_t c = 4 * (l + 64 * i);
        if (c + 4 <= M) {
            v[i] = __builtin_nontemporal_load(reinterpret_cast<const f4v *>(w + c));
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) v[i][e] = (c + e < M) ? w[c + e] : -INFINITY;
        }
    }
    if (argmax) {
        // each lane visits its columns in increasing order, so the strict
        // comparison keeps its lowest maximal index; padding (-inf) never wins
        float m = -INFINITY;
        int mi = 0;
#pragma unroll
        for (int i = 0; i < V4; ++i)
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (v[i][e] > m) { m = v[i][e]; mi = 4 * (l + 64 * i) + e; }
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) {
            const float m2 = __shfl_xor(m, o);
            const int i2 = __shfl_xor(mi, o);
            fold_max(m, mi, m2, i2);
        }
        if (l == 0) argmax[row] = mi;
    }
    if (!A) return;
    float mb = -INFINITY;
#pragma unroll
    for (int i = 0; i < V4; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            v[i][e] = (4 * (l + 64 * i) + e < M) ? beta * v[i][e] : -INFINITY;
            mb = fmaxf(mb, v[i][e]);
        }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) mb = fmaxf(mb, __shfl_xor(mb, o));
    float z = 0.f;
#pragma unroll
    for (int i = 0; i < V4; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            v[i][e] = __expf(v[i][e] - mb);          // exp(-inf) = 0 past the row's end
            z += v[i][e];
        }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) z += __shfl_xor(z, o);
    const float iz = 1.f / z;
    float *a = A + row * lda;
#pragma unroll
    for (int i = 0; i < V4; ++i) {
        const int64_t c = 4 * (l + 64 * i);
        const f4v q = v[i] * iz;
        if (c + 4 <= M) {
            __builtin_nontemporal_store(q, reinterpret_cast<f4v *>(a + c));
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (c + e < M) a[c + e] = q[e];
        }
    }
}

// The same for any M and alignment: one wave per row, three sweeps (maximum
// and its index, sum of exponentials, weights).  In place is safe: each
// element is read and written by the same lane.
__global__ void __launch_bounds__(256) rows_sim_attn_kernel(const float *W, int64_t ldw, int64_t B, int64_t M,
                                                           int32_t *argmax, float beta, float *A, int64_t lda) {
    const int l = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= B) return;
    const float *w = W + row * ldw;
    float m = -INFINITY, mb = -INFINITY;
    int mi = 0;
    for (int64_t c = l; c < M; c += 64) {
        const float x = w[c];
        if (x > m) { m = x; mi = (int)c; }
        mb = fmaxf(mb, beta * x);
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const float m2 = __shfl_xor(m, o);
        const int i2 = __shfl_xor(mi, o);
        fold_max(m, mi, m2, i2);
        mb = fmaxf(mb, __shfl_xor(mb, o));
    }
    if (argmax && l == 0) argmax[row] = mi;
    if (!A) return;
    float z = 0.f;
    for (int64_t c = l; c < M; c += 64) z += __expf(beta * w[c] - mb);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) z += __shfl_xor(z, o);
    const float iz = 1.f / z;
    float *a = A + row * lda;
    for (int64_t c = l; c < M; c += 64) a[c] = __expf(beta * w[c] - mb) * iz;
}

// Scores of a few query rows (A, g.M rows) against every codebook row (B
// stored N x K): one work-group per (query row, J codebook rows), the K range
// split over its 256 threads, which also sum the squares for cosine norms
// not given.  out[b, j] = scale * <a_b, b_j> (/ (||a_b|| ||b_j||) for cosine,
// 0 if a norm is 0).
template <typename T, int J>
__global__ void __launch_bounds__(256) few_rows_kernel(GemmArgs g) {
    constexpr int NV = 2 * J + 1;   // J products, J codebook squares, the query square
    const int64_t b = blockIdx.y;
    const int64_t j0 = (int64_t)blockIdx.x * J;
    const int nj = (g.N - j0 < J) ? (int)(g.N - j0) : J;
    const T *x = static_cast<const T *>(g.A) + b * g.lda;
    const T *Bm = static_cast<const T *>(g.B) + j0 * g.ldb;
    float v[NV];
#pragma unroll
    for (int i = 0; i < NV; ++i) v[i] = 0.f;
    for (int64_t k = threadIdx.x; k < g.K; k += 256) {
        const float xv = ld_f32<T>(x, k);
        v[2 * J] += xv * xv;
#pragma unroll
        for (int j = 0; j < J; ++j)
            if (j < nj) {
                const float c = ld_f32<T>(Bm, (int64_t)j * g.ldb + k);
                v[j] += xv * c;
                v[J + j] += c * c;
            }
    }
#pragma unroll
    for (int i = 0; i < NV; ++i)
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) v[i] += __shfl_xor(v[i], o);
    __shared__ float part[4][NV];
    const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
    if (l == 0) {
#pragma unroll
        for (int i = 0; i < NV; ++i) part[w][i] = v[i];
    }
    __syncthreads();
    if ((int)threadIdx.x < nj) {
        const int j = threadIdx.x;
        const float dot = part[0][j] + part[1][j] + part[2][j] + part[3][j];
        float f = g.scale;
        if (g.cosine) {
            const float n2 = g.qnorm2 ? g.qnorm2[b] : part[0][2 * J] + part[1][2 * J] + part[2][2 * J] + part[3][2 * J];
            const float c = g.cnorm ? g.cnorm[j0 + j]
                                    : sqrtf(part[0][J + j] + part[1][J + j] + part[2][J + j] + part[3][J + j]);
            f = (n2 > 0.f && c > 0.f) ? g.scale / (sqrtf(n2) * c) : 0.f;
        }
        static_cast<float *>(g.C)[b * g.ldc + j0 + j] = dot * f;
    }
}

template <typename T, bool SOFTMAX, bool ROWN, bool COLN>
hipError_t launch_sweep(const GemmArgs &a, hipStream_t s) {
    const int64_t nM = (a.M + TM - 1) / TM;
    const dim3 grid((unsigned)(8 * ((nM + 7) / 8)));
    const void *k = reinterpret_cast<const void *>(sweep256_kernel<T, SOFTMAX, ROWN, COLN>);
    hipError_t e = raise_lds_limit(k, SWEEP_LDS_BYTES);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((sweep256_kernel<T, SOFTMAX, ROWN, COLN>), grid, dim3(NTH), SWEEP_LDS_BYTES, s, a);
    return hipGetLastError();
}

template <typename T, bool SOFTMAX>
hipError_t launch_sweep_norms(const GemmArgs &a, hipStream_t s) {
    const bool rown = a.cosine && a.qnorm2 == nullptr, coln = a.cosine && a.cnorm == nullptr;
    if (rown) return coln ? launch_sweep<T, SOFTMAX, true, true>(a, s) : launch_sweep<T, SOFTMAX, true, false>(a, s);
    return coln ? launch_sweep<T, SOFTMAX, false, true>(a, s) : launch_sweep<T, SOFTMAX, false, false>(a, s);
}

template <typename T, int FUSE>
hipError_t launch_scores_fuse(const GemmArgs &b, hipStream_t s) {
    const int64_t total = ((b.M + TM - 1) / TM) * ((b.N + TN - 1) / TN);
    const dim3 grid((unsigned)(8 * ((total + 7) / 8)));
    const size_t lds = FUSE == FUSE_NONE ? SCORES_LDS_BYTES : SCORES_FUSED_LDS_BYTES;
    const void *k = reinterpret_cast<const void *>(scores256_kernel<T, FUSE>);
    hipError_t e = raise_lds_limit(k, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((scores256_kernel<T, FUSE>), grid, dim3(Waves<GEMM_NW>::NTHR), lds, s, b);
    return hipGetLastError();
}

// `fused`: the row pass was folded into the epilogue (whole rows per tile).
template <typename T>
hipError_t launch_scores(const GemmArgs &a, bool softmax, bool &fused, hipStream_t s) {
    GemmArgs b = a;
    if (softmax) b.scale = a.scale * a.beta;      // the softmax acts on beta * score
    fused = a.N <= TN && (softmax || a.argmax);
    if (!fused) return launch_scores_fuse<T, FUSE_NONE>(b, s);
    return softmax ? launch_scores_fuse<T, FUSE_SOFTMAX>(b, s) : launch_scores_fuse<T, FUSE_ARGMAX>(b, s);
}

}  // namespace

hipError_t launch_scores256(gs_dtype t, const GemmArgs &a, bool softmax, hipStream_t s) {
    if (a.M == 0 || a.N == 0) return hipSuccess;
    bool fused = false;
    hipError_t e = (t == GS_BF16) ? launch_scores<bf16_t>(a, softmax, fused, s)
                                  : launch_scores<float>(a, softmax, fused, s);
    if (e != hipSuccess || fused) return e;
    return launch_rows_pass(softmax, static_cast<float *>(a.C), a.ldc, a.M, a.N, softmax ? nullptr : a.argmax, s);
}

hipError_t launch_few_rows(gs_dtype t, const GemmArgs &a, bool softmax, hipStream_t s) {
    if (a.M == 0 || a.N == 0) return hipSuccess;
    GemmArgs b = a;
    if (softmax) b.scale = a.scale * a.beta;      // the softmax acts on beta * score
    // 8 codebook rows per work-group while that still gives a round of 256
    // work-groups, else one (more work-groups, each reading its query again)
    if (a.M * ((a.N + 7) / 8) >= 256) {
        const dim3 grid((unsigned)((a.N + 7) / 8), (unsigned)a.M);
        if (t == GS_BF16) hipLaunchKernelGGL((few_rows_kernel<bf16_t, 8>), grid, dim3(256), 0, s, b);
        else hipLaunchKernelGGL((few_rows_kernel<float, 8>), grid, dim3(256), 0, s, b);
    } else {
        const dim3 grid((unsigned)a.N, (unsigned)a.M);
        if (t == GS_BF16) hipLaunchKernelGGL((few_rows_kernel<bf16_t, 1>), grid, dim3(256), 0, s, b);
        else hipLaunchKernelGGL((few_rows_kernel<float, 1>), grid, dim3(256), 0, s, b);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_rows_pass(softmax, static_cast<float *>(a.C), a.ldc, a.M, a.N, softmax ? nullptr : a.argmax, s);
}

hipError_t launch_rows_pass(bool softmax, float *out, int64_t ld, int64_t B, int64_t M, int32_t *argmax,
                            hipStream_t s) {
    if (B == 0 || M == 0) return hipSuccess;
    const dim3 rgrid((unsigned)((B + 3) / 4));
    if (softmax) {
        // rows in registers when they fit (16-byte aligned rows of up to 2048)
        const bool aligned = (reinterpret_cast<uintptr_t>(out) & 15) == 0 && ld % 4 == 0;
        if (aligned && M <= 512) hipLaunchKernelGGL((rows_softmax_reg_kernel<2>), rgrid, dim3(256), 0, s, out, ld, B, M);
        else if (aligned && M <= 2048) hipLaunchKernelGGL((rows_softmax_reg_kernel<8>), rgrid, dim3(256), 0, s, out, ld, B, M);
        else hipLaunchKernelGGL(rows_softmax_kernel, rgrid, dim3(256), 0, s, out, ld, B, M);
        return hipGetLastError();
    }
    if (argmax) {
        hipLaunchKernelGGL(rows_argmax_kernel, rgrid, dim3(256), 0, s, out, ld, B, M, argmax);
        return hipGetLastError();
    }
    return hipSuccess;
}

hipError_t launch_sim_attn_pass(const float *W, int64_t ldw, int64_t B, int64_t M, int32_t *argmax, float beta,
                                float *A, int64_t lda, hipStream_t s) {
    if (B == 0 || M == 0 || (!argmax && !A)) return hipSuccess;
    const dim3 rgrid((unsigned)((B + 3) / 4));
    const auto al = [](const float *p, int64_t ld) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0 && ld % 4 == 0; };
    const bool aligned = al(W, ldw) && (!A || al(A, lda));
    if (aligned && M <= 512)
        hipLaunchKernelGGL((rows_sim_attn_reg_kernel<2>), rgrid, dim3(256), 0, s, W, ldw, B, M, argmax, beta, A, lda);
    else if (aligned && M <= 2048)
        hipLaunchKernelGGL((rows_sim_attn_reg_kernel<8>), rgrid, dim3(256), 0, s, W, ldw, B, M, argmax, beta, A, lda);
    else
        hipLaunchKernelGGL(rows_sim_attn_kernel, rgrid, dim3(256), 0, s, W, ldw, B, M, argmax, beta, A, lda);
    return hipGetLastError();
}

bool sweep256_fits(gs_dtype t, const GemmArgs &a) {
    // at least one 256-row block per CU; offsets within the buffer resources
    // below 2^31
    if ((a.M + TM - 1) / TM < 256) return false;
    const int64_t es = elt_bytes(t), lim = ((int64_t)1 << 31) - 8192;
    return es * (TM * a.lda + a.K + 8) < lim && es * (TN * a.ldb + a.K + 8) < lim;
}

hipError_t launch_sweep256(gs_dtype t, bool softmax, const GemmArgs &a, hipStream_t s) {
    if (a.M == 0 || a.N == 0) return hipSuccess;
    if (t == GS_BF16) return softmax ? launch_sweep_norms<bf16_t, true>(a, s) : launch_sweep_norms<bf16_t, false>(a, s);
    return softmax ? launch_sweep_norms<float, true>(a, s) : launch_sweep_norms<float, false>(a, s);
}

bool gemm256_fits(gs_dtype t, const GemmArgs &a, bool b_nn) {
    // at least one full round of 256 x 256 tiles over the 256 CUs; smaller
    // products keep the 128 x 128 tiles, which spread over more CUs
    const int64_t total = ((a.M + TM - 1) / TM) * ((a.N + TN - 1) / TN);
    if (total < 256) return false;
    // byte offsets within a tile's buffer resources stay below 2^31
    const int64_t es = elt_bytes(t), lim = ((int64_t)1 << 31) - 8192;
    if (es * (TM * a.lda + a.K + 8) >= lim) return false;
    if (b_nn) return es * (a.K * a.ldb + TN) < lim;
    return es * (TN * a.ldb + a.K + 8) < lim;
}

hipError_t launch_gemm256(gs_dtype t, gs_dtype tout, bool b_nn, const GemmArgs &a, hipStream_t s) {
    if (a.M == 0 || a.N == 0) return hipSuccess;
    if (t == GS_BF16) return (tout == GS_BF16) ? launch_to<bf16_t, bf16_t>(b_nn, a, s) : launch_to<bf16_t, float>(b_nn, a, s);
    return (tout == GS_BF16) ? launch_to<float, bf16_t>(b_nn, a, s) : launch_to<float, float>(b_nn, a, s);
}

}  // namespace gs
