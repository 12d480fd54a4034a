// Binding of two coordinate batches through the original domain in one pass:
// Z = ((T Q) .* (T2 Q)) Q^T for r <= 256 (fp32), the restored and bound
// vectors never leaving the chip.
//
// A work-group of four waves owns 128 batch rows, a wave 32 of them, and
// walks D in chunks of 32 columns.  Per chunk the r x 32 slice of Q is staged
// in LDS twice (d-major and r-major, rows padded against bank conflicts);
// then each wave
//   (1) forms Y1^T = Qc^T T^T and Y2^T = Qc^T T2^T for its rows (32 x 32
//       each, one 32x32x2 fp32 MFMA block, K = r), the T and T2 values read
//       from memory four consecutive k at a time,
//   (2) multiplies them element by element (Y^T = Y1^T .* Y2^T, in
//       registers),
//   (3) adds Y Qc^T to its r/32 accumulator blocks of Z (K = 32).
// The k order of the products is chosen so that no data moves between lanes:
// in (1) MFMA step (t, u) pairs k = 8t + u and 8t + 4 + u (the k-halves of a
// lane hold four consecutive k of one row); in (3) step s pairs
// d = 8(s/4) + (s%4) and d + 4, which is where the accumulator of (1) holds
// row i's value in register s, so Y^T's registers are the A operand of (3)
// as they are.  Each sum over D runs chunk by chunk in order.
#include "gs_internal.h"

namespace gs {
namespace {

constexpr int BC_WAVES = 4;
constexpr int BC_THREADS = 64 * BC_WAVES;
constexpr int BC_ROWS = 32 * BC_WAVES;      // batch rows per work-group
constexpr int BC_DC = 32;                   // columns of D per chunk

typedef float f4v __attribute__((ext_vector_type(4)));
typedef float f16v __attribute__((ext_vector_type(16)));

// LDS layout of a chunk for r padded to RB (a multiple of 32): qd[d][k] =
// Q[k][d0 + d] with rows of RB + 4 floats, qn[n][d] = Q[n][d0 + d] with rows
// of 36 floats; entries past r or past D are zero.
template <int RB> struct ChunkLayout {
    static constexpr int QD = RB + 4, QN = BC_DC + 4;
    static constexpr size_t BYTES = (size_t)(BC_DC * QD + RB * QN) * sizeof(float);
};

template <int RB>
__global__ void __launch_bounds__(BC_THREADS, 2) bind_coords_kernel(BindCoordsArgs a) {
    typedef ChunkLayout<RB> Ly;
    constexpr int NB = RB / 32;
    extern __shared__ float lds_bc[];
    float *qd = lds_bc;
    float *qn = lds_bc + BC_DC * Ly::QD;
    const int tid = threadIdx.x, l = tid & 63, w = tid >> 6, h = l >> 5, ln = l & 31;
    const float *T = a.T, *T2 = a.T2, *Q = a.Q;
    const int64_t r = a.r, D = a.D;
    const int64_t row0 = (int64_t)blockIdx.x * BC_ROWS + 32 * w;
    // this lane's row of T and T2 (the B operand of step 1); rows past the
    // batch reuse the last one and are not stored
    const int64_t brow = (row0 + ln < a.B) ? row0 + ln : a.B - 1;
    const float *trow = T + brow * a.ldt, *t2row = T2 + brow * a.ldt2;
    const bool vec = a.vec;                 // 16-byte aligned rows of T and T2
    f16v z[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) z[b] = f16v{};

    // Q[0..RB)[d0..d0+32): this thread's RB / 32 pieces of four columns,
    // read into registers (the next chunk's while the current one is
    // multiplied, when they fit) and written to LDS in both layouts
    constexpr int NP = RB * (BC_DC / 4) / BC_THREADS;
    constexpr bool PREFETCH = RB <= 128;
    f4v pre[NP];
    auto fetch = [&](int64_t d0) {
#pragma unroll
        for (int j = 0; j < NP; ++j) {
            const int i = tid + j * BC_THREADS;
            const int k = i / (BC_DC / 4), d4 = 4 * (i % (BC_DC / 4));
            f4v v = f4v{0.f, 0.f, 0.f, 0.f};
            if (k < r) {
                const float *q = Q + (int64_t)k * a.ldq + d0 + d4;
                if (a.qvec && d0 + d4 + 4 <= D) {
                    v = *reinterpret_cast<const f4v *>(q);
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e) v[e] = (d0 + d4 + e < D) ? q[e] : 0.f;
                }
            }
            pre[j] = v;
        }
    };
    auto stage = [&]() {
#pragma unroll
        for (int j = 0; j < NP; ++j) {
            const int i = tid + j * BC_THREADS;
            const int k = i / (BC_DC / 4), d4 = 4 * (i % (BC_DC / 4));
            *reinterpret_cast<f4v *>(qn + k * Ly::QN + d4) = pre[j];
#pragma unroll
            for (int e = 0; e < 4; ++e) qd[(d4 + e) * Ly::QD + k] = pre[j][e];
        }
    };
    if (PREFETCH) {
        fetch(0);
        stage();
        __syncthreads();
    }

    for (int64_t d0 = 0; d0 < D; d0 += BC_DC) {
        const bool more = d0 + BC_DC < D;
        if (!PREFETCH) {
            fetch(d0);
            stage();
            __syncthreads();
        } else if (more) {
            fetch(d0 + BC_DC);           // in flight during this chunk's products
        }

        // (1) Y1^T and Y2^T: C[d][row] over k = 8t + 4h + u
        f16v y1 = f16v{}, y2 = f16v{};
#pragma unroll 4
        for (int t = 0; t < RB / 8; ++t) {
            const int k0 = 8 * t + 4 * h;
            f4v tv, t2v;
            if (vec && k0 + 4 <= r) {
                tv = *reinterpret_cast<const f4v *>(trow + k0);
                t2v = *reinterpret_cast<const f4v *>(t2row + k0);
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    tv[e] = (k0 + e < r) ? trow[k0 + e] : 0.f;
                    t2v[e] = (k0 + e < r) ? t2row[k0 + e] : 0.f;
                }
            }
            const f4v qv = *reinterpret_cast<const f4v *>(qd + ln * Ly::QD + k0);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                y1 = __builtin_amdgcn_mfma_f32_32x32x2f32(qv[u], tv[u], y1, 0, 0, 0);
                y2 = __builtin_amdgcn_mfma_f32_32x32x2f32(qv[u], t2v[u], y2, 0, 0, 0);
            }
        }
        // (2) the bound values, still in the accumulator layout: register g
        // of lane (ln, h) holds Y[row ln][d = 8 (g / 4) + 4 h + g % 4]
        f16v y;
#pragma unroll
        for (int g = 0; g < 16; ++g) y[g] = y1[g] * y2[g];
        // (3) Z[row][n] += sum_d Y[row][d] Q[n][d0 + d]
#pragma unroll
        for (int a4 = 0; a4 < 4; ++a4) {
            f4v qv[NB];
#pragma unroll
            for (int b = 0; b < NB; ++b)
                qv[b] = *reinterpret_cast<const f4v *>(qn + (32 * b + ln) * Ly::QN + 8 * a4 + 4 * h);
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int b = 0; b < NB; ++b)
                    z[b] = __builtin_amdgcn_mfma_f32_32x32x2f32(y[4 * a4 + u], qv[b][u], z[b], 0, 0, 0);
        }
        __syncthreads();                  // every wave is done with this chunk
        if (PREFETCH && more) {
            stage();
            __syncthreads();
        }
    }

    // register g of block b holds Z[row0 + 8 (g / 4) + 4 h + g % 4][32 b + ln]
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        const int64_t col = 32 * b + ln;
#pragma unroll
        for (int g = 0; g < 16; ++g) {
            const int64_t row = row0 + 8 * (g >> 2) + 4 * h + (g & 3);
            if (row < a.B && col < r) a.Z[row * a.ldz + col] = z[b][g];
        }
    }
}

template <int RB>
hipError_t launch_rb(const BindCoordsArgs &a, hipStream_t s) {
    const size_t lds = ChunkLayout<RB>::BYTES;
    const void *k = reinterpret_cast<const void *>(bind_coords_kernel<RB>);
    hipError_t e = raise_lds_limit(k, lds);
    if (e != hipSuccess) return e;
    const dim3 grid((unsigned)((a.B + BC_ROWS - 1) / BC_ROWS));
    hipLaunchKernelGGL((bind_coords_kernel<RB>), grid, dim3(BC_THREADS), lds, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_bind_coords(const BindCoordsArgs &a_in, hipStream_t s) {
    if (a_in.B == 0) return hipSuccess;
    BindCoordsArgs a = a_in;
    const auto al = [](const void *p, int64_t ld) { return ((uintptr_t)p & 15) == 0 && ld % 4 == 0; };
    a.vec = al(a.T, a.ldt) && al(a.T2, a.ldt2);
    a.qvec = al(a.Q, a.ldq);
    if (a.r <= 32) return launch_rb<32>(a, s);
    if (a.r <= 64) return launch_rb<64>(a, s);
    if (a.r <= 128) return launch_rb<128>(a, s);
    if (a.r <= 256) return launch_rb<256>(a, s);
    return hipErrorInvalidValue;
}

}  // namespace gs
